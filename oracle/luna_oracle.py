"""LUNA attention, plain float64 CPU oracle.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
or run this module.  The GPU library never calls it, and it shares no code with
the GPU library: it imports nothing but NumPy.  It is written for a reader who
checks it against the paper by eye, so it is slow and direct on purpose.

What it computes (paper: "Learning Kernels for Linear Attention", section 3):

* ``project``      u_i = w_i . x + b_i, the scalar projections of eq. (11) of Section 3.2
                   with the per-projection bias that the Fig. 3 caption and
                   Listing 1's task-specific projection module add.
* ``psi``          the channel functions psi_l, each a scalar MLP
                   1 -> hidden -> 1 (ReLU activation, optional ReLU on the
                   output), evaluated literally, as in Listing 1's scalar MLP.
* ``featuremap``   phi(x) = (1/sqrt(M)) [psi_l(u_i)]_{i,l} of eq. (11) of Section 3.2
                   with the envelope h = 1 (the "no gate" default of Table 5);
                   feature index i*L + l (channel index fastest), Listing 1's
                   view(B,H,N,M,L) -> reshape(..., M*L).
* ``attn_noncausal``  eq. (9) of Section 3.1: phi(Q) (phi(K)^T V) / phi(Q) (phi(K)^T 1),
                   denominator per row, with the sufficient statistics
                   S = phi(K)^T V and z = phi(K)^T 1 of the runtime section.
* ``attn_causal``  the streaming (prefix) form: S_t and z_t summed over s <= t,
                   evaluated one token at a time.
* ``causal_state`` / ``attn_causal_step``  the same streaming form split at any
                   token: the prefix state (S, z) of the first tokens, and the
                   recurrence continued from a given state over new tokens.
* ``attn_quadratic`` / ``attn_quadratic_rows``  the kernel form
                   out_t = sum_s k(q_t, k_s) v_s / sum_s k(q_t, k_s) with the
                   kernel of eq. (10) of Section 3.2, k(x, y) = (1/M) sum_i <psi(u_i(x)), psi(u_i(y))>
                   (optionally restricted to s <= t).
* ``attn_causal_chunked``  the chunked prefix scan (intra-chunk masked block
                   plus inter-chunk state carry), an exact regrouping of the
                   causal sums.
* ``pwl_tables`` / ``psi_pwl``  the exact piecewise-linear form of a ReLU
                   channel MLP (a derived identity, not in the paper).
* ``featuremap_backward``, ``attn_noncausal_backward``, ``attn_causal_backward``
                   gradients of a loss L = sum(dO * out) (dO the upstream gradient)
                   with respect to Q, K, V and every feature-map parameter, by the
                   chain rule through the definitions above, for training the
                   feature map end to end (section 5.1) and for the conversion
                   fine-tuning (section 5.2).  ReLU'(0) is taken as 0.

Readings where the paper is silent (each is listed in the design notes):
the MLP activation is ReLU; h = 1; the causal prefix includes the diagonal
(s <= t); the denominator gets an additive eps (out = num / (den + eps)), the
same eps on every path; the parameters are shared across heads unless a
leading head axis is given.

Parameter dictionaries hold NumPy arrays W [M, d], b [M], fc1_w [C1, hidden],
fc1_b [C1, hidden], fc2_w [L, hidden], fc2_b [L] (C1 = L for per-channel MLPs,
C1 = 1 for one MLP whose first layer is shared by all channels), or the same
with a leading head axis when ``per_head`` is true, plus the scalars M, L,
hidden, nonneg, shared_channels, per_head.

Parity: every function here is pinned by the oracle tests (values derived by
hand from the definitions, closed forms, special cases that reduce to library
routines, brute force, invariants); none is "parity unpinned".
"""

from __future__ import annotations

import math

import numpy as np

_PSI_CHUNK = 1 << 16  # scalars per block when evaluating the channel MLPs


def _f64(x):
    return np.asarray(x, dtype=np.float64)


# ---------------------------------------------------------------------------
# feature map, eq. (11) of Section 3.2
# ---------------------------------------------------------------------------

def project(X, W, b):
    """u[..., t, i] = w_i . x_t + b_i for X [..., n, d], W [M, d], b [M]."""
    X, W, b = _f64(X), _f64(W), _f64(b)
    return X @ W.T + b


def psi(u, fc1_w, fc1_b, fc2_w, fc2_b, nonneg=True):
    """Channel MLPs on the scalar u; returns an array of shape u.shape + (L,).

    Channel l: hidden_k = relu(a_k u + c_k) with (a, c) the first layer of
    channel l (or the shared first layer), then y_l = g_l + sum_k f_lk hidden_k,
    then relu(y_l) when ``nonneg`` (Listing 1's scalar MLP forward).
    """
    u = _f64(u)
    a_all, c_all = _f64(fc1_w), _f64(fc1_b)
    f_all, g_all = _f64(fc2_w), _f64(fc2_b)
    L = f_all.shape[0]
    shared = a_all.shape[0] == 1
    flat = u.reshape(-1)
    out = np.empty((flat.size, L), dtype=np.float64)
    for s in range(0, flat.size, _PSI_CHUNK):
        uu = flat[s:s + _PSI_CHUNK]
        for l in range(L):
            a = a_all[0 if shared else l]
            c = c_all[0 if shared else l]
            hid = np.maximum(uu[:, None] * a[None, :] + c[None, :], 0.0)
            y = hid @ f_all[l] + g_all[l]
            out[s:s + _PSI_CHUNK, l] = np.maximum(y, 0.0) if nonneg else y
    return out.reshape(u.shape + (L,))


def _head_params(p, h):
    """Parameters of head h (the same dict when they are shared)."""
    if not p.get("per_head", False):
        return p
    q = dict(p)
    for k in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b"):
        q[k] = p[k][h]
    q["per_head"] = False
    return q


def featuremap(X, p):
    """phi(X) for X [..., H, n, d] (or [n, d] with shared parameters).

    Returns [..., n, M*L] with feature index i*L + l and the 1/sqrt(M) scale.
    """
    X = _f64(X)
    if p.get("per_head", False):
        H = X.shape[-3]
        return np.stack([featuremap(X[..., h, :, :], _head_params(p, h)) for h in range(H)], axis=-3)
    u = project(X, p["W"], p["b"])                                   # [..., n, M]
    y = psi(u, p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"], p["nonneg"])  # [..., n, M, L]
    M, L = y.shape[-2], y.shape[-1]
    return y.reshape(y.shape[:-2] + (M * L,)) / math.sqrt(M)


# ---------------------------------------------------------------------------
# linear attention, eq. (9) of Section 3.1 and the runtime section's statistics
# ---------------------------------------------------------------------------

def sufficient_statistics(phiK, V):
    """S = phi(K)^T V  [..., D, dv] and z = phi(K)^T 1  [..., D]."""
    phiK, V = _f64(phiK), _f64(V)
    return np.swapaxes(phiK, -1, -2) @ V, phiK.sum(axis=-2)


def attn_noncausal(Q, K, V, p, eps=1e-6):
    """out = phi(Q) S / (phi(Q) z + eps), row by row."""
    phiQ, phiK = featuremap(Q, p), featuremap(K, p)
    S, z = sufficient_statistics(phiK, V)
    num = phiQ @ S
    den = (phiQ @ z[..., :, None])[..., 0]
    return num / (den + eps)[..., None]


def attn_causal(Q, K, V, p, eps=1e-6):
    """Streaming form: out_t = phi(q_t)^T S_t / (phi(q_t)^T z_t + eps) with
    S_t = sum_{s<=t} phi(k_s) v_s^T and z_t = sum_{s<=t} phi(k_s), one token at a time."""
    phiQ, phiK, V = featuremap(Q, p), featuremap(K, p), _f64(V)
    lead, n, D = phiQ.shape[:-2], phiQ.shape[-2], phiQ.shape[-1]
    dv = V.shape[-1]
    S = np.zeros(lead + (D, dv))
    z = np.zeros(lead + (D,))
    out = np.empty(lead + (n, dv))
    for t in range(n):
        S += phiK[..., t, :, None] * V[..., t, None, :]
        z += phiK[..., t, :]
        q = phiQ[..., t, :]
        num = (q[..., None, :] @ S)[..., 0, :]
        den = (q * z).sum(axis=-1)
        out[..., t, :] = num / (den + eps)[..., None]
    return out


def causal_state(K, V, p):
    """The prefix state of the streaming form after the tokens of K, V: the
    key-side statistics S = phi(K)^T V and z = phi(K)^T 1 of the runtime section."""
    return sufficient_statistics(featuremap(K, p), V)


def attn_causal_step(Q, K, V, p, S, z, eps=1e-6):
    """The streaming form continued from a prefix state (S, z): for each new token t in
    order, S += phi(k_t) v_t^T and z += phi(k_t), then out_t = phi(q_t)^T S /
    (phi(q_t)^T z + eps).  Returns (out, S, z) after the new tokens; S = z = 0 gives
    ``attn_causal``."""
    phiQ, phiK, V = featuremap(Q, p), featuremap(K, p), _f64(V)
    S, z = _f64(S).copy(), _f64(z).copy()
    lead, m, dv = phiQ.shape[:-2], phiQ.shape[-2], V.shape[-1]
    out = np.empty(lead + (m, dv))
    for t in range(m):
        S += phiK[..., t, :, None] * V[..., t, None, :]
        z += phiK[..., t, :]
        q = phiQ[..., t, :]
        out[..., t, :] = (q[..., None, :] @ S)[..., 0, :] / ((q * z).sum(axis=-1) + eps)[..., None]
    return out, S, z


def attn_causal_chunked(Q, K, V, p, chunk, eps=1e-6):
    """Chunked prefix scan: per chunk c, P = tril(phi(Q_c) phi(K_c)^T) including the
    diagonal, num = P V_c + phi(Q_c) S, den = P 1 + phi(Q_c) z, then S += phi(K_c)^T V_c
    and z += phi(K_c)^T 1.  A regrouping of ``attn_causal``'s sums."""
    phiQ, phiK, V = featuremap(Q, p), featuremap(K, p), _f64(V)
    lead, n, D = phiQ.shape[:-2], phiQ.shape[-2], phiQ.shape[-1]
    dv = V.shape[-1]
    S = np.zeros(lead + (D, dv))
    z = np.zeros(lead + (D,))
    out = np.empty(lead + (n, dv))
    for s0 in range(0, n, chunk):
        s1 = min(n, s0 + chunk)
        q, k, v = phiQ[..., s0:s1, :], phiK[..., s0:s1, :], V[..., s0:s1, :]
        P = np.tril(q @ np.swapaxes(k, -1, -2))
        num = P @ v + q @ S
        den = P.sum(axis=-1) + (q @ z[..., :, None])[..., 0]
        out[..., s0:s1, :] = num / (den + eps)[..., None]
        S = S + np.swapaxes(k, -1, -2) @ v
        z = z + k.sum(axis=-2)
    return out


# ---------------------------------------------------------------------------
# kernel (quadratic) form, eq. (10) of Section 3.2 with the kernel-attention normaliser
# ---------------------------------------------------------------------------

def kernel_matrix(Xq, Xk, p):
    """k(q_t, k_s) = (1/M) sum_i sum_l psi_l(w_i.q_t + b_i) psi_l(w_i.k_s + b_i)
    for Xq [n1, d], Xk [n2, d] of one head; returns [n1, n2]."""
    yq = psi(project(Xq, p["W"], p["b"]), p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"], p["nonneg"])
    yk = psi(project(Xk, p["W"], p["b"]), p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"], p["nonneg"])
    M = yq.shape[-2]
    A = np.zeros((yq.shape[0], yk.shape[0]))
    for i in range(M):  # average over the M projections w_i
        A += yq[:, i, :] @ yk[:, i, :].T
    return A / M


def attn_quadratic_rows(Q, K, V, p, rows, eps=1e-6, causal=False):
    """Kernel form for selected query rows of one head: Q, K [n, d], V [n, dv].

    out_t = sum_s k(q_t, k_s) v_s / (sum_s k(q_t, k_s) + eps), s over all
    tokens, or over s <= t when ``causal``.  Returns [len(rows), dv].
    """
    rows = np.asarray(rows, dtype=np.int64)
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    kmax = int(rows.max()) + 1 if causal else K.shape[0]
    A = kernel_matrix(Q[rows], K[:kmax], p)
    if causal:
        A = np.where(np.arange(kmax)[None, :] <= rows[:, None], A, 0.0)
    return (A @ V[:kmax]) / (A.sum(axis=-1) + eps)[:, None]


def attn_quadratic(Q, K, V, p, eps=1e-6, causal=False):
    """Kernel form for every row of every head: Q, K, V [..., H, n, d]."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    if Q.ndim == 2:
        return attn_quadratic_rows(Q, K, V, p, np.arange(Q.shape[0]), eps, causal)
    lead = Q.shape[:-2]
    out = np.empty(lead + (Q.shape[-2], V.shape[-1]))
    for idx in np.ndindex(*lead):
        ph = _head_params(p, idx[-1])  # idx[-1] is the head index
        out[idx] = attn_quadratic_rows(Q[idx], K[idx], V[idx], ph, np.arange(Q.shape[-2]), eps, causal)
    return out


# ---------------------------------------------------------------------------
# exact piecewise-linear form of a ReLU channel MLP (derived identity)
# ---------------------------------------------------------------------------

def pwl_tables(fc1_w, fc1_b, fc2_w, fc2_b):
    """Breakpoints and per-segment affine coefficients of the pre-ReLU channel outputs.

    Unit k of channel l switches at beta_k = -c_k / a_k (a_k != 0).  With the
    breakpoints sorted, on the open interval between two neighbours every unit is
    either on or off, so y_l(u) = s_l u + t_l there.  Returns (bp [nbp],
    s [nbp+1, L], t [nbp+1, L]); segment j covers bp[j-1] < u <= bp[j].
    """
    a_all, c_all = _f64(fc1_w), _f64(fc1_b)
    f_all, g_all = _f64(fc2_w), _f64(fc2_b)
    L = f_all.shape[0]
    shared = a_all.shape[0] == 1
    units = []  # (channel or -1 for shared, a, c)
    for ch in range(a_all.shape[0]):
        for k in range(a_all.shape[1]):
            units.append((ch, k, a_all[ch, k], c_all[ch, k]))
    bp = np.sort(np.array([-c / a for (_, _, a, c) in units if a != 0.0], dtype=np.float64))
    nseg = bp.size + 1
    # a point inside every segment (segment ends are finite breakpoints)
    if bp.size == 0:
        mids = np.array([0.0])
    else:
        inner = 0.5 * (bp[:-1] + bp[1:])
        pad0, pad1 = max(1.0, abs(bp[0])), max(1.0, abs(bp[-1]))
        mids = np.concatenate([[bp[0] - pad0], inner, [bp[-1] + pad1]])
    s = np.zeros((nseg, L))
    t = np.tile(g_all[None, :], (nseg, 1))
    for (ch, k, a, c) in units:
        on = (a * mids + c) > 0.0  # unit state on each segment
        for l in range(L):
            if not shared and l != ch:
                continue
            f = f_all[l, k]
            s[:, l] += np.where(on, f * a, 0.0)
            t[:, l] += np.where(on, f * c, 0.0)
    return bp, s, t


def psi_pwl(u, tables, nonneg=True):
    """Evaluate the channel MLPs through ``pwl_tables``: segment search, then s u + t."""
    bp, s, t = tables
    u = _f64(u)
    j = np.searchsorted(bp, u, side="left")  # number of breakpoints < u
    y = s[j] * u[..., None] + t[j]
    return np.maximum(y, 0.0) if nonneg else y


# ---------------------------------------------------------------------------
# gradients (chain rule through the definitions above; ReLU'(0) = 0)
# ---------------------------------------------------------------------------

PARAM_NAMES = ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")


def _psi_backward(u, dpsi, fc1_w, fc1_b, fc2_w, fc2_b, nonneg=True):
    """Gradients of sum(dpsi * psi(u)) for scalars u [N] and dpsi [N, L]: returns
    (du [N], dfc1_w, dfc1_b, dfc2_w, dfc2_b).  Channel l: pre_k = a_k u + c_k,
    h_k = relu(pre_k), y_l = g_l + sum_k f_lk h_k, psi_l = relu(y_l) when ``nonneg``."""
    u = _f64(u)
    a_all, c_all = _f64(fc1_w), _f64(fc1_b)
    f_all, g_all = _f64(fc2_w), _f64(fc2_b)
    L = f_all.shape[0]
    shared = a_all.shape[0] == 1
    du = np.zeros(u.shape)
    d1w, d1b = np.zeros(a_all.shape), np.zeros(c_all.shape)
    d2w, d2b = np.zeros(f_all.shape), np.zeros(g_all.shape)
    for s in range(0, u.size, _PSI_CHUNK):
        uu, dp = u[s:s + _PSI_CHUNK], dpsi[s:s + _PSI_CHUNK]
        for l in range(L):
            i = 0 if shared else l
            pre = uu[:, None] * a_all[i][None, :] + c_all[i][None, :]
            hid = np.maximum(pre, 0.0)
            y = hid @ f_all[l] + g_all[l]
            dy = dp[:, l] * (y > 0.0) if nonneg else dp[:, l]
            d2w[l] += hid.T @ dy
            d2b[l] += dy.sum()
            dpre = (dy[:, None] * f_all[l][None, :]) * (pre > 0.0)
            d1w[i] += (dpre * uu[:, None]).sum(axis=0)
            d1b[i] += dpre.sum(axis=0)
            du[s:s + _PSI_CHUNK] += dpre @ a_all[i]
    return du, d1w, d1b, d2w, d2b


def featuremap_backward(X, p, dphi):
    """Gradients of sum(dphi * featuremap(X, p)): returns (dX, grads) with dX shaped
    like X and grads a dict of the parameter gradients (PARAM_NAMES, shaped like the
    parameters), summed over every row.  phi_{iL+l} = psi_l(u_i) / sqrt(M) with
    u = X W^T + b."""
    X, dphi = _f64(X), _f64(dphi)
    if p.get("per_head", False):
        H = X.shape[-3]
        dX = np.empty(X.shape)
        grads = {k: np.zeros(np.shape(p[k])) for k in PARAM_NAMES}
        for h in range(H):
            dXh, gh = featuremap_backward(X[..., h, :, :], _head_params(p, h), dphi[..., h, :, :])
            dX[..., h, :, :] = dXh
            for k in PARAM_NAMES:
                grads[k][h] += gh[k]
        return dX, grads
    W = _f64(p["W"])
    M, L = W.shape[0], _f64(p["fc2_b"]).shape[0]
    u = project(X, p["W"], p["b"])                                        # [..., n, M]
    dpsi = dphi.reshape(u.shape + (L,)) / math.sqrt(M)
    du, d1w, d1b, d2w, d2b = _psi_backward(u.reshape(-1), dpsi.reshape(-1, L), p["fc1_w"], p["fc1_b"],
                                           p["fc2_w"], p["fc2_b"], p["nonneg"])
    du = du.reshape(u.shape)
    dX = du @ W
    grads = {
        "W": du.reshape(-1, M).T @ X.reshape(-1, X.shape[-1]),
        "b": du.reshape(-1, M).sum(axis=0),
        "fc1_w": d1w, "fc1_b": d1b, "fc2_w": d2w, "fc2_b": d2b,
    }
    return dX, grads


def _add_grads(g1, g2):
    return {k: g1[k] + g2[k] for k in PARAM_NAMES}


def attn_noncausal_backward(Q, K, V, p, dO, eps=1e-6):
    """Gradients of L = sum(dO * attn_noncausal(Q, K, V, p, eps)) with respect to Q, K,
    V and the feature-map parameters: returns (dQ, dK, dV, grads).

    With num = phi(Q) S, den = phi(Q) z + eps and out = num / den per row:
    dnum = dO / den, dden = -(dO . num) / den^2, dphi(Q) = dnum S^T + dden z^T,
    dS = phi(Q)^T dnum, dz = phi(Q)^T dden, dphi(K) = V dS^T + 1 dz^T, dV = phi(K) dS."""
    V, dO = _f64(V), _f64(dO)
    phiQ, phiK = featuremap(Q, p), featuremap(K, p)
    S, z = sufficient_statistics(phiK, V)
    num = phiQ @ S
    den = (phiQ @ z[..., :, None])[..., 0] + eps
    dnum = dO / den[..., None]
    dden = -(dO * num).sum(axis=-1) / den ** 2
    dphiQ = dnum @ np.swapaxes(S, -1, -2) + dden[..., None] * z[..., None, :]
    dS = np.swapaxes(phiQ, -1, -2) @ dnum
    dz = (np.swapaxes(phiQ, -1, -2) @ dden[..., None])[..., 0]
    dphiK = V @ np.swapaxes(dS, -1, -2) + dz[..., None, :]
    dV = phiK @ dS
    dQ, gq = featuremap_backward(Q, p, dphiQ)
    dK, gk = featuremap_backward(K, p, dphiK)
    return dQ, dK, dV, _add_grads(gq, gk)


def attn_causal_backward(Q, K, V, p, dO, eps=1e-6):
    """Gradients of L = sum(dO * attn_causal(Q, K, V, p, eps)): returns (dQ, dK, dV, grads).

    Query t sees the prefix state (S_t, z_t) over s <= t, so dphi(q_t) = S_t dnum_t +
    z_t dden_t, taken in a forward pass over the tokens; key s feeds every query t >= s,
    so with the suffix sums dS_s = sum_{t >= s} phi(q_t) dnum_t^T and dz_s = sum_{t >= s}
    phi(q_t) dden_t, dphi(k_s) = dS_s v_s + dz_s and dv_s = dS_s^T phi(k_s), taken in a
    backward pass."""
    V, dO = _f64(V), _f64(dO)
    phiQ, phiK = featuremap(Q, p), featuremap(K, p)
    lead, n, D = phiQ.shape[:-2], phiQ.shape[-2], phiQ.shape[-1]
    dv = V.shape[-1]
    S = np.zeros(lead + (D, dv))
    z = np.zeros(lead + (D,))
    dnum = np.empty(lead + (n, dv))
    dden = np.empty(lead + (n,))
    dphiQ = np.empty(phiQ.shape)
    for t in range(n):
        S += phiK[..., t, :, None] * V[..., t, None, :]
        z += phiK[..., t, :]
        q = phiQ[..., t, :]
        num = (q[..., None, :] @ S)[..., 0, :]
        den = (q * z).sum(axis=-1) + eps
        dnum[..., t, :] = dO[..., t, :] / den[..., None]
        dden[..., t] = -(dO[..., t, :] * num).sum(axis=-1) / den ** 2
        dphiQ[..., t, :] = (S @ dnum[..., t, :, None])[..., 0] + z * dden[..., t, None]
    dS = np.zeros(lead + (D, dv))
    dz = np.zeros(lead + (D,))
    dphiK = np.empty(phiK.shape)
    dV = np.empty(V.shape)
    for t in range(n - 1, -1, -1):
        dS += phiQ[..., t, :, None] * dnum[..., t, None, :]
        dz += phiQ[..., t, :] * dden[..., t, None]
        dphiK[..., t, :] = (dS @ V[..., t, :, None])[..., 0] + dz
        dV[..., t, :] = (phiK[..., t, None, :] @ dS)[..., 0, :]
    dQ, gq = featuremap_backward(Q, p, dphiQ)
    dK, gk = featuremap_backward(K, p, dphiK)
    return dQ, dK, dV, _add_grads(gq, gk)
