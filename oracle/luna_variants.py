"""Feature-map variants, plain float64 CPU oracle.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import or
run this module; the GPU library never does and shares no code with it.

The learned map of eq. (11) of Section 3.2, phi(x) = h(x)/sqrt(M) [psi_l(w_i . x +
b_i)]_{i,l}, is a template: fixing h and the psi_l by hand recovers the random-feature
maps of Section 3.1, and the ablation of Section 5.4 (Table 5) changes its form.  The
variants here, each a different psi / h stage on the same projection u = W x + b:

* ``rff_cos``        random Fourier features (Section 3.1): sqrt(2/M) cos(u_i), one
                     feature per projection (the phase b_i is the projection bias).
* ``rff_sincos``     Table 5's fixed sin/cos features: (1/sqrt(M)) [sin(u_i), cos(u_i)],
                     two channels per projection, sin first.
* ``performer``      Performer positive features (Section 3.1): (1/sqrt(M))
                     exp(u_i - |x|^2 / (2 sqrt(d))), i.e. psi = exp and the envelope
                     h(x) = exp(-|x|^2 / (2 sqrt(d))); with w_i = omega_i / d^(1/4) and
                     omega_i ~ N(0, I) the feature inner product is an unbiased estimate
                     of exp(x . y / sqrt(d)).
* ``mlp_variant``    Listing 1's channel MLPs with a smooth hidden activation (act in
                     relu, gelu, silu, tanh), and optionally Table 5's envelope-gated
                     form h(x) (.) psi(x) with a tokenwise envelope in [0, 1]^L
                     (sigmoid(G x + c), one value per channel), Listing 1's channel RMS
                     normalisation (ch_rms) and Table 5's Bank+Coef form (the channels of
                     each projection summed with global coefficients w_l, one feature per
                     projection).  Order: psi, envelope, channel RMS, bank sum, 1/sqrt(M).
* ``attn_from_features``  eq. (9) of Section 3.1 (and its causal prefix form) for
                     given feature matrices.

Readings (listed in the design notes): the hidden activation names follow
PyTorch's definitions (gelu in its erf form); the envelope is sigmoid of an affine
map of x, one value per channel, multiplying that channel of every projection; the
Performer sampling variance is the one that makes the estimate unbiased for the
feature formula as printed (omega ~ N(0, I) with x scaled by d^(-1/4), folded into
W); channel RMS: per channel, rms = sqrt(mean over every (batch, head, token,
projection) of y^2 + 1e-6), y *= min(target / (rms + 1e-6), 1).
"""

from __future__ import annotations

import math

import numpy as np

from .luna_oracle import _f64, project


def _act(name, z):
    """The hidden activation of Listing 1's scalar MLP, by name."""
    if name == "relu":
        return np.maximum(z, 0.0)
    if name == "gelu":  # z Phi(z), Phi the standard normal distribution function
        erf = np.vectorize(math.erf)
        return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))
    if name == "silu":  # z sigmoid(z)
        return z / (1.0 + np.exp(-z))
    if name == "tanh":
        return np.tanh(z)
    raise ValueError(name)


def psi_act(u, fc1_w, fc1_b, fc2_w, fc2_b, nonneg=True, act="relu"):
    """Channel MLPs 1 -> hidden -> 1 with the hidden activation ``act``; returns
    u.shape + (L,).  Channel l: y_l = g_l + sum_k f_lk act(a_k u + c_k), (a, c) its
    own first layer (or the shared one), then relu(y_l) when ``nonneg``."""
    u = _f64(u)
    a_all, c_all, f_all, g_all = _f64(fc1_w), _f64(fc1_b), _f64(fc2_w), _f64(fc2_b)
    L = f_all.shape[0]
    shared = a_all.shape[0] == 1
    flat = u.reshape(-1)
    out = np.empty((flat.size, L))
    for l in range(L):
        a, c = a_all[0 if shared else l], c_all[0 if shared else l]
        hid = _act(act, flat[:, None] * a[None, :] + c[None, :])
        y = hid @ f_all[l] + g_all[l]
        out[:, l] = np.maximum(y, 0.0) if nonneg else y
    return out.reshape(u.shape + (L,))


def _per_head(fn, X, p, *rest):
    """fn applied head by head when the parameters have a leading head axis."""
    if not p.get("per_head", False):
        return fn(X, p, *rest)
    H = X.shape[-3]
    outs = []
    for h in range(H):
        q = dict(p)
        for k in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b", "env_w", "env_b", "bank"):
            if k in p and p[k] is not None:
                q[k] = p[k][h]
        q["per_head"] = False
        outs.append(fn(X[..., h, :, :], q, *rest))
    return np.stack(outs, axis=X.ndim - 3)  # the head axis where X has it


def rff_cos(X, p):
    """sqrt(2/M) [cos(w_i . x + b_i)]_i for X [..., n, d]."""
    X = _f64(X)
    if p.get("per_head", False):
        return _per_head(rff_cos, X, p)
    u = project(X, p["W"], p["b"])
    return math.sqrt(2.0 / u.shape[-1]) * np.cos(u)


def rff_sincos(X, p):
    """(1/sqrt(M)) [sin(u_i), cos(u_i)]_i, feature 2i + l (sin at l = 0)."""
    X = _f64(X)
    if p.get("per_head", False):
        return _per_head(rff_sincos, X, p)
    u = project(X, p["W"], p["b"])
    M = u.shape[-1]
    y = np.stack([np.sin(u), np.cos(u)], axis=-1)
    return y.reshape(u.shape[:-1] + (2 * M,)) / math.sqrt(M)


def performer(X, p):
    """(1/sqrt(M)) [exp(w_i . x + b_i - |x|^2 / (2 sqrt(d)))]_i."""
    X = _f64(X)
    if p.get("per_head", False):
        return _per_head(performer, X, p)
    d = X.shape[-1]
    u = project(X, p["W"], p["b"])
    sq = (X * X).sum(axis=-1, keepdims=True)
    return np.exp(u - sq / (2.0 * math.sqrt(d))) / math.sqrt(u.shape[-1])


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def ch_rms(y, target, eps=1e-6):
    """Listing 1's channel RMS normalisation of y [..., M, L] (all leading axes and the
    projections pooled): y_l * min(target / (rms_l + eps), 1), rms_l = sqrt(mean y_l^2 + eps)."""
    y = _f64(y)
    L = y.shape[-1]
    rms = np.sqrt((y.reshape(-1, L) ** 2).mean(axis=0) + eps)
    s = np.minimum(target / (rms + eps), 1.0)
    return y * s


def _mlp_channels(X, p):
    """psi (with the activation), then the envelope, for X [..., n, d]: [..., n, M, L]."""
    u = project(X, p["W"], p["b"])
    y = psi_act(u, p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"], p["nonneg"], p.get("act", "relu"))
    if p.get("env_w") is not None:
        env = _sigmoid(X @ _f64(p["env_w"]).T + _f64(p["env_b"]))  # [..., n, L]
        y = y * env[..., None, :]
    return y


def mlp_variant(X, p):
    """The channel-MLP map with the options of ``p``: "act", "env_w" [L, d] / "env_b"
    [L] (envelope), "ch_rms" (bool) / "ch_rms_target", "bank" [L] (Bank+Coef).
    Returns [..., n, M*L] (feature i*L + l), or [..., n, M] with a bank."""
    X = _f64(X)
    y = _per_head(_mlp_channels, X, p)  # [..., n, M, L]
    if p.get("ch_rms", False):
        y = ch_rms(y, p.get("ch_rms_target", 0.1))
    M, L = y.shape[-2], y.shape[-1]
    if p.get("bank") is not None:
        w = _f64(p["bank"])
        if p.get("per_head", False):  # [H, L] coefficients, head axis at -4 of y
            out = np.einsum("...hnml,hl->...hnm", y, w)
        else:
            out = y @ w
        return out / math.sqrt(M)
    return y.reshape(y.shape[:-2] + (M * L,)) / math.sqrt(M)


def featuremap_variant(X, p):
    """Dispatch on p["kind"]: "mlp", "rff_cos", "rff_sincos", "performer"."""
    kind = p.get("kind", "mlp")
    return {"mlp": mlp_variant, "rff_cos": rff_cos, "rff_sincos": rff_sincos, "performer": performer}[kind](X, p)


def attn_from_features(phiQ, phiK, V, eps=1e-6, causal=False):
    """out_t = phi(q_t) S / (phi(q_t) z + eps) with S = sum_s phi(k_s) v_s^T and
    z = sum_s phi(k_s), over every s or over s <= t (eq. (9) of Section 3.1 and its
    prefix form), for given features phiQ, phiK [..., n, D] and V [..., n, dv]."""
    phiQ, phiK, V = _f64(phiQ), _f64(phiK), _f64(V)
    if not causal:
        S = np.swapaxes(phiK, -1, -2) @ V
        z = phiK.sum(axis=-2)
        return (phiQ @ S) / ((phiQ @ z[..., :, None]) + eps)
    lead, n, D = phiQ.shape[:-2], phiQ.shape[-2], phiQ.shape[-1]
    S = np.zeros(lead + (D, V.shape[-1]))
    z = np.zeros(lead + (D,))
    out = np.empty(lead + (n, V.shape[-1]))
    for t in range(n):
        S += phiK[..., t, :, None] * V[..., t, None, :]
        z += phiK[..., t, :]
        q = phiQ[..., t, :]
        out[..., t, :] = (q[..., None, :] @ S)[..., 0, :] / ((q * z).sum(axis=-1) + eps)[..., None]
    return out
