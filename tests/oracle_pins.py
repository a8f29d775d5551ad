"""Pins that tie the float64 oracle to something other than itself.

Each ``pin_*`` function takes the oracle module and raises AssertionError (or
any exception) when the oracle disagrees with what the paper or the mathematics
fixes: values worked out by hand, closed forms, special cases that reduce to a
library routine, brute force on tiny inputs, invariants.  ``tests/test_oracle_pins.py``
runs them against the real oracle; ``tests/test_oracle_mutations.py`` plants
plausible mistakes in the oracle and checks that some pin fails for each.
"""

from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _params(rng, M, L, d, hidden=8, shared=False, nonneg=True, scale=None, per_head=0):
    s = (1.0 / math.sqrt(d)) if scale is None else scale
    C1 = 1 if shared else L
    lead = (per_head,) if per_head else ()
    p = {
        "W": rng.standard_normal(lead + (M, d)) * s,
        "b": rng.standard_normal(lead + (M,)) * s,
        "fc1_w": rng.standard_normal(lead + (C1, hidden)) * s,
        "fc1_b": rng.standard_normal(lead + (C1, hidden)) * s,
        "fc2_w": rng.standard_normal(lead + (L, hidden)) * s,
        "fc2_b": rng.standard_normal(lead + (L,)) * s,
        "M": M, "L": L, "hidden": hidden, "nonneg": nonneg,
        "shared_channels": shared, "per_head": bool(per_head),
    }
    return p


def _qkv(rng, shape, dv=None):
    Q = rng.standard_normal(shape)
    K = rng.standard_normal(shape)
    V = rng.standard_normal(shape[:-1] + ((dv or shape[-1]),))
    return Q, K, V


def _rel(a, b):
    a, b = np.asarray(a, float), np.asarray(b, float)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def _frac(x):
    return np.array([[float(Fraction(v)) for v in row] for row in x])


# ---------------------------------------------------------------------------

def pin_golden_hand_example(o):
    """Values worked out by hand (tests/golden/hand_example.md)."""
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    p = {k: np.array(g[k], dtype=float) for k in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")}
    p.update(M=2, L=2, hidden=2, nonneg=True, shared_channels=False, per_head=False)
    Q, K, V = (np.array(g[k], dtype=float) for k in ("Q", "K", "V"))
    assert np.allclose(o.featuremap(Q, p) * math.sqrt(2), _frac(g["phi_q_times_sqrtM"]), rtol=0, atol=1e-15)
    assert np.allclose(o.featuremap(K, p) * math.sqrt(2), _frac(g["phi_k_times_sqrtM"]), rtol=0, atol=1e-15)
    assert np.allclose(o.kernel_matrix(Q, K, p), _frac(g["kernel"]), rtol=0, atol=1e-15)
    for f in (lambda: o.attn_noncausal(Q, K, V, p, eps=0.0),
              lambda: o.attn_quadratic(Q, K, V, p, eps=0.0, causal=False)):
        assert np.allclose(f(), _frac(g["out_noncausal"]), rtol=0, atol=1e-15)
    for f in (lambda: o.attn_causal(Q, K, V, p, eps=0.0),
              lambda: o.attn_causal_chunked(Q, K, V, p, 1, eps=0.0),
              lambda: o.attn_quadratic(Q, K, V, p, eps=0.0, causal=True)):
        assert np.allclose(f(), _frac(g["out_causal"]), rtol=0, atol=1e-15)


def pin_single_unit_psi_by_hand(o):
    """One hidden unit, a=2, c=-1, f=3, g=-1/2: psi(u) = relu(3 relu(2u-1) - 1/2)."""
    a, c, f, g = [[2.0]], [[-1.0]], [[3.0]], [-0.5]
    u = np.array([0.0, 1.0, -1.0, 0.75])
    assert np.array_equal(o.psi(u, a, c, f, g, nonneg=True)[:, 0], [0.0, 2.5, 0.0, 1.0])
    assert np.array_equal(o.psi(u, a, c, f, g, nonneg=False)[:, 0], [-0.5, 2.5, -0.5, 1.0])


def pin_relu_channels_layout(o):
    """psi_0(u) = relu(u), psi_1(u) = relu(-u), psi_2(u) = relu(u - 1) + 1 fix
    phi = [relu(u_i), relu(-u_i), relu(u_i - 1) + 1]_i / sqrt(M) with index i*L + l."""
    rng = np.random.default_rng(7)
    M, L, d, n = 3, 3, 4, 5
    W, b = rng.standard_normal((M, d)), rng.standard_normal(M)
    p = {"W": W, "b": b,
         "fc1_w": np.array([[1.0, 0.0], [-1.0, 0.0], [1.0, 0.0]]),
         "fc1_b": np.array([[0.0, 0.0], [0.0, 0.0], [-1.0, 1.0]]),
         "fc2_w": np.array([[1.0, 0.0], [1.0, 0.0], [1.0, 1.0]]),
         "fc2_b": np.array([0.0, 0.0, 0.0]),
         "M": M, "L": L, "hidden": 2, "nonneg": True, "shared_channels": False, "per_head": False}
    X = rng.standard_normal((n, d))
    u = np.einsum("nd,md->nm", X, W) + b
    want = np.empty((n, M * L))
    for i in range(M):
        want[:, i * L + 0] = np.maximum(u[:, i], 0)
        want[:, i * L + 1] = np.maximum(-u[:, i], 0)
        want[:, i * L + 2] = np.maximum(u[:, i] - 1, 0) + 1
    assert np.allclose(o.featuremap(X, p), want / math.sqrt(M), rtol=1e-14, atol=1e-14)


def pin_linear_equals_quadratic(o):
    """Associativity: phi(Q)(phi(K)^T V) / phi(Q)(phi(K)^T 1) equals the kernel form."""
    rng = np.random.default_rng(1)
    for (M, L, d, n, hidden, shared, nonneg) in [(4, 3, 6, 37, 5, False, True), (2, 8, 5, 20, 7, True, True),
                                                 (3, 2, 4, 11, 3, False, False)]:
        p = _params(rng, M, L, d, hidden, shared, nonneg)
        Q, K, V = _qkv(rng, (2, 3, n, d), dv=7)
        a = o.attn_noncausal(Q, K, V, p, eps=0.0)
        b = o.attn_quadratic(Q, K, V, p, eps=0.0, causal=False)
        assert _rel(a, b) < 1e-10, _rel(a, b)
        a = o.attn_noncausal(Q, K, V, p, eps=1e-3)
        b = o.attn_quadratic(Q, K, V, p, eps=1e-3, causal=False)
        assert _rel(a, b) < 1e-10


def pin_causal_equals_masked(o):
    """Prefix recurrence equals the kernel form restricted to s <= t."""
    rng = np.random.default_rng(2)
    p = _params(rng, 4, 4, 8, 6)
    Q, K, V = _qkv(rng, (2, 2, 41, 8), dv=5)
    a = o.attn_causal(Q, K, V, p, eps=1e-6)
    b = o.attn_quadratic(Q, K, V, p, eps=1e-6, causal=True)
    assert _rel(a, b) < 1e-10
    rows = np.array([0, 5, 40])
    c = o.attn_quadratic_rows(Q[1, 0], K[1, 0], V[1, 0], p, rows, eps=1e-6, causal=True)
    assert _rel(c, a[1, 0, rows]) < 1e-10


def pin_step_continues_the_prefix(o):
    """The streaming form split at any token: from the state of the first n0 tokens,
    steps over the rest give the masked kernel form's rows n0.. and, at the end, the
    statistics of the whole sequence; from a zero state, the whole masked form."""
    rng = np.random.default_rng(31)
    p = _params(rng, 3, 4, 6, 5)
    n = 23
    Q, K, V = _qkv(rng, (2, 2, n, 6), dv=5)
    full = o.attn_quadratic(Q, K, V, p, eps=1e-6, causal=True)
    D = 3 * 4
    out, S, z = o.attn_causal_step(Q, K, V, p, np.zeros((2, 2, D, 5)), np.zeros((2, 2, D)), eps=1e-6)
    assert _rel(out, full) < 1e-10
    for n0 in (0, 1, 9, 22):
        S0, z0 = o.causal_state(K[..., :n0, :], V[..., :n0, :], p)
        parts, St, zt = [], S0, z0
        for a, b in ((n0, min(n, n0 + 4)), (min(n, n0 + 4), n)):  # two steps
            y, St, zt = o.attn_causal_step(Q[..., a:b, :], K[..., a:b, :], V[..., a:b, :], p, St, zt, eps=1e-6)
            parts.append(y)
        assert _rel(np.concatenate(parts, axis=-2), full[..., n0:, :]) < 1e-10
        # the state after the last token: phi(K)^T V and phi(K)^T 1 by brute force over the tokens
        phiK = o.featuremap(K, p)
        Sb = sum(np.einsum("...f,...v->...fv", phiK[..., t, :], V[..., t, :]) for t in range(n))
        zb = sum(phiK[..., t, :] for t in range(n))
        assert _rel(St, Sb) < 1e-12 and _rel(zt, zb) < 1e-12
    # the step does not modify the state it is given
    S0, z0 = o.causal_state(K[..., :5, :], V[..., :5, :], p)
    S1, z1 = S0.copy(), z0.copy()
    o.attn_causal_step(Q[..., 5:9, :], K[..., 5:9, :], V[..., 5:9, :], p, S0, z0)
    assert np.array_equal(S0, S1) and np.array_equal(z0, z1)


def pin_chunked_equals_recurrence(o):
    """Chunk sizes 1, 3, 16 and n (n not a multiple of the chunk) give the recurrence."""
    rng = np.random.default_rng(3)
    p = _params(rng, 2, 8, 8, 4)
    n = 29
    Q, K, V = _qkv(rng, (1, 2, n, 8), dv=6)
    ref = o.attn_causal(Q, K, V, p, eps=1e-6)
    for C in (1, 3, 16, n, 64):
        assert _rel(o.attn_causal_chunked(Q, K, V, p, C, eps=1e-6), ref) < 1e-10


def pin_positivity_and_pd(o):
    """ReLU output gives phi >= 0; the kernel's Gram matrix is symmetric PSD (Prop. 1)."""
    rng = np.random.default_rng(4)
    p = _params(rng, 5, 4, 6, 8, scale=1.0)
    X = rng.standard_normal((40, 6))
    phi = o.featuremap(X, p)
    assert (phi >= 0).all() and (phi == 0).any()
    G = o.kernel_matrix(X, X, p)
    assert np.allclose(G, G.T, rtol=1e-13, atol=1e-13)
    ev = np.linalg.eigvalsh(0.5 * (G + G.T))
    assert ev.min() >= -1e-12 * np.trace(G)
    assert np.allclose(G, phi @ phi.T, rtol=1e-12, atol=1e-13)


def pin_constant_psi_gives_mean(o):
    """psi = 1 for every channel: non-causal output is the mean of V, causal the running mean."""
    rng = np.random.default_rng(5)
    M, L, d = 3, 2, 4
    p = {"W": rng.standard_normal((M, d)), "b": rng.standard_normal(M),
         "fc1_w": np.zeros((L, 1)), "fc1_b": np.ones((L, 1)), "fc2_w": np.ones((L, 1)),
         "fc2_b": np.zeros(L), "M": M, "L": L, "hidden": 1, "nonneg": True,
         "shared_channels": False, "per_head": False}
    Q, K, V = _qkv(rng, (2, 13, d), dv=3)
    out = o.attn_noncausal(Q, K, V, p, eps=0.0)
    assert np.allclose(out, np.broadcast_to(V.mean(axis=-2, keepdims=True), out.shape), rtol=1e-13, atol=1e-13)
    run = np.cumsum(V, axis=-2) / np.arange(1, 14)[:, None]
    assert np.allclose(o.attn_causal(Q, K, V, p, eps=0.0), run, rtol=1e-13, atol=1e-13)
    assert np.allclose(o.attn_causal_chunked(Q, K, V, p, 4, eps=0.0), run, rtol=1e-13, atol=1e-13)


def pin_single_feature_weighted_average(o):
    """M = L = 1: out_t is the average of the v_s weighted by phi(k_s), whatever q_t is."""
    rng = np.random.default_rng(6)
    p = _params(rng, 1, 1, 5, 6, scale=1.0)
    p["fc2_b"] = np.array([0.3])  # keeps phi(q) > 0 somewhere
    Q, K, V = _qkv(rng, (30, 5), dv=4)
    phiq, phik = o.featuremap(Q, p)[:, 0], o.featuremap(K, p)[:, 0]
    assert (phik > 0).any() and (phiq > 0).any()
    out = o.attn_noncausal(Q, K, V, p, eps=0.0)
    want = np.average(V, axis=0, weights=phik)
    for t in np.nonzero(phiq > 0)[0]:
        assert np.allclose(out[t], want, rtol=1e-12, atol=1e-13)


def pin_convexity(o):
    """Constant V rows are reproduced; each output coordinate lies within the range of V (eps = 0)."""
    rng = np.random.default_rng(8)
    p = _params(rng, 4, 3, 6, 5)
    Q, K, _ = _qkv(rng, (2, 25, 6))
    V = np.tile(rng.standard_normal(5), (2, 25, 1))
    for out in (o.attn_noncausal(Q, K, V, p, eps=0.0), o.attn_causal(Q, K, V, p, eps=0.0)):
        ok = np.isfinite(out).all(axis=-1)
        assert ok.mean() > 0.5
        assert np.allclose(out[ok], V[ok], rtol=1e-12, atol=1e-12)
    V = rng.standard_normal((2, 25, 5))
    out = o.attn_noncausal(Q, K, V, p, eps=0.0)
    ok = np.isfinite(out).all(axis=-1)
    lo, hi = V.min(axis=-2, keepdims=True), V.max(axis=-2, keepdims=True)
    assert ((out >= lo - 1e-12) | ~ok[..., None]).all() and ((out <= hi + 1e-12) | ~ok[..., None]).all()


def pin_permutation_and_scale(o):
    """Non-causal: permuting (K, V) rows leaves the output unchanged, permuting Q rows
    permutes it; scaling the channel outputs by alpha > 0 scales phi and leaves out unchanged."""
    rng = np.random.default_rng(9)
    p = _params(rng, 3, 4, 5, 6)
    Q, K, V = _qkv(rng, (17, 5))
    ref = o.attn_noncausal(Q, K, V, p, eps=0.0)
    perm = rng.permutation(17)
    assert np.allclose(o.attn_noncausal(Q, K[perm], V[perm], p, eps=0.0), ref, rtol=1e-12, atol=1e-13)
    assert np.allclose(o.attn_noncausal(Q[perm], K, V, p, eps=0.0), ref[perm], rtol=1e-12, atol=1e-13)
    q = dict(p)
    q["fc2_w"], q["fc2_b"] = 2.5 * p["fc2_w"], 2.5 * p["fc2_b"]
    assert np.allclose(o.featuremap(Q, q), 2.5 * o.featuremap(Q, p), rtol=1e-13, atol=1e-14)
    assert np.allclose(o.attn_noncausal(Q, K, V, q, eps=0.0), ref, rtol=1e-12, atol=1e-13)


def pin_zero_features_give_zero(o):
    """psi = 0 everywhere (g = -1, f = 0): numerator and denominator vanish, out = 0/(0+eps) = 0."""
    rng = np.random.default_rng(10)
    M, L, d = 2, 3, 4
    p = {"W": rng.standard_normal((M, d)), "b": np.zeros(M), "fc1_w": np.ones((L, 2)),
         "fc1_b": np.zeros((L, 2)), "fc2_w": np.zeros((L, 2)), "fc2_b": -np.ones(L),
         "M": M, "L": L, "hidden": 2, "nonneg": True, "shared_channels": False, "per_head": False}
    Q, K, V = _qkv(rng, (9, d))
    assert np.array_equal(o.attn_noncausal(Q, K, V, p, eps=1e-6), np.zeros((9, d)))
    assert np.array_equal(o.attn_causal(Q, K, V, p, eps=1e-6), np.zeros((9, d)))


def pin_shared_first_layer(o):
    """Shared first layer equals per-channel MLPs whose first layers are all the same."""
    rng = np.random.default_rng(11)
    p = _params(rng, 3, 4, 5, 6, shared=True)
    q = dict(p)
    q["fc1_w"] = np.repeat(p["fc1_w"], 4, axis=0)
    q["fc1_b"] = np.repeat(p["fc1_b"], 4, axis=0)
    q["shared_channels"] = False
    X = rng.standard_normal((11, 5))
    assert np.array_equal(o.featuremap(X, p), o.featuremap(X, q))


def pin_per_head_parameters(o):
    """Per-head parameters: head h of the batched result equals a run with head h's parameters."""
    rng = np.random.default_rng(12)
    H = 3
    p = _params(rng, 2, 4, 6, 5, per_head=H)
    Q, K, V = _qkv(rng, (2, H, 9, 6))
    a = o.attn_noncausal(Q, K, V, p, eps=1e-6)
    c = o.attn_causal(Q, K, V, p, eps=1e-6)
    for h in range(H):
        ph = {k: (v[h] if k in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b") else v) for k, v in p.items()}
        ph["per_head"] = False
        assert np.allclose(a[:, h], o.attn_quadratic(Q[:, h], K[:, h], V[:, h], ph, eps=1e-6), rtol=1e-10, atol=1e-12)
        assert np.allclose(c[:, h], o.attn_quadratic(Q[:, h], K[:, h], V[:, h], ph, eps=1e-6, causal=True),
                           rtol=1e-10, atol=1e-12)


def pin_pwl_identity(o):
    """The ReLU MLP equals its piecewise-linear form on a dense grid and next to every breakpoint."""
    rng = np.random.default_rng(13)
    for shared, nonneg, hidden, L in ((False, True, 64, 8), (True, False, 64, 8), (False, False, 5, 3)):
        C1 = 1 if shared else L
        a = rng.standard_normal((C1, hidden)) * 0.125
        a[0, 0] = 0.0  # a unit without a breakpoint
        c = rng.standard_normal((C1, hidden)) * 0.125
        f = rng.standard_normal((L, hidden)) * 0.125
        g = rng.standard_normal(L) * 0.125
        tab = o.pwl_tables(a, c, f, g)
        bp = tab[0]
        assert bp.size == C1 * hidden - 1 and np.all(np.diff(bp) >= 0)
        u = np.concatenate([np.linspace(-8, 8, 4001), bp, np.nextafter(bp, np.inf), np.nextafter(bp, -np.inf),
                            [-1e6, 1e6]])
        want = o.psi(u, a, c, f, g, nonneg)
        got = o.psi_pwl(u, tab, nonneg)
        scale = np.maximum(1.0, np.abs(u))[:, None]
        assert np.max(np.abs(got - want) / scale) < 1e-12


# ---------------------------------------------------------------------------
# gradients
# ---------------------------------------------------------------------------

def _grad_problems(rng):
    """Tiny problems for the gradient pins: (causal, p, Q, K, V, dO), with per-channel
    and shared first layers, output ReLU on and off (denominators kept away from 0)."""
    out = []
    for causal in (False, True):
        for shared, nonneg in ((False, True), (True, False)):
            p = _params(rng, M=2, L=3, d=4, hidden=5, shared=shared, nonneg=nonneg, scale=0.7)
            if not nonneg:
                p["fc2_b"] = p["fc2_b"] + 2.0
            Q, K, V = _qkv(rng, (1, 2, 6, 4), dv=3)
            dO = rng.standard_normal((1, 2, 6, 3))
            out.append((causal, p, Q, K, V, dO))
    return out


def _grads(o, causal, p, Q, K, V, dO, eps):
    f = o.attn_causal_backward if causal else o.attn_noncausal_backward
    dQ, dK, dV, g = f(Q, K, V, p, dO, eps=eps)
    return {"Q": dQ, "K": dK, "V": dV, **g}


def pin_backward_finite_differences(o):
    """Every gradient of L = sum(dO * out) against central differences of the oracle's
    own forward pass (both forms, per-channel and shared first layers, output ReLU
    on and off), element by element."""
    rng = np.random.default_rng(21)
    eps, h = 1e-6, 1e-6
    for causal, p, Q, K, V, dO in _grad_problems(rng):
        fwd = o.attn_causal if causal else o.attn_noncausal
        g = _grads(o, causal, p, Q, K, V, dO, eps)
        inputs = {"Q": Q, "K": K, "V": V}

        def loss(inp, prm):
            return float((fwd(inp["Q"], inp["K"], inp["V"], prm, eps=eps) * dO).sum())

        for name in list(inputs) + ["W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b"]:
            base = inputs[name] if name in inputs else p[name]
            fd = np.zeros(np.shape(base))
            for idx in np.ndindex(*np.shape(base)):
                vals = []
                for sgn in (1.0, -1.0):
                    x = np.array(base, dtype=np.float64, copy=True)
                    x[idx] += sgn * h
                    inp, prm = dict(inputs), dict(p)
                    if name in inputs:
                        inp[name] = x
                    else:
                        prm[name] = x
                    vals.append(loss(inp, prm))
                fd[idx] = (vals[0] - vals[1]) / (2 * h)
            assert _rel(g[name], fd) < 1e-5, (causal, name, _rel(g[name], fd))


def _torch_forward(torch, Q, K, V, prm, causal, eps, nonneg):
    """The forward pass written with torch operations (float64, CPU), for autograd."""
    def phi(X):
        u = X @ prm["W"].T + prm["b"]
        shared = prm["fc1_w"].shape[0] == 1
        L = prm["fc2_w"].shape[0]
        chans = []
        for l in range(L):
            i = 0 if shared else l
            hid = torch.relu(u[..., None] * prm["fc1_w"][i] + prm["fc1_b"][i])
            y = hid @ prm["fc2_w"][l] + prm["fc2_b"][l]
            chans.append(torch.relu(y) if nonneg else y)
        y = torch.stack(chans, dim=-1)                       # [..., n, M, L]
        return y.reshape(y.shape[:-2] + (-1,)) / math.sqrt(prm["W"].shape[0])
    pq, pk = phi(Q), phi(K)
    if causal:
        S = torch.cumsum(pk[..., :, :, None] * V[..., :, None, :], dim=-3)   # [..., n, D, dv]
        z = torch.cumsum(pk, dim=-2)
        num = (pq[..., :, :, None] * S).sum(dim=-2)
        den = (pq * z).sum(dim=-1)
    else:
        S = pk.transpose(-1, -2) @ V
        z = pk.sum(dim=-2)
        num = pq @ S
        den = pq @ z[..., :, None]
        den = den[..., 0]
    return num / (den + eps)[..., None]


def pin_backward_matches_autograd(o):
    """The oracle's gradients against torch autograd of the forward written with torch
    operations (float64), including rows whose pre-activations are exactly 0, where both
    take ReLU'(0) = 0."""
    import torch
    rng = np.random.default_rng(22)
    eps = 1e-6
    problems = _grad_problems(rng)
    # kinks: x = 0 rows, b = 0 and c = 0 for one unit give pre-activations a u + c = 0
    causal, p, Q, K, V, dO = problems[0]
    p = dict(p)
    p["b"] = np.zeros_like(p["b"])
    p["fc1_b"] = p["fc1_b"].copy()
    p["fc1_b"][:, 0] = 0.0
    Q, K = Q.copy(), K.copy()
    Q[..., 1, :] = 0.0
    K[..., 2, :] = 0.0
    problems.append((causal, p, Q, K, V, dO))
    for causal, p, Q, K, V, dO in problems:
        g = _grads(o, causal, p, Q, K, V, dO, eps)
        t = {k: torch.tensor(np.asarray(v, dtype=np.float64), requires_grad=True)
             for k, v in (("Q", Q), ("K", K), ("V", V), *((n, p[n]) for n in ("W", "b", "fc1_w", "fc1_b", "fc2_w",
                                                                              "fc2_b")))}
        out = _torch_forward(torch, t["Q"], t["K"], t["V"], t, causal, eps, p["nonneg"])
        (out * torch.tensor(dO)).sum().backward()
        for name, tv in t.items():
            assert _rel(g[name], tv.grad.numpy()) < 1e-12, (causal, name, _rel(g[name], tv.grad.numpy()))


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
