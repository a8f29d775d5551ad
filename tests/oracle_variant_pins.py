"""Pins of the feature-map variants of the oracle (oracle/luna_variants.py) to what
the paper and the mathematics fix: the kernels that random Fourier and Performer
features estimate (closed forms, Monte Carlo within its error), the cos(a - b)
identity of sin/cos features, special cases that reduce to the pinned base map,
values worked out by hand.  Each pin takes the variants module."""

from __future__ import annotations

import math

import numpy as np

from oracle import luna_oracle as base


def _rel(a, b):
    a, b = np.asarray(a, float), np.asarray(b, float)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def _mlp_params(rng, M, L, d, hidden=8, shared=False, nonneg=True):
    s = 1.0 / math.sqrt(d)
    C1 = 1 if shared else L
    return {"kind": "mlp", "W": rng.standard_normal((M, d)) * s, "b": rng.standard_normal(M) * s,
            "fc1_w": rng.standard_normal((C1, hidden)), "fc1_b": rng.standard_normal((C1, hidden)),
            "fc2_w": rng.standard_normal((L, hidden)) * s, "fc2_b": rng.standard_normal(L) * s + 0.5,
            "M": M, "L": L, "hidden": hidden, "nonneg": nonneg, "shared_channels": shared, "per_head": False}


def pin_rff_cos_estimates_gaussian_kernel(v):
    """Section 3.1: with w_i ~ N(0, sigma^2 I) and phases b_i ~ U(0, 2 pi), E[phi(x) . phi(y)]
    = exp(-sigma^2 |x - y|^2 / 2) (the Gaussian kernel, Bochner); Monte Carlo with M =
    40000 features lands within 5 standard errors (the variance of 2 cos a cos b is <= 2)."""
    rng = np.random.default_rng(31)
    d, M, sigma = 6, 40000, 0.7
    p = {"W": rng.standard_normal((M, d)) * sigma, "b": rng.uniform(0, 2 * math.pi, M)}
    X = rng.standard_normal((5, d)) * 0.8
    phi = v.rff_cos(X, p)
    est = phi @ phi.T
    diff = X[:, None, :] - X[None, :, :]
    exact = np.exp(-0.5 * sigma ** 2 * (diff ** 2).sum(-1))
    assert np.max(np.abs(est - exact)) < 5 * math.sqrt(2.0 / M), np.max(np.abs(est - exact))
    # one feature by hand: W = [[1, 0]], b = [pi / 3], x = (pi / 6, 5): sqrt(2) cos(pi / 2) = 0
    one = v.rff_cos(np.array([[math.pi / 6, 5.0]]), {"W": np.array([[1.0, 0.0]]), "b": np.array([math.pi / 3])})
    assert abs(one[0, 0]) < 1e-15
    two = v.rff_cos(np.array([[0.0, 0.0]]), {"W": np.ones((2, 2)), "b": np.zeros(2)})
    assert np.allclose(two, 1.0)  # sqrt(2/2) cos 0 = 1


def pin_rff_sincos_cos_difference(v):
    """sin a sin b + cos a cos b = cos(a - b): the sin/cos map's kernel is exactly
    (1/M) sum_i cos(u_i(x) - u_i(y)), with the sin feature first in each pair."""
    rng = np.random.default_rng(32)
    d, M = 5, 7
    p = {"W": rng.standard_normal((M, d)), "b": rng.standard_normal(M)}
    X, Y = rng.standard_normal((4, d)), rng.standard_normal((3, d))
    ux, uy = X @ p["W"].T + p["b"], Y @ p["W"].T + p["b"]
    kern = np.cos(ux[:, None, :] - uy[None, :, :]).mean(-1)
    assert _rel(v.rff_sincos(X, p) @ v.rff_sincos(Y, p).T, kern) < 1e-13
    # layout by hand: u = (pi/2, pi/6) gives features (sin, cos) of u_0, then of u_1:
    # (1, 0, 1/2, sqrt(3)/2) / sqrt(2)
    f = v.rff_sincos(np.zeros((1, d)), {"W": np.zeros((2, d)), "b": np.array([math.pi / 2, math.pi / 6])})
    assert np.max(np.abs(f[0] * math.sqrt(2) - np.array([1.0, 0.0, 0.5, math.sqrt(3) / 2]))) < 1e-15


def pin_performer_estimates_exp_kernel(v):
    """Section 3.1: Performer features with w_i = omega_i / d^(1/4), omega_i ~ N(0, I)
    give E[phi(x) . phi(y)] = exp(x . y / sqrt(d)) (a Gaussian moment); Monte Carlo
    within 6 standard errors, estimated from the samples themselves; positive features."""
    rng = np.random.default_rng(33)
    d, M = 4, 60000
    p = {"W": rng.standard_normal((M, d)) / d ** 0.25, "b": np.zeros(M)}
    X = rng.standard_normal((4, d)) * 0.6
    phi = v.performer(X, p)
    assert (phi > 0).all()
    est = phi @ phi.T
    exact = np.exp(X @ X.T / math.sqrt(d))
    terms = (phi[:, None, :] * phi[None, :, :]) * M  # per-sample products, mean = est
    se = terms.std(axis=-1) / math.sqrt(M)
    assert (np.abs(est - exact) < 6 * se + 1e-12).all(), np.max(np.abs(est - exact) / se)
    # by hand: d = 4, x = (1, 1, 1, 1), one projection w = 0, b = 0: exp(-4 / (2 * 2)) = e^-1
    one = v.performer(np.ones((1, 4)), {"W": np.zeros((1, 4)), "b": np.zeros(1)})
    assert abs(one[0, 0] - math.exp(-1.0)) < 1e-15


def pin_activations_by_hand(v):
    """The hidden activations at points with known values: gelu(1) = Phi(1) =
    0.8413447460685429, gelu(-1) = -0.15865525393145707 (normal table), silu(1) =
    1 / (1 + e^-1) = 0.7310585786300049, silu(2) = 2 / (1 + e^-2) = 1.7615941559557646,
    tanh(0.5) = 0.46211715726000974; relu
    through the activation path equals the pinned ReLU channel MLPs."""
    z = np.array([1.0, -1.0])
    assert _rel(v._act("gelu", z), [0.8413447460685429, -0.15865525393145707]) < 1e-15
    assert _rel(v._act("silu", np.array([1.0, 2.0])), [0.7310585786300049, 1.7615941559557646]) < 1e-15
    assert abs(v._act("tanh", np.array([0.5]))[0] - 0.46211715726000974) < 1e-15
    rng = np.random.default_rng(34)
    p = _mlp_params(rng, 3, 4, 5)
    X = rng.standard_normal((6, 5))
    assert _rel(v.mlp_variant(X, p), base.featuremap(X, p)) < 1e-14
    # one tanh unit by hand: psi(u) = g + f tanh(a u + c) with a = 2, c = -1, f = 3, g = 0.25
    q = {"W": np.array([[1.0]]), "b": np.array([0.0]), "fc1_w": np.array([[2.0]]), "fc1_b": np.array([[-1.0]]),
         "fc2_w": np.array([[3.0]]), "fc2_b": np.array([0.25]), "nonneg": False, "act": "tanh"}
    got = v.mlp_variant(np.array([[0.75]]), q)[0, 0]
    assert abs(got - (0.25 + 3.0 * 0.46211715726000974)) < 1e-14  # tanh(0.5)


def pin_envelope_special_cases(v):
    """Table 5's envelope-gated map h(x) (.) psi(x): with G = 0 the envelope is
    sigmoid(c); c = 0 halves every feature, a large c leaves the base map, a very
    negative c removes it; one channel's envelope by hand."""
    rng = np.random.default_rng(35)
    M, L, d = 3, 4, 6
    p = _mlp_params(rng, M, L, d)
    X = rng.standard_normal((5, d))
    base_phi = base.featuremap(X, p)
    q = dict(p, env_w=np.zeros((L, d)), env_b=np.zeros(L))
    assert _rel(v.mlp_variant(X, q), 0.5 * base_phi) < 1e-14
    q = dict(p, env_w=np.zeros((L, d)), env_b=np.full(L, 60.0))
    assert _rel(v.mlp_variant(X, q), base_phi) < 1e-14
    q = dict(p, env_w=np.zeros((L, d)), env_b=np.full(L, -800.0))
    assert np.max(np.abs(v.mlp_variant(X, q))) == 0.0
    # channel 1 gated by sigmoid(x_0) with x_0 = ln 3: 3/4 of the base value; the others by 1/2
    G = np.zeros((L, d))
    G[1, 0] = 1.0
    x = np.zeros((1, d))
    x[0, 0] = math.log(3.0)
    got = v.mlp_variant(x, dict(p, env_w=G, env_b=np.zeros(L))).reshape(M, L)
    ref = base.featuremap(x, p).reshape(M, L)
    assert _rel(got[:, 1], 0.75 * ref[:, 1]) < 1e-14 and _rel(got[:, 0], 0.5 * ref[:, 0]) < 1e-14


def pin_bank_coef_selects_and_mixes(v):
    """Table 5's Bank+Coef map sum_l w_l phi_l(x): a one-hot w picks channel l of the
    base map for every projection, and the map is linear in w."""
    rng = np.random.default_rng(36)
    M, L, d = 4, 3, 5
    p = _mlp_params(rng, M, L, d)
    X = rng.standard_normal((6, d))
    ref = base.featuremap(X, p).reshape(6, M, L)
    for l in range(L):
        w = np.zeros(L)
        w[l] = 1.0
        assert _rel(v.mlp_variant(X, dict(p, bank=w)), ref[:, :, l]) < 1e-14
    w1, w2 = rng.standard_normal(L), rng.standard_normal(L)
    mix = v.mlp_variant(X, dict(p, bank=2 * w1 - w2))
    assert _rel(mix, 2 * v.mlp_variant(X, dict(p, bank=w1)) - v.mlp_variant(X, dict(p, bank=w2))) < 1e-12


def pin_channel_rms(v):
    """Listing 1's ch_rms by hand: channel values y = (3, 4) over two positions have
    rms sqrt(12.5 + 1e-6); target 0.5 scales them by 0.5 / (rms + 1e-6); a channel
    whose rms is below the target is unchanged; after scaling the rms is the target
    up to the eps terms."""
    y = np.zeros((2, 1, 2))
    y[:, 0, 0] = [3.0, 4.0]
    y[:, 0, 1] = [0.01, 0.02]
    out = v.ch_rms(y, 0.5)
    rms0 = math.sqrt(12.5 + 1e-6)
    assert _rel(out[:, 0, 0], np.array([3.0, 4.0]) * (0.5 / (rms0 + 1e-6))) < 1e-15
    assert np.array_equal(out[:, 0, 1], y[:, 0, 1])
    assert abs(math.sqrt((out[:, 0, 0] ** 2).mean()) - 0.5) < 1e-6
    # through the map: pooled over tokens and projections (and every head), per channel
    rng = np.random.default_rng(37)
    p = _mlp_params(rng, 3, 2, 4)
    X = rng.standard_normal((2, 3, 8, 4))  # [B, H, n, d]
    q = dict(p, ch_rms=True, ch_rms_target=0.05)
    got = v.mlp_variant(X, q).reshape(2, 3, 8, 3, 2) * math.sqrt(3)
    yb = base.featuremap(X, p).reshape(2, 3, 8, 3, 2) * math.sqrt(3)
    rms = np.sqrt((yb.reshape(-1, 2) ** 2).mean(0) + 1e-6)
    assert _rel(got, yb * np.minimum(0.05 / (rms + 1e-6), 1.0)) < 1e-14


def pin_attention_from_features(v):
    """eq. (9) of Section 3.1 for given features equals the pinned oracle on the base
    map's features (both forms), and for signed features (sin/cos) the quadratic kernel
    form computed by brute force."""
    rng = np.random.default_rng(38)
    p = _mlp_params(rng, 3, 4, 5)
    Q, K, V = rng.standard_normal((2, 9, 5)), rng.standard_normal((2, 9, 5)), rng.standard_normal((2, 9, 3))
    fq, fk = base.featuremap(Q, p), base.featuremap(K, p)
    assert _rel(v.attn_from_features(fq, fk, V), base.attn_noncausal(Q, K, V, p)) < 1e-13
    assert _rel(v.attn_from_features(fq, fk, V, causal=True), base.attn_causal(Q, K, V, p)) < 1e-13
    r = {"W": rng.standard_normal((6, 5)) * 0.2, "b": rng.standard_normal(6) * 0.2}
    fq, fk = v.rff_sincos(Q[0], r), v.rff_sincos(K[0], r)
    A = np.cos((Q[0] @ r["W"].T + r["b"])[:, None, :] - (K[0] @ r["W"].T + r["b"])[None, :, :]).mean(-1)
    for causal in (False, True):
        Am = np.tril(A) if causal else A
        ref = (Am @ V[0]) / (Am.sum(-1) + 1e-6)[:, None]
        assert _rel(v.attn_from_features(fq, fk, V[0], causal=causal), ref) < 1e-12


def pin_per_head_variants(v):
    """Per-head parameters: head h of the output equals the map with head h's
    parameters, for every kind."""
    rng = np.random.default_rng(39)
    H, M, L, d = 3, 2, 2, 4
    X = rng.standard_normal((2, H, 5, d))
    heads = [_mlp_params(rng, M, L, d) for _ in range(H)]
    stacked = {k: np.stack([h[k] for h in heads]) for k in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")}
    stacked.update({k: heads[0][k] for k in ("M", "L", "hidden", "nonneg", "shared_channels")}, per_head=True)
    stacked["env_w"] = rng.standard_normal((H, L, d))
    stacked["env_b"] = rng.standard_normal((H, L))
    for kind in ("mlp", "rff_cos", "rff_sincos", "performer"):
        q = dict(stacked, kind=kind)
        got = v.featuremap_variant(X, q)
        for h in range(H):
            one = dict(heads[h], kind=kind, env_w=stacked["env_w"][h], env_b=stacked["env_b"][h])
            assert _rel(got[:, h], v.featuremap_variant(X[:, h], one)) < 1e-14, kind


ALL_PINS = [f for k, f in sorted(globals().items()) if k.startswith("pin_")]
