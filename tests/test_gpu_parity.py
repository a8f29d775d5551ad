"""HIP path (through the C ABI) against the float64 oracle, element by element.

Small problems span several tiles, chunks and a ragged tail and are compared in
full; the five measured problems run at full size in the launch configuration the
benchmark times and are compared on sampled heads / rows.  Tolerance: normwise per
(b, h) slice, 1e-4 for fp32 and 2e-2 for bf16 inputs with fp32 accumulation.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from gpu_util import assert_close, assert_close_rows, inputs, oracle_per_batch, say, small_workload, to_np, upload
from paper_2512_08061_amd import luna
from paper_2512_08061_amd import workloads as wl

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    luna.load_library()
    yield
    torch.cuda.synchronize()


def _sync():
    import torch
    torch.cuda.synchronize()


# ---------------------------------------------------------------------------
# feature map
# ---------------------------------------------------------------------------

FM_CASES = [
    ("f32", 32, 8, 8, 100), ("f32", 64, 16, 8, 77), ("bf16", 64, 16, 8, 300), ("bf16", 128, 32, 8, 65),
    ("bf16", 64, 64, 1, 33), ("bf16", 32, 5, 4, 50), ("f32", 128, 3, 16, 20), ("bf16", 64, 8, 2, 1),
    ("bf16", 64, 128, 1, 70), ("bf16", 128, 256, 1, 33), ("f32", 32, 100, 2, 130),  # more than 64 projections
]


@pytest.mark.parametrize("dtype,d,M,L,n", FM_CASES)
def test_featuremap_small(dtype, d, M, L, n):
    w = small_workload(dtype, B=2, H=2, n=n, d=d, M=M, L=L, hidden=64 if L < 16 else 16)
    say(f"featuremap {w.name}")
    Q, K, V, p = inputs(w, seed=1)
    (Xt,), pt = upload(w, [Q], p)
    phi = to_np(luna.featuremap(Xt, pt))
    ref = oracle.featuremap(Q, p)
    assert_close(phi, ref, dtype, "phi")
    if dtype == "bf16":  # fp32 output from bf16 input is checked at the fp32 bar
        import torch
        phi32 = to_np(luna.featuremap(Xt, pt, out_dtype=torch.float32))
        assert_close(phi32, ref, "f32", "phi fp32 out")


@pytest.mark.parametrize("shared,nonneg", [(False, True), (True, False), (False, False)])
def test_featuremap_psi_sweep(shared, nonneg):
    """u swept over [-50, 50] and onto every breakpoint (and its fp32 neighbours):
    every segment of the piecewise-linear tables is hit."""
    w = small_workload("f32", B=1, H=1, n=8, d=32, M=1, L=8, shared_channels=shared, nonneg=nonneg)
    p = wl.make_params(w, seed=12)
    p = dict(p)
    p["W"] = np.zeros((1, 32), np.float32)
    p["W"][0, 0] = 1.0  # u = x_0 + b
    p["b"] = np.zeros(1, np.float32)
    a, c = p["fc1_w"].astype(np.float64), p["fc1_b"].astype(np.float64)
    bp = (-c / a).ravel().astype(np.float32)
    u = np.concatenate([np.linspace(-50, 50, 4001, dtype=np.float32), bp, np.nextafter(bp, np.float32(np.inf)),
                        np.nextafter(bp, np.float32(-np.inf)), np.float32([0, 1e-30, -1e-30, 1e4, -1e4])])
    X = np.zeros((1, 1, u.size, 32), np.float32)
    X[0, 0, :, 0] = u
    (Xt,), pt = upload(w.with_(n=u.size), [X], p)
    phi = to_np(luna.featuremap(Xt, pt))[0, 0]
    ref = oracle.featuremap(X[0, 0], p)
    err = np.abs(phi - ref) / np.maximum(1.0, np.abs(u.astype(np.float64)))[:, None]
    assert err.max() < 2e-6 * max(1.0, np.abs(ref).max()), err.max()


# bucket layout of the kernels' table search: magnitudes in [2^-BUCKET_EXP,
# 2^BUCKET_EXP) split by exponent and BUCKET_MANT mantissa bits
BUCKET_EXP, BUCKET_MANT = 6, 7


def _bucket_of(u):
    """Bucket index of each float32 u, in the kernels' order (sign, then magnitude)."""
    bits = np.asarray(u, np.float32).view(np.uint32).astype(np.int64)
    mag = (bits >> (23 - BUCKET_MANT)) & ((1 << (31 - 23 + BUCKET_MANT)) - 1)
    nmag = 2 * BUCKET_EXP * (1 << BUCKET_MANT) + 2
    m = np.clip(mag - ((127 - BUCKET_EXP) << BUCKET_MANT) + 1, 0, nmag - 1)
    return np.where(bits >> 31, nmag - 1 - m, nmag + m)


def _bucket_edges():
    """Every boundary of the float-bit buckets the kernels index the breakpoints by
    (powers of two and 2^-BUCKET_MANT mantissa steps over [2^-6, 2^6]), both signs,
    with the fp32 neighbours of each, plus zeros and denormals."""
    steps = 1 << BUCKET_MANT
    mags = [np.float32(2.0) ** e * np.float32(1 + k / steps) for e in range(-BUCKET_EXP, BUCKET_EXP)
            for k in range(steps)]
    mags.append(np.float32(64.0))
    mags = np.array(mags, np.float32)
    vals = np.concatenate([mags, np.nextafter(mags, np.float32(0)), np.nextafter(mags, np.float32(np.inf))])
    return np.concatenate([vals, -vals, np.float32([0.0, -0.0, 1e-40, -1e-40, 3e-39, -3e-39, 1e6, -1e6])])


def _featuremap_exact(p, u, shared=False, nonneg=True):
    w = small_workload("f32", B=1, H=1, n=u.size, d=32, M=1, L=p["L"], shared_channels=shared, nonneg=nonneg,
                       hidden=p["hidden"])
    p = dict(p)
    p["W"] = np.zeros((1, 32), np.float32)
    p["W"][0, 0] = 1.0  # u = x_0
    p["b"] = np.zeros(1, np.float32)
    X = np.zeros((1, 1, u.size, 32), np.float32)
    X[0, 0, :, 0] = u
    (Xt,), pt = upload(w, [X], p)
    phi = to_np(luna.featuremap(Xt, pt))[0, 0]
    ref = oracle.featuremap(X[0, 0], p)
    err = np.abs(phi - ref) / np.maximum(1.0, np.abs(u.astype(np.float64)))[:, None]
    assert err.max() < 2e-6 * max(1.0, np.abs(ref).max()), err.max()


@pytest.mark.parametrize("layout", ["random", "clustered", "all_equal", "wide", "zero_and_tiny"])
def test_featuremap_bucket_edges(layout):
    """psi at every bucket boundary (and its fp32 neighbours) and at every breakpoint,
    for breakpoint sets that leave buckets sparse, crowd one bucket, make all
    breakpoints equal, spread them over many decades, or sit at 0 and below 2^-6."""
    w = small_workload("f32", B=1, H=1, n=8, d=32, M=1, L=8)
    p = dict(wl.make_params(w, seed=21))
    rng = np.random.default_rng(22)
    a = p["fc1_w"].astype(np.float64).copy()
    if layout == "clustered":      # 300 of the 512 breakpoints inside [0.5, 0.5 + 1/128)
        beta = np.where(rng.random(a.shape) < 0.6, 0.5 + rng.random(a.shape) / 128, rng.standard_cauchy(a.shape))
    elif layout == "all_equal":
        beta = np.full(a.shape, -0.3)
    elif layout == "wide":
        beta = rng.choice([-1, 1], a.shape) * 10.0 ** rng.uniform(-9, 9, a.shape)
    elif layout == "zero_and_tiny":
        beta = np.where(rng.random(a.shape) < 0.5, 0.0, rng.uniform(-2 ** -6, 2 ** -6, a.shape))
    else:
        beta = -p["fc1_b"].astype(np.float64) / a
    p["fc1_b"] = (-beta * a).astype(np.float32)
    bp = (-p["fc1_b"].astype(np.float64) / p["fc1_w"].astype(np.float64)).ravel().astype(np.float32)
    bp = bp[np.isfinite(bp)]
    u = np.concatenate([_bucket_edges(), bp, np.nextafter(bp, np.float32(np.inf)), np.nextafter(bp, np.float32(-np.inf)),
                        np.linspace(-3, 3, 601, dtype=np.float32)])
    say(f"bucket edges {layout}: {u.size} values")
    _featuremap_exact(p, u)


@pytest.mark.parametrize("L,hidden,shared", [(1, 63, False), (8, 61, False), (16, 19, False), (16, 33, True),
                                             (4, 64, True)])
def test_featuremap_unit_counts(L, hidden, shared):
    """Tables built from odd and uneven numbers of hidden units (the rank sort's
    padded last pair, one or two units per thread), per-channel and shared first
    layers, at every breakpoint and its fp32 neighbours."""
    w = small_workload("f32", B=1, H=1, n=8, d=32, M=1, L=L, hidden=hidden, shared_channels=shared)
    p = dict(wl.make_params(w, seed=41))
    bp = (-p["fc1_b"].astype(np.float64) / p["fc1_w"].astype(np.float64)).ravel().astype(np.float32)
    bp = bp[np.isfinite(bp)]
    u = np.concatenate([bp, np.nextafter(bp, np.float32(np.inf)), np.nextafter(bp, np.float32(-np.inf)),
                        np.linspace(-4, 4, 401, dtype=np.float32)])
    say(f"unit counts L={L} hidden={hidden} shared={shared}: {u.size} values")
    _featuremap_exact(p, u, shared=shared)


def _breakpoints(p):
    bp = (-p["fc1_b"].astype(np.float64) / p["fc1_w"].astype(np.float64)).ravel().astype(np.float32)
    bp = bp[np.isfinite(bp)]
    return np.where(bp == 0, np.float32(0), bp)


@pytest.mark.parametrize("layout,most_range", [("spread", (1, 4)), ("six", (5, 8)), ("crowded", (9, 10 ** 6))])
def test_attn_causal_search_paths(layout, most_range):
    """The bf16 causal kernel's table search, on u placed exactly on breakpoints and
    at small offsets from them, for breakpoint layouts whose fullest bucket holds at
    most 4 keys (one 4-key group per search), 5 to 8 (two groups) or more (halving
    search).  W has one nonzero column, so u = x_0 + b exactly when x_0 = 0."""
    w = small_workload("bf16", B=1, H=2, n=200, d=128, M=32, L=8, causal=True)
    Q, K, V, p = inputs(w, seed=31)
    Q, K, p = Q.copy(), K.copy(), dict(p)
    rng = np.random.default_rng(32)
    a = p["fc1_w"].astype(np.float64).copy()
    beta = -p["fc1_b"].astype(np.float64) / a
    if layout == "six":     # six breakpoints of channel 0 inside one otherwise empty bucket near 37.3
        beta[0, :6] = 37.3 + 1e-3 * np.arange(6)
    elif layout == "crowded":  # three channels' breakpoints all inside one bucket near 0.3
        beta[:3] = 0.3 + 1e-5 * rng.random(beta[:3].shape)
    p["fc1_b"] = (-beta * a).astype(np.float32)
    bp = _breakpoints(p)
    most = np.bincount(_bucket_of(bp)).max()
    assert most_range[0] <= most <= most_range[1], most
    p["W"] = np.zeros_like(p["W"])
    p["W"][:, 0] = 1.0
    p["b"] = rng.choice(np.concatenate([bp, _bucket_edges()[::17]]), size=p["b"].shape).astype(np.float32)
    for X in (Q, K):
        X[..., 0] = rng.choice(np.float32([0, 0, 0, 2.0 ** -20, -2.0 ** -20, 2.0 ** -9, -2.0 ** -9, 0.75, -1.5]),
                               size=X.shape[:-1])
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=64, eps=w.eps))
    assert_close(out, oracle.attn_causal(Q, K, V, p, eps=w.eps), "bf16", f"search {layout}")


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_featuremap_workload_full_size(name):
    w = wl.WORKLOADS[name]
    say(f"featuremap full size {name}")
    Q, K, V, p = inputs(w, seed=0)
    (Qt,), pt = upload(w, [Q], p)
    phi = luna.featuremap(Qt, pt)
    _sync()
    rng = np.random.default_rng(5)
    for _ in range(2):
        b, h = int(rng.integers(w.B)), int(rng.integers(w.H))
        assert_close(to_np(phi[b, h]), oracle.featuremap(Q[b, h], p), w.dtype, f"phi[{b},{h}]")
    del phi


# ---------------------------------------------------------------------------
# non-causal attention
# ---------------------------------------------------------------------------

NC_CASES = [
    ("f32", 32, 8, 8), ("f32", 64, 16, 8), ("bf16", 32, 16, 8), ("bf16", 64, 8, 8), ("bf16", 64, 16, 8),
    ("bf16", 64, 32, 8), ("bf16", 64, 16, 4), ("bf16", 64, 64, 1), ("bf16", 128, 16, 8),
    # one channel per projection, M = D = 128 (fused); shapes on the fp32 GEMM path
    ("bf16", 64, 128, 1), ("bf16", 64, 100, 1), ("bf16", 128, 256, 1), ("f32", 128, 16, 8), ("f32", 64, 32, 4),
]


@pytest.mark.parametrize("dtype,d,M,L", NC_CASES)
@pytest.mark.parametrize("n", [1, 97, 600])
def test_attn_noncausal_small(dtype, d, M, L, n):
    w = small_workload(dtype, B=2, H=2, n=n, d=d, M=M, L=L)
    say(f"noncausal {w.name}")
    Q, K, V, p = inputs(w, seed=2)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd(Qt, Kt, Vt, pt, eps=w.eps))
    assert_close(out, oracle.attn_noncausal(Q, K, V, p, eps=w.eps), dtype, "out")


# enough heads for the one-pass kernel (one workgroup per head), with ragged lengths
@pytest.mark.parametrize("dtype,d,M,L,n", [("f32", 64, 16, 8, 77), ("bf16", 64, 16, 8, 333), ("bf16", 64, 8, 8, 1),
                                           ("bf16", 32, 16, 8, 200), ("f32", 32, 8, 2, 45),
                                           # at most 8 projections: half of the fused kernel's
                                           # 16-projection block is padding
                                           ("bf16", 64, 8, 8, 333), ("bf16", 32, 5, 8, 100), ("bf16", 64, 3, 8, 47),
                                           ("bf16", 64, 8, 8, 16), ("bf16", 64, 1, 8, 40)])
def test_attn_noncausal_many_heads(dtype, d, M, L, n):
    w = small_workload(dtype, B=16, H=13, n=n, d=d, M=M, L=L)
    say(f"noncausal many heads {w.name}")
    Q, K, V, p = inputs(w, seed=5)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd(Qt, Kt, Vt, pt, eps=w.eps))
    assert_close(out, oracle.attn_noncausal(Q, K, V, p, eps=w.eps), dtype, "out")


@pytest.mark.parametrize("name", ["tiny_f32", "text_encoder", "vision_encoder", "long_noncausal"])
def test_attn_noncausal_workload_full_size(name):
    """Every head of every non-causal workload, in the launch configuration the
    benchmark times, against the oracle's linear form."""
    w = wl.WORKLOADS[name]
    say(f"noncausal full size {name}: all {w.B * w.H} heads")
    Q, K, V, p = inputs(w, seed=0)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd(Qt, Kt, Vt, pt, eps=w.eps))
    ref = oracle_per_batch(oracle.attn_noncausal, Q, K, V, p, w.eps)
    assert_close(out, ref, w.dtype, "out, every head")
    if name == "tiny_f32":  # also against the O(n^2) kernel form
        ref = oracle.attn_quadratic(Q, K, V, p, eps=w.eps)
        assert_close(out, ref, w.dtype, "out vs kernel form")


# ---------------------------------------------------------------------------
# causal attention
# ---------------------------------------------------------------------------

CS_CASES = [
    ("f32", 32, 8, 8), ("f32", 64, 16, 8), ("bf16", 32, 16, 8), ("bf16", 64, 16, 8), ("bf16", 64, 32, 8),
    ("bf16", 128, 16, 8), ("bf16", 128, 32, 8),
    # one channel per projection (M = D = 256, 128: features mapped beforehand, then the
    # scan kernel); the fp32 GEMM path: fp32 at d = 128, L = 2 with M > 16, L = 4, 128 features at d = 128
    ("bf16", 128, 256, 1), ("bf16", 64, 128, 1), ("f32", 128, 16, 8), ("f32", 32, 24, 2), ("bf16", 64, 16, 4),
    ("bf16", 128, 128, 1),
]


@pytest.mark.parametrize("dtype,d,M,L", CS_CASES)
@pytest.mark.parametrize("n", [1, 64, 65, 333])
def test_attn_causal_small(dtype, d, M, L, n):
    w = small_workload(dtype, B=1, H=3, n=n, d=d, M=M, L=L, causal=True)
    say(f"causal {w.name}")
    Q, K, V, p = inputs(w, seed=3)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=64, eps=w.eps))
    assert_close_rows(out, oracle.attn_causal(Q, K, V, p, eps=w.eps), dtype, "out")


@pytest.mark.parametrize("M,L", [(32, 8), (256, 1)])
@pytest.mark.parametrize("B,H,n", [(1, 3, 1000), (4, 25, 650), (8, 20, 300)])
def test_attn_causal_state_pieces(B, H, n, M, L):
    """With fewer than 256 heads each head is cut at x (n/2 rounded down to whole
    chunks) and the state of [0, x) is summed in pieces, one workgroup per head and
    piece: seven one-chunk pieces (3 heads), two pieces (160 heads); 100 heads take the
    staged form (two scan launches) instead.
    Checked against the oracle on sampled heads (the parameters are shared).  M = 256,
    L = 1: the features are mapped beforehand and the kernel reads them."""
    w = small_workload("bf16", B=B, H=H, n=n, d=128, M=M, L=L, causal=True)
    say(f"causal state pieces B={B} H={H} n={n} M={M} L={L}")
    Q, K, V, p = inputs(w, seed=51)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=64, eps=w.eps))
    bs, hs = sorted({0, B - 1}), sorted({0, H // 2, H - 1})
    pick = lambda X: X[bs][:, hs]  # noqa: E731
    ref = oracle.attn_causal(pick(Q), pick(K), pick(V), p, eps=w.eps)
    assert_close_rows(pick(out), ref, "bf16", "out")


@pytest.mark.parametrize("dtype,d,M,B,H,n", [("bf16", 128, 32, 8, 16, 1000), ("bf16", 64, 16, 4, 25, 321),
                                               ("f32", 64, 16, 1, 100, 400), ("bf16", 128, 32, 2, 64, 4096)])
def test_attn_causal_staged(dtype, d, M, B, H, n):
    """97 to 128 heads: two scan launches, the first scanning chunks [0, A) beside a
    state-only part over [A, A + B), the second scanning [A, A + B) and [A + B, nch)
    from the exported states (A = nch / 5, B = C = 2 nch / 5).  Every row of sampled
    heads against the oracle's token recurrence, so that both part boundaries and the
    ragged last chunk are covered."""
    w = small_workload(dtype, B=B, H=H, n=n, d=d, M=M, L=8, causal=True)
    say(f"causal staged {dtype} d={d} M={M} B={B} H={H} n={n}")
    Q, K, V, p = inputs(w, seed=61)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=64, eps=w.eps))
    bs, hs = sorted({0, B - 1}), sorted({0, H // 3, H - 1})
    pick = lambda X: X[bs][:, hs]  # noqa: E731
    ref = oracle.attn_causal(pick(Q), pick(K), pick(V), p, eps=w.eps)
    assert_close_rows(pick(out), ref, dtype, "out")


def test_attn_causal_workload_full_size():
    w = wl.WORKLOADS["long_causal"]
    say("causal full size long_causal")
    Q, K, V, p = inputs(w, seed=0)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=w.chunk, eps=w.eps)
    _sync()
    # masked kernel form on the first 512 tokens of every head
    pre = 512
    got = to_np(out[:, :, :pre])
    for b in range(w.B):
        ref = oracle.attn_quadratic(Q[b, :, :pre], K[b, :, :pre], V[b, :, :pre], p, eps=w.eps, causal=True)
        assert_close_rows(got[b], ref, w.dtype, f"prefix b={b}")
    # whole sequences (every row of both parts of the split: the second starts from
    # the state pieces) of four heads, against the oracle's chunked scan (pinned to
    # the token recurrence and the masked kernel form)
    rng = np.random.default_rng(11)
    heads = [(0, 0), (w.B - 1, w.H - 1), (int(rng.integers(w.B)), int(rng.integers(w.H))), (3, 5)]
    full = to_np(out[[b for b, _ in heads], [h for _, h in heads]])
    for i, (b, h) in enumerate(heads):
        ref = oracle.attn_causal_chunked(Q[b, h], K[b, h], V[b, h], p, chunk=w.chunk, eps=w.eps)
        assert_close_rows(full[i], ref, w.dtype, f"all rows of ({b},{h})")
    # rows deep into the sequence, kernel form one row at a time
    for b, h in heads[:2]:
        rows = np.sort(np.concatenate([rng.integers(0, w.n, 12), [w.n - 1, 8191, 8192]]))
        ref = oracle.attn_quadratic_rows(Q[b, h], K[b, h], V[b, h], p, rows, eps=w.eps, causal=True)
        assert_close_rows(to_np(out[b, h, rows]), ref, w.dtype, f"rows of ({b},{h})")


def test_attn_noncausal_one_channel_full_size():
    """The one-channel variant of the long non-causal problem (L = 1, M = D = 128),
    every head, on the launch the benchmark times."""
    w = wl.WORKLOADS["long_noncausal"].with_(M=128, L=1)
    say(f"noncausal full size one-channel: all {w.B * w.H} heads")
    Q, K, V, p = inputs(w, seed=0)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd(Qt, Kt, Vt, pt, eps=w.eps))
    ref = oracle_per_batch(oracle.attn_noncausal, Q, K, V, p, w.eps)
    assert_close(out, ref, w.dtype, "out, every head")


def test_attn_causal_one_channel_full_size():
    """The one-channel variant of the long causal problem (L = 1, M = D = 256, fp32
    GEMM path): the masked kernel form on the first 512 tokens of every head, whole
    sequences of two heads against the chunked scan, and single rows deep in them."""
    w = wl.WORKLOADS["long_causal"].with_(M=256, L=1)
    say("causal full size one-channel")
    Q, K, V, p = inputs(w, seed=0)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=w.chunk, eps=w.eps)
    _sync()
    pre = 512
    got = to_np(out[:, :, :pre])
    for b in range(w.B):
        ref = oracle.attn_quadratic(Q[b, :, :pre], K[b, :, :pre], V[b, :, :pre], p, eps=w.eps, causal=True)
        assert_close_rows(got[b], ref, w.dtype, f"prefix b={b}")
    heads = [(0, 0), (w.B - 1, w.H - 1)]
    full = to_np(out[[b for b, _ in heads], [h for _, h in heads]])
    rng = np.random.default_rng(12)
    for i, (b, h) in enumerate(heads):
        ref = oracle.attn_causal_chunked(Q[b, h], K[b, h], V[b, h], p, chunk=w.chunk, eps=w.eps)
        assert_close_rows(full[i], ref, w.dtype, f"all rows of ({b},{h})")
        rows = np.sort(np.concatenate([rng.integers(0, w.n, 8), [w.n - 1]]))
        ref = oracle.attn_quadratic_rows(Q[b, h], K[b, h], V[b, h], p, rows, eps=w.eps, causal=True)
        assert_close_rows(to_np(out[b, h, rows]), ref, w.dtype, f"rows of ({b},{h})")


# ---------------------------------------------------------------------------
# hand-worked example, edge cases, options
# ---------------------------------------------------------------------------

def _golden_problem():
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    d = 32  # the example has d = 2; zero columns leave every projection unchanged
    pad = lambda x: np.pad(np.array(x, dtype=np.float32), ((0, 0), (0, d - 2)))  # noqa: E731
    Q, K, V = pad(g["Q"])[None, None], pad(g["K"])[None, None], pad(g["V"])[None, None]
    p = {"W": pad(g["W"]), "b": np.array(g["b"], np.float32), "fc1_w": np.array(g["fc1_w"], np.float32),
         "fc1_b": np.array(g["fc1_b"], np.float32), "fc2_w": np.array(g["fc2_w"], np.float32),
         "fc2_b": np.array(g["fc2_b"], np.float32), "M": 2, "L": 2, "hidden": 2}
    frac = lambda x: np.array([[float(Fraction(v)) for v in row] for row in x])  # noqa: E731
    return g, Q, K, V, p, frac


def test_golden_hand_example_on_gpu():
    g, Q, K, V, p, frac = _golden_problem()
    w = small_workload("f32", B=1, H=1, n=2, d=32, M=2, L=2, hidden=2)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    phi = to_np(luna.featuremap(Qt, pt))[0, 0]
    assert np.allclose(phi * math.sqrt(2), frac(g["phi_q_times_sqrtM"]), rtol=0, atol=1e-6)
    out = to_np(luna.attn_fwd(Qt, Kt, Vt, pt, eps=0.0))[0, 0, :, :2]
    assert np.allclose(out, frac(g["out_noncausal"]), rtol=0, atol=1e-6)
    outc = to_np(luna.attn_fwd_causal(Qt, Kt, Vt, pt, eps=0.0))[0, 0, :, :2]
    assert np.allclose(outc, frac(g["out_causal"]), rtol=0, atol=1e-6)


@pytest.mark.parametrize("causal", [False, True])
def test_zero_features_give_zero(causal):
    w = small_workload("bf16", B=1, H=2, n=70, d=64, M=16, L=8, causal=causal)
    Q, K, V, p = inputs(w, seed=4)
    p = dict(p)
    p["fc2_w"] = np.zeros_like(p["fc2_w"])
    p["fc2_b"] = -np.ones_like(p["fc2_b"])  # psi = relu(-1) = 0 everywhere
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    f = luna.attn_fwd_causal if causal else luna.attn_fwd
    out = to_np(f(Qt, Kt, Vt, pt, eps=1e-6))
    assert np.array_equal(out, np.zeros_like(out))


# (dtype, d, M, L): the fused kernels; one channel per projection (causal: features
# mapped first, then the scan kernel; non-causal: the fp32 GEMM path); fp32 at d = 128
# (the fp32 GEMM path)
OPTION_SHAPES = [("bf16", 64, 16, 8), ("bf16", 128, 256, 1), ("f32", 128, 16, 8)]


@pytest.mark.parametrize("dtype,d,M,L", OPTION_SHAPES)
@pytest.mark.parametrize("causal", [False, True])
def test_options_per_head_shared_signed(causal, dtype, d, M, L):
    # per-head parameters, one shared first layer, no output relu
    w = small_workload(dtype, B=2, H=3, n=150, d=d, M=M, L=L, causal=causal, per_head=True,
                       shared_channels=True, nonneg=False)
    say(f"options {w.name} causal={causal}")
    Q, K, V, p = inputs(w, seed=6)
    # keep denominators away from zero when features may be negative
    p = dict(p)
    p["fc2_b"] = p["fc2_b"] + 1.0
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    f = luna.attn_fwd_causal if causal else luna.attn_fwd
    out = to_np(f(Qt, Kt, Vt, pt, eps=w.eps))
    ref = (oracle.attn_causal if causal else oracle.attn_noncausal)(Q, K, V, p, eps=w.eps)
    (assert_close_rows if causal else assert_close)(out, ref, dtype, "options")
    phi = to_np(luna.featuremap(Qt, pt))
    assert_close(phi, oracle.featuremap(Q, p), dtype, "phi options")


@pytest.mark.parametrize("M", [8, 6])
def test_attn_noncausal_few_projections_options(M):
    """The fused kernel (208 heads) with at most 8 projections, so that half of its
    projection block is padding, with per-head parameters, one shared first layer and
    no output relu."""
    w = small_workload("bf16", B=16, H=13, n=150, d=64, M=M, L=8, per_head=True, shared_channels=True,
                       nonneg=False)
    say(f"few projections, options {w.name}")
    Q, K, V, p = inputs(w, seed=8)
    p = dict(p)
    p["fc2_b"] = p["fc2_b"] + 1.0  # denominators away from zero with signed features
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd(Qt, Kt, Vt, pt, eps=w.eps))
    assert_close(out, oracle.attn_noncausal(Q, K, V, p, eps=w.eps), "bf16", "few projections, options")


@pytest.mark.parametrize("per_head", [False, True])
def test_featuremap_many_tiles(per_head):
    """More 64-row tiles than workgroups (each workgroup loops over tiles, loading a
    table when the parameter set changes): 313 tiles per head, six heads; checked on
    sampled rows of every head."""
    w = small_workload("bf16", B=2, H=3, n=20000, d=64, M=16, L=8, per_head=per_head)
    say(f"featuremap many tiles per_head={per_head}")
    Q, K, V, p = inputs(w, seed=8)
    (Xt,), pt = upload(w, [Q], p)
    phi = to_np(luna.featuremap(Xt, pt))
    rows = np.concatenate([np.arange(0, 20000, 97), [19999]])
    assert_close(phi[:, :, rows], oracle.featuremap(Q[:, :, rows], p), "bf16", "phi sampled")


def test_nan_propagates():
    w = small_workload("f32", B=1, H=1, n=130, d=32, M=8, L=8)
    Q, K, V, p = inputs(w, seed=8)
    Q = Q.copy()
    Q[0, 0, 5, 3] = np.nan
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    out = to_np(luna.attn_fwd(Qt, Kt, Vt, pt))[0, 0]
    assert np.isnan(out[5]).all() and np.isfinite(np.delete(out, 5, axis=0)).all()
    K = K.copy()
    K[0, 0, 70, 0] = np.nan
    (Qt, Kt, Vt), pt = upload(w, [np.nan_to_num(Q), K, V], p)
    outc = to_np(luna.attn_fwd_causal(Qt, Kt, Vt, pt))[0, 0]
    assert np.isfinite(outc[:70]).all() and np.isnan(outc[70:]).all()


@pytest.mark.parametrize("causal", [False, True])
def test_deterministic(causal):
    w = small_workload("bf16", B=2, H=4, n=1100, d=64, M=16, L=8, causal=causal)
    Q, K, V, p = inputs(w, seed=9)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    f = luna.attn_fwd_causal if causal else luna.attn_fwd
    a = f(Qt, Kt, Vt, pt).clone()
    b = f(Qt, Kt, Vt, pt).clone()
    import torch
    assert torch.equal(a, b)
