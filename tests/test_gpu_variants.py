"""Feature-map variants and attention from given features (HIP path through the C
ABI) against the float64 oracle of the variants (oracle/luna_variants.py).

Inputs are rounded to the call's dtype before the oracle sees them (X and W), so
that the comparison measures the kernels' arithmetic.  Tolerances as everywhere:
normwise per (b, h) slice (per row for causal outputs), 1e-4 for fp32, 2e-2 for bf16.
"""
import math
import zlib

import numpy as np
import pytest

from gpu_util import assert_close, assert_close_rows, say, to_np, torch_dtype
from oracle import luna_variants as VAR
from paper_2512_08061_amd import luna

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    luna.load_library()
    yield
    torch.cuda.synchronize()


def _variant_params(rng, kind, M, d, L=4, hidden=16, act="relu", shared=False, nonneg=True, env=False, bank=False,
                    ch_rms=False, per_head=0):
    lead = (per_head,) if per_head else ()
    s = 1.0 / math.sqrt(d)
    p = {"kind": kind, "act": act, "M": M, "per_head": bool(per_head)}
    if kind == "performer":  # omega / d^(1/4), omega ~ N(0, I): unbiased for exp(x . y / sqrt(d))
        p["W"] = rng.standard_normal(lead + (M, d)) / d ** 0.25
        p["b"] = np.zeros(lead + (M,))
    elif kind in ("rff_cos", "rff_sincos"):
        p["W"] = rng.standard_normal(lead + (M, d)) * s
        p["b"] = rng.uniform(0, 2 * math.pi, lead + (M,))
    else:
        C1 = 1 if shared else L
        p.update(W=rng.standard_normal(lead + (M, d)) * s, b=rng.standard_normal(lead + (M,)) * s,
                 fc1_w=rng.standard_normal(lead + (C1, hidden)), fc1_b=rng.standard_normal(lead + (C1, hidden)),
                 fc2_w=rng.standard_normal(lead + (L, hidden)) * 0.3, fc2_b=rng.standard_normal(lead + (L,)) * 0.3 + 0.2,
                 L=L, hidden=hidden, nonneg=nonneg, shared_channels=shared)
        if env:
            p["env_w"] = rng.standard_normal(lead + (L, d)) * s
            p["env_b"] = rng.standard_normal(lead + (L,))
        if bank:
            p["bank"] = rng.standard_normal(lead + (L,))
        if ch_rms:
            p["ch_rms"], p["ch_rms_target"] = True, 0.05
    return p


def _upload_rounded(x, dtype):
    """x on the device in dtype, and the same values (rounded) for the oracle."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(torch_dtype(dtype)).contiguous()
    return t, to_np(t)


def _run_variant(p, X, dtype, out_dtype=None):
    import torch
    Xt, Xr = _upload_rounded(X, dtype)
    v = luna.PhiVariant.from_arrays(p, torch.device("cuda:0"), torch_dtype(dtype))
    q = dict(p, W=to_np(v.base.W))  # the oracle takes W as the device holds it
    got = to_np(luna.featuremap_variant(Xt, v, out_dtype))
    return got, VAR.featuremap_variant(Xr, q)


MAP_CASES = [  # (kind, act, dtype, d, M, options)
    ("rff_cos", "relu", "f32", 64, 40, {}), ("rff_cos", "relu", "bf16", 128, 128, {}),
    ("rff_sincos", "relu", "f32", 32, 24, {}), ("rff_sincos", "relu", "bf16", 64, 64, {}),
    ("performer", "relu", "f32", 64, 48, {}), ("performer", "relu", "bf16", 128, 256, {}),
    ("mlp", "relu", "f32", 64, 16, {}), ("mlp", "gelu", "f32", 64, 16, {}), ("mlp", "silu", "bf16", 64, 20, {}),
    ("mlp", "tanh", "f32", 128, 9, dict(shared=True, nonneg=False)),
    ("mlp", "gelu", "f32", 32, 16, dict(env=True)), ("mlp", "relu", "bf16", 64, 16, dict(env=True, shared=True)),
    ("mlp", "silu", "f32", 64, 33, dict(bank=True)), ("mlp", "relu", "f32", 64, 16, dict(env=True, bank=True)),
    ("mlp", "tanh", "f32", 64, 12, dict(per_head=3, env=True)),
    ("rff_sincos", "relu", "f32", 64, 16, dict(per_head=3)),
]


@pytest.mark.parametrize("kind,act,dtype,d,M,opts", MAP_CASES)
def test_featuremap_variant(kind, act, dtype, d, M, opts):
    say(f"variant map {kind} act={act} {dtype} d={d} M={M} {opts}")
    rng = np.random.default_rng(zlib.crc32(f"{kind}/{act}/{d}/{M}/{sorted(opts)}".encode()))
    p = _variant_params(rng, kind, M, d, act=act, **opts)
    X = rng.standard_normal((2, 3, 77, d))
    got, ref = _run_variant(p, X, dtype)
    assert_close(got, ref, dtype, "phi")
    if dtype == "bf16":  # fp32 output from bf16 input at the fp32 bar
        import torch
        got32, _ = _run_variant(p, X, dtype, torch.float32)
        assert_close(got32, ref, "f32", "phi, fp32 out")


@pytest.mark.parametrize("dtype,bank", [("f32", False), ("bf16", False), ("f32", True)])
def test_featuremap_variant_channel_rms(dtype, bank):
    """Listing 1's channel RMS over the whole call (two passes), with channels both
    above the target (scaled down) and below it (unchanged)."""
    say(f"variant channel RMS {dtype} bank={bank}")
    rng = np.random.default_rng(41)
    p = _variant_params(rng, "mlp", 16, 64, L=4, act="gelu", ch_rms=True, bank=bank)
    p["fc2_b"] = np.array([2.0, 0.01, 0.5, 0.0])  # channel 0 large, channel 1 tiny
    p["ch_rms_target"] = 0.3
    X = rng.standard_normal((2, 3, 200, 64))
    got, ref = _run_variant(p, X, dtype)
    assert_close(got, ref, dtype, "phi with channel RMS")


ATTN_CASES = [  # (feature dtype, value dtype, d, D, n, causal)
    ("f32", "f32", 64, 64, 97, False), ("f32", "f32", 64, 100, 333, True), ("bf16", "bf16", 128, 256, 700, False),
    ("bf16", "bf16", 128, 256, 1000, True), ("bf16", "bf16", 64, 128, 333, True), ("bf16", "f32", 32, 48, 129, True),
    ("f32", "bf16", 128, 256, 65, True),
]


@pytest.mark.parametrize("fdt,vdt,d,D,n,causal", ATTN_CASES)
def test_attn_from_features(fdt, vdt, d, D, n, causal):
    """Positive random features (exp of a Gaussian projection), so that denominators
    stay away from 0; the bf16 causal cases with (d, D) = (128, 256) and (64, 128) run
    on the causal scan kernel (with state pieces at n >= 256), the others on the fp32
    GEMM path."""
    say(f"attention from features {fdt}/{vdt} d={d} D={D} n={n} causal={causal}")
    rng = np.random.default_rng(42 + n)
    B, H = 2, 3
    fq = np.exp(rng.standard_normal((B, H, n, D)) * 0.5) / math.sqrt(D)
    fk = np.exp(rng.standard_normal((B, H, n, D)) * 0.5) / math.sqrt(D)
    V = rng.standard_normal((B, H, n, d))
    (tq, rq), (tk, rk), (tv, rv) = (_upload_rounded(a, dt) for a, dt in ((fq, fdt), (fk, fdt), (V, vdt)))
    got = to_np(luna.attn_fwd_features(tq, tk, tv, causal=causal))
    ref = VAR.attn_from_features(rq, rk, rv, causal=causal)
    tol_dt = "f32" if (fdt == "f32" and vdt == "f32") else "bf16"
    (assert_close_rows if causal else assert_close)(got, ref, tol_dt, "out")


@pytest.mark.parametrize("kind,causal", [("performer", False), ("performer", True), ("rff_sincos", True),
                                         ("mlp", False)])
def test_variant_attention_end_to_end(kind, causal):
    """A variant map of Q and K, then attention from the features, against the oracle's
    composition.  The sin/cos features are taken at small inputs, where the kernel
    cos(u_x - u_y) stays near 1 (positive denominators)."""
    import torch
    say(f"variant attention {kind} causal={causal}")
    rng = np.random.default_rng(43)
    B, H, n, d = 2, 2, 150, 64
    p = _variant_params(rng, kind, 32, d, L=4, act="silu", env=(kind == "mlp"))
    scale = 0.2 if kind == "rff_sincos" else 0.7
    Q, K = rng.standard_normal((B, H, n, d)) * scale, rng.standard_normal((B, H, n, d)) * scale
    V = rng.standard_normal((B, H, n, d))
    v = luna.PhiVariant.from_arrays(p, torch.device("cuda:0"), torch.float32)
    tq, tk, tv = (torch.from_numpy(a).float().cuda().contiguous() for a in (Q, K, V))
    out = to_np(luna.attn_fwd_features(luna.featuremap_variant(tq, v), luna.featuremap_variant(tk, v), tv,
                                       causal=causal))
    ref = VAR.attn_from_features(VAR.featuremap_variant(Q, p), VAR.featuremap_variant(K, p), V, causal=causal)
    (assert_close_rows if causal else assert_close)(out, ref, "f32", "out")


def test_features_of_the_base_map():
    """luna_featuremap's own output through attention from features equals luna_attn_fwd
    (the same eq. (9) on the same features, to the bf16 bar)."""
    import torch
    from gpu_util import inputs, small_workload, upload
    w = small_workload("bf16", B=2, H=3, n=300, d=64, M=16, L=8)
    Q, K, V, p = inputs(w, seed=44)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    f32 = torch.float32
    out = to_np(luna.attn_fwd_features(luna.featuremap(Qt, pt, f32), luna.featuremap(Kt, pt, f32), Vt))
    assert_close(out, to_np(luna.attn_fwd(Qt, Kt, Vt, pt)), "bf16", "features vs fused")
