"""The backward pass (luna_attn_bwd) on the GPU, through the C ABI, against the float64
oracle's gradients (pinned to finite differences and to autograd): dQ, dK, dV per
(b, h) slice and every feature-map parameter gradient, non-causal and causal, with
ragged chunk tails, per-channel and shared first layers, per-head parameters and the
output ReLU off.  Tolerance: normwise, 1e-4 for fp32 and 2e-2 for bf16 inputs."""
import numpy as np
import pytest

import oracle
from gpu_util import TOL, assert_close, inputs, say, small_workload, to_np, upload
from paper_2512_08061_amd import luna

pytestmark = pytest.mark.gpu

NAMES = ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    luna.load_library()
    yield
    torch.cuda.synchronize()


def _check(w, seed, causal, **opt):
    import torch
    Q, K, V, p = inputs(w, seed=seed)
    if not w.nonneg:  # keep denominators away from zero when features may be negative
        p = dict(p)
        p["fc2_b"] = p["fc2_b"] + 1.0
    rng = np.random.default_rng(seed + 100)
    dO = rng.standard_normal(Q.shape).astype(np.float32)
    if w.dtype == "bf16":
        from paper_2512_08061_amd import workloads as wl
        dO = wl.round_bf16(dO)
    (Qt, Kt, Vt, dOt), pt = upload(w, [Q, K, V, dO], p)
    dQ, dK, dV, g = luna.attn_bwd(Qt, Kt, Vt, dOt, pt, causal=causal, eps=w.eps)
    f = oracle.attn_causal_backward if causal else oracle.attn_noncausal_backward
    rQ, rK, rV, rg = f(Q, K, V, p, dO, eps=w.eps)
    tol = TOL[w.dtype]
    errs = {}
    grads_qkv = (("dQ", dQ, rQ), ("dK", dK, rK), ("dV", dV, rV))
    scales = {}
    if w.n == 1:
        # One token: out = a v / (a + eps) with a = phi(q).phi(k), so every gradient but
        # dV is of the order of eps / a, the difference of two terms of dphi (dnum S^T and
        # dden z^T for the query; dS v and dz for the key), each of the order of 1 / a.
        # Those errors are bounded against the size of the first term's contribution.
        phiQ, phiK = oracle.featuremap(Q, p), oracle.featuremap(K, p)
        S, z = oracle.sufficient_statistics(phiK, V)
        den = (phiQ @ z[..., :, None])[..., 0] + w.eps
        dnum = np.asarray(dO, np.float64) / den[..., None]
        dS = np.swapaxes(phiQ, -1, -2) @ dnum
        gq = oracle.featuremap_backward(Q, p, dnum @ np.swapaxes(S, -1, -2))
        gk = oracle.featuremap_backward(K, p, np.asarray(V, np.float64) @ np.swapaxes(dS, -1, -2))
        scales = {"dQ": np.abs(gq[0]).max(), "dK": np.abs(gk[0]).max()}
        scales.update({name: np.abs(gq[1][name]).max() + np.abs(gk[1][name]).max() for name in NAMES})
        for name, got, ref in grads_qkv[:2]:
            err = np.abs(to_np(got) - ref).max() / scales[name]
            errs[name] = float(err)
            assert err <= tol, f"{name} (one token): error {err:.3e} of the terms' size > {tol}"
        grads_qkv = grads_qkv[2:]
    for name, got, ref in grads_qkv:
        errs[name] = assert_close(to_np(got), ref, w.dtype, name)
    for name in NAMES:
        got, ref = to_np(g[name]).ravel(), np.asarray(rg[name], np.float64).ravel()
        err = np.abs(got - ref).max() / max(scales.get(name, np.abs(ref).max()), 1e-30)
        errs[name] = float(err)
        assert np.isfinite(got).all() and err <= tol, f"d{name}: normwise error {err:.3e} > {tol}"
    say("  " + ", ".join(f"{k} {v:.1e}" for k, v in errs.items()))


CASES = [  # (dtype, d, M, L, n)
    ("f32", 32, 8, 8, 1), ("f32", 32, 8, 8, 37), ("f32", 64, 16, 8, 130), ("f32", 128, 32, 8, 70),
    ("f32", 64, 64, 1, 65), ("f32", 64, 8, 4, 200), ("bf16", 64, 16, 8, 333), ("bf16", 128, 32, 8, 150),
    ("bf16", 128, 256, 1, 100), ("f32", 64, 128, 1, 70),  # one channel per projection, M = D
]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dtype,d,M,L,n", CASES)
def test_attn_bwd(dtype, d, M, L, n, causal):
    w = small_workload(dtype, B=2, H=2, n=n, d=d, M=M, L=L, causal=causal)
    say(f"backward {'causal' if causal else 'non-causal'} {w.name}")
    _check(w, seed=31 + n, causal=causal)


@pytest.mark.parametrize("causal", [False, True])
def test_attn_bwd_options(causal):
    """Per-head parameters, one shared first layer, no output ReLU."""
    w = small_workload("f32", B=2, H=3, n=90, d=64, M=16, L=8, causal=causal, per_head=True, shared_channels=True,
                       nonneg=False)
    say(f"backward options causal={causal}")
    _check(w, seed=37, causal=causal)


def test_attn_bwd_rejects_bad_arguments():
    import torch
    w = small_workload("f32", B=1, H=1, n=8, d=64, M=16, L=8)
    Q, K, V, p = inputs(w, seed=1)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    with pytest.raises(luna.LunaError):
        luna.attn_bwd(Qt, Kt, Vt, Qt[..., :32].contiguous(), pt)
    with pytest.raises(luna.LunaError):
        luna.attn_bwd(Qt, Kt, Vt, Qt.to(torch.bfloat16), pt)
