"""The streaming form of causal attention on the GPU, through the C ABI, against the
float64 oracle: the causal state of a sequence (luna_attn_state) and the recurrent
step over new tokens (luna_attn_causal_step), alone and chained (state of a prefix,
then steps), with ragged step sizes, one-token decode and partial last chunks.
Tolerance: normwise per (b, h) slice, 1e-4 for fp32 and 2e-2 for bf16 inputs."""
import numpy as np
import pytest

import oracle
from gpu_util import assert_close, assert_close_rows, inputs, say, small_workload, to_np, upload
from paper_2512_08061_amd import luna

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    luna.load_library()
    yield
    torch.cuda.synchronize()


def _col(z):
    """z [..., D] as [..., D, 1], so that the normwise check runs per (b, h)."""
    return np.asarray(z)[..., None]


# (dtype, d, M, L, n, B, H): the first ones take the non-causal state pass, the
# (bf16, 128, 32, 8) ones the causal kernel's state launch (pieces, then export), the
# last ones the fp32 GEMM path
STATE_CASES = [
    ("f32", 32, 8, 8, 100, 2, 3), ("f32", 64, 16, 8, 65, 1, 2), ("bf16", 64, 16, 8, 300, 2, 3),
    ("bf16", 64, 32, 8, 130, 1, 3), ("bf16", 64, 64, 1, 97, 1, 2),
    ("bf16", 128, 32, 8, 1, 2, 2), ("bf16", 128, 32, 8, 64, 1, 3), ("bf16", 128, 32, 8, 200, 1, 1),
    ("bf16", 128, 32, 8, 700, 2, 5),
    # the fp32 GEMM path (512-token pieces, the last ragged)
    ("bf16", 128, 256, 1, 1100, 2, 3), ("f32", 128, 16, 8, 600, 1, 2), ("bf16", 64, 100, 1, 97, 1, 2),
]


@pytest.mark.parametrize("dtype,d,M,L,n,B,H", STATE_CASES)
def test_attn_state(dtype, d, M, L, n, B, H):
    import torch
    w = small_workload(dtype, B=B, H=H, n=n, d=d, M=M, L=L, causal=True)
    say(f"state {w.name} B={B} H={H}")
    Q, K, V, p = inputs(w, seed=7)
    (Kt, Vt), pt = upload(w, [K, V], p)
    S, z = luna.attn_state(Kt, Vt, pt)
    Sr, zr = oracle.causal_state(K, V, p)
    assert_close(to_np(S), Sr, dtype, "S")
    assert_close(_col(to_np(z)), _col(zr), dtype, "z")
    # accumulate onto a given state: S0 + state
    rng = np.random.default_rng(1)
    S0 = rng.standard_normal(Sr.shape) * np.abs(Sr).max()
    z0 = np.abs(rng.standard_normal(zr.shape)) * np.abs(zr).max()
    St = torch.from_numpy(S0).float().cuda().contiguous()
    zt = torch.from_numpy(z0).float().cuda().contiguous()
    luna.attn_state(Kt, Vt, pt, St, zt, accumulate=True)
    assert_close(to_np(St), S0 + Sr, dtype, "S accumulated")
    assert_close(_col(to_np(zt)), _col(z0 + zr), dtype, "z accumulated")


# (dtype, d, M, L, n, m): every step but the last has m tokens; steps of 16 tokens or
# more run on the matrix cores (stages of 16 tokens, the last ragged), shorter ones on
# the VALU
STEP_CASES = [
    ("f32", 32, 8, 8, 37, 5), ("f32", 64, 16, 8, 20, 1), ("bf16", 64, 16, 8, 100, 16), ("bf16", 128, 32, 8, 70, 33),
    ("bf16", 32, 5, 4, 20, 1), ("bf16", 64, 64, 4, 40, 17), ("bf16", 128, 3, 8, 9, 4),
    ("f32", 32, 8, 8, 37, 16), ("bf16", 32, 5, 4, 40, 16), ("f32", 128, 32, 8, 50, 64), ("bf16", 64, 7, 2, 30, 8),
    ("bf16", 64, 7, 2, 45, 22),
]


@pytest.mark.parametrize("dtype,d,M,L,n,m", STEP_CASES)
def test_causal_step_from_zero(dtype, d, M, L, n, m):
    """Steps of m tokens from the empty prefix give the causal form and, at the end,
    the state of the whole sequence."""
    import torch
    w = small_workload(dtype, B=2, H=2, n=n, d=d, M=M, L=L, causal=True)
    say(f"step {w.name} m={m}")
    Q, K, V, p = inputs(w, seed=11)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    D = M * L
    S = torch.zeros((2, 2, D, d), dtype=torch.float32, device="cuda")
    z = torch.zeros((2, 2, D), dtype=torch.float32, device="cuda")
    outs = []
    for a in range(0, n, m):
        b = min(n, a + m)
        sl = lambda X: X[:, :, a:b].contiguous()  # noqa: E731
        outs.append(to_np(luna.attn_causal_step(sl(Qt), sl(Kt), sl(Vt), pt, S, z, eps=w.eps)))
    out = np.concatenate(outs, axis=2)
    assert_close_rows(out, oracle.attn_causal(Q, K, V, p, eps=w.eps), dtype, "out")
    Sr, zr = oracle.causal_state(K, V, p)
    assert_close(to_np(S), Sr, dtype, "S")
    assert_close(_col(to_np(z)), _col(zr), dtype, "z")


@pytest.mark.parametrize("dtype,d,M,L,n0", [("bf16", 128, 32, 8, 150), ("bf16", 64, 16, 8, 64), ("f32", 32, 8, 8, 33)])
def test_prefill_then_decode(dtype, d, M, L, n0):
    """The state of a prefix from luna_attn_state, then one-token steps: the rows of
    the causal form after the prefix, and the same rows as the chunked scan."""
    w = small_workload(dtype, B=1, H=3, n=n0 + 8, d=d, M=M, L=L, causal=True)
    say(f"prefill {n0} then decode 8: {w.name}")
    Q, K, V, p = inputs(w, seed=13)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    S, z = luna.attn_state(Kt[:, :, :n0].contiguous(), Vt[:, :, :n0].contiguous(), pt)
    outs = []
    for t in range(n0, n0 + 8):
        sl = lambda X: X[:, :, t:t + 1].contiguous()  # noqa: E731
        outs.append(to_np(luna.attn_causal_step(sl(Qt), sl(Kt), sl(Vt), pt, S, z, eps=w.eps)))
    out = np.concatenate(outs, axis=2)
    ref = oracle.attn_causal(Q, K, V, p, eps=w.eps)[:, :, n0:]
    assert_close_rows(out, ref, dtype, "decoded rows")
    scan = to_np(luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=64, eps=w.eps))[:, :, n0:]
    assert_close_rows(out, scan, dtype, "decoded rows against the chunked scan")


@pytest.mark.parametrize("m", [3, 20])
def test_step_many_heads_from_state(m):
    """Enough heads that the step kernel's grid runs in several rounds of workgroups
    (2048 heads x 4 column blocks): every column block of a head must read z as it was
    before the call, although the head's block 0 rewrites z in place.  Started from a
    random state, against the oracle's recurrence; 3 tokens on the VALU, 20 on the
    matrix cores."""
    import torch
    B, H, d, M, L = 16, 128, 128, 32, 8
    w = small_workload("bf16", B=B, H=H, n=m, d=d, M=M, L=L, causal=True)
    say(f"step from a random state, {B * H} heads: {w.name}")
    Q, K, V, p = inputs(w, seed=29)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    D = M * L
    rng = np.random.default_rng(3)
    S0 = rng.standard_normal((B, H, D, d)) * 0.05
    z0 = rng.random((B, H, D)) + 0.5
    S = torch.from_numpy(S0).float().cuda().contiguous()
    z = torch.from_numpy(z0).float().cuda().contiguous()
    S0 = to_np(S)
    z0 = to_np(z)
    out = to_np(luna.attn_causal_step(Qt, Kt, Vt, pt, S, z, eps=w.eps))
    ro, rS, rz = oracle.attn_causal_step(Q, K, V, p, S0, z0, eps=w.eps)
    assert_close_rows(out, ro, "bf16", "out")
    assert_close(to_np(S), rS, "bf16", "S")
    assert_close(_col(to_np(z)), _col(rz), "bf16", "z")
    # z is summed once per call: a second read of the rewritten z would add the new
    # keys' features twice, which this bound (far below one key's share) rules out
    assert np.abs(to_np(z) - rz).max() <= 1e-3 * np.abs(rz - z0).max(), "z updated more than once"


@pytest.mark.parametrize("dtype,d,M,L", [("bf16", 128, 32, 8), ("f32", 32, 8, 8), ("bf16", 64, 128, 1)])
@pytest.mark.parametrize("m", [1, 4, 6])
def test_step_options_from_state(dtype, d, M, L, m):
    """Per-head parameters, one shared first layer and no output relu, from a random
    state, for one, a few and more tokens per head, against the oracle's recurrence."""
    import torch
    B, H = 2, 3
    w = small_workload(dtype, B=B, H=H, n=m, d=d, M=M, L=L, causal=True, per_head=True, shared_channels=True,
                       nonneg=False)
    say(f"step options {w.name} m={m}")
    Q, K, V, p = inputs(w, seed=41)
    p = dict(p)
    p["fc2_b"] = p["fc2_b"] + 1.0  # denominators away from zero with signed features
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    D = M * L
    rng = np.random.default_rng(5)
    S = torch.from_numpy(rng.standard_normal((B, H, D, d)) * 0.05).float().cuda().contiguous()
    z = torch.from_numpy(rng.random((B, H, D)) + 0.5).float().cuda().contiguous()
    S0, z0 = to_np(S), to_np(z)
    out = to_np(luna.attn_causal_step(Qt, Kt, Vt, pt, S, z, eps=w.eps))
    ro, rS, rz = oracle.attn_causal_step(Q, K, V, p, S0, z0, eps=w.eps)
    assert_close_rows(out, ro, dtype, "out")
    assert_close(to_np(S), rS, dtype, "S")
    assert_close(_col(to_np(z)), _col(rz), dtype, "z")


def test_step_rejects_bad_state():
    """Malformed state tensors are refused before anything runs."""
    import torch
    w = small_workload("bf16", B=1, H=2, n=5, d=64, M=16, L=8, causal=True)
    Q, K, V, p = inputs(w, seed=17)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    S = torch.zeros((1, 2, 128, 64), dtype=torch.float32, device="cuda")
    z = torch.zeros((1, 2, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(luna.LunaError):
        luna.attn_causal_step(Qt, Kt, Vt, pt, S[:, :, :64].contiguous(), z, eps=w.eps)
    with pytest.raises(luna.LunaError):
        luna.attn_causal_step(Qt, Kt, Vt, pt, S.half(), z, eps=w.eps)


def test_step_plan_reuses_tables():
    """Steps through a plan (tables built by the first call, reused after) give the
    same bits as steps that build the tables every time."""
    import torch
    w = small_workload("bf16", B=2, H=3, n=12, d=128, M=32, L=8, causal=True)
    Q, K, V, p = inputs(w, seed=19)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    D = 256
    Sa = torch.zeros((2, 3, D, 128), dtype=torch.float32, device="cuda")
    za = torch.zeros((2, 3, D), dtype=torch.float32, device="cuda")
    Sb, zb = Sa.clone(), za.clone()
    plan = luna.StepPlan(pt, 2, 3, 4, 128, torch.bfloat16, Qt.device, eps=w.eps)
    for a in range(0, 12, 4):
        sl = lambda X: X[:, :, a:a + 4].contiguous()  # noqa: E731
        oa = luna.attn_causal_step(sl(Qt), sl(Kt), sl(Vt), pt, Sa, za, eps=w.eps)
        ob = plan.run(sl(Qt), sl(Kt), sl(Vt), Sb, zb, torch.empty_like(sl(Qt)))
        assert torch.equal(oa, ob)
    assert torch.equal(Sa, Sb) and torch.equal(za, zb)
    assert plan.tables_ready == 1


def test_step_graph_replays():
    """A streaming call captured in a HIP graph (tables already built) and replayed
    advances the state exactly as eager calls do, replay after replay, with eager
    work and synchronisations between the replays."""
    import torch
    w = small_workload("bf16", B=2, H=3, n=4, d=128, M=32, L=8, causal=True)
    Q, K, V, p = inputs(w, seed=23)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    D = 256
    S0 = torch.randn((2, 3, D, 128), device="cuda") * 0.1
    z0 = torch.rand((2, 3, D), device="cuda") + 1.0
    Se, ze = S0.clone(), z0.clone()
    Sg, zg = S0.clone(), z0.clone()
    plan_e = luna.StepPlan(pt, 2, 3, 4, 128, torch.bfloat16, Qt.device, eps=w.eps)
    plan_g = luna.StepPlan(pt, 2, 3, 4, 128, torch.bfloat16, Qt.device, eps=w.eps)
    out_g = torch.empty_like(Qt)
    # first call outside the graph: it builds the tables
    Sw, zw = Sg.clone(), zg.clone()
    plan_g.run(Qt, Kt, Vt, Sw, zw, torch.empty_like(Qt))
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        plan_g.run(Qt, Kt, Vt, Sg, zg, out_g)
    torch.cuda.synchronize()
    Sg.copy_(S0)
    zg.copy_(z0)
    for rep in range(4):
        out_e = plan_e.run(Qt, Kt, Vt, Se, ze, torch.empty_like(Qt))
        graph.replay()
        torch.cuda.synchronize()
        _ = (Qt.float() * 2).sum().item()  # eager work between replays
        assert torch.equal(out_g, out_e), f"replay {rep}: output"
        assert torch.equal(Sg, Se) and torch.equal(zg, ze), f"replay {rep}: state"
