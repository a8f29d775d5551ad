"""luna_attn_fwd_causal_noalloc (the causal forward with the library's static scratch
as its workspace) against luna_attn_fwd_causal (a workspace from the caller) on the
same inputs: two calls in a row, the second on a smaller problem, each bitwise equal
to the workspace entry point (same kernels; the scratch keeps the first call's
contents, which the second must not depend on).  Also: a problem beyond the scratch
is refused before anything is enqueued."""
import numpy as np
import pytest

from gpu_util import inputs, say, small_workload, upload
from paper_2512_08061_amd import luna

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    luna.load_library()
    yield
    torch.cuda.synchronize()


def _pair(B, H, n, d, M, L, seed):
    import torch
    w = small_workload("bf16", B=B, H=H, n=n, d=d, M=M, L=L, causal=True)
    say(f"noalloc vs workspace: {w.name} B={B} H={H}")
    Q, K, V, p = inputs(w, seed=seed)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    ref = luna.attn_fwd_causal(Qt, Kt, Vt, pt, chunk=64, eps=w.eps)
    out = torch.full_like(Qt, float("nan"))
    luna.attn_fwd_causal_noalloc(Qt, Kt, Vt, pt, chunk=64, eps=w.eps, out=out)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    assert torch.equal(out, ref), f"max diff {(out.float() - ref.float()).abs().max().item()}"


def test_noalloc_matches_workspace_entry_point_twice():
    # first: 32 heads, so the call cuts every head in two and sums the first halves'
    # state in 8 pieces per head in the scratch; second: a smaller problem (2 heads)
    _pair(2, 16, 2048, 128, 32, 8, seed=41)
    _pair(1, 2, 300, 128, 32, 8, seed=43)


def test_noalloc_refuses_problems_beyond_the_scratch():
    import torch
    lib = luna.load_library()
    cap = luna.noalloc_scratch_bytes()
    assert cap == 64 << 20
    # per-head parameters: one 70+ KB table per head, beyond the scratch at 1024 heads
    w = small_workload("bf16", B=1, H=1024, n=64, d=128, M=32, L=8, causal=True, per_head=True)
    Q, K, V, p = inputs(w, seed=47)
    (Qt, Kt, Vt), pt = upload(w, [Q, K, V], p)
    pc = pt.c()
    need = lib.luna_workspace_bytes(luna.OP_ATTN_CAUSAL, luna.LUNA_BF16, 1, 1024, 64, 128, pc, 64)
    assert need > cap
    out = torch.zeros_like(Qt)
    with pytest.raises(luna.LunaError) as e:
        luna.attn_fwd_causal_noalloc(Qt, Kt, Vt, pt, out=out)
    assert e.value.status == luna.LUNA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert not out.any()
