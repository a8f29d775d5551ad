"""The feature map as the bf16 attention kernels evaluate it, element by element,
against the float64 oracle, on channel MLPs whose breakpoints sit at 2 <= |beta| <= 64
and rows whose projections fall just past them (where fp16 intercepts would cancel).

* phi itself: the state of a one-token sequence is z = phi(k) (rounded to bf16 as a
  matrix-core operand, summed in fp32), exported by luna_attn_state from the
  non-causal state pass (d = 64) and from the causal kernel's state launch (d = 128).
* attention weights: with one-hot value rows (v_t = e_{t mod d}) the output is the
  normalised kernel matrix summed per value column, which checks the phi of queries
  and keys inside the fused non-causal kernel, the split readout and both launches of
  the causal scan, element by element.

Bounds (tests/phi_bounds.py): per phi element 2^-8 |phi| (bf16 operand) plus 2^-11 of
the channel's local size on its segment (fp16 slope and value at the anchor) plus the
slope times the fp32 error of the projection; propagated through the sums of
non-negative terms, with one more bf16 rounding of the statistics or P operands, the
fp32 sums and the bf16 output."""
import numpy as np
import pytest

import oracle
import phi_bounds as pb
from gpu_util import say, to_np
from paper_2512_08061_amd import luna

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    luna.load_library()
    yield
    torch.cuda.synchronize()


def _dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda().to(torch.bfloat16).contiguous()


@pytest.mark.parametrize("d,M,nonneg,outliers", [(64, 16, True, False), (64, 16, False, False),
                                                  (128, 32, True, False), (128, 32, False, False),
                                                  (64, 16, True, True), (128, 32, False, True)])
def test_phi_elementwise_through_state(d, M, nonneg, outliers):
    """z of one-token sequences = bf16(phi(k)) against the oracle's phi, per element;
    with outliers, one breakpoint per channel at |beta| = 1e20."""
    import torch
    L, B, H = 8, 2, 128
    p = pb.wide_params(d, M, L, nonneg=nonneg, seed=d + int(nonneg), outliers=outliers)
    X = pb.rows_near_breakpoints(p, B * H, seed=d + 10 * int(nonneg))
    say(f"phi through luna_attn_state: d={d} M={M} L={L} nonneg={nonneg}, {B * H} one-token heads")
    Kt = _dev(X.reshape(B, H, 1, d))
    Vt = torch.zeros_like(Kt)
    pt = luna.PhiParams.from_arrays(p, Kt.device, torch.bfloat16)
    _, z = luna.attn_state(Kt, Vt, pt)
    got = to_np(z).reshape(B * H, M * L)
    phi, local, slope_du = pb.local_terms(X, p)
    bound = pb.phi_bound(phi, local, slope_du)
    err = np.abs(got - phi)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    say(f"  max err/bound {float((err / bound).max()):.3f} at {worst}; max |phi| {np.abs(phi).max():.3g}")
    assert np.isfinite(got).all()
    assert (err <= bound).all(), f"{int((err > bound).sum())} elements beyond the bound, worst {worst}"


def _weights_case(B, H, n, d, M, causal, seed):
    import torch
    L = 8
    p = pb.wide_params(d, M, L, nonneg=True, seed=seed)
    Q = pb.rows_near_breakpoints(p, B * H * n, seed=seed + 1).reshape(B, H, n, d)
    K = pb.rows_near_breakpoints(p, B * H * n, seed=seed + 2).reshape(B, H, n, d)
    V = np.zeros((B, H, n, d), np.float32)
    V[..., np.arange(n), np.arange(n) % d] = 1.0
    eps = 1e-6
    Qt, Kt, Vt = _dev(Q), _dev(K), _dev(V)
    pt = luna.PhiParams.from_arrays(p, Qt.device, torch.bfloat16)
    f = luna.attn_fwd_causal if causal else luna.attn_fwd
    got = to_np(f(Qt, Kt, Vt, pt, eps=eps)).reshape(B * H, n, d)
    cls = np.zeros((n, d))
    cls[np.arange(n), np.arange(n) % d] = 1.0
    mask = np.tril(np.ones((n, n))) if causal else np.ones((n, n))
    worst = 0.0
    for h in range(B * H):
        q, k = Q.reshape(B * H, n, d)[h], K.reshape(B * H, n, d)[h]
        A = oracle.kernel_matrix(q, k, p) * mask                   # the oracle's kernel form
        num, den = A @ cls, A.sum(1)
        ref = num / (den + eps)[:, None]
        pq, lq, sq = pb.local_terms(q, p)
        pk, lk, sk = pb.local_terms(k, p)
        dq, dk = pb.phi_bound(pq, lq, sq), pb.phi_bound(pk, lk, sk)
        dA = (pq @ dk.T + dq @ pk.T + dq @ dk.T) * mask
        dnum = dA @ cls
        dden = dA.sum(1)
        dnum = dnum + (pb.U_BF16 + 1e-4) * (num + dnum)          # bf16 S / P operand, fp32 sums
        dden = dden + (pb.U_BF16 + 1e-4) * (den + dden)          # bf16 z operand, fp32 sums
        dout = (dnum + np.abs(ref) * dden[:, None]) / (den + eps - dden)[:, None]
        bound = dout + pb.U_BF16 * (np.abs(ref) + dout)          # bf16 output
        assert (den + eps - dden > 0).all()
        err = np.abs(got[h] - ref)
        worst = max(worst, float((err / np.maximum(bound, 1e-30)).max()))
        assert (err <= bound).all(), f"head {h}: {int((err > bound).sum())} weights beyond the bound"
    say(f"  max err/bound {worst:.3f}")


@pytest.mark.parametrize("B,H,n,d,M,causal", [
    (1, 256, 64, 64, 16, False),   # fused non-causal kernel (>= 192 heads)
    (1, 8, 64, 64, 16, False),     # split path: state pass, reduce, readout kernel
    (1, 4, 384, 128, 32, True),    # causal: state launch pieces, then both scan parts
    (1, 256, 128, 128, 32, True),  # causal: one scan part per head
])
def test_attention_weights_elementwise(B, H, n, d, M, causal):
    say(f"one-hot values: B={B} H={H} n={n} d={d} M={M} causal={causal}")
    _weights_case(B, H, n, d, M, causal, seed=7 * n + H)
