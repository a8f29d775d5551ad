"""The GPU tests' comparison of causal outputs, checked on the CPU against a defect
planted in the oracle's output: part 1 of a split head starting from a state whose z
misses one piece (one chunk's worth of keys of the first half).  Applied per row, the
tolerance catches it; a bound per head would not, because the rows that go wrong are
small next to the head's largest row (row 0 is v_0)."""
import numpy as np

import oracle
from gpu_util import TOL, row_errors, slice_errors
from paper_2512_08061_amd import workloads as wl


def test_row_metric_catches_a_seed_missing_one_pieces_z():
    w = wl.Workload("metric", 1, 2, 1000, 64, 16, 8, "bf16", "iid", True)
    Q, K, V = wl.make_inputs(w, seed=5)
    p = wl.make_params(w, seed=5)
    x, p0, p1 = 448, 128, 192           # split token, and the piece [p0, p1) whose z is lost
    good = oracle.attn_causal(Q, K, V, p, eps=w.eps)
    S, z = oracle.causal_state(K[:, :, :x], V[:, :, :x], p)
    _, zp = oracle.causal_state(K[:, :, p0:p1], V[:, :, p0:p1], p)
    bad_tail, _, _ = oracle.attn_causal_step(Q[:, :, x:], K[:, :, x:], V[:, :, x:], p, S, z - zp, eps=w.eps)
    bad = good.copy()
    bad[:, :, x:] = bad_tail
    assert np.allclose(bad[:, :, :x], good[:, :, :x])
    assert row_errors(bad, good).max() > 2 * TOL["bf16"]
    # (the same defect measured per head stays within the bf16 tolerance)
    assert slice_errors(bad, good).max() < TOL["bf16"]
