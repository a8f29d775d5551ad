"""Host checks of the element-wise phi bound that the GPU tests of the bf16 attention
paths use (tests/phi_bounds.py): on parameters with breakpoints far from zero and rows
whose projections sit just past them, fp16 rows of (slope, value at the segment's
anchor) stay inside the bound, while fp16 rows of (slope, intercept) -- the rounding of
an intercept that cancels against slope u -- break it.  So a GPU test against the bound
tells the two forms apart."""
import numpy as np
import pytest

import phi_bounds as pb


@pytest.mark.parametrize("nonneg", [True, False])
def test_bound_separates_anchored_rows_from_intercepts(nonneg):
    p = pb.wide_params(64, 16, 8, nonneg=nonneg, seed=1)
    X = pb.rows_near_breakpoints(p, 256, seed=1)
    phi, local, slope_du = pb.local_terms(X, p)
    bound = pb.phi_bound(phi, local, slope_du)
    anchored = np.abs(pb.fp16_rows_emulated(X, p, anchored=True) - phi)
    intercept = np.abs(pb.fp16_rows_emulated(X, p, anchored=False) - phi)
    assert (anchored <= bound).all(), float((anchored / bound).max())
    ratio = intercept / bound
    assert (ratio > 1).sum() >= 10 and ratio.max() > 5, (int((ratio > 1).sum()), float(ratio.max()))


def test_rows_land_next_to_breakpoints():
    p = pb.wide_params(128, 32, 8, seed=2)
    X = pb.rows_near_breakpoints(p, 64, seed=2)
    u = X.astype(np.float64) @ np.asarray(p["W"], np.float64).T + p["b"]
    beta = np.sort((-p["fc1_b"] / p["fc1_w"]).ravel().astype(np.float64))
    j = np.clip(np.searchsorted(beta, u), 1, beta.size - 1)
    gap = np.minimum(np.abs(u - beta[j - 1]), np.abs(u - beta[j]))
    assert np.median(gap) < 0.2 and np.abs(u).max() > 16
