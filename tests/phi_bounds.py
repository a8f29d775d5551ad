"""Element-wise error bounds for the feature map as the bf16 attention kernels
evaluate it, and the inputs that stress them.  CPU only (NumPy); used by the GPU
tests of the attention paths' phi and by the host test that the bound separates the
anchored fp16 rows from a (slope, intercept) fp16 form.

The bf16 kernels evaluate channel l of projection i on the segment j of u_i as
    psi_l = slope_l (u - a_j) + value_l,
with slope and value rounded to fp16 (unit roundoff 2^-11) and the anchor a_j the
segment's left breakpoint (the first segment's right one), clamped to [-64, 64],
then round phi to bf16
(unit roundoff 2^-8) as a matrix-core operand.  Per element that gives
    |phi_gpu - phi| <= 2^-8 |phi| + (2^-11 (|slope (u - a)| + |value|) + |slope| du) / sqrt(M)
up to fp32 roundings, where du bounds the fp32 error of the projection u.  The
slope, anchor and value come from the oracle's exact piecewise-linear form of the
channel MLPs (pwl_tables, pinned to the literal MLP)."""
from __future__ import annotations

import math

import numpy as np

import oracle
from paper_2512_08061_amd import workloads as wl

U_BF16 = 2.0 ** -8
U_FP16 = 2.0 ** -11
U_FP32 = 2.0 ** -24
ANCHOR_MAX = 64.0  # anchors (segment breakpoints) are clamped to [-64, 64]


def wide_params(d: int, M: int, L: int, hidden: int = 64, nonneg: bool = True, seed: int = 0,
                outliers: bool = False) -> dict:
    """Channel MLPs whose breakpoints -c/a all lie at 2 <= |beta| <= 64 (slopes of order
    one), projections N(0, 1/d): far from u = 0 a segment's intercept is much larger
    than the channel's value there, which is where an fp16 intercept loses it.  With
    `outliers`, one unit per channel breaks at |beta| = 1e20 (a tiny first-layer
    weight), whose far segment must not set the scale of the fp16 rows."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 2000]))
    a = rng.standard_normal((L, hidden))
    beta = rng.uniform(2.0, 64.0, (L, hidden)) * rng.choice([-1.0, 1.0], (L, hidden))
    if outliers:
        a[:, 0] = 1e-20 * rng.choice([-1.0, 1.0], L)
        beta[:, 0] = 1e20 * rng.choice([-1.0, 1.0], L)
    p = {
        "W": wl.round_bf16(rng.standard_normal((M, d)) / math.sqrt(d)),
        "b": (rng.standard_normal(M) / math.sqrt(d)).astype(np.float32),
        "fc1_w": a.astype(np.float32),
        "fc1_b": (-a * beta).astype(np.float32),
        "fc2_w": (rng.standard_normal((L, hidden)) / math.sqrt(hidden)).astype(np.float32),
        "fc2_b": (0.5 * rng.standard_normal(L)).astype(np.float32),
    }
    p.update(M=M, L=L, hidden=hidden, shared_channels=False, nonneg=nonneg, per_head=False)
    return p


def rows_near_breakpoints(p: dict, rows: int, seed: int = 0) -> np.ndarray:
    """bf16 rows x [rows, d] whose projections u_i = w_i.x + b_i fall just past (or at)
    randomly chosen breakpoints of the channel MLPs: min-norm solutions of
    W x = target - b, rounded to bf16 (which moves u by a fraction of the segment)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 2001]))
    W = np.asarray(p["W"], np.float64)
    b = np.asarray(p["b"], np.float64)
    beta = (-np.asarray(p["fc1_b"], np.float64) / np.asarray(p["fc1_w"], np.float64)).ravel()
    beta = beta[np.abs(beta) <= 64.0]  # (outlying breakpoints are not targets)
    M = W.shape[0]
    target = rng.choice(beta, (rows, M)) + rng.uniform(0.0, 0.05, (rows, M))
    X = np.linalg.lstsq(W, (target - b).T, rcond=None)[0].T
    return wl.round_bf16(X.astype(np.float32)).astype(np.float32)


def local_terms(X: np.ndarray, p: dict):
    """Per element of phi(X) [..., n, M*L] (feature i*L + l): |phi|, the local size
    |slope (u - a)| + |value| / sqrt(M) and |slope| du / sqrt(M) of the anchored form."""
    bp, s, t = oracle.pwl_tables(p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"])
    W = np.asarray(p["W"], np.float64)
    b = np.asarray(p["b"], np.float64)
    X = np.asarray(X, np.float64)
    u = X @ W.T + b                                                    # [..., n, M]
    du = (X.shape[-1] + 2) * U_FP32 * (np.abs(X) @ np.abs(W).T + np.abs(b))
    j = np.searchsorted(bp, u, side="left")                            # segment
    anchor = np.clip(np.where(j > 0, bp[np.maximum(j - 1, 0)], bp[0] if bp.size else 0.0), -ANCHOR_MAX, ANCHOR_MAX)
    sj, tj = s[j], t[j]                                                # [..., n, M, L]
    value = sj * anchor[..., None] + tj
    M, L = W.shape[0], s.shape[1]
    scale = 1.0 / math.sqrt(M)
    local = (np.abs(sj * (u - anchor)[..., None]) + np.abs(value)) * scale
    slope_du = np.abs(sj) * du[..., None] * scale
    phi = oracle.featuremap(X, p)
    shp = u.shape[:-1] + (M * L,)
    return phi, local.reshape(shp), slope_du.reshape(shp)


def fp16_rows_emulated(X: np.ndarray, p: dict, anchored: bool) -> np.ndarray:
    """phi(X) evaluated as a bf16 kernel would from fp16 rows scaled by 2^e (largest
    magnitude in [2^13, 2^14)): anchored, slope (u - a) + value at the anchor; or not,
    slope u + intercept.  fp64 otherwise, so the difference to phi is the rows' rounding
    (phi is not rounded to bf16 here)."""
    bp, s, t = oracle.pwl_tables(p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"])
    W = np.asarray(p["W"], np.float64)
    u = np.asarray(X, np.float64) @ W.T + np.asarray(p["b"], np.float64)
    j = np.searchsorted(bp, u, side="left")
    M = W.shape[0]
    seg_anchor = np.clip(np.concatenate([[bp[0] if bp.size else 0.0], bp]), -ANCHOR_MAX, ANCHOR_MAX)
    v = s * seg_anchor[:, None] + t if anchored else t
    e = 14 - math.frexp(max(np.abs(s).max(), np.abs(v).max()) / math.sqrt(M))[1]
    q16 = lambda x: np.ldexp(np.ldexp(x / math.sqrt(M), e).astype(np.float16).astype(np.float64), -e)  # noqa: E731
    sj, vj = q16(s)[j], q16(v)[j]
    arg = (u - seg_anchor[j]) if anchored else u
    y = sj * arg[..., None] + vj
    if p["nonneg"]:
        y = np.maximum(y, 0.0)
    return y.reshape(u.shape[:-1] + (M * s.shape[1],))


def phi_bound(phi: np.ndarray, local: np.ndarray, slope_du: np.ndarray) -> np.ndarray:
    """Element-wise bound on |phi_gpu - phi| for the bf16 attention kernels."""
    return U_BF16 * np.abs(phi) + 1.01 * (U_FP16 * local + slope_du) + 2.0 ** -20 * local
