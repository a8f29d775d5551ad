"""Seeded synthetic inputs for LUNA attention.

This module is shared by the tests, the smoke check and the benchmark, and it
is the only code that the GPU path and the CPU oracle have in common.  It holds
none of the method's arithmetic: it draws random numbers, shapes them, rounds
them to the storage dtype and returns plain NumPy arrays.  Both sides then read
exactly the same stored values (the oracle upcasts them to float64, the GPU path
uploads them unchanged).

Recipe (all streams are NumPy PCG64 seeded through ``SeedSequence``):

* Q, K, V: one independent stream per (tensor, batch index b), entropy
  ``[seed, tensor_id, b]`` with tensor_id 0/1/2 for Q/K/V.  Each stream fills
  the ``[H, n, d]`` block of its batch index.  Distributions:

  - ``"iid"``: every element N(0, 1).
  - ``"token_correlated"``: a per-(tensor, b) mean vector mu ~ N(0, 1) of shape
    ``[d]`` is drawn first, then every row is ``mu + 0.5 * N(0, 1)``; rows of
    one batch item share mu, as the patch tokens of one image do.
  - ``"l2norm"``: rows drawn N(0, 1), divided by their L2 norm and multiplied
    by sqrt(d) (every row has norm sqrt(d)).

* feature-map parameters: one stream with entropy ``[seed, 1000]`` draws, in
  this order, W [P, M, d], b [P, M], fc1_w [P, C1, hidden], fc1_b [P, C1, hidden],
  fc2_w [P, L, hidden], fc2_b [P, L], every element N(0, 1/d).  P is H when
  the parameters are per head and 1 otherwise (the leading axis is then
  dropped); C1 is L for per-channel MLPs and 1 for one shared first layer.

* storage: ``"f32"`` rounds to float32; ``"bf16"`` rounds Q, K, V and W to
  bfloat16 (round to nearest, ties to even, via float32) and keeps b and the MLP
  parameters in float32.  Arrays are returned as float32 NumPy arrays whose
  values are exactly representable in the storage dtype.
"""

from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "round_bf16",
    "make_inputs",
    "make_params",
    "workload",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and input recipe of one synthetic LUNA attention problem."""

    name: str
    B: int
    H: int
    n: int
    d: int
    M: int  # projections w_i
    L: int  # channels per projection
    dtype: str  # "f32" | "bf16"
    dist: str  # "iid" | "token_correlated" | "l2norm"
    causal: bool
    hidden: int = 64
    chunk: int = 64
    shared_channels: bool = False
    nonneg: bool = True
    per_head: bool = False
    eps: float = 1e-6

    @property
    def D(self) -> int:
        return self.M * self.L

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five problems the hot path is measured and checked on.  Feature count
# D = M*L with L = 8 channels per projection (the paper's default L).
WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", 1, 1, 256, 32, 8, 8, "f32", "iid", False),
    "text_encoder": Workload("text_encoder", 32, 12, 512, 64, 8, 8, "bf16", "iid", False),
    "vision_encoder": Workload("vision_encoder", 64, 12, 197, 64, 16, 8, "bf16", "token_correlated", False),
    "long_noncausal": Workload("long_noncausal", 32, 8, 4096, 64, 16, 8, "bf16", "l2norm", False),
    "long_causal": Workload("long_causal", 8, 16, 16384, 128, 32, 8, "bf16", "iid", True),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned as float32."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = (b + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    nan = np.isnan(x)
    out = r.view(np.float32)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32)
    return round_bf16(x) if dtype == "bf16" else x


def _fill_block(seed: int, tensor_id: int, b: int, shape, dist: str, dtype: str, out: np.ndarray) -> None:
    rng = np.random.default_rng(np.random.SeedSequence([seed, tensor_id, b]))
    H, n, d = shape
    if dist == "iid":
        x = rng.standard_normal((H, n, d), dtype=np.float32)
    elif dist == "token_correlated":
        mu = rng.standard_normal(d, dtype=np.float32)
        x = mu[None, None, :] + np.float32(0.5) * rng.standard_normal((H, n, d), dtype=np.float32)
    elif dist == "l2norm":
        x = rng.standard_normal((H, n, d), dtype=np.float32).astype(np.float64)
        x *= np.sqrt(d) / np.linalg.norm(x, axis=-1, keepdims=True)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    out[...] = _store(x, dtype)


def make_inputs(w: Workload, seed: int = 0, threads: int | None = None):
    """Return (Q, K, V) as float32 arrays of shape [B, H, n, d]."""
    shape = (w.H, w.n, w.d)
    arrs = [np.empty((w.B,) + shape, dtype=np.float32) for _ in range(3)]
    jobs = [(t, b) for t in range(3) for b in range(w.B)]
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))
    if threads <= 1 or len(jobs) == 1:
        for t, b in jobs:
            _fill_block(seed, t, b, shape, w.dist, w.dtype, arrs[t][b])
    else:
        with _cf.ThreadPoolExecutor(threads) as ex:
            futs = [ex.submit(_fill_block, seed, t, b, shape, w.dist, w.dtype, arrs[t][b]) for t, b in jobs]
            for f in futs:
                f.result()
    return tuple(arrs)


def make_params(w: Workload, seed: int = 0) -> dict:
    """Feature-map parameters, every element N(0, 1/d)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 1000]))
    P = w.H if w.per_head else 1
    C1 = 1 if w.shared_channels else w.L
    s = 1.0 / np.sqrt(w.d)

    def draw(*shape):
        return (rng.standard_normal(shape) * s).astype(np.float32)

    p = {
        "W": draw(P, w.M, w.d),
        "b": draw(P, w.M),
        "fc1_w": draw(P, C1, w.hidden),
        "fc1_b": draw(P, C1, w.hidden),
        "fc2_w": draw(P, w.L, w.hidden),
        "fc2_b": draw(P, w.L),
    }
    if w.dtype == "bf16":
        p["W"] = round_bf16(p["W"])
    if not w.per_head:
        p = {k: v[0] for k, v in p.items()}
    p.update(M=w.M, L=w.L, hidden=w.hidden, shared_channels=w.shared_channels,
             nonneg=w.nonneg, per_head=w.per_head)
    return p


def make_variant_params(kind: str, M: int, d: int, L: int = 8, hidden: int = 64, act: str = "relu",
                        shared: bool = False, env: bool = False, bank: bool = False, ch_rms: bool = False,
                        seed: int = 0) -> dict:
    """Parameters of a feature-map variant, as the variant calls take them.  Random
    Fourier features: W rows N(0, I/d), phases b uniform in [0, 2 pi).  Performer:
    W = omega / d^(1/4) with omega ~ N(0, I), b = 0.  Channel MLPs: every element
    N(0, 1/d) as in make_params, an envelope G x + c with G N(0, 1/d) and c N(0, 1),
    bank coefficients N(0, 1), channel RMS target 0.1."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 2000]))
    s = 1.0 / np.sqrt(d)
    p = {"kind": kind, "act": act, "M": M}
    if kind == "performer":
        p.update(W=(rng.standard_normal((M, d)) / d ** 0.25).astype(np.float32), b=np.zeros(M, np.float32))
        return p
    if kind in ("rff_cos", "rff_sincos"):
        p.update(W=(rng.standard_normal((M, d)) * s).astype(np.float32),
                 b=rng.uniform(0.0, 2.0 * np.pi, M).astype(np.float32))
        return p
    C1 = 1 if shared else L

    def draw(*shape):
        return (rng.standard_normal(shape) * s).astype(np.float32)

    p.update(W=draw(M, d), b=draw(M), fc1_w=draw(C1, hidden), fc1_b=draw(C1, hidden), fc2_w=draw(L, hidden),
             fc2_b=draw(L), L=L, hidden=hidden, nonneg=True, shared_channels=shared)
    if env:
        p.update(env_w=draw(L, d), env_b=rng.standard_normal(L).astype(np.float32))
    if bank:
        p["bank"] = rng.standard_normal(L).astype(np.float32)
    if ch_rms:
        p.update(ch_rms=True, ch_rms_target=0.1)
    return p
