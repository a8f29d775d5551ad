"""Helpers shared by the GPU parity tests: upload seeded inputs, run the HIP path
through the C ABI, and compare with the float64 oracle."""
from __future__ import annotations

import sys

import numpy as np

from paper_2512_08061_amd import luna
from paper_2512_08061_amd import workloads as wl

# normwise tolerance per (b, h) slice: max|gpu - ref| / max|ref|
TOL = {"f32": 1e-4, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def upload(w: wl.Workload, arrays, p: dict):
    import torch
    dev = torch.device("cuda:0")
    tdt = torch_dtype(w.dtype)
    ts = [torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(tdt).contiguous() for a in arrays]
    return ts, luna.PhiParams.from_arrays(p, dev, tdt)


def to_np(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def slice_errors(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Normwise error of every leading slice (all but the last two axes)."""
    g = gpu.reshape((-1,) + gpu.shape[-2:])
    r = ref.reshape((-1,) + ref.shape[-2:])
    num = np.abs(g - r).reshape(g.shape[0], -1).max(axis=1)
    den = np.maximum(np.abs(r).reshape(r.shape[0], -1).max(axis=1), 1e-30)
    return num / den


def assert_close(gpu, ref, dtype: str, what: str = ""):
    gpu, ref = np.asarray(gpu, np.float64), np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.isfinite(gpu).all(), f"{what}: non-finite GPU output"
    err = slice_errors(gpu, ref)
    tol = TOL[dtype]
    assert err.max() <= tol, f"{what}: normwise error {err.max():.3e} > {tol} (worst slice {int(err.argmax())})"
    return float(err.max())


def row_errors(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Normwise error of every row (the last axis): max|gpu - ref| / max|ref| per row."""
    g = gpu.reshape(-1, gpu.shape[-1])
    r = ref.reshape(-1, ref.shape[-1])
    return np.abs(g - r).max(axis=1) / np.maximum(np.abs(r).max(axis=1), 1e-30)


def assert_close_rows(gpu, ref, dtype: str, what: str = ""):
    """The tolerance applied to every output row on its own.  Causal rows are averages
    over prefixes of different lengths (row 0 is v_0, late rows are much smaller), so a
    bound on a whole head would let late rows drift by many times the tolerance."""
    gpu, ref = np.asarray(gpu, np.float64), np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.isfinite(gpu).all(), f"{what}: non-finite GPU output"
    err = row_errors(gpu, ref)
    tol = TOL[dtype]
    assert err.max() <= tol, f"{what}: row error {err.max():.3e} > {tol} (worst row {int(err.argmax())})"
    return float(err.max())


def oracle_per_batch(fn, Q, K, V, p, eps, threads: int = 8):
    """fn(Q[b], K[b], V[b], p, eps=eps) for every batch entry, in a thread pool (NumPy
    releases the interpreter lock in its array operations)."""
    import concurrent.futures as cf
    out = np.empty(Q.shape[:-1] + (V.shape[-1],), np.float64)

    def job(b):
        out[b] = fn(Q[b], K[b], V[b], p, eps=eps)

    with cf.ThreadPoolExecutor(max(1, min(threads, Q.shape[0]))) as ex:
        list(ex.map(job, range(Q.shape[0])))
    return out


def small_workload(dtype="bf16", B=2, H=3, n=300, d=64, M=16, L=8, causal=False, **kw) -> wl.Workload:
    return wl.Workload(f"small_{dtype}_{d}_{M}x{L}_{n}", B, H, n, d, M, L, dtype, kw.pop("dist", "iid"), causal,
                       **kw)


def inputs(w: wl.Workload, seed=0):
    Q, K, V = wl.make_inputs(w, seed)
    p = wl.make_params(w, seed)
    return Q, K, V, p
