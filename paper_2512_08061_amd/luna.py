"""Python binding of libluna.so (ctypes), argument marshalling only.

Every function here checks shapes and dtypes, allocates the outputs and the
workspace with torch on the tensors' device, and calls the C entry point of the
same name on the current torch stream.  All arithmetic runs in the HIP kernels of
libluna.so; there is no other code path.  If the library is missing the calls
raise instead of computing anything.
"""

from __future__ import annotations

import ctypes
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libluna.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "luna.h")

LUNA_OK, LUNA_ERR_INVALID_ARG, LUNA_ERR_UNSUPPORTED, LUNA_ERR_WORKSPACE, LUNA_ERR_HIP = range(5)
LUNA_F32, LUNA_BF16 = 0, 1
OP_FEATUREMAP, OP_ATTN, OP_ATTN_CAUSAL, OP_STATE, OP_CAUSAL_STEP, OP_ATTN_BWD, OP_ATTN_CAUSAL_BWD = range(7)


class LunaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


class PhiParamsC(ctypes.Structure):
    _fields_ = [
        ("M", ctypes.c_int32), ("L", ctypes.c_int32), ("hidden", ctypes.c_int32),
        ("shared_channels", ctypes.c_int32), ("nonneg", ctypes.c_int32), ("per_head", ctypes.c_int32),
        ("W", ctypes.c_void_p), ("b", ctypes.c_void_p),
        ("fc1_w", ctypes.c_void_p), ("fc1_b", ctypes.c_void_p),
        ("fc2_w", ctypes.c_void_p), ("fc2_b", ctypes.c_void_p),
    ]


class PhiGradsC(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libluna.so (raises LunaError if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise LunaError(LUNA_ERR_HIP, f"{path} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(PhiParamsC)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.luna_workspace_bytes.argtypes = [i32, i32, i64, i64, i64, i64, P, i32]
    lib.luna_workspace_bytes.restype = sz
    lib.luna_featuremap.argtypes = [vp, i32, i64, i64, i64, i64, P, vp, i32, vp, sz, vp]
    lib.luna_featuremap.restype = i32
    lib.luna_attn_fwd.argtypes = [vp, vp, vp, i32, i64, i64, i64, i64, P, ctypes.c_float, vp, vp, sz, vp]
    lib.luna_attn_fwd.restype = i32
    lib.luna_attn_fwd_causal.argtypes = [vp, vp, vp, i32, i64, i64, i64, i64, P, i32, ctypes.c_float, vp, vp,
                                         sz, vp]
    lib.luna_attn_fwd_causal.restype = i32
    lib.luna_attn_fwd_causal_noalloc.argtypes = [vp, vp, vp, i32, i64, i64, i64, i64, P, i32, ctypes.c_float,
                                                 vp, vp]
    lib.luna_attn_fwd_causal_noalloc.restype = i32
    lib.luna_noalloc_scratch_bytes.argtypes = []
    lib.luna_noalloc_scratch_bytes.restype = sz
    PV = ctypes.POINTER(PhiVariantC)
    lib.luna_phi_variant_features.argtypes = [PV]
    lib.luna_phi_variant_features.restype = i64
    lib.luna_featuremap_variant_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, PV]
    lib.luna_featuremap_variant_workspace_bytes.restype = sz
    lib.luna_featuremap_variant.argtypes = [vp, i32, i64, i64, i64, i64, PV, vp, i32, vp, sz, vp]
    lib.luna_featuremap_variant.restype = i32
    lib.luna_attn_features_workspace_bytes.argtypes = [i32, i32, i64, i64, i64, i64, i64, i32, i32]
    lib.luna_attn_features_workspace_bytes.restype = sz
    lib.luna_attn_fwd_features.argtypes = [vp, vp, i32, vp, i32, i64, i64, i64, i64, i64, i32, i32, ctypes.c_float,
                                           vp, vp, sz, vp]
    lib.luna_attn_fwd_features.restype = i32
    lib.luna_attn_state.argtypes = [vp, vp, i32, i64, i64, i64, i64, P, i32, vp, vp, vp, sz, vp]
    lib.luna_attn_state.restype = i32
    lib.luna_attn_causal_step.argtypes = [vp, vp, vp, i32, i64, i64, i64, i64, P, ctypes.c_float, i32, vp, vp, vp,
                                          vp, sz, vp]
    lib.luna_attn_causal_step.restype = i32
    lib.luna_attn_bwd.argtypes = [vp, vp, vp, vp, i32, i64, i64, i64, i64, P, i32, ctypes.c_float, vp, vp, vp,
                                  ctypes.POINTER(PhiGradsC), vp, sz, vp]
    lib.luna_attn_bwd.restype = i32
    lib.luna_distill_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, P, i32]
    lib.luna_distill_workspace_bytes.restype = sz
    lib.luna_distill.argtypes = [vp, vp, i32, i64, i64, i64, i64, P, i32, ctypes.c_float, vp,
                                 ctypes.POINTER(PhiGradsC), vp, sz, vp]
    lib.luna_distill.restype = i32
    lib.luna_status_string.argtypes = [i32]
    lib.luna_status_string.restype = ctypes.c_char_p
    lib.luna_last_error.argtypes = []
    lib.luna_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def header_functions(path: str = HEADER) -> list[str]:
    """Names of the functions include/luna.h declares."""
    txt = open(path).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(luna_[a-z_]+)\s*\(", txt)))


def _check(status: int) -> None:
    if status != LUNA_OK:
        lib = load_library()
        raise LunaError(status, f"{lib.luna_status_string(status).decode()}: {lib.luna_last_error().decode()}")


# ---------------------------------------------------------------------------
# torch-facing helpers
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dt(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return LUNA_BF16
    if t.dtype == torch.float32:
        return LUNA_F32
    raise LunaError(LUNA_ERR_INVALID_ARG, f"unsupported dtype {t.dtype}")


class PhiParams:
    """Device-resident feature-map parameters (see luna_phi_params in include/luna.h)."""

    def __init__(self, W, b, fc1_w, fc1_b, fc2_w, fc2_b, M, L, hidden, shared_channels=False, nonneg=True,
                 per_head=False):
        self.W, self.b, self.fc1_w, self.fc1_b, self.fc2_w, self.fc2_b = W, b, fc1_w, fc1_b, fc2_w, fc2_b
        self.M, self.L, self.hidden = int(M), int(L), int(hidden)
        self.shared_channels, self.nonneg, self.per_head = bool(shared_channels), bool(nonneg), bool(per_head)
        for name in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b"):
            t = getattr(self, name)
            if not t.is_contiguous():
                raise LunaError(LUNA_ERR_INVALID_ARG, f"{name} must be contiguous")
        torch = _torch()
        for name in ("b", "fc1_w", "fc1_b", "fc2_w", "fc2_b"):
            if getattr(self, name).dtype != torch.float32:
                raise LunaError(LUNA_ERR_INVALID_ARG, f"{name} must be float32")

    @classmethod
    def from_arrays(cls, p: dict, device, dtype):
        """Upload a parameter dict (NumPy arrays + scalars, as the workload generator returns)."""
        torch = _torch()
        f32 = lambda x: torch.as_tensor(x, dtype=torch.float32).contiguous().to(device)  # noqa: E731
        W = torch.as_tensor(p["W"], dtype=torch.float32).to(dtype).contiguous().to(device)
        return cls(W, f32(p["b"]), f32(p["fc1_w"]), f32(p["fc1_b"]), f32(p["fc2_w"]), f32(p["fc2_b"]),
                   p["M"], p["L"], p["hidden"], p.get("shared_channels", False), p.get("nonneg", True),
                   p.get("per_head", False))

    def c(self) -> PhiParamsC:
        return PhiParamsC(self.M, self.L, self.hidden, int(self.shared_channels), int(self.nonneg),
                          int(self.per_head), self.W.data_ptr(), self.b.data_ptr(), self.fc1_w.data_ptr(),
                          self.fc1_b.data_ptr(), self.fc2_w.data_ptr(), self.fc2_b.data_ptr())


def workspace_bytes(op: int, dtype: int, B: int, H: int, n: int, d: int, p: PhiParams | PhiParamsC,
                    chunk: int = 64) -> int:
    lib = load_library()
    pc = p.c() if isinstance(p, PhiParams) else p
    return int(lib.luna_workspace_bytes(op, dtype, B, H, n, d, ctypes.byref(pc), chunk))


def _workspace(nbytes: int, device):
    torch = _torch()
    ws = torch.empty(max(nbytes, 256) + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws, ws.data_ptr() + off, max(nbytes, 256)


def _stream_ptr(device) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _qkv_shape(*ts):
    B, H, n, d = ts[0].shape
    for t in ts:
        if tuple(t.shape) != (B, H, n, d) or not t.is_contiguous() or t.dtype != ts[0].dtype:
            raise LunaError(LUNA_ERR_INVALID_ARG, "Q, K, V must be contiguous [B, H, n, d] of one dtype")
    return B, H, n, d


def featuremap(X, p: PhiParams, out_dtype=None):
    """phi(X) for X [B, H, n, d]; returns [B, H, n, M*L] (feature i*L + l)."""
    torch = _torch()
    lib = load_library()
    if X.dim() != 4 or not X.is_contiguous():
        raise LunaError(LUNA_ERR_INVALID_ARG, "X must be a contiguous [B, H, n, d] tensor")
    B, H, n, d = X.shape
    out_dtype = X.dtype if out_dtype is None else out_dtype
    out = torch.empty((B, H, n, p.M * p.L), dtype=out_dtype, device=X.device)
    pc = p.c()
    dt = _dt(X)
    nb = lib.luna_workspace_bytes(OP_FEATUREMAP, dt, B, H, n, d, ctypes.byref(pc), 64)
    if nb == 0:
        _check(lib.luna_featuremap(X.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), out.data_ptr(), _dt(out),
                                   None, 0, None))
    ws, wsp, wsn = _workspace(nb, X.device)
    _check(lib.luna_featuremap(X.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), out.data_ptr(), _dt(out), wsp, wsn,
                               _stream_ptr(X.device)))
    out._luna_ws = ws  # keep the workspace alive until the output is
    return out


# ---------------------------------------------------------------------------
# feature-map variants and attention from given features
# ---------------------------------------------------------------------------

PHI_MLP, PHI_RFF_COS, PHI_RFF_SINCOS, PHI_PERFORMER = 0, 1, 2, 3
ACTS = {"relu": 0, "gelu": 1, "silu": 2, "tanh": 3}
KINDS = {"mlp": PHI_MLP, "rff_cos": PHI_RFF_COS, "rff_sincos": PHI_RFF_SINCOS, "performer": PHI_PERFORMER}


class PhiVariantC(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("act", ctypes.c_int32), ("base", ctypes.POINTER(PhiParamsC)),
                ("env_w", ctypes.c_void_p), ("env_b", ctypes.c_void_p), ("bank", ctypes.c_void_p),
                ("ch_rms", ctypes.c_int32), ("ch_rms_target", ctypes.c_float)]


class PhiVariant:
    """Device-resident description of a feature-map variant (luna_phi_variant)."""

    def __init__(self, kind: str, base: PhiParams, act: str = "relu", env_w=None, env_b=None, bank=None,
                 ch_rms: bool = False, ch_rms_target: float = 0.1):
        self.kind, self.act, self.base = kind, act, base
        self.env_w, self.env_b, self.bank = env_w, env_b, bank
        self.ch_rms, self.ch_rms_target = bool(ch_rms), float(ch_rms_target)
        self._pc = base.c()

    @classmethod
    def from_arrays(cls, p: dict, device, dtype):
        """Upload a variant dict as the oracle takes it ("kind", "act", W, b, the channel
        MLP for "mlp", optional env_w / env_b / bank / ch_rms / ch_rms_target)."""
        import numpy as np

        torch = _torch()
        f32 = lambda x: None if x is None else torch.as_tensor(x, dtype=torch.float32).contiguous().to(device)  # noqa: E731
        q = dict(p)
        if q.get("kind", "mlp") != "mlp":  # the projection only: a placeholder channel MLP
            lead = q["W"].shape[:-2]
            q.update(fc1_w=np.zeros(lead + (1, 1)), fc1_b=np.zeros(lead + (1, 1)), fc2_w=np.zeros(lead + (1, 1)),
                     fc2_b=np.zeros(lead + (1,)), L=1, hidden=1, M=q["W"].shape[-2])
        base = PhiParams.from_arrays(q, device, dtype)
        return cls(q.get("kind", "mlp"), base, q.get("act", "relu"), f32(q.get("env_w")), f32(q.get("env_b")),
                   f32(q.get("bank")), q.get("ch_rms", False), q.get("ch_rms_target", 0.1))

    def c(self) -> PhiVariantC:
        ptr = lambda t: None if t is None else t.data_ptr()  # noqa: E731
        return PhiVariantC(KINDS[self.kind], ACTS[self.act], ctypes.pointer(self._pc), ptr(self.env_w),
                           ptr(self.env_b), ptr(self.bank), int(self.ch_rms), self.ch_rms_target)

    def features(self) -> int:
        D = int(load_library().luna_phi_variant_features(ctypes.byref(self.c())))
        if D < 0:
            raise LunaError(LUNA_ERR_INVALID_ARG, load_library().luna_last_error().decode())
        return D


def featuremap_variant(X, v: PhiVariant, out_dtype=None, out=None):
    """The variant map of every row of X [B, H, n, d]; returns [B, H, n, D] (into out
    when given: a contiguous tensor of that shape)."""
    torch = _torch()
    lib = load_library()
    if X.dim() != 4 or not X.is_contiguous():
        raise LunaError(LUNA_ERR_INVALID_ARG, "X must be a contiguous [B, H, n, d] tensor")
    B, H, n, d = X.shape
    vc = v.c()
    D = int(lib.luna_phi_variant_features(ctypes.byref(vc)))
    if D < 0:
        raise LunaError(LUNA_ERR_INVALID_ARG, lib.luna_last_error().decode())
    if out is None:
        out = torch.empty((B, H, n, D), dtype=X.dtype if out_dtype is None else out_dtype, device=X.device)
    elif tuple(out.shape) != (B, H, n, D) or not out.is_contiguous():
        raise LunaError(LUNA_ERR_INVALID_ARG, f"out must be a contiguous [{B}, {H}, {n}, {D}] tensor")
    nb = int(lib.luna_featuremap_variant_workspace_bytes(_dt(X), B, H, n, d, ctypes.byref(vc)))
    ws, wsp, wsn = _workspace(nb, X.device)
    _check(lib.luna_featuremap_variant(X.data_ptr(), _dt(X), B, H, n, d, ctypes.byref(vc), out.data_ptr(), _dt(out),
                                       wsp, wsn, _stream_ptr(X.device)))
    out._luna_ws = ws
    return out


def attn_fwd_features(phiQ, phiK, V, causal: bool = False, eps: float = 1e-6, chunk: int = 64, out=None):
    """Kernel attention for given features phiQ, phiK [B, H, n, D] and V [B, H, n, d]."""
    torch = _torch()
    lib = load_library()
    for t in (phiQ, phiK, V):
        if t.dim() != 4 or not t.is_contiguous():
            raise LunaError(LUNA_ERR_INVALID_ARG, "inputs must be contiguous [B, H, n, *] tensors")
    B, H, n, D = phiQ.shape
    d = V.shape[-1]
    if phiK.shape != phiQ.shape or V.shape[:3] != phiQ.shape[:3] or phiK.dtype != phiQ.dtype:
        raise LunaError(LUNA_ERR_INVALID_ARG, "shapes or dtypes do not match")
    out = torch.empty_like(V) if out is None else out
    nb = int(lib.luna_attn_features_workspace_bytes(_dt(phiQ), _dt(V), B, H, n, d, D, int(causal), chunk))
    ws, wsp, wsn = _workspace(nb, V.device)
    _check(lib.luna_attn_fwd_features(phiQ.data_ptr(), phiK.data_ptr(), _dt(phiQ), V.data_ptr(), _dt(V), B, H, n, d,
                                      D, int(causal), chunk, eps, out.data_ptr(), wsp, wsn, _stream_ptr(V.device)))
    out._luna_ws = ws
    return out


def attn_fwd(Q, K, V, p: PhiParams, eps: float = 1e-6, out=None):
    """Non-causal LUNA attention; returns out [B, H, n, d] in Q's dtype."""
    torch = _torch()
    lib = load_library()
    B, H, n, d = _qkv_shape(Q, K, V)
    out = torch.empty_like(Q) if out is None else out
    pc = p.c()
    dt = _dt(Q)
    nb = lib.luna_workspace_bytes(OP_ATTN, dt, B, H, n, d, ctypes.byref(pc), 64)
    if nb == 0:
        _check(lib.luna_attn_fwd(Q.data_ptr(), K.data_ptr(), V.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), eps,
                                 out.data_ptr(), None, 0, None))
    ws, wsp, wsn = _workspace(nb, Q.device)
    _check(lib.luna_attn_fwd(Q.data_ptr(), K.data_ptr(), V.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), eps,
                             out.data_ptr(), wsp, wsn, _stream_ptr(Q.device)))
    out._luna_ws = ws
    return out


def attn_fwd_causal(Q, K, V, p: PhiParams, chunk: int = 64, eps: float = 1e-6, out=None):
    """Causal LUNA attention (chunked prefix scan); returns out [B, H, n, d]."""
    torch = _torch()
    lib = load_library()
    B, H, n, d = _qkv_shape(Q, K, V)
    out = torch.empty_like(Q) if out is None else out
    pc = p.c()
    dt = _dt(Q)
    nb = lib.luna_workspace_bytes(OP_ATTN_CAUSAL, dt, B, H, n, d, ctypes.byref(pc), chunk)
    if nb == 0:
        _check(lib.luna_attn_fwd_causal(Q.data_ptr(), K.data_ptr(), V.data_ptr(), dt, B, H, n, d, ctypes.byref(pc),
                                        chunk, eps, out.data_ptr(), None, 0, None))
    ws, wsp, wsn = _workspace(nb, Q.device)
    _check(lib.luna_attn_fwd_causal(Q.data_ptr(), K.data_ptr(), V.data_ptr(), dt, B, H, n, d, ctypes.byref(pc),
                                    chunk, eps, out.data_ptr(), wsp, wsn, _stream_ptr(Q.device)))
    out._luna_ws = ws
    return out


def attn_fwd_causal_noalloc(Q, K, V, p: PhiParams, chunk: int = 64, eps: float = 1e-6, out=None):
    """luna_attn_fwd_causal_noalloc: the causal forward with the library's static
    scratch as workspace (no allocation in the call; pass ``out`` to allocate nothing
    here either).  Returns out [B, H, n, d]."""
    torch = _torch()
    lib = load_library()
    B, H, n, d = _qkv_shape(Q, K, V)
    if out is None:
        out = torch.empty_like(Q)
    elif out.shape != Q.shape or out.dtype != Q.dtype or not out.is_contiguous() or out.device != Q.device:
        raise LunaError(LUNA_ERR_INVALID_ARG, "out must be a contiguous tensor of Q's shape, dtype and device")
    pc = p.c()
    _check(lib.luna_attn_fwd_causal_noalloc(Q.data_ptr(), K.data_ptr(), V.data_ptr(), _dt(Q), B, H, n, d,
                                            ctypes.byref(pc), chunk, eps, out.data_ptr(), _stream_ptr(Q.device)))
    return out


def noalloc_scratch_bytes() -> int:
    """Bytes of the static scratch behind attn_fwd_causal_noalloc."""
    return int(load_library().luna_noalloc_scratch_bytes())


def attn_bwd(Q, K, V, dO, p: PhiParams, causal: bool = False, eps: float = 1e-6, param_grads: bool = True):
    """Backward pass of attn_fwd (causal False) or attn_fwd_causal (causal True) for the
    upstream gradient dO: returns (dQ, dK, dV, grads) with dQ, dK, dV like Q and grads a
    dict of fp32 parameter gradients shaped like p's arrays (None if not param_grads)."""
    torch = _torch()
    lib = load_library()
    B, H, n, d = _qkv_shape(Q, K, V)
    if dO.shape != Q.shape or dO.dtype != Q.dtype or not dO.is_contiguous():
        raise LunaError(LUNA_ERR_INVALID_ARG, "dO must be a contiguous tensor of Q's shape and dtype")
    dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    grads, gc = None, None
    if param_grads:
        grads = {name: torch.empty(getattr(p, name).shape, dtype=torch.float32, device=Q.device)
                 for name in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")}
        gc = PhiGradsC(*(grads[k].data_ptr() for k in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")))
    pc = p.c()
    dt = _dt(Q)
    op = OP_ATTN_CAUSAL_BWD if causal else OP_ATTN_BWD
    nb = lib.luna_workspace_bytes(op, dt, B, H, n, d, ctypes.byref(pc), 64)
    args = (Q.data_ptr(), K.data_ptr(), V.data_ptr(), dO.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), int(causal), eps,
            dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(), ctypes.byref(gc) if gc is not None else None)
    if nb == 0:
        _check(lib.luna_attn_bwd(*args, None, 0, None))
    ws, wsp, wsn = _workspace(nb, Q.device)
    _check(lib.luna_attn_bwd(*args, wsp, wsn, _stream_ptr(Q.device)))
    dQ._luna_ws = ws
    return dQ, dK, dV, grads


def distill(Q, K, p: PhiParams, causal: bool = False, eps: float = 1e-6, param_grads: bool = True):
    """Attention-distillation loss (luna_distill): returns (row_loss, grads) with
    row_loss the fp32 [B, H, n] soft cross-entropy of the softmax teacher against LUNA's
    smoothed weights per query row, and grads a dict of fp32 gradients of its mean with
    respect to p's arrays (None if not param_grads)."""
    torch = _torch()
    lib = load_library()
    for t in (Q, K):
        if t.dim() != 4 or not t.is_contiguous():
            raise LunaError(LUNA_ERR_INVALID_ARG, "Q and K must be contiguous [B, H, n, d] tensors")
    if Q.shape != K.shape or Q.dtype != K.dtype:
        raise LunaError(LUNA_ERR_INVALID_ARG, "Q and K must have one shape and dtype")
    B, H, n, d = Q.shape
    row_loss = torch.empty((B, H, n), dtype=torch.float32, device=Q.device)
    grads, gc = None, None
    if param_grads:
        grads = {name: torch.empty(getattr(p, name).shape, dtype=torch.float32, device=Q.device)
                 for name in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")}
        gc = PhiGradsC(*(grads[k].data_ptr() for k in ("W", "b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")))
    pc = p.c()
    dt = _dt(Q)
    nb = int(lib.luna_distill_workspace_bytes(dt, B, H, n, d, ctypes.byref(pc), int(param_grads)))
    args = (Q.data_ptr(), K.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), int(causal), eps, row_loss.data_ptr(),
            ctypes.byref(gc) if gc is not None else None)
    if nb == 0:
        _check(lib.luna_distill(*args, None, 0, None))
    ws, wsp, wsn = _workspace(nb, Q.device)
    _check(lib.luna_distill(*args, wsp, wsn, _stream_ptr(Q.device)))
    row_loss._luna_ws = ws
    return row_loss, grads


def _state_tensors(B, H, D, d, device, S, z):
    torch = _torch()
    if S is None:
        S = torch.zeros((B, H, D, d), dtype=torch.float32, device=device)
    if z is None:
        z = torch.zeros((B, H, D), dtype=torch.float32, device=device)
    if tuple(S.shape) != (B, H, D, d) or S.dtype != torch.float32 or not S.is_contiguous():
        raise LunaError(LUNA_ERR_INVALID_ARG, "S must be a contiguous fp32 [B, H, M*L, d] tensor")
    if tuple(z.shape) != (B, H, D) or z.dtype != torch.float32 or not z.is_contiguous():
        raise LunaError(LUNA_ERR_INVALID_ARG, "z must be a contiguous fp32 [B, H, M*L] tensor")
    return S, z


def attn_state(K, V, p: PhiParams, S=None, z=None, accumulate: bool = False):
    """Causal state of the tokens of K, V: S = phi(K)^T V [B, H, M*L, d] and z = phi(K)^T 1
    [B, H, M*L] (fp32), written into S, z (allocated when None) or added to them."""
    lib = load_library()
    B, H, n, d = _qkv_shape(K, V)
    S, z = _state_tensors(B, H, p.M * p.L, d, K.device, S, z)
    pc = p.c()
    dt = _dt(K)
    nb = lib.luna_workspace_bytes(OP_STATE, dt, B, H, n, d, ctypes.byref(pc), 64)
    if nb == 0:
        _check(lib.luna_attn_state(K.data_ptr(), V.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), int(accumulate),
                                   S.data_ptr(), z.data_ptr(), None, 0, None))
    ws, wsp, wsn = _workspace(nb, K.device)
    _check(lib.luna_attn_state(K.data_ptr(), V.data_ptr(), dt, B, H, n, d, ctypes.byref(pc), int(accumulate),
                               S.data_ptr(), z.data_ptr(), wsp, wsn, _stream_ptr(K.device)))
    S._luna_ws = ws
    return S, z


def attn_causal_step(Q, K, V, p: PhiParams, S, z, eps: float = 1e-6, out=None):
    """One streaming step over the m new tokens of Q, K, V [B, H, m, d] from the state
    (S, z), which is updated in place; returns out [B, H, m, d]."""
    torch = _torch()
    lib = load_library()
    B, H, m, d = _qkv_shape(Q, K, V)
    S, z = _state_tensors(B, H, p.M * p.L, d, Q.device, S, z)
    out = torch.empty_like(Q) if out is None else out
    pc = p.c()
    dt = _dt(Q)
    nb = lib.luna_workspace_bytes(OP_CAUSAL_STEP, dt, B, H, m, d, ctypes.byref(pc), 64)
    if nb == 0:
        _check(lib.luna_attn_causal_step(Q.data_ptr(), K.data_ptr(), V.data_ptr(), dt, B, H, m, d,
                                         ctypes.byref(pc), eps, 0, S.data_ptr(), z.data_ptr(), out.data_ptr(), None,
                                         0, None))
    ws, wsp, wsn = _workspace(nb, Q.device)
    _check(lib.luna_attn_causal_step(Q.data_ptr(), K.data_ptr(), V.data_ptr(), dt, B, H, m, d, ctypes.byref(pc), eps,
                                     0, S.data_ptr(), z.data_ptr(), out.data_ptr(), wsp, wsn, _stream_ptr(Q.device)))
    out._luna_ws = ws
    return out


class StepPlan:
    """Streaming steps of m tokens per head with one persistent workspace: the first
    ``run`` builds the channel tables in it, later ones reuse them (tables_ready = 1).
    The parameters must stay unchanged between runs."""

    def __init__(self, p: PhiParams, B: int, H: int, m: int, d: int, dtype, device, eps: float = 1e-6):
        self.lib = load_library()
        self.p, self.pc = p, p.c()
        self.B, self.H, self.m, self.d, self.eps = B, H, m, d, float(eps)
        self.dt = LUNA_BF16 if str(dtype).endswith("bfloat16") else LUNA_F32
        nb = self.lib.luna_workspace_bytes(OP_CAUSAL_STEP, self.dt, B, H, m, d, ctypes.byref(self.pc), 64)
        if nb == 0:
            raise LunaError(LUNA_ERR_UNSUPPORTED, "no streaming step for this problem")
        self.ws, self.wsp, self.wsn = _workspace(nb, device)
        self.tables_ready = 0

    def run(self, Q, K, V, S, z, out, stream=None):
        if _qkv_shape(Q, K, V) != (self.B, self.H, self.m, self.d) or _dt(Q) != self.dt:
            raise LunaError(LUNA_ERR_INVALID_ARG, "Q, K, V do not match the plan")
        _state_tensors(self.B, self.H, self.p.M * self.p.L, self.d, Q.device, S, z)
        s = stream if stream is not None else _stream_ptr(Q.device)
        _check(self.lib.luna_attn_causal_step(Q.data_ptr(), K.data_ptr(), V.data_ptr(), self.dt, self.B, self.H,
                                              self.m, self.d, ctypes.byref(self.pc), self.eps, self.tables_ready,
                                              S.data_ptr(), z.data_ptr(), out.data_ptr(), self.wsp, self.wsn, s))
        self.tables_ready = 1
        return out


class Plan:
    """A reusable call: output, workspace and the C parameter struct allocated once.

    ``run()`` only enqueues the kernels (for timing loops and graph capture).
    """

    def __init__(self, op: int, Q, K, V, p: PhiParams, eps: float = 1e-6, chunk: int = 64):
        torch = _torch()
        self.lib = load_library()
        self.op, self.Q, self.K, self.V, self.p = op, Q, K, V, p
        self.B, self.H, self.n, self.d = _qkv_shape(Q, K, V)
        self.dt = _dt(Q)
        self.eps, self.chunk = float(eps), int(chunk)
        self.pc = p.c()
        self.out = torch.empty_like(Q)
        nb = self.lib.luna_workspace_bytes(op, self.dt, self.B, self.H, self.n, self.d, ctypes.byref(self.pc), chunk)
        if nb == 0:
            self._call(None, 0, None)  # raises with the reason
        self.ws, self.wsp, self.wsn = _workspace(nb, Q.device)
        self.ws_bytes = nb

    def _call(self, wsp, wsn, stream):
        q, k, v, o = self.Q.data_ptr(), self.K.data_ptr(), self.V.data_ptr(), self.out.data_ptr()
        if self.op == OP_ATTN:
            st = self.lib.luna_attn_fwd(q, k, v, self.dt, self.B, self.H, self.n, self.d, ctypes.byref(self.pc),
                                        self.eps, o, wsp, wsn, stream)
        else:
            st = self.lib.luna_attn_fwd_causal(q, k, v, self.dt, self.B, self.H, self.n, self.d,
                                               ctypes.byref(self.pc), self.chunk, self.eps, o, wsp, wsn, stream)
        _check(st)

    def run(self, stream=None):
        s = stream if stream is not None else _stream_ptr(self.Q.device)
        self._call(self.wsp, self.wsn, s)
        return self.out
