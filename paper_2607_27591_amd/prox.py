"""Thin ctypes binding of libprox.so (declared in include/prox.h).

Argument marshalling only: every step of the decode FFN runs in the HIP
kernels of libprox.  PyTorch provides device memory and streams.  There is no
fallback: if the library is missing or a call fails, this module raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import List, Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libprox.so")

F16, BF16 = 0, 1
INT8, INT4, NONE = 0, 1, 2   # NONE: unquantised 16-bit proxy (group = d_model)
MAX_BATCH = 64   # PROX_MAX_BATCH of include/prox.h
SPARSE_STAGES = 3

_TORCH_DT = {torch.float16: F16, torch.bfloat16: BF16}
_DT_TORCH = {F16: torch.float16, BF16: torch.bfloat16}


class ProxError(RuntimeError):
    """A libprox entry point returned a status other than PROX_OK."""

    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {strerror(status)} (status {status})")


class _Weights(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int), ("d_ff", ctypes.c_int), ("dtype", ctypes.c_int),
                ("w_gate", ctypes.c_void_p), ("w_up", ctypes.c_void_p),
                ("w_down", ctypes.c_void_p), ("act", ctypes.c_int)]


SILU, GELU = 0, 1   # gate activations: SwiGLU, GeGLU


class _Proxy(ctypes.Structure):
    _fields_ = [("fmt", ctypes.c_int), ("group", ctypes.c_int), ("blob", ctypes.c_void_p),
                ("bytes", ctypes.c_size_t)]


class _W4(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("d_model", ctypes.c_int), ("d_ff", ctypes.c_int),
                ("group", ctypes.c_int), ("act", ctypes.c_int), ("blob", ctypes.c_void_p),
                ("bytes", ctypes.c_size_t)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libprox.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_27591_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I, S, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_float
        WP, PP = ctypes.POINTER(_Weights), ctypes.POINTER(_Proxy)
        L.prox_proxy_bytes.argtypes = [I, I, I, I]
        L.prox_proxy_bytes.restype = S
        L.prox_pack_proxy.argtypes = [WP, PP, P]
        L.prox_unpack_proxy.argtypes = [PP, I, I, P, P, P, P, P]
        L.prox_workspace_bytes.argtypes = [I, I, I]
        L.prox_workspace_bytes.restype = S
        L.prox_w4_workspace_bytes.argtypes = [I, I, I]
        L.prox_w4_workspace_bytes.restype = S
        L.prox_stage1_mfma_rows.argtypes = [I, I, I, I, I]
        L.prox_stage1_mfma_rows.restype = I
        L.prox_stage2_rows.argtypes = [I, I, I, I]
        L.prox_stage2_rows.restype = I
        L.prox_ffn_dense.argtypes = [WP, P, I, P, P, S, P]
        L.prox_ffn_sparse.argtypes = [WP, PP, P, I, I, I, P, P, P, P, P, S, P]
        L.prox_ffn_sparse_noalloc.argtypes = [WP, PP, P, I, I, I, P, P, P, P, P]
        L.prox_noalloc_max_bytes.argtypes = []
        L.prox_noalloc_max_bytes.restype = S
        L.prox_ffn_sparse_staged.argtypes = [WP, PP, P, I, I, I, P, P, P, P, P, S, P, P]
        L.prox_ffn_sparse_tau.argtypes = [WP, PP, P, I, Z, Z, P, P, P, P, P, P, S, P]
        L.prox_reservoir_add.argtypes = [P, S, P, P, S, P]
        L.prox_quantile_threshold.argtypes = [P, S, ctypes.c_double, P]
        Dd = ctypes.c_double
        L.prox_effective_sparsity.argtypes = [Dd, Dd, Dd]
        L.prox_effective_sparsity.restype = Dd
        L.prox_allocate_sparsity.argtypes = [Dd, Dd, Dd, Dd, Dd, P, P]
        L.prox_sparse_stage_name.argtypes = [I]
        L.prox_sparse_stage_name.restype = ctypes.c_char_p
        L.prox_add_rmsnorm.argtypes = [P, P, I, I, I, Z, P, P]
        QP = ctypes.POINTER(_W4)
        L.prox_w4_bytes.argtypes = [I, I, I]
        L.prox_w4_bytes.restype = S
        L.prox_pack_w4.argtypes = [WP, QP, P]
        L.prox_unpack_w4.argtypes = [QP, I, P, P, P]
        L.prox_ffn_dense_w4.argtypes = [QP, P, I, P, P, S, P]
        L.prox_ffn_sparse_w4.argtypes = [QP, PP, P, I, I, I, P, P, P, P, P, S, P, P]
        L.prox_ffn_sparse_tau_w4.argtypes = [QP, PP, P, I, Z, Z, P, P, P, P, P, P, S, P]
        L.prox_strerror.argtypes = [I]
        L.prox_strerror.restype = ctypes.c_char_p
        for name in ("prox_pack_proxy", "prox_unpack_proxy", "prox_ffn_dense", "prox_ffn_sparse",
                     "prox_ffn_sparse_staged", "prox_ffn_sparse_tau", "prox_add_rmsnorm",
                     "prox_reservoir_add", "prox_quantile_threshold", "prox_allocate_sparsity",
                     "prox_pack_w4", "prox_unpack_w4", "prox_ffn_dense_w4", "prox_ffn_sparse_w4",
                     "prox_ffn_sparse_tau_w4"):
            getattr(L, name).restype = I
        _lib = L
    return _lib


def strerror(status: int) -> str:
    return lib().prox_strerror(int(status)).decode()


def stage_names() -> List[str]:
    return [lib().prox_sparse_stage_name(i).decode() for i in range(SPARSE_STAGES)]


def _check(status: int, where: str) -> None:
    if status != 0:
        raise ProxError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dev_tensor(t: torch.Tensor, what: str, dtype=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{what} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what} must have dtype {dtype}, got {t.dtype}")
    return t


@dataclasses.dataclass
class Weights:
    """Channel-major gated-FFN weights, each [d_ff][d_model] in fp16 or bf16;
    act is the gate activation (SILU: SwiGLU, GELU: GeGLU)."""
    w_gate: torch.Tensor
    w_up: torch.Tensor
    w_down: torch.Tensor
    act: int = SILU

    @property
    def d_ff(self) -> int:
        return self.w_gate.shape[0]

    @property
    def d_model(self) -> int:
        return self.w_gate.shape[1]

    @property
    def dtype(self) -> torch.dtype:
        return self.w_gate.dtype

    def struct(self) -> _Weights:
        dt = _TORCH_DT.get(self.w_gate.dtype)
        if dt is None:
            raise ValueError("weights must be float16 or bfloat16")
        for name in ("w_gate", "w_up", "w_down"):
            t = _dev_tensor(getattr(self, name), name, self.w_gate.dtype)
            if tuple(t.shape) != (self.d_ff, self.d_model):
                raise ValueError(f"{name} must be [d_ff][d_model]")
        return _Weights(self.d_model, self.d_ff, dt, self.w_gate.data_ptr(),
                        self.w_up.data_ptr(), self.w_down.data_ptr(), int(self.act))


@dataclasses.dataclass
class Proxy:
    """A packed proxy blob (opaque device bytes) with its format."""
    blob: torch.Tensor
    fmt: int
    group: int

    def struct(self) -> _Proxy:
        _dev_tensor(self.blob, "proxy blob", torch.uint8)
        return _Proxy(self.fmt, self.group, self.blob.data_ptr(), self.blob.numel())


def proxy_bytes(d_model: int, d_ff: int, fmt: int, group: int) -> int:
    return int(lib().prox_proxy_bytes(d_model, d_ff, fmt, group))


def stage1_mfma_rows(d_model: int, fmt: int, group: int, batch: int, k_in: int) -> int:
    """Batch rows per matrix-core Stage-1 launch, 0 when the dot-product
    kernel runs (threshold mode: pass k_in = d_model)."""
    return int(lib().prox_stage1_mfma_rows(d_model, fmt, group, batch, k_in))


def stage2_rows(d_model: int, d_ff: int, w4: bool, batch: int) -> int:
    """Batch rows per Stage-2 launch: 16 on the matrix-core kernel, else the
    VALU kernel's row count; 0 for an unsupported shape or batch."""
    return int(lib().prox_stage2_rows(d_model, d_ff, int(w4), batch))


def workspace_bytes(d_model: int, d_ff: int, batch: int, w4: bool = False) -> int:
    """prox_workspace_bytes, or prox_w4_workspace_bytes for INT4 base weights."""
    f = lib().prox_w4_workspace_bytes if w4 else lib().prox_workspace_bytes
    return int(f(d_model, d_ff, batch))


def new_workspace(d_model: int, d_ff: int, batch: int, device="cuda", w4: bool = False) -> torch.Tensor:
    n = workspace_bytes(d_model, d_ff, batch, w4)
    if n == 0:
        raise ProxError(2, "prox_w4_workspace_bytes" if w4 else "prox_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def pack_proxy(w: Weights, fmt: int = INT4, group: int = 128) -> Proxy:
    if fmt == NONE:
        group = w.d_model   # the unquantised proxy has one unit scale per channel
    n = proxy_bytes(w.d_model, w.d_ff, fmt, group)
    if n == 0:
        raise ProxError(2, "prox_proxy_bytes")
    p = Proxy(torch.empty(n, dtype=torch.uint8, device=w.w_gate.device), fmt, group)
    ws, ps = w.struct(), p.struct()
    _check(lib().prox_pack_proxy(ctypes.byref(ws), ctypes.byref(ps), _stream(w.w_gate.device)),
           "prox_pack_proxy")
    return p


def unpack_proxy(p: Proxy, d_model: int, d_ff: int):
    """(codes_gate int8 [f][d], scales_gate fp16-bits int16 [f][d/g], codes_up, scales_up)."""
    dev = p.blob.device
    ng = d_model // p.group
    cg = torch.empty((d_ff, d_model), dtype=torch.int8, device=dev)
    cu = torch.empty_like(cg)
    sg = torch.empty((d_ff, ng), dtype=torch.int16, device=dev)
    su = torch.empty_like(sg)
    ps = p.struct()
    _check(lib().prox_unpack_proxy(ctypes.byref(ps), d_model, d_ff, _ptr(cg), _ptr(sg), _ptr(cu),
                                   _ptr(su), _stream(dev)), "prox_unpack_proxy")
    return cg, sg, cu, su


def _as_batch(x: torch.Tensor, w: Weights) -> torch.Tensor:
    x = _dev_tensor(x, "x", w.dtype)
    if x.dim() == 1:
        x = x.view(1, -1)
    if x.dim() != 2 or x.shape[1] != w.d_model:
        raise ValueError("x must be [batch][d_model]")
    return x


def ffn_dense(w: Weights, x: torch.Tensor, y: Optional[torch.Tensor] = None,
              ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    x = _as_batch(x, w)
    B = x.shape[0]
    y = torch.empty_like(x) if y is None else _dev_tensor(y, "y", w.dtype)
    ws = new_workspace(w.d_model, w.d_ff, B, x.device) if ws is None else ws
    wst = w.struct()
    _check(lib().prox_ffn_dense(ctypes.byref(wst), _ptr(x), B, _ptr(y), _ptr(ws), ws.numel(),
                                _stream(x.device)), "prox_ffn_dense")
    return y


def ffn_sparse(w: Weights, p: Proxy, x: torch.Tensor, k_in: int, k_ff: int, *,
               y: Optional[torch.Tensor] = None, mask: Optional[torch.Tensor] = None,
               in_mask: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
               ws: Optional[torch.Tensor] = None,
               events: Optional[Sequence[torch.cuda.Event]] = None):
    """Prox sparse decode step.  Returns (y, mask).  ``in_mask`` / ``scores``
    are filled when given.  ``events`` (PROX_SPARSE_STAGES + 1 timing events,
    already recorded once so they exist) selects the staged entry point."""
    x = _as_batch(x, w)
    B = x.shape[0]
    dev = x.device
    y = torch.empty_like(x) if y is None else _dev_tensor(y, "y", w.dtype)
    mask = (torch.empty(w.d_ff, dtype=torch.uint8, device=dev) if mask is None
            else _dev_tensor(mask, "mask", torch.uint8))
    if in_mask is not None:
        _dev_tensor(in_mask, "in_mask", torch.uint8)
    if scores is not None:
        _dev_tensor(scores, "scores", torch.float32)
    ws = new_workspace(w.d_model, w.d_ff, B, dev) if ws is None else ws
    wst, pst = w.struct(), p.struct()
    args = [ctypes.byref(wst), ctypes.byref(pst), _ptr(x), B, int(k_in), int(k_ff), _ptr(y),
            _ptr(mask), _ptr(in_mask), _ptr(scores), _ptr(ws), ws.numel()]
    if events is None:
        _check(lib().prox_ffn_sparse(*args, _stream(dev)), "prox_ffn_sparse")
    else:
        if len(events) != SPARSE_STAGES + 1:
            raise ValueError(f"need {SPARSE_STAGES + 1} events")
        arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
        _check(lib().prox_ffn_sparse_staged(*args, arr, _stream(dev)), "prox_ffn_sparse_staged")
    return y, mask


def ffn_sparse_noalloc(w: Weights, p: Proxy, x: torch.Tensor, k_in: int, k_ff: int, *,
                       y: Optional[torch.Tensor] = None, mask: Optional[torch.Tensor] = None,
                       in_mask: Optional[torch.Tensor] = None,
                       scores: Optional[torch.Tensor] = None):
    """prox_ffn_sparse_noalloc: the sparse decode step on the library's own
    device scratch (no workspace argument; the C call allocates nothing).
    Returns (y, mask); y and mask are allocated here when not given."""
    x = _as_batch(x, w)
    B = x.shape[0]
    dev = x.device
    y = torch.empty_like(x) if y is None else _dev_tensor(y, "y", w.dtype)
    mask = (torch.empty(w.d_ff, dtype=torch.uint8, device=dev) if mask is None
            else _dev_tensor(mask, "mask", torch.uint8))
    if in_mask is not None:
        _dev_tensor(in_mask, "in_mask", torch.uint8)
    if scores is not None:
        _dev_tensor(scores, "scores", torch.float32)
    wst, pst = w.struct(), p.struct()
    _check(lib().prox_ffn_sparse_noalloc(ctypes.byref(wst), ctypes.byref(pst), _ptr(x), B,
                                         int(k_in), int(k_ff), _ptr(y), _ptr(mask),
                                         _ptr(in_mask), _ptr(scores), _stream(dev)),
           "prox_ffn_sparse_noalloc")
    return y, mask


def noalloc_max_bytes() -> int:
    """Scratch bytes per GPU of prox_ffn_sparse_noalloc (the workspace of a call
    must fit)."""
    return int(lib().prox_noalloc_max_bytes())


def ffn_sparse_tau(w: Weights, p: Proxy, x: torch.Tensor, tau_x: float, tau_s: float, *,
                   y: Optional[torch.Tensor] = None, mask: Optional[torch.Tensor] = None,
                   in_mask: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
                   counts: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """Prox decode step with layer-wise thresholds (keep |x| >= tau_x and
    score >= tau_s).  Returns (y, mask, counts) with counts an int32 [2]
    device tensor (k_in, k_ff realised by this call)."""
    x = _as_batch(x, w)
    B = x.shape[0]
    dev = x.device
    y = torch.empty_like(x) if y is None else _dev_tensor(y, "y", w.dtype)
    mask = (torch.empty(w.d_ff, dtype=torch.uint8, device=dev) if mask is None
            else _dev_tensor(mask, "mask", torch.uint8))
    counts = (torch.empty(2, dtype=torch.int32, device=dev) if counts is None
              else _dev_tensor(counts, "counts", torch.int32))
    if in_mask is not None:
        _dev_tensor(in_mask, "in_mask", torch.uint8)
    if scores is not None:
        _dev_tensor(scores, "scores", torch.float32)
    ws = new_workspace(w.d_model, w.d_ff, B, dev) if ws is None else ws
    wst, pst = w.struct(), p.struct()
    _check(lib().prox_ffn_sparse_tau(ctypes.byref(wst), ctypes.byref(pst), _ptr(x), B,
                                     float(tau_x), float(tau_s), _ptr(y), _ptr(mask),
                                     _ptr(in_mask), _ptr(scores), _ptr(counts), _ptr(ws),
                                     ws.numel(), _stream(dev)), "prox_ffn_sparse_tau")
    return y, mask, counts


@dataclasses.dataclass
class W4Weights:
    """INT4 copy of the three FFN matrices for Stage 2 (W4A16): an opaque
    device blob in the layout include/prox.h describes."""
    blob: torch.Tensor
    dtype: torch.dtype
    d_model: int
    d_ff: int
    group: int
    act: int = SILU

    def struct(self) -> _W4:
        _dev_tensor(self.blob, "W4 blob", torch.uint8)
        return _W4(_TORCH_DT[self.dtype], self.d_model, self.d_ff, self.group, int(self.act),
                   self.blob.data_ptr(), self.blob.numel())


def w4_bytes(d_model: int, d_ff: int, group: int = 128) -> int:
    return int(lib().prox_w4_bytes(d_model, d_ff, group))


def pack_w4(w: Weights, group: int = 128) -> W4Weights:
    n = w4_bytes(w.d_model, w.d_ff, group)
    if n == 0:
        raise ProxError(2, "prox_w4_bytes")
    q = W4Weights(torch.empty(n, dtype=torch.uint8, device=w.w_gate.device), w.dtype, w.d_model,
                  w.d_ff, group, w.act)
    ws, qs = w.struct(), q.struct()
    _check(lib().prox_pack_w4(ctypes.byref(ws), ctypes.byref(qs), _stream(w.w_gate.device)),
           "prox_pack_w4")
    return q


def unpack_w4(q: W4Weights, matrix: int):
    """(codes int8 [d_ff][d_model], scales fp16 bits int16 [d_ff][d_model / group]) of
    matrix 0 (gate), 1 (up) or 2 (down)."""
    dev = q.blob.device
    codes = torch.empty((q.d_ff, q.d_model), dtype=torch.int8, device=dev)
    scales = torch.empty((q.d_ff, q.d_model // q.group), dtype=torch.int16, device=dev)
    qs = q.struct()
    _check(lib().prox_unpack_w4(ctypes.byref(qs), int(matrix), _ptr(codes), _ptr(scales),
                                _stream(dev)), "prox_unpack_w4")
    return codes, scales


def _as_batch_w4(x: torch.Tensor, q: W4Weights) -> torch.Tensor:
    x = _dev_tensor(x, "x", q.dtype)
    if x.dim() == 1:
        x = x.view(1, -1)
    if x.dim() != 2 or x.shape[1] != q.d_model:
        raise ValueError("x must be [batch][d_model]")
    return x


def ffn_dense_w4(q: W4Weights, x: torch.Tensor, y: Optional[torch.Tensor] = None,
                 ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The dense FFN on the INT4 weights."""
    x = _as_batch_w4(x, q)
    B = x.shape[0]
    y = torch.empty_like(x) if y is None else _dev_tensor(y, "y", q.dtype)
    ws = new_workspace(q.d_model, q.d_ff, B, x.device, w4=True) if ws is None else ws
    qs = q.struct()
    _check(lib().prox_ffn_dense_w4(ctypes.byref(qs), _ptr(x), B, _ptr(y), _ptr(ws), ws.numel(),
                                   _stream(x.device)), "prox_ffn_dense_w4")
    return y


def ffn_sparse_w4(q: W4Weights, p: Proxy, x: torch.Tensor, k_in: int, k_ff: int, *,
                  y: Optional[torch.Tensor] = None, mask: Optional[torch.Tensor] = None,
                  in_mask: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
                  ws: Optional[torch.Tensor] = None,
                  events: Optional[Sequence[torch.cuda.Event]] = None):
    """The sparse decode step with Stage 2 on the INT4 weights.  Returns
    (y, mask); arguments as ffn_sparse."""
    x = _as_batch_w4(x, q)
    B = x.shape[0]
    dev = x.device
    y = torch.empty_like(x) if y is None else _dev_tensor(y, "y", q.dtype)
    mask = (torch.empty(q.d_ff, dtype=torch.uint8, device=dev) if mask is None
            else _dev_tensor(mask, "mask", torch.uint8))
    if in_mask is not None:
        _dev_tensor(in_mask, "in_mask", torch.uint8)
    if scores is not None:
        _dev_tensor(scores, "scores", torch.float32)
    ws = new_workspace(q.d_model, q.d_ff, B, dev, w4=True) if ws is None else ws
    arr = None
    if events is not None:
        if len(events) != SPARSE_STAGES + 1:
            raise ValueError(f"need {SPARSE_STAGES + 1} events")
        arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    qs, pst = q.struct(), p.struct()
    _check(lib().prox_ffn_sparse_w4(ctypes.byref(qs), ctypes.byref(pst), _ptr(x), B, int(k_in),
                                    int(k_ff), _ptr(y), _ptr(mask), _ptr(in_mask), _ptr(scores),
                                    _ptr(ws), ws.numel(), arr, _stream(dev)), "prox_ffn_sparse_w4")
    return y, mask


def ffn_sparse_tau_w4(q: W4Weights, p: Proxy, x: torch.Tensor, tau_x: float, tau_s: float, *,
                      y: Optional[torch.Tensor] = None, mask: Optional[torch.Tensor] = None,
                      in_mask: Optional[torch.Tensor] = None,
                      scores: Optional[torch.Tensor] = None,
                      counts: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """Threshold-mode step with Stage 2 on the INT4 weights.  Returns
    (y, mask, counts) like ffn_sparse_tau."""
    x = _as_batch_w4(x, q)
    B = x.shape[0]
    dev = x.device
    y = torch.empty_like(x) if y is None else _dev_tensor(y, "y", q.dtype)
    mask = (torch.empty(q.d_ff, dtype=torch.uint8, device=dev) if mask is None
            else _dev_tensor(mask, "mask", torch.uint8))
    counts = (torch.empty(2, dtype=torch.int32, device=dev) if counts is None
              else _dev_tensor(counts, "counts", torch.int32))
    if in_mask is not None:
        _dev_tensor(in_mask, "in_mask", torch.uint8)
    if scores is not None:
        _dev_tensor(scores, "scores", torch.float32)
    ws = new_workspace(q.d_model, q.d_ff, B, dev, w4=True) if ws is None else ws
    qs, pst = q.struct(), p.struct()
    _check(lib().prox_ffn_sparse_tau_w4(ctypes.byref(qs), ctypes.byref(pst), _ptr(x), B,
                                        float(tau_x), float(tau_s), _ptr(y), _ptr(mask),
                                        _ptr(in_mask), _ptr(scores), _ptr(counts), _ptr(ws),
                                        ws.numel(), _stream(dev)), "prox_ffn_sparse_tau_w4")
    return y, mask, counts


def effective_sparsity(s1: float, s2: float, alpha: float = 1.0 / 3.0) -> float:
    """Sec. 4.2 effective sparsity of stage sparsities (s1, s2)."""
    return float(lib().prox_effective_sparsity(float(s1), float(s2), float(alpha)))


def allocate_sparsity(e: float, alpha: float = 1.0 / 3.0, s_ref: float = 0.7,
                      s1_min: float = 0.0, s1_max: float = 0.7):
    """Sec. 4.2 allocation of a target effective sparsity: (s1, s2)."""
    a, b = ctypes.c_double(), ctypes.c_double()
    _check(lib().prox_allocate_sparsity(float(e), float(alpha), float(s_ref), float(s1_min),
                                        float(s1_max), ctypes.byref(a), ctypes.byref(b)),
           "prox_allocate_sparsity")
    return a.value, b.value


def add_rmsnorm(x: torch.Tensor, y: torch.Tensor, eps: float = 1e-6,
                out: Optional[torch.Tensor] = None) -> torch.Tensor:
    dt = _TORCH_DT.get(x.dtype)
    if dt is None:
        raise ValueError("x must be float16 or bfloat16")
    x = _dev_tensor(x, "x")
    y = _dev_tensor(y, "y", x.dtype)
    x2 = x.view(1, -1) if x.dim() == 1 else x
    out = torch.empty_like(x) if out is None else _dev_tensor(out, "out", x.dtype)
    _check(lib().prox_add_rmsnorm(_ptr(x), _ptr(y), x2.shape[0], x2.shape[1], dt,
                                  ctypes.c_float(eps), _ptr(out), _stream(x.device)),
           "prox_add_rmsnorm")
    return out


def from_bits(bits, dtype_code: int, device="cuda") -> torch.Tensor:
    """numpy uint16 bit patterns -> device tensor of the matching 16-bit dtype."""
    import numpy as np
    t = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    return t.to(device).view(_DT_TORCH[dtype_code])


def to_bits(t: torch.Tensor):
    """Device 16-bit tensor -> numpy uint16 bit patterns."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view("uint16")
