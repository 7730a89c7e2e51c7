"""ctypes binding of ``include/skewadam.h``: argument marshalling only.

Every step of the optimizer runs in the HIP library ``libskewadam.so``. PyTorch
supplies device memory (the caller's bf16 weights and gradients, and the state and
workspace buffers this wrapper allocates) and the HIP stream. There is no fallback:
without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Iterable, List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libskewadam.so")

SKEW_OK, SKEW_EINVAL, SKEW_ENOSPACE, SKEW_EHIP, SKEW_ENOMEM, SKEW_ESTALE, SKEW_ETOOBIG = 0, -1, -2, -3, -4, -5, -6
STATIC_WORKSPACE_BYTES = 64 << 20   # SKEW_STATIC_WORKSPACE_BYTES
BACKBONE, EXPERT, ROUTER = 0, 1, 2
FLAG_EXACT_CLIP = 1
STATE_MOMENTUM, STATE_FACTORED, STATE_FP32 = 1, 2, 4   # tier variants (SKEW_STATE_*)
FLAG_EXACT_ULP = 2
TIERS = {"backbone": BACKBONE, "expert": EXPERT, "router": ROUTER}
ABI_VERSION = 4

# names every build of the library exports (checked by the CPU test suite)
EXPORTS = ("skew_state_bytes", "skew_state_init", "skew_state_init_static", "skew_step", "skew_destroy", "skew_strerror",
           "skew_abi_version", "skew_timing_enable", "skew_timing_read", "skew_launch_name", "skew_clip_info")


class SkewError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {_strerror(status)} (status {status})")
        self.status = status


class TensorDesc(ctypes.Structure):
    _fields_ = [
        ("tier", ctypes.c_int32), ("ndim", ctypes.c_int32),
        ("rows", ctypes.c_int64), ("cols", ctypes.c_int64), ("ld", ctypes.c_int64),
        ("tensor_id", ctypes.c_uint64),
        ("w", ctypes.c_void_p), ("g", ctypes.c_void_p),
        ("m", ctypes.c_void_p), ("v", ctypes.c_void_p), ("r", ctypes.c_void_p), ("c", ctypes.c_void_p),
        ("batch", ctypes.c_int64), ("state_flags", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
    ]


class HParams(ctypes.Structure):
    _fields_ = [
        ("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float), ("clip_threshold", ctypes.c_float), ("flags", ctypes.c_int32),
        ("step", ctypes.c_int64), ("seed", ctypes.c_uint64),
        ("weight_decay", ctypes.c_float), ("max_grad_norm", ctypes.c_float),
    ]


_LIB = None


def lib():
    """Load the in-tree HIP library; raise if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; "
                               "g.build()'` (hipcc, gfx950); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        L.skew_state_bytes.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t),
                                       ctypes.POINTER(ctypes.c_size_t)]
        L.skew_state_bytes.restype = ctypes.c_int
        L.skew_state_init.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_int,
                                      ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_size_t,
                                      ctypes.c_void_p]
        L.skew_state_init.restype = ctypes.c_int
        L.skew_state_init_static.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_int,
                                             ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.skew_state_init_static.restype = ctypes.c_int
        L.skew_step.argtypes = [ctypes.c_void_p, ctypes.POINTER(HParams), ctypes.c_void_p]
        L.skew_step.restype = ctypes.c_int
        L.skew_destroy.argtypes = [ctypes.c_void_p]
        L.skew_destroy.restype = None
        L.skew_strerror.argtypes = [ctypes.c_int]
        L.skew_strerror.restype = ctypes.c_char_p
        L.skew_abi_version.restype = ctypes.c_int
        L.skew_timing_enable.argtypes = [ctypes.c_void_p, ctypes.c_int]
        L.skew_timing_enable.restype = ctypes.c_int
        L.skew_timing_read.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_double), ctypes.c_int,
                                       ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)]
        L.skew_timing_read.restype = ctypes.c_int
        L.skew_launch_name.argtypes = [ctypes.c_void_p, ctypes.c_int]
        L.skew_launch_name.restype = ctypes.c_char_p
        L.skew_clip_info.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_int32),
                                     ctypes.c_int, ctypes.c_void_p]
        L.skew_clip_info.restype = ctypes.c_int
        if L.skew_abi_version() != ABI_VERSION:
            raise RuntimeError("libskewadam.so ABI version mismatch")
        _LIB = L
    return _LIB


def _strerror(status: int) -> str:
    try:
        return lib().skew_strerror(status).decode()
    except Exception:  # the library itself may be what failed to load
        return "status"


def make_desc(tier: int, ndim: int, rows: int, cols: int, ld: int, tensor_id: int, w_ptr: int = 0,
              g_ptr: int = 0, batch: int = 0, state_flags: int = 0) -> TensorDesc:
    return TensorDesc(tier, ndim, rows, cols, ld, tensor_id & (2**64 - 1), w_ptr or None, g_ptr or None,
                      None, None, None, None, batch, state_flags, 0)


def state_bytes(descs: Sequence[TensorDesc]):
    """(state_bytes, workspace_bytes) for a descriptor table; host only, needs no GPU."""
    arr = (TensorDesc * max(1, len(descs)))(*descs)
    sb, wb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    rc = lib().skew_state_bytes(arr, len(descs), ctypes.byref(sb), ctypes.byref(wb))
    if rc != SKEW_OK:
        raise SkewError(rc, "skew_state_bytes")
    return sb.value, wb.value


def _desc_for(tier: int, w, g, tensor_id: int, state_flags: int = 0) -> TensorDesc:
    import torch
    want = torch.float32 if state_flags & STATE_FP32 else torch.bfloat16
    if w.dtype != want or g.dtype != want:
        raise TypeError(f"weights and gradients must be {want} for these state flags")
    if w.device.type != "cuda" or g.device != w.device:
        raise TypeError("weights and gradients must live on the same HIP device")
    if w.shape != g.shape or w.stride() != g.stride():
        raise ValueError("weight and gradient must have the same shape and strides")
    if w.dim() == 1:
        if w.numel() > 1 and w.stride(0) != 1:
            raise ValueError("vectors must be contiguous")
        return make_desc(tier, 1, 1, w.shape[0], max(1, w.shape[0]), tensor_id, w.data_ptr(), g.data_ptr(),
                         state_flags=state_flags)
    if w.dim() == 3:
        # stacked (E, n, m): slices at a stride of n * ld elements
        E, n, m = w.shape
        if m > 1 and w.stride(2) != 1:
            raise ValueError("stacked matrices must be row-major (unit column stride)")
        ld = w.stride(1) if n > 1 else max(1, m)
        if n > 1 and m > 0 and ld < m:
            # rows that overlap (an expanded or unfolded view): the kernels write rows * ld
            # elements in place, so such a view is refused rather than widened
            raise ValueError(f"row stride {ld} is smaller than the row length {m} (overlapping rows)")
        ld = max(ld, 1)
        if E > 1 and n * m > 0 and w.stride(0) != n * ld:   # (a tensor with no elements has no layout)
            raise ValueError("stacked slices must follow each other (slice stride rows * ld)")
        return make_desc(tier, 3, n, m, ld, tensor_id, w.data_ptr(), g.data_ptr(), batch=E,
                         state_flags=state_flags)
    if w.dim() != 2:
        raise ValueError("only vectors, matrices and stacked matrices are supported")
    n, m = w.shape
    if m > 1 and w.stride(1) != 1:
        raise ValueError("matrices must be row-major (unit column stride)")
    ld = w.stride(0) if n > 1 else max(1, m)
    if n > 1 and m > 0 and ld < m:
        raise ValueError(f"row stride {ld} is smaller than the row length {m} (overlapping rows)")
    return make_desc(tier, 2, n, m, max(ld, 1), tensor_id, w.data_ptr(), g.data_ptr(), state_flags=state_flags)


class SkewAdam:
    """One SkewAdam context over a fixed set of (tier, weight, gradient) tensors.

    ``params`` is a list of ``(tier, w, g, tensor_id)`` or ``(tier, w, g, tensor_id,
    state_flags)`` with bf16 CUDA/HIP tensors: vectors, matrices or stacked (E, n, m)
    matrices; ``state_flags`` takes STATE_MOMENTUM / STATE_FACTORED (tier variants).
    The state and workspace are allocated here as torch byte tensors on the same
    device; weights, gradients and these buffers must outlive the object.
    ``static_workspace=True`` sets the context up with skew_state_init_static: the
    library's own static workspace replaces the workspace buffer (one such context per
    GPU at a time; see include/skewadam.h).
    """

    def __init__(self, params: Iterable, stream=None, static_workspace: bool = False):
        import torch
        params = list(params)
        self._keep = params
        self.descs = [_desc_for(TIERS.get(p[0], p[0]), p[1], p[2], p[3], p[4] if len(p) > 4 else 0)
                      for p in params]
        self.device = params[0][1].device if params else torch.device("cuda", torch.cuda.current_device())
        sb, wb = state_bytes(self.descs)
        self.state = torch.empty(max(sb, 1), dtype=torch.uint8, device=self.device)
        self.workspace = None if static_workspace else torch.empty(max(wb, 1), dtype=torch.uint8, device=self.device)
        self.state_nbytes, self.workspace_nbytes = sb, wb
        self._arr = (TensorDesc * max(1, len(self.descs)))(*self.descs)
        ctx = ctypes.c_void_p()
        s = self._stream(stream)
        if static_workspace:
            rc = lib().skew_state_init_static(ctypes.byref(ctx), self._arr, len(self.descs), self.state.data_ptr(),
                                              self.state.numel(), s)
            what = "skew_state_init_static"
        else:
            rc = lib().skew_state_init(ctypes.byref(ctx), self._arr, len(self.descs), self.state.data_ptr(),
                                       self.state.numel(), self.workspace.data_ptr(), self.workspace.numel(), s)
            what = "skew_state_init"
        if rc != SKEW_OK:
            raise SkewError(rc, what)
        self._ctx = ctx
        self._lib = lib()

    @staticmethod
    def _stream(stream) -> Optional[int]:
        import torch
        if stream is None:
            stream = torch.cuda.current_stream()
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream

    def step(self, step: int, lr: float = 3e-4, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
             clip_threshold: float = 1.0, seed: int = 0, stream=None, flags: int = 0, weight_decay: float = 0.0,
             max_grad_norm: float = 0.0) -> None:
        hp = HParams(lr, beta1, beta2, eps, clip_threshold, int(flags), int(step), int(seed) & (2**64 - 1),
                     weight_decay, max_grad_norm)
        rc = self._lib.skew_step(self._ctx, ctypes.byref(hp), self._stream(stream))
        if rc != SKEW_OK:
            raise SkewError(rc, "skew_step")

    def timing_enable(self, max_steps: int) -> None:
        """Record HIP events around each of the library's kernels for the next max_steps steps."""
        rc = self._lib.skew_timing_enable(self._ctx, int(max_steps))
        if rc != SKEW_OK:
            raise SkewError(rc, "skew_timing_enable")

    def timing_read(self) -> dict:
        """{kernel name: summed milliseconds} over the recorded steps, plus '_steps'."""
        ms = (ctypes.c_double * 16)()
        nl, ns = ctypes.c_int(), ctypes.c_int()
        rc = self._lib.skew_timing_read(self._ctx, ms, 16, ctypes.byref(nl), ctypes.byref(ns))
        if rc != SKEW_OK:
            raise SkewError(rc, "skew_timing_read")
        out = {self._lib.skew_launch_name(self._ctx, j).decode(): ms[j] for j in range(nl.value)}
        out["_steps"] = ns.value
        return out

    def clip_info(self, stream=None):
        """(k, route) lists of the last step, one entry per tensor (see skew_clip_info)."""
        n = max(1, len(self.descs))
        k = (ctypes.c_float * n)()
        route = (ctypes.c_int32 * n)()
        rc = self._lib.skew_clip_info(self._ctx, k, route, n, self._stream(stream))
        if rc != SKEW_OK:
            raise SkewError(rc, "skew_clip_info")
        return list(k)[:len(self.descs)], list(route)[:len(self.descs)]

    def state_views(self, i: int) -> dict:
        """float32 torch views of tensor i's state slices (m, v, r, c; absent ones omitted)."""
        import torch
        d = self._arr[i]
        n, m = (1, d.rows * d.cols) if d.ndim == 1 else (d.rows, d.cols)
        E = d.batch if d.ndim == 3 else 1
        shape = {"m": (E * n * m,), "v": (E * n * m,), "r": (E * n,), "c": (E * m,)}
        base = self.state.data_ptr()
        out = {}
        for name in ("m", "v", "r", "c"):
            p = getattr(d, name)
            if p:
                off = p - base
                cnt = shape[name][0]
                out[name] = self.state[off:off + 4 * cnt].view(torch.float32)
        return out

    def close(self) -> None:
        if getattr(self, "_ctx", None):
            self._lib.skew_destroy(self._ctx)
            self._ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
