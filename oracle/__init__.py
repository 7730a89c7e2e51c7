"""TEST INFRASTRUCTURE ONLY: the CPU oracle of one SkewAdam step.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package. It shares no code with the GPU library: the step itself
is plain C in ``skew_oracle.c`` (loaded through ctypes), and the closed-form state
model of Eq. 2 / Table 6 is plain Python below.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field
from typing import Iterable, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libskew_oracle.so")
SRC_PATH = os.path.join(HERE, "skew_oracle.c")

BACKBONE, EXPERT, ROUTER = 0, 1, 2
TIER_NAMES = {"backbone": BACKBONE, "expert": EXPERT, "router": ROUTER}

# Paper defaults (Alg. 1 caption, Table 5): beta = (0.9, 0.999), eps = 1e-8,
# lr = 3e-4; update clipping at RMS 1 (Sec. 3).
DEFAULTS = dict(lr=3e-4, beta1=0.9, beta2=0.999, eps=1e-8, clip_threshold=1.0)
# tier variants of the ablation (Table 3): momentum in any tier; router matrices factored;
# float32 master weights and gradients for exact-moment tensors (fp32 router and norms)
STATE_MOMENTUM, STATE_FACTORED, STATE_FP32 = 1, 2, 4


def build(verbose: bool = False) -> str:
    """Compile the oracle with plain IEEE float semantics (no contraction, no fast-math)."""
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
           "-std=c11", "-Wall", "-o", LIB_PATH + ".tmp", SRC_PATH, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd, cwd=HERE)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


class _Tensor(ctypes.Structure):
    _fields_ = [
        ("tier", ctypes.c_int32), ("ndim", ctypes.c_int32),
        ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
        ("tensor_id", ctypes.c_uint64),
        ("w", ctypes.c_void_p), ("g", ctypes.c_void_p),
        ("m", ctypes.c_void_p), ("v", ctypes.c_void_p),
        ("r", ctypes.c_void_p), ("c", ctypes.c_void_p),
        ("u_out", ctypes.c_void_p), ("x_out", ctypes.c_void_p), ("y_out", ctypes.c_void_p),
        ("rms_out", ctypes.c_void_p),
        ("batch", ctypes.c_int64), ("state_flags", ctypes.c_uint32),
    ]


class _HParams(ctypes.Structure):
    _fields_ = [
        ("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float), ("clip_threshold", ctypes.c_float),
        ("step", ctypes.c_int64), ("seed", ctypes.c_uint64),
        ("weight_decay", ctypes.c_float), ("max_grad_norm", ctypes.c_float), ("gsq_total", ctypes.c_double),
        ("exact_ulp", ctypes.c_int32), ("rbar_min_only", ctypes.c_int32),
    ]


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        L.skew_oracle_step.argtypes = [ctypes.POINTER(_HParams), ctypes.POINTER(_Tensor), ctypes.c_int]
        L.skew_oracle_step.restype = ctypes.c_int
        L.skew_oracle_step_gcoef.argtypes = [ctypes.POINTER(_HParams), ctypes.POINTER(_Tensor), ctypes.c_int,
                                             ctypes.POINTER(ctypes.c_float)]
        L.skew_oracle_step_gcoef.restype = ctypes.c_int
        L.skew_oracle_f32_to_bf16.argtypes = [ctypes.c_float]
        L.skew_oracle_f32_to_bf16.restype = ctypes.c_uint16
        L.skew_oracle_f32_to_bf16_array.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        L.skew_oracle_mix64.argtypes = [ctypes.c_uint64]
        L.skew_oracle_mix64.restype = ctypes.c_uint64
        L.skew_oracle_fmix32.argtypes = [ctypes.c_uint32]
        L.skew_oracle_fmix32.restype = ctypes.c_uint32
        L.skew_oracle_key.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_uint64]
        L.skew_oracle_key.restype = ctypes.c_uint64
        L.skew_oracle_u16.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.skew_oracle_u16.restype = ctypes.c_uint32
        L.skew_oracle_u16_array.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p]
        L.skew_oracle_threads.restype = ctypes.c_int
        L.skew_oracle_sumsq_bf16.argtypes = [ctypes.c_void_p, ctypes.c_int64]
        L.skew_oracle_sumsq_bf16.restype = ctypes.c_double
        L.skew_oracle_set_threads.argtypes = [ctypes.c_int]
        L.skew_oracle_set_threads.restype = None
        _LIB = L
    return _LIB


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


@dataclass
class Tensor:
    """One parameter tensor and its state, as dense row-major numpy arrays."""
    tier: int
    w: np.ndarray                 # uint16 bf16 bits, shape (rows, cols) or (n,)
    g: np.ndarray                 # uint16 bf16 bits, same shape
    tensor_id: int
    m: Optional[np.ndarray] = None
    v: Optional[np.ndarray] = None
    r: Optional[np.ndarray] = None
    c: Optional[np.ndarray] = None
    u_out: Optional[np.ndarray] = field(default=None, repr=False)
    x_out: Optional[np.ndarray] = field(default=None, repr=False)
    y_out: Optional[np.ndarray] = field(default=None, repr=False)
    rms: float = float("nan")
    state_flags: int = 0          # STATE_MOMENTUM | STATE_FACTORED (tier variants, Table 3)

    @property
    def ndim(self) -> int:
        return self.w.ndim

    @property
    def batch(self) -> int:
        """E for a stacked (E, rows, cols) tensor, else 1."""
        return int(self.w.shape[0]) if self.w.ndim == 3 else 1

    @property
    def rows_cols(self):
        if self.w.ndim == 1:
            return 1, int(self.w.shape[0])
        return int(self.w.shape[-2]), int(self.w.shape[-1])

    @property
    def exact(self) -> bool:
        return (self.tier == ROUTER and not (self.state_flags & STATE_FACTORED)) or self.ndim == 1

    @property
    def momentum(self) -> bool:
        return self.tier == BACKBONE or bool(self.state_flags & STATE_MOMENTUM)

    def init_state(self):
        """Allocate zeroed state for this tensor's tier (Fig. 1, Table 6) and variant
        (Table 3); a stacked tensor keeps R [E, rows] and C [E, cols]."""
        n, m = self.rows_cols
        shape = self.w.shape
        if self.momentum:
            self.m = np.zeros(shape, np.float32)
        if self.exact:
            self.v = np.zeros(shape, np.float32)
        else:
            self.r = np.zeros((self.batch, n) if self.ndim == 3 else n, np.float32)
            self.c = np.zeros((self.batch, m) if self.ndim == 3 else m, np.float32)
        return self


def step(tensors: Iterable[Tensor], step: int, seed: int = 0, lr: float = DEFAULTS["lr"],
         beta1: float = DEFAULTS["beta1"], beta2: float = DEFAULTS["beta2"], eps: float = DEFAULTS["eps"],
         clip_threshold: float = DEFAULTS["clip_threshold"], want_u: bool = False, want_x: bool = False,
         want_y: bool = False, weight_decay: float = 0.0, max_grad_norm: float = 0.0,
         gsq_total: Optional[float] = None, exact_ulp: bool = False, rbar_min_only: bool = False) -> int:
    """Run one oracle step over ``tensors`` in place. Returns the C status.

    weight_decay: lambda of the decoupled decay (router tier exempt). max_grad_norm > 0
    scales every gradient by min(1, max_grad_norm / (||G|| + 1e-6)) over all the tensors
    given, or over a larger set whose sum of squares is ``gsq_total``. The scale used is
    returned by ``last_gcoef()``. exact_ulp: the dither spans the exact bf16 ulp of w.
    Tensors with STATE_FP32 hold float32 w and g (the arrays' dtype) and skip the cast.
    rbar_min_only: the other reading of Alg. 1's eps-clamps (mean(R) guarded at FLT_MIN
    instead of clamped at eps), for the sensitivity check of that reading only."""
    tensors = list(tensors)
    arr = (_Tensor * max(1, len(tensors)))()
    rms = np.full(max(1, len(tensors)), np.nan, np.float64)
    keep = []
    for k, t in enumerate(tensors):
        for name in ("w", "g", "m", "v", "r", "c"):
            a = getattr(t, name)
            if a is not None:
                assert a.flags["C_CONTIGUOUS"], name
        want = np.float32 if t.state_flags & STATE_FP32 else np.uint16
        assert t.w.dtype == want and t.g.dtype == want and t.w.shape == t.g.shape
        n, m = t.rows_cols
        E = t.batch
        if n * m > 0:
            if t.momentum:
                assert t.m is not None and t.m.dtype == np.float32 and t.m.size == E * n * m
            if t.exact:
                assert t.v is not None and t.v.dtype == np.float32 and t.v.size == E * n * m
            else:
                assert t.r is not None and t.r.size == E * n and t.c is not None and t.c.size == E * m
        if want_u:
            t.u_out = np.empty(t.w.shape, np.float32)
        if want_x:
            t.x_out = np.empty(t.w.shape, np.float32)
        if want_y:
            t.y_out = np.empty(t.w.shape, np.float32)
        arr[k] = _Tensor(t.tier, t.ndim, n, m, t.tensor_id, _ptr(t.w), _ptr(t.g), _ptr(t.m), _ptr(t.v),
                         _ptr(t.r), _ptr(t.c), _ptr(t.u_out), _ptr(t.x_out), _ptr(t.y_out),
                         rms.ctypes.data + 8 * k, E if t.ndim == 3 else 0, int(t.state_flags))
        keep.append(t)
    hp = _HParams(lr, beta1, beta2, eps, clip_threshold, int(step), int(seed) & (2**64 - 1),
                  weight_decay, max_grad_norm, -1.0 if gsq_total is None else float(gsq_total), int(exact_ulp),
                  int(rbar_min_only))
    gc = ctypes.c_float(0.0)
    rc = lib().skew_oracle_step_gcoef(ctypes.byref(hp), arr, len(tensors), ctypes.byref(gc))
    global _LAST_GCOEF
    _LAST_GCOEF = float(gc.value)
    for k, t in enumerate(tensors):
        t.rms = float(rms[k])
    return rc


_LAST_GCOEF = 1.0


def last_gcoef() -> float:
    """The gradient scale of the last ``step`` (1.0 without max_grad_norm)."""
    return _LAST_GCOEF


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bits, round to nearest even (the cast of Alg. 1)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().skew_oracle_f32_to_bf16_array(x.ctypes.data, out.ctypes.data, x.size)
    return out


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def mix64(z: int) -> int:
    return int(lib().skew_oracle_mix64(z & (2**64 - 1)))


def fmix32(h: int) -> int:
    return int(lib().skew_oracle_fmix32(h & 0xFFFFFFFF))


def dither_key(seed: int, step: int, tensor_id: int) -> int:
    return int(lib().skew_oracle_key(seed & (2**64 - 1), step, tensor_id & (2**64 - 1)))


def dither_u16(key: int, idx0: int, n: int) -> np.ndarray:
    out = np.empty(n, np.uint32)
    lib().skew_oracle_u16_array(key, idx0, n, out.ctypes.data)
    return out


def threads() -> int:
    return int(lib().skew_oracle_threads())


def sumsq_bf16(g: np.ndarray) -> float:
    """Sum of squares in double of bf16 values (uint16 bits): a set's squared gradient norm."""
    g = np.ascontiguousarray(g, np.uint16)
    return float(lib().skew_oracle_sumsq_bf16(g.ctypes.data, g.size))


def set_threads(n: int) -> None:
    """OpenMP threads of later oracle steps (the results do not depend on the count)."""
    lib().skew_oracle_set_threads(int(n))


# ----------------------------------------------------------------------------------------
# Closed-form state model: Eq. 2 plus the exact-v term of the vector parameters (Table 6).
# ----------------------------------------------------------------------------------------
POLICIES = ("skewadam", "expert_momentum", "factored_router", "uniform")


def tensor_state_parts(tier: int, shape, policy: str = "skewadam") -> dict:
    """fp32 state entries one tensor keeps under a tier policy, split by kind.

    ``m``: momentum; ``v``: exact second moment; ``rc``: factored row + column
    statistics (Fig. 1; Sec. 3 "The tiers"; Table 3 for the variant policies).
    """
    assert policy in POLICIES
    dims = tuple(int(s) for s in shape)
    N = int(np.prod(dims, dtype=np.int64)) if dims else 1
    parts = {"m": 0, "v": 0, "rc": 0}
    if N == 0:
        return parts
    momentum = tier == BACKBONE or (tier == EXPERT and policy in ("expert_momentum", "uniform")) \
        or (tier == ROUTER and policy == "uniform")
    if len(dims) == 1:
        parts["v"] = N                     # vectors keep an exact v (Alg. 1)
    elif tier == ROUTER and policy not in ("factored_router", "uniform"):
        parts["v"] = N                     # the router keeps an exact v (Sec. 3, "The tiers")
    else:
        n, m = dims[-2], dims[-1]
        lead = N // (n * m)                # stacked (E, n, m) tensors factor over the last two axes
        parts["rc"] = lead * (n + m)       # Eq. 1: R in R^n, C in R^m
    if momentum:
        parts["m"] = N
    return parts


def tensor_state_floats(tier: int, shape, policy: str = "skewadam") -> int:
    return sum(tensor_state_parts(tier, shape, policy).values())


def state_bytes(tensors, policy: str = "skewadam") -> int:
    """Eq. 2 (plus vector v): 4 bytes per fp32 state entry; ``tensors`` = iterable of (tier, shape)."""
    return 4 * sum(tensor_state_floats(t, s, policy) for t, s in tensors)


def adamw_state_bytes(tensors) -> int:
    """AdamW keeps two fp32 moments per parameter (8 bytes, Sec. 1)."""
    return 8 * sum(int(np.prod(s, dtype=np.int64)) for _, s in tensors)
