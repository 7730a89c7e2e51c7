"""GPU-vs-oracle parity harness.

Bar (per step, per compared tensor):
  M, V        bit-identical (no reduction feeds them; same fma sites on both sides)
  R, C        |gpu - oracle| <= 1e-5 |oracle| elementwise
  W (bf16)    bit-identical, except where the oracle's pre-round float y lies within
              1e-6 |y| of a round-to-nearest-even boundary; such a mismatch must be one
              bf16 step. The share of mismatched elements is reported and must be <= 1e-4.
After each compared step the oracle takes the GPU's weight wherever the two differ (an
allowed one-step mismatch): the next update depends on W (the dither scales with |W| and
the decay with W), so both sides start every step from the same weights and every element
stays compared at every step.
"""
from __future__ import annotations

import sys
import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch

import oracle
from paper_2607_19058_amd import SkewAdam
from paper_2607_19058_amd import workloads as W

REL_STATE = 1e-5
REL_WINDOW = 1e-6
MAX_MISMATCH_FRACTION = 1e-4


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def near_boundary(y: np.ndarray, rel: float = REL_WINDOW) -> np.ndarray:
    """True where float32 y lies within rel*|y| of the bf16 rounding boundary above its
    truncation (the only boundary between the two bf16 values around y)."""
    y = np.ascontiguousarray(y, np.float32)
    mid = ((y.view(np.uint32) & np.uint32(0xFFFF0000)) | np.uint32(0x8000)).view(np.float32)
    return np.abs(y.astype(np.float64) - mid.astype(np.float64)) <= rel * np.abs(y.astype(np.float64))


@dataclass
class Stats:
    compared: int = 0
    mismatched: int = 0
    outside_window: int = 0
    not_one_step: int = 0
    state_bad: Dict[str, int] = field(default_factory=dict)
    max_rel_rc: float = 0.0

    def fraction(self) -> float:
        return self.mismatched / max(1, self.compared)

    def ok(self) -> bool:
        return (self.outside_window == 0 and self.not_one_step == 0 and not self.state_bad
                and self.fraction() <= MAX_MISMATCH_FRACTION)

    def __str__(self):
        return (f"compared={self.compared} mismatched={self.mismatched} frac={self.fraction():.3g} "
                f"outside_window={self.outside_window} not_one_step={self.not_one_step} "
                f"max_rel_RC={self.max_rel_rc:.3g} state_bad={self.state_bad}")


def compare_tensor(name: str, o: "oracle.Tensor", gpu_w: np.ndarray, gpu_state: Dict[str, np.ndarray],
                   st: Stats) -> None:
    """Compare one tensor after a step: the oracle's arrays (``o``, stepped with want_y)
    against the GPU's weight (bf16 bits, or float32 values for float32 masters) and state
    arrays (float32, by name m, v, r, c), to the bar of this module. Where the weights
    differ by an allowed one-step mismatch, the oracle takes the GPU's weight."""
    for key in ("m", "v"):
        ref = getattr(o, key)
        if ref is None:
            assert key not in gpu_state, (name, key)
            continue
        got = gpu_state[key]
        bad = int(np.count_nonzero(got.view(np.uint32) != ref.ravel().view(np.uint32)))
        if bad:
            st.state_bad[f"{name}.{key}"] = bad
    for key in ("r", "c"):
        ref = getattr(o, key)
        if ref is None:
            assert key not in gpu_state, (name, key)
            continue
        got = gpu_state[key].astype(np.float64)
        r = ref.ravel().astype(np.float64)
        with np.errstate(invalid="ignore"):   # inf - inf where both are infinite
            err = np.abs(got - r)
        lim = REL_STATE * np.abs(r)
        same = (got == r) | (np.isnan(got) & np.isnan(r))   # equal infinities, NaN for NaN
        bad = int(np.count_nonzero(~((err <= lim) | same)))
        with np.errstate(invalid="ignore", divide="ignore"):
            rel = np.where(r != 0, err / np.abs(r), np.where(err == 0, 0.0, np.inf))
        if rel.size and not np.all(np.isnan(rel)):
            st.max_rel_rc = max(st.max_rel_rc, float(np.nanmax(rel)))
        if bad:
            st.state_bad[f"{name}.{key}"] = bad
    if o.w.dtype == np.float32:
        # float32 masters: the oracle's own float sequence, bit for bit
        gwf = gpu_w.reshape(o.w.shape)
        bad = int(np.count_nonzero(gwf.view(np.uint32) != o.w.view(np.uint32)))
        st.compared += o.w.size
        if bad:
            st.state_bad[f"{name}.w32"] = bad
        return
    gw = gpu_w.reshape(o.w.shape)
    ow = o.w
    mism = gw != ow
    both_nan = np.isnan(oracle.bf16_to_f32(gw)) & np.isnan(oracle.bf16_to_f32(ow))
    mism &= ~both_nan
    n_new = int(np.count_nonzero(mism))
    st.compared += int(ow.size)
    st.mismatched += n_new
    if n_new:
        y = o.y_out.reshape(ow.shape)[mism]
        outside = ~near_boundary(y)
        st.outside_window += int(np.count_nonzero(outside))
        if outside.any():
            pos = np.argwhere(mism)[outside][:4]
            for q in pos:
                q = tuple(q)
                yy = float(o.y_out.reshape(ow.shape)[q])
                log(f"    outside window: {name} idx={q} y_oracle={yy!r} gpu=0x{int(gw[q]):04x} "
                    f"oracle=0x{int(ow[q]):04x}")
        step_dist = np.abs(gw[mism].astype(np.int32) - ow[mism].astype(np.int32))
        st.not_one_step += int(np.count_nonzero(step_dist != 1))
        ow[mism] = gw[mism]   # both sides take the next step from the same weights


def merge(into: Stats, st: Stats) -> None:
    into.compared += st.compared
    into.mismatched += st.mismatched
    into.outside_window += st.outside_window
    into.not_one_step += st.not_one_step
    into.max_rel_rc = max(into.max_rel_rc, st.max_rel_rc)
    for key, v in st.state_bad.items():
        into.state_bad[key] = into.state_bad.get(key, 0) + v


class ParityRun:
    """Runs the HIP step over every tensor of a workload and the oracle over a sample."""

    def __init__(self, wl: W.Workload, sample: Optional[List[int]] = None, device="cuda", seed: int = 0,
                 hp: Optional[dict] = None, specs: Optional[List[W.Spec]] = None, flags: int = 0,
                 weights: Optional[List[torch.Tensor]] = None, grads: Optional[List[torch.Tensor]] = None):
        """weights, grads: the caller's tensors (e.g. strided or unaligned views), with the
        initial weights already in them; by default they are allocated here."""
        self.wl, self.device, self.seed, self.flags = wl, torch.device(device), seed, flags
        self.hp = dict(oracle.DEFAULTS) if hp is None else dict(hp)
        self.specs = specs if specs is not None else wl.specs
        self.W = weights if weights is not None else [W.init_weight(s, wl, self.device) for s in self.specs]
        self.G = grads if grads is not None else [
            torch.zeros(s.shape, dtype=torch.float32 if s.state_flags & oracle.STATE_FP32 else torch.bfloat16,
                        device=self.device) for s in self.specs]
        self.opt = SkewAdam([(s.tier, self.W[k], self.G[k], s.tensor_id, s.state_flags)
                             for k, s in enumerate(self.specs)])
        idx = list(range(len(self.specs))) if sample is None else list(sample)
        self.sample = idx
        self.O = {}
        for k in idx:
            s = self.specs[k]
            w = self._host(self.W[k])
            self.O[k] = oracle.Tensor(tier=s.tier, w=w.copy(), g=np.zeros_like(w), tensor_id=s.tensor_id,
                                      state_flags=s.state_flags).init_state()
        self.stats = Stats()

    def step(self, t: int, check: bool = True, mutate=None) -> Stats:
        scales = W.expert_scales(self.wl, t)
        for k, s in enumerate(self.specs):
            W.fill_grad(s, self.wl, t, self.G[k], scales)
        if mutate is not None:   # a test's change to this step's gradients (both sides see it)
            mutate(t, self.G)
        for k in self.sample:
            self.O[k].g = self._host(self.G[k])
        torch.cuda.synchronize()
        t0 = time.time()
        # the gradient-norm scaling couples every tensor: an oracle step over a sample gets the
        # whole set's sum of squares, formed here on the host from the bf16 bits
        extra = {}
        if self.hp.get("max_grad_norm", 0.0) > 0.0 and len(self.sample) < len(self.specs):
            extra["gsq_total"] = sum(oracle.sumsq_bf16(bits(G)) if G.dtype == torch.bfloat16 else
                                     float(np.sum(G.detach().cpu().numpy().astype(np.float64) ** 2))
                                     for G in self.G)
        self.opt.step(t, seed=self.seed, flags=self.flags, **self.hp)
        torch.cuda.synchronize()
        t1 = time.time()
        if self.flags & 2:   # the exact-ulp dither
            extra["exact_ulp"] = True
        oracle.step([self.O[k] for k in self.sample], t, seed=self.seed, want_y=True, **self.hp, **extra)
        t2 = time.time()
        st = Stats()
        if check:
            for k in self.sample:
                self._compare(k, st)
        merge(self.stats, st)
        log(f"  step {t}: gpu {1e3 * (t1 - t0):.1f} ms, oracle {t2 - t1:.2f} s; {st}")
        return st

    @staticmethod
    def _host(t: torch.Tensor) -> np.ndarray:
        """bf16 bits (uint16), or float32 values for float32 masters."""
        return t.detach().cpu().numpy().copy() if t.dtype == torch.float32 else bits(t)

    def _compare(self, k: int, st: Stats):
        views = {name: v.cpu().numpy() for name, v in self.opt.state_views(k).items()}
        gw = self.W[k]
        gpu_w = gw.detach().cpu().numpy() if gw.dtype == torch.float32 else bits(gw)
        compare_tensor(self.specs[k].name, self.O[k], gpu_w, views, st)


class StreamParity:
    """Every tensor of a full-size workload compared at chosen steps, without an oracle
    trajectory in host memory. Before a step that may be compared, the GPU's weights and
    state are copied to the host; after it, each tensor's oracle step starts from those
    copies and its result is compared with the GPU's (so each compared step checks the
    GPU's step from the very inputs it had). Host memory holds the snapshot and one tensor's
    oracle arrays at a time."""

    ROUTES = {0: "fast sums", 4: "re-check with the exact floor split", 2: "re-check with the exact float sequence"}

    def __init__(self, wl: W.Workload, device="cuda", seed: int = 0, hp: Optional[dict] = None, flags: int = 0):
        self.wl, self.device, self.seed, self.flags = wl, torch.device(device), seed, flags
        self.hp = dict(oracle.DEFAULTS) if hp is None else dict(hp)
        assert self.hp.get("max_grad_norm", 0.0) == 0.0, "the gradient-norm mode couples tensors"
        self.specs = wl.specs
        self.W = [W.init_weight(s, wl, self.device) for s in self.specs]
        self.G = [torch.zeros(s.shape, dtype=torch.bfloat16, device=self.device) for s in self.specs]
        self.opt = SkewAdam([(s.tier, self.W[k], self.G[k], s.tensor_id, s.state_flags)
                             for k, s in enumerate(self.specs)])
        self.snap_w = None
        self.snap_state = None
        self.t = 0
        self.stats = Stats()

    def _state_slices(self, k: int, buf: np.ndarray) -> Dict[str, np.ndarray]:
        """tensor k's state arrays (m, v, r, c present) as float32 views of a host copy of the
        state buffer (offsets as the set-up carved it)."""
        d = self.opt._arr[k]
        n, m = (1, d.rows * d.cols) if d.ndim == 1 else (d.rows, d.cols)
        E = d.batch if d.ndim == 3 else 1
        cnt = {"m": E * n * m, "v": E * n * m, "r": E * n, "c": E * m}
        base = self.opt.state.data_ptr()
        out = {}
        for key in ("m", "v", "r", "c"):
            ptr = getattr(d, key)
            if ptr:
                off = ptr - base
                out[key] = buf[off:off + 4 * cnt[key]].view(np.float32)
        return out

    def step(self, t: int, snapshot: bool = True) -> List[int]:
        """One GPU step on fresh gradients; returns each tensor's clip route (bits 0..3)."""
        scales = W.expert_scales(self.wl, t)
        for k, s in enumerate(self.specs):
            W.fill_grad(s, self.wl, t, self.G[k], scales)
        torch.cuda.synchronize()
        if snapshot:
            self.snap_w = [bits(w) for w in self.W]
            self.snap_state = self.opt.state.cpu().numpy()
        else:
            self.snap_w = self.snap_state = None
        self.opt.step(t, seed=self.seed, flags=self.flags, **self.hp)
        torch.cuda.synchronize()
        self.t = t
        _, route = self.opt.clip_info()
        return [r & 0xF for r in route]

    def compare_last(self) -> Stats:
        """Every tensor of the last step against the oracle stepped from the snapshot."""
        assert self.snap_w is not None, "the last step took no snapshot"
        t0 = time.time()
        post_state = self.opt.state.cpu().numpy()
        st = Stats()
        for k, s in enumerate(self.specs):
            if s.numel == 0:
                continue
            g = bits(self.G[k])

            def oracle_step(want_y):
                pre = {key: a.copy() for key, a in self._state_slices(k, self.snap_state).items()}
                o = oracle.Tensor(tier=s.tier, w=self.snap_w[k].reshape(s.shape).copy(), g=g,
                                  tensor_id=s.tensor_id, state_flags=s.state_flags, **pre)
                oracle.step([o], self.t, seed=self.seed, want_y=want_y, exact_ulp=bool(self.flags & 2), **self.hp)
                return o

            gw = bits(self.W[k])
            o = oracle_step(False)
            if np.any(gw.reshape(o.w.shape) != o.w):
                o = oracle_step(True)   # the pre-cast values, for the window test of the mismatches
            compare_tensor(s.name, o, gw, self._state_slices(k, post_state), st)
            del o
        merge(self.stats, st)
        log(f"  step {self.t}: every tensor, {time.time() - t0:.1f} s; {st}")
        return st


def run(wl: W.Workload, steps: Optional[int] = None, sample=None, **kw) -> Stats:
    pr = ParityRun(wl, sample=sample, **kw)
    for t in range(1, (steps or wl.steps) + 1):
        pr.step(t)
    log(f"  total: {pr.stats}")
    return pr.stats
