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


class ParityRun:
    """Runs the HIP step over every tensor of a workload and the oracle over a sample."""

    def __init__(self, wl: W.Workload, sample: Optional[List[int]] = None, device="cuda", seed: int = 0,
                 hp: Optional[dict] = None, specs: Optional[List[W.Spec]] = None, flags: int = 0):
        self.wl, self.device, self.seed, self.flags = wl, torch.device(device), seed, flags
        self.hp = dict(oracle.DEFAULTS) if hp is None else dict(hp)
        self.specs = specs if specs is not None else wl.specs
        self.W = [W.init_weight(s, wl, self.device) for s in self.specs]
        self.G = [torch.zeros(s.shape, dtype=torch.float32 if s.state_flags & oracle.STATE_FP32 else torch.bfloat16,
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
            extra["gsq_total"] = float(sum(float(torch.sum(G.cpu().double() ** 2)) for G in self.G))
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
        self.stats.compared += st.compared
        self.stats.mismatched += st.mismatched
        self.stats.outside_window += st.outside_window
        self.stats.not_one_step += st.not_one_step
        self.stats.max_rel_rc = max(self.stats.max_rel_rc, st.max_rel_rc)
        for key, v in st.state_bad.items():
            self.stats.state_bad[key] = self.stats.state_bad.get(key, 0) + v
        log(f"  step {t}: gpu {1e3 * (t1 - t0):.1f} ms, oracle {t2 - t1:.2f} s; {st}")
        return st

    @staticmethod
    def _host(t: torch.Tensor) -> np.ndarray:
        """bf16 bits (uint16), or float32 values for float32 masters."""
        return t.detach().cpu().numpy().copy() if t.dtype == torch.float32 else bits(t)

    def _compare(self, k: int, st: Stats):
        o, s = self.O[k], self.specs[k]
        views = self.opt.state_views(k)
        for name in ("m", "v"):
            ref = getattr(o, name)
            if ref is None:
                assert name not in views, (s.name, name)
                continue
            got = views[name].cpu().numpy()
            bad = int(np.count_nonzero(got.view(np.uint32) != ref.ravel().view(np.uint32)))
            if bad:
                st.state_bad[f"{s.name}.{name}"] = bad
        for name in ("r", "c"):
            ref = getattr(o, name)
            if ref is None:
                assert name not in views, (s.name, name)
                continue
            got = views[name].cpu().numpy().astype(np.float64)
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
                st.state_bad[f"{s.name}.{name}"] = bad
        if o.w.dtype == np.float32:
            # float32 masters: the oracle's own float sequence, bit for bit
            gwf = self.W[k].detach().cpu().numpy().reshape(o.w.shape)
            bad = int(np.count_nonzero(gwf.view(np.uint32) != o.w.view(np.uint32)))
            st.compared += o.w.size
            if bad:
                st.state_bad[f"{s.name}.w32"] = bad
            return
        gw = bits(self.W[k]).reshape(o.w.shape)
        ow = o.w
        mism = gw != ow
        both_nan = np.isnan(oracle.bf16_to_f32(gw)) & np.isnan(oracle.bf16_to_f32(ow))
        mism &= ~both_nan
        new = mism
        n_new = int(np.count_nonzero(new))
        st.compared += int(ow.size)
        st.mismatched += n_new
        if n_new:
            y = o.y_out.reshape(ow.shape)[new]
            outside = ~near_boundary(y)
            st.outside_window += int(np.count_nonzero(outside))
            if outside.any():
                pos = np.argwhere(new)[outside][:4]
                for p in pos:
                    p = tuple(p)
                    yy = float(o.y_out.reshape(ow.shape)[p])
                    log(f"    outside window: {s.name} idx={p} y_oracle={yy!r} gpu=0x{int(gw[p]):04x} "
                        f"oracle=0x{int(ow[p]):04x}")
            step_dist = np.abs(gw[new].astype(np.int32) - ow[new].astype(np.int32))
            st.not_one_step += int(np.count_nonzero(step_dist != 1))
            ow[new] = gw[new]   # both sides take the next step from the same weights


def run(wl: W.Workload, steps: Optional[int] = None, sample=None, **kw) -> Stats:
    pr = ParityRun(wl, sample=sample, **kw)
    for t in range(1, (steps or wl.steps) + 1):
        pr.step(t)
    log(f"  total: {pr.stats}")
    return pr.stats
