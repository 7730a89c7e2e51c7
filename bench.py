#!/usr/bin/env python3
"""Benchmark of the SkewAdam optimizer step on one MI355X.

Workload: the full 6,784,327,680-parameter synthetic MoE parameter set (432 tensors:
backbone 341,352,448 / experts 6,442,450,944 / router 524,288 parameters, the tier
sizes of the paper's model), bf16 weights and gradients resident in HBM.

One timed step is one call of skew_step over every tensor, i.e. the whole hot path
(row-band statistics, fold, update sums, clip factor, update and dithered write-back).
Every step, warm-up and timed, draws fresh seeded gradients first (Sec. 4: each training
step takes a new batch); HIP events on the launch stream bracket each step's skew_step
alone, so the draws are not timed and the inputs are resident in HBM when a step starts.
The headline is the mean of the K timed steps. Prints one JSON line.

Reported alongside the headline (parameters updated per second):
  step          the step's algorithmic bytes (Table 6's state by tier: G read 2 B, W read and
                written 4 B, fp32 momentum and exact V 8 B each per parameter) and its
                effective GB/s and fraction of the 8 TB/s peak; median, min and max of the
                timed steps; the warm-up steps (steps 1.. of the run) one by one
  roofline      the dominant kernel's achieved algorithmic GB/s against 8 TB/s, from HIP
                events around each of the library's kernels over a separate pass of steps
                (so the headline's steps carry no per-kernel events); `traffic` from the
                committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary when the kernel source
                still matches it
  tiers         per tier: parameters, algorithmic bytes, and the update kernel's measured
                HBM bytes from the committed per-tier counter summary (same source check)
  ceilings      a plain device copy of 2 GiB, timed in this process
  cpu_baseline  the CPU oracle (plain C, OpenMP) over one whole step of the same workload
                on this host's cores, and single-threaded on a sample (extrapolated)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Gparams/s per SkewAdam step + achieved HBM GB/s (% of peak), 6.78B MoE"
PEAK_GBPS = 8000.0
# Algorithmic bytes per parameter and tier: G read 2, W read + write 4, fp32 M read + write 8,
# fp32 exact V read + write 8 (the factored R, C and per-tensor scalars are negligible).
BYTES_PER_PARAM = {"expert": 6, "backbone_matrix": 14, "backbone_vector": 22, "router": 14,
                   "expert_vector": 14, "router_vector": 14}
KERNEL_SRC = os.path.join(ROOT, "paper_2607_19058_amd", "csrc", "skew_kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_full.json")
TIER_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_full_tiers.json")
TIER_NAMES = {0: "backbone", 1: "expert", 2: "router"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def tier_class(spec) -> str:
    from paper_2607_19058_amd import workloads as W
    vec = len(spec.shape) == 1
    if spec.tier == W.EXPERT:
        return "expert_vector" if vec else "expert"
    if spec.tier == W.ROUTER:
        return "router_vector" if vec else "router"
    return "backbone_vector" if vec else "backbone_matrix"


def bytes_per_param(spec) -> int:
    """G read (2) + W read and written (4) + fp32 momentum read and written (8) where the
    tier or its variant keeps one + the exact second moment read and written (8)."""
    from paper_2607_19058_amd import workloads as W
    flags = getattr(spec, "state_flags", 0)
    vec = len(spec.shape) == 1
    momentum = spec.tier == W.BACKBONE or bool(flags & 1)
    exact = vec or (spec.tier == W.ROUTER and not flags & 2)
    wbytes = 12 if flags & 4 else 6    # float32 master: G 4 + W 8
    return wbytes + (8 if momentum else 0) + (8 if exact else 0)


def algorithmic_bytes(specs) -> int:
    total = sum(bytes_per_param(s) * s.numel for s in specs)
    assert all(bytes_per_param(s) == BYTES_PER_PARAM[tier_class(s)] for s in specs
               if not getattr(s, "state_flags", 0))
    return total


# comments and C string/char literals of the kernel source, in source order
_C_TOKENS = re.compile(r'//[^\n]*|/\*.*?\*/|"(?:\\.|[^"\\\n])*"|\'(?:\\.|[^\'\\\n])*\'', re.S)


def code_hash(src: str) -> str:
    """sha256[:16] of C/C++ source with its comments removed and whitespace collapsed."""
    code = _C_TOKENS.sub(lambda mt: " " if mt.group(0)[0] == "/" else mt.group(0), src)
    return hashlib.sha256(" ".join(code.split()).encode()).hexdigest()[:16]


def kernel_sha() -> str:
    """The kernel source's code hash: the stored counters stay tied to the code they were
    taken on, not to its comments."""
    return code_hash(open(KERNEL_SRC, encoding="utf-8").read())


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(wl, Wt, G, t: int, single_budget_s: float = 8.0) -> dict:
    """The CPU oracle as it stands: one whole step over every tensor of the workload (the
    weights and step-t gradients copied from the GPU, zero state) on this host's OpenMP
    threads; then single-threaded on a sample of the workload's tensors, extrapolated."""
    import numpy as np
    import torch
    import oracle

    def host(x):
        return x.detach().view(torch.int16).cpu().numpy().view(np.uint16)

    T = [oracle.Tensor(tier=s.tier, w=host(Wt[k]), g=host(G[k]), tensor_id=s.tensor_id,
                       state_flags=s.state_flags).init_state() for k, s in enumerate(wl.specs)]
    params = sum(s.numel for s in wl.specs)
    threads = oracle.threads()
    t0 = time.perf_counter()
    oracle.step(T, t)
    dt = time.perf_counter() - t0
    del T
    # single thread: two expert matrices (both orientations), an attention matrix, a norm
    # vector and a router, stepped until the budget is spent
    from paper_2607_19058_amd import workloads as W
    pick = []
    for cond in (lambda s: s.tier == W.EXPERT and s.shape[0] < s.shape[-1],
                 lambda s: s.tier == W.EXPERT and s.shape[0] > s.shape[-1],
                 lambda s: s.tier == W.BACKBONE and len(s.shape) == 2 and s.shape[0] == s.shape[1],
                 lambda s: s.tier == W.BACKBONE and len(s.shape) == 1,
                 lambda s: s.tier == W.ROUTER):
        ks = [k for k, s in enumerate(wl.specs) if cond(s)]
        if ks:
            pick.append(ks[0])
    S = [oracle.Tensor(tier=wl.specs[k].tier, w=host(Wt[k]), g=host(G[k]), tensor_id=wl.specs[k].tensor_id,
                       state_flags=wl.specs[k].state_flags).init_state() for k in pick]
    sparams = sum(wl.specs[k].numel for k in pick)
    oracle.set_threads(1)
    try:
        t1 = time.perf_counter()
        steps = 0
        while True:
            steps += 1
            oracle.step(S, t + steps - 1)
            if time.perf_counter() - t1 >= single_budget_s or steps >= 50:
                break
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_threads(threads)
    one = sparams * steps / dt1 / 1e9
    return {"value": round(params / dt / 1e9, 4), "unit": "Gparams/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": len(os.sched_getaffinity(0)),
            "sample": f"one whole step of the workload ({len(wl.specs)} tensors, {params:,} params; weights and "
                      f"step-{t} gradients copied from the GPU, zero state): {dt:.1f} s wall on {threads} OpenMP threads",
            "single_thread": {"value": round(one, 4), "unit": "Gparams/s",
                              "sample": f"{len(pick)} tensors ({sparams:,} params: "
                                        + ", ".join(wl.specs[k].name for k in pick)
                                        + f"), {steps} steps, {dt1:.1f} s on 1 thread",
                              "extrapolated_all_cores": round(one * threads, 4),
                              "note": "single-thread rate times the thread count: an extrapolation, not a measurement"}}


def stream_ceilings(dev) -> dict:
    """A plain device copy (read 2 GiB + write 2 GiB of bf16) with torch's own kernel, best
    of 5: context for the step's rates."""
    import torch
    a = torch.ones(1 << 30, dtype=torch.bfloat16, device=dev)
    b = torch.empty_like(a)
    out = {}
    for name, fn, nbytes in (("copy", lambda: b.copy_(a), 4 << 30),):
        fn()
        best = 1e30
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
        out[f"{name}_GBps"] = round(nbytes / (best * 1e-3) / 1e9, 1)
    out["note"] = "torch copy_ of 2 GiB of bf16 (2 GiB read + 2 GiB written), best of 5, in this process"
    del a, b
    torch.cuda.empty_cache()
    return out


def tier_table(wl) -> dict:
    """Per tier: parameters and algorithmic bytes (Table 6's state by tier), with the update
    kernel's measured HBM bytes from the committed per-tier counter summary when the kernel
    source still matches it."""
    measured = {}
    if os.path.exists(TIER_TRAFFIC_FILE):
        tr = json.load(open(TIER_TRAFFIC_FILE))
        if tr.get("kernel_src_sha") == kernel_sha() and tr.get("workload") == wl.name:
            measured = tr.get("tiers", {})
    out = {}
    for tier, name in TIER_NAMES.items():
        specs = [s for s in wl.specs if s.tier == tier]
        if not specs:
            continue
        params = sum(s.numel for s in specs)
        alg = algorithmic_bytes(specs)
        row = {"params": params, "algorithmic_bytes": alg, "bytes_per_param": round(alg / params, 3)}
        m = measured.get(name)
        if m:
            row["p3_measured_bytes"] = m["hbm_bytes_per_launch"]
            row["p3_measured_over_algorithmic"] = round(m["hbm_bytes_per_launch"] / alg, 4)
        out[name] = row
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="full")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--weight-decay", type=float, default=0.0,
                    help="decoupled weight decay lambda fused into the update (router exempt)")
    ap.add_argument("--max-grad-norm", type=float, default=0.0,
                    help="> 0: the step scales the gradients by the global-norm factor (two-pass "
                         "statistics); the bench also times torch's unfused clip_grad_norm_ on the same G")
    ap.add_argument("--variant", default="skewadam", choices=["skewadam", "expert_momentum", "factored_router",
                                                              "uniform"],
                    help="tier variant of the ablation (state flags per tier)")
    ap.add_argument("--stacked", action="store_true",
                    help="each expert projection as one stacked (E, n, m) tensor")
    ap.add_argument("--exact-ulp", action="store_true", help="dither of one exact bf16 ulp")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run three plain 1 GiB device-to-device copies (read 1 GiB, write 1 GiB "
                         "each), whose FETCH_SIZE / WRITE_SIZE counters calibrate the traffic figures")
    ap.add_argument("--tier", default="all", choices=["all", "backbone", "expert", "router"],
                    help="only this tier's tensors of the workload (the per-tier traffic counters)")
    ap.add_argument("--kernel-steps", type=int, default=5,
                    help="steps of the separate pass that times each kernel with HIP events")
    ap.add_argument("--no-ceilings", action="store_true", help="skip the in-process copy/read ceilings")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0 or args.kernel_steps < 1:
        ap.error("--steps and --kernel-steps must be at least 1 and --warmup at least 0 (the roofline's "
                 "per-kernel times come from the --kernel-steps pass)")
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} (WORLD_SIZE {world}) is not supported: "
              "the optimizer step is measured on one MI355X's share", file=sys.stderr, flush=True)
        return 2

    import torch
    from paper_2607_19058_amd import SkewAdam
    from paper_2607_19058_amd import workloads as W

    if not torch.cuda.is_available():
        log("bench.py needs a HIP device")
        return 1
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    if args.calibrate_copy:
        src = torch.empty(1 << 29, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("[bench] calibration copies done (3 x 1 GiB)")
    ceilings = None if args.no_ceilings else stream_ceilings(dev)
    wl = W.get(args.workload)
    if args.stacked:
        wl = W.stacked(wl)
    wl = W.with_variant(wl, args.variant)
    if args.tier != "all":
        import dataclasses
        keep = {v: k for k, v in TIER_NAMES.items()}[args.tier]
        wl = dataclasses.replace(wl, specs=[s for s in wl.specs if s.tier == keep])
    log(f"[bench] workload {wl.name}: {len(wl.specs)} tensors, {wl.numel:,} params; allocating")
    Wt = [W.init_weight(s, wl, dev) for s in wl.specs]
    G = [torch.empty(s.shape, dtype=torch.bfloat16, device=dev) for s in wl.specs]
    opt = SkewAdam([(s.tier, Wt[k], G[k], s.tensor_id, s.state_flags) for k, s in enumerate(wl.specs)])

    def draw(t):
        sc = W.expert_scales(wl, t)
        for k, s in enumerate(wl.specs):
            W.fill_grad(s, wl, t, G[k], sc)

    hp = dict(lr=3e-4, beta1=0.9, beta2=0.999, eps=1e-8, clip_threshold=1.0, seed=0,
              weight_decay=args.weight_decay, max_grad_norm=args.max_grad_norm,
              flags=2 if args.exact_ulp else 0)
    stream = torch.cuda.current_stream()

    def steps(t_from, count):
        """count steps from step t_from, each on a fresh draw; events bracket skew_step alone"""
        ev = []
        for t in range(t_from, t_from + count):
            draw(t)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            opt.step(t, **hp)
            b.record(stream)
            ev.append((a, b))
        return ev

    first = steps(1, args.warmup)
    torch.cuda.synchronize()
    first_ms = [round(a.elapsed_time(b), 3) for a, b in first]
    log(f"[bench] warmup done ({args.warmup} steps); timing {args.steps} steps, fresh gradients each")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    timed = steps(args.warmup + 1, args.steps)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = [a.elapsed_time(b) for a, b in timed]
    ms_per_step = sum(step_ms) / len(step_ms)
    step_sorted = sorted(step_ms)
    # per-kernel times: a separate pass of steps with HIP events around each kernel
    t_next = args.warmup + args.steps + 1
    opt.timing_enable(args.kernel_steps)
    steps(t_next, args.kernel_steps)
    torch.cuda.synchronize()
    per_kernel = opt.timing_read()
    steps_rec = per_kernel.pop("_steps")
    opt.timing_enable(0)
    t_last = t_next + args.kernel_steps - 1
    unfused_ms = None
    if args.max_grad_norm > 0:
        # what the fused scaling replaces: torch's clip_grad_norm_ on the same bf16 gradients
        # (a norm read of G, then an in-place scale), timed on copies so G stays unchanged
        Gc = [g.clone() for g in G]

        def torch_clip():   # torch.nn.utils.clip_grad_norm_'s foreach path, on the tensors themselves
            norms = torch._foreach_norm(Gc, 2.0)
            total = torch.linalg.vector_norm(torch.stack([n_.float() for n_ in norms]), 2.0)
            coef = torch.clamp(args.max_grad_norm / (total + 1e-6), max=1.0)
            torch._foreach_mul_(Gc, coef.to(Gc[0].dtype))

        torch_clip()
        torch.cuda.synchronize()
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record(stream)
        for _ in range(3):
            torch_clip()
        c1.record(stream)
        torch.cuda.synchronize()
        unfused_ms = c0.elapsed_time(c1) / 3
        del Gc

    params = wl.numel
    alg = algorithmic_bytes(wl.specs)
    kern_avg = {k: v / max(1, steps_rec) for k, v in per_kernel.items()}
    dom = max(kern_avg, key=kern_avg.get)
    # the apply kernel alone reads G, W (and M or V) and writes W (and M or V) once:
    # its algorithmic bytes per launch are the step's; the other kernels re-read G
    dom_bytes = {"p3_apply_dither": alg}.get(dom, 0)
    achieved = dom_bytes / (kern_avg[dom] * 1e-3) / 1e9
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        tr = json.load(open(TRAFFIC_FILE))
        if tr.get("kernel_src_sha") == kernel_sha() and tr.get("kernel") == dom and tr.get("workload") == wl.name:
            traffic = tr.get("hbm_bytes_per_launch")
    roof = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / PEAK_GBPS, 4), "traffic": traffic,
            "algorithmic_bytes_per_launch": dom_bytes, "avg_launch_ms": round(kern_avg[dom], 4)}
    step_gbps = alg / (ms_per_step * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(params / (ms_per_step * 1e-3) / 1e9, 2),
        "unit": "Gparams/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "achieved_GBps": round(step_gbps, 1),
        "frac_of_peak": round(step_gbps / PEAK_GBPS, 4),
        "config": {"workload": f"{wl.name}: {params:,}-parameter synthetic MoE parameter set, {len(wl.specs)} tensors "
                               "(bf16 weights and gradients, fp32 state)"
                               + ("" if args.tier == "all" else f", {args.tier} tier only"),
                   "params": params, "tensors": len(wl.specs), "state_bytes": opt.state_nbytes,
                   "workspace_bytes": opt.workspace_nbytes, "weight_decay": args.weight_decay,
                   "max_grad_norm": args.max_grad_norm, "variant": args.variant, "stacked": args.stacked,
                   "exact_ulp": args.exact_ulp, "tier": args.tier,
                   "gradients": "fresh seeded draw before every step (not timed)"},
        "roofline": roof,
        "step": {"algorithmic_bytes": alg, "bytes_per_param": round(alg / params, 3),
                 "effective_GBps": round(step_gbps, 1), "frac_of_peak": round(step_gbps / PEAK_GBPS, 4),
                 "ms_mean": round(ms_per_step, 4), "ms_median": round(step_sorted[len(step_sorted) // 2], 4),
                 "ms_min": round(step_sorted[0], 4), "ms_max": round(step_sorted[-1], 4),
                 "wall_ms_per_step_with_draws": round(1e3 * wall / args.steps, 4),
                 "warmup_steps_ms": first_ms,   # steps 1.. of the run, before the timed region
                 "kernel_ms_per_step": {k: round(v, 4) for k, v in kern_avg.items()},
                 "kernel_pass_steps": steps_rec},
        "tiers": tier_table(wl),
        **({"ceilings": ceilings} if ceilings else {}),
        **({"torch_clip_grad_norm_ms": round(unfused_ms, 4)} if unfused_ms is not None else {}),
    }
    if not args.no_cpu_baseline:
        del opt
        log("[bench] timing the CPU oracle: one whole step, then single-threaded on a sample")
        out["cpu_baseline"] = cpu_baseline(wl, Wt, G, t_last)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
