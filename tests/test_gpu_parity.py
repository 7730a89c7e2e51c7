"""GPU parity: the HIP step against the CPU oracle on the same seeded inputs.

Workloads: the tiny one-layer MoE on every tensor, unit shapes (odd, ragged, strided,
unaligned, vectors), and the full-size workloads (one MoE layer at width 2048, the
heavy-tailed stress case, the ragged tier mix, and the 6.78B parameter set) with every
tensor compared at chosen steps (each compared step starts the oracle from the GPU's
weights and state before it), plus sampled tensors followed over all steps of the 6.78B
and ragged runs. Every test calls the library through its C ABI.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2607_19058_amd import SkewAdam
from paper_2607_19058_amd import workloads as W

from parity_util import ParityRun, StreamParity, bits, log, run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    torch.cuda.init()


def test_tiny_every_tensor():
    log("[parity] tiny: 21 tensors, 10 steps, all compared")
    st = run(W.get("tiny"))
    assert st.ok(), st


def _unit_workload():
    specs = []
    shapes = [(1, 1), (1, 7), (7, 1), (3, 5), (13, 17), (256, 8), (64, 520), (33, 1031), (5,), (1,), (4097,),
              (2, 2048), (300, 2056)]
    for tier in (W.BACKBONE, W.EXPERT, W.ROUTER):
        for sh in shapes:
            specs.append(W.Spec(f"t{tier}_{'x'.join(map(str, sh))}", tier, sh, len(specs)))
    return W.Workload("unit", specs, 3)


def test_tiny_exact_clip_everywhere():
    """The exact re-check of the clip factor's sum, forced for every tensor at every step,
    gives the same bits as the oracle (it is the path the clip stage takes when the fast
    estimate cannot decide k's rounding)."""
    from paper_2607_19058_amd.skewadam import FLAG_EXACT_CLIP
    log("[parity] tiny with the exact clip re-check forced on every tensor")
    st = run(W.get("tiny"), flags=FLAG_EXACT_CLIP)
    assert st.ok(), st


def test_unit_shapes_all_tiers():
    log("[parity] unit shapes: odd, ragged and vector shapes in every tier, 3 steps")
    st = run(_unit_workload(), hp=dict(oracle.DEFAULTS, lr=1e-2))
    assert st.ok(), st


def test_strided_and_unaligned_tensors():
    """Row stride larger than the width, and pointers off 16-byte alignment (the scalar
    paths): weights and every state array against the oracle on the dense copy, to the same
    bar as every other parity test; the padding around each view stays untouched."""
    log("[parity] strided / unaligned tensors")
    dev = torch.device("cuda")
    wl = W.Workload("strided", [W.Spec("a", W.EXPERT, (37, 200), 0), W.Spec("b", W.BACKBONE, (64, 1024), 1),
                                W.Spec("c", W.ROUTER, (16, 24), 2), W.Spec("d", W.EXPERT, (40, 1031), 3),
                                W.Spec("e", W.BACKBONE, (33, 520), 4)], 3)
    pads, offs = (56, 8, 3, 5, 16), (0, 1, 1, 3, 8)
    bases, Ws, Gs = [], [], []
    for s, pad, off in zip(wl.specs, pads, offs):
        n, m = s.shape
        wb = torch.zeros((n, m + pad + off), dtype=torch.bfloat16, device=dev)
        gb = torch.zeros_like(wb)
        w = wb[:, off:off + m]
        w.copy_(W.init_weight(s, wl, dev))
        bases.append((wb, gb))
        Ws.append(w)
        Gs.append(gb[:, off:off + m])
    pr = ParityRun(wl, weights=Ws, grads=Gs, hp=dict(oracle.DEFAULTS, lr=1e-2))
    for t in range(1, 4):
        pr.step(t)
    assert pr.stats.ok(), pr.stats
    assert pr.stats.compared == 3 * sum(s.numel for s in wl.specs)
    for k, s in enumerate(wl.specs):
        wb, gb = bases[k]
        n, m = s.shape
        assert torch.count_nonzero(wb[:, :offs[k]]) == 0
        assert torch.count_nonzero(wb[:, offs[k] + m:]) == 0


def _route_log(routes, specs):
    counts = {r: sum(1 for q, s in zip(routes, specs) if q == r and s.numel > 0) for r in (0, 4, 2)}
    return ", ".join(f"{StreamParity.ROUTES[r]}: {c}" for r, c in counts.items())


def _every_tensor(wl, compare_steps, max_steps, need_routes=False):
    """Run `wl` on the GPU and compare every tensor at the steps in compare_steps, and (with
    need_routes) at further steps until each way of deciding the clip factor (fast sums,
    floor-split re-check, exact re-check; no forcing flag) has been taken by a compared
    tensor. Returns the routes seen on compared steps."""
    sp = StreamParity(wl)
    seen = set()
    done = 0
    for t in range(1, max_steps + 1):
        routes = sp.step(t, snapshot=True)
        here = {r for r, s in zip(routes, wl.specs) if s.numel > 0}
        want = t in compare_steps or (need_routes and not here <= seen)
        if want:
            st = sp.compare_last()
            assert st.ok(), (t, st)
            log(f"    routes at step {t}: {_route_log(routes, wl.specs)}")
            seen |= here
            done += 1
        if done >= len(compare_steps) and (not need_routes or seen >= {0, 2, 4}):
            break
    log(f"  total: {sp.stats}")
    assert sp.stats.ok(), sp.stats
    return seen


@pytest.mark.timeout(900)
def test_layer_every_tensor():
    """One MoE layer at full width (263 tensors, 4.35B parameters), 5 steps, every tensor
    compared at the last."""
    wl = W.get("layer")
    log("[parity] layer: 263 tensors (4.35B params), 5 steps, every tensor compared at step 5")
    _every_tensor(wl, {5}, 5)


@pytest.mark.timeout(900)
def test_layer_stacked_every_tensor_and_partial_split():
    """The layer with each expert projection stacked into one (128, n, m) tensor that shares
    one clip factor: when a stack's sum is open, the floor-split re-check re-reads only its
    open slices (and its first) and keeps the others' fast sums. Every tensor compared at
    step 2 and, until a stack has taken that re-check on a compared step, at later ones."""
    wl = W.stacked(W.get("layer"))
    log("[parity] layer with stacked experts: every tensor compared, a stack decided by the floor split")
    sp = StreamParity(wl)
    stacks = [k for k, s in enumerate(wl.specs) if len(s.shape) == 3]
    assert stacks
    split_seen = False
    for t in range(1, 6):
        routes = sp.step(t, snapshot=t >= 2)
        if t >= 2:
            st = sp.compare_last()
            assert st.ok(), (t, st)
            log(f"    routes at step {t}: {_route_log(routes, wl.specs)}; stacks {[routes[k] for k in stacks]}")
            split_seen |= any(routes[k] == 4 for k in stacks)
            if split_seen:
                break
    assert sp.stats.ok(), sp.stats
    assert split_seen, "no stack took the floor-split re-check on a compared step"


@pytest.mark.timeout(900)
def test_stress_every_tensor_and_clip_routes():
    """Heavy-tailed stress (Student-t(2), 0.1% outliers x100, 90% sparse experts): every
    tensor at each of its 5 steps, and each way of deciding the clip factor taken by at least
    one compared tensor (fast sums, floor-split re-check, exact re-check), unforced."""
    wl = W.get("stress")
    log("[parity] stress: 263 tensors, 5 steps, every tensor compared")
    seen = _every_tensor(wl, {1, 2, 3, 4, 5}, 5)
    assert seen >= {0, 2, 4}, f"clip routes taken on compared steps: {sorted(seen)}"


@pytest.mark.timeout(900)
def test_full_every_tensor_and_clip_routes():
    """The benchmark workload (6.78B parameters, 432 tensors; tok_embed and the untied head
    included) in bench.py's launch configuration: every tensor compared at steps 1-3 and at
    later steps until each way of deciding the clip factor has been taken by a compared
    tensor (unforced)."""
    wl = W.get("full")
    log("[parity] full 6.78B: 432 tensors, every tensor compared at steps 1-3 and until every clip route is seen")
    seen = _every_tensor(wl, {1, 2, 3}, 20, need_routes=True)
    assert seen >= {0, 2, 4}, f"clip routes taken on compared steps: {sorted(seen)}"


@pytest.mark.timeout(900)
def test_ragged_every_tensor():
    """The ragged tier mix (269 tensors, 7.05B parameters: 1536/6144/4096/11008-column
    matrices, 1-D vectors on the exact fallback): every tensor compared at step 2 (a sample is
    followed over all 50 steps below)."""
    wl = W.get("ragged")
    log("[parity] ragged: 269 tensors (7.05B params), every tensor compared at step 2")
    _every_tensor(wl, {2}, 2)


def test_determinism_order_and_resume():
    """Bit-identical across runs, descriptor orders and a checkpoint/resume split."""
    log("[parity] determinism, descriptor order, resume")
    dev = torch.device("cuda")
    wl = W.get("tiny")
    G = [torch.empty(s.shape, dtype=torch.bfloat16, device=dev) for s in wl.specs]

    def run_steps(order, t_from, t_to, Wt, opt=None):
        if opt is None:
            opt = SkewAdam([(wl.specs[k].tier, Wt[k], G[k], wl.specs[k].tensor_id) for k in order])
        for t in range(t_from, t_to + 1):
            sc = W.expert_scales(wl, t)
            for k, s in enumerate(wl.specs):
                W.fill_grad(s, wl, t, G[k], sc)
            opt.step(t, seed=5)
        torch.cuda.synchronize()
        return opt

    def fresh():
        return [W.init_weight(s, wl, dev) for s in wl.specs]

    Wa = fresh()
    a = run_steps(list(range(len(wl.specs))), 1, 10, Wa)
    Wb = fresh()
    run_steps(list(range(len(wl.specs))), 1, 10, Wb)
    Wc = fresh()
    run_steps(list(reversed(range(len(wl.specs)))), 1, 10, Wc)
    Wd = fresh()
    d = run_steps(list(range(len(wl.specs))), 1, 5, Wd)
    saved = d.state.clone()
    d.close()
    d2 = SkewAdam([(s.tier, Wd[k], G[k], s.tensor_id) for k, s in enumerate(wl.specs)])
    d2.state.copy_(saved)
    run_steps(None, 6, 10, Wd, opt=d2)
    for k in range(len(wl.specs)):
        assert torch.equal(Wa[k].view(torch.int16), Wb[k].view(torch.int16)), "run to run"
        assert torch.equal(Wa[k].view(torch.int16), Wc[k].view(torch.int16)), "descriptor order"
        assert torch.equal(Wa[k].view(torch.int16), Wd[k].view(torch.int16)), "resume"
    assert torch.equal(a.state, d2.state)


def test_hparam_errors_launch_nothing():
    dev = torch.device("cuda")
    w = torch.ones((4, 8), dtype=torch.bfloat16, device=dev)
    g = torch.ones_like(w)
    opt = SkewAdam([(W.EXPERT, w, g, 0)])
    from paper_2607_19058_amd import SkewError
    for bad in (dict(step=0), dict(step=1, eps=0.0), dict(step=1, beta2=1.0), dict(step=1, beta1=-0.1),
                dict(step=1, clip_threshold=0.0), dict(step=1, lr=float("nan"))):
        with pytest.raises(SkewError):
            opt.step(**bad)
    torch.cuda.synchronize()
    assert torch.equal(w, torch.ones_like(w))


def test_full_6p78b_sampled():
    """The benchmark workload (6,784,327,680 parameters, 432 tensors), all 20 steps, in the
    launch configuration bench.py times; the oracle follows a sample of tensors from every
    tier (norm vector, attention, positions, the 50304x2048 embedding and the untied
    2048x50304 head, expert matrices of both orientations including a zero-gradient one, a
    router)."""
    wl = W.get("full")
    names = {s.name: s.tensor_id for s in wl.specs}
    sc = W.expert_scales(wl, 1)[0]
    zero_e = int(np.flatnonzero(sc == 0)[0])
    sample = [names["norm.3"], names["attn.7"], names["pos_embed"], names["tok_embed"], names["lm_head"],
              names["ex5.gate"], names["ex77.down"], names[f"ex{zero_e}.up"], names["router.1"]]
    log(f"[parity] full 6.78B: 432 tensors, 20 steps, sampled {sample}")
    st = run(wl, sample=sample)
    assert st.ok(), st


def test_ragged_sampled():
    """Non-power-of-two widths (1536, 6144, 4096, 11008), 1-D bias and norm vectors on the
    exact fallback, a 4096x64 router; 50 steps."""
    wl = W.get("ragged")
    names = {s.name: s.tensor_id for s in wl.specs}
    sample = [names["norm.1"], names["bias.2"], names["attn.0"], names["exA3.up"], names["exA9.down"],
              names["exB40.down"], names["exB7.up"], names["router"]]
    log(f"[parity] ragged: 269 tensors (7.05B params), 50 steps, sampled {sample}")
    st = run(wl, sample=sample)
    assert st.ok(), st


def test_more_than_2p31_elements():
    """A 65537 x 32768 expert matrix (2,147,516,416 elements > 2^31) and a backbone vector of
    2^31 + 3 elements: 64-bit sizes and element indices through the whole step."""
    wl = W.Workload("big", [W.Spec("big", W.EXPERT, (65537, 32768), 0), W.Spec("vec", W.BACKBONE, ((1 << 31) + 3,), 1)], 2)
    log("[parity] > 2^31 elements: 65537x32768 expert matrix and a (2^31+3)-element backbone vector, 2 steps")
    st = run(wl)
    assert st.ok(), st
    assert st.compared >= 2 * ((1 << 31) + 65537 * 32768)
