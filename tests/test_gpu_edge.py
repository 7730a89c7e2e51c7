"""GPU edge cases of the descriptor table, checked against the CPU oracle: tensors with no
elements (a zero row or column count, an empty vector, a stacked tensor of no slices or of
empty slices) in every tier, mixed into a table of ordinary tensors, and a table that holds
nothing but empty tensors. Empty tensors keep no state and take no work; the others must
match the oracle as they do without them (also with the gradient-norm scaling, whose norm
runs over every tensor of the table, and the decay)."""
import pytest
import torch

import oracle
from paper_2607_19058_amd import SkewAdam
from paper_2607_19058_amd import workloads as W

from parity_util import ParityRun, log, run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    torch.cuda.init()


def _mixed():
    shapes = [("bb.empty_rows", W.BACKBONE, (0, 64)), ("bb", W.BACKBONE, (256, 256)),
              ("bb.empty_vec", W.BACKBONE, (0,)), ("bb.vec", W.BACKBONE, (257,)),
              ("ex.empty_cols", W.EXPERT, (64, 0)), ("ex", W.EXPERT, (128, 520)),
              ("ex.no_slices", W.EXPERT, (0, 64, 64)), ("ex.empty_slices", W.EXPERT, (3, 0, 16)),
              ("ex.stack", W.EXPERT, (3, 64, 96)),
              ("rt.empty", W.ROUTER, (0, 8)), ("rt", W.ROUTER, (256, 8)), ("rt.empty_vec", W.ROUTER, (0,))]
    specs = [W.Spec(name, tier, shape, k) for k, (name, tier, shape) in enumerate(shapes)]
    wl = W.Workload("mixed_empty", specs, 4)
    sample = [k for k, s in enumerate(specs) if s.numel > 0]
    return wl, sample


@pytest.mark.parametrize("hp", [oracle.DEFAULTS, dict(oracle.DEFAULTS, weight_decay=0.05, max_grad_norm=1e-3)],
                         ids=["plain", "gnorm+decay"])
def test_empty_tensors_mixed_into_every_tier(hp):
    wl, sample = _mixed()
    log(f"[parity] {len(wl.specs)} tensors, {len(wl.specs) - len(sample)} of them empty, {hp}; "
        f"non-empty ones compared")
    st = run(wl, sample=sample, hp=hp)
    assert st.ok(), st
    assert st.compared > 0


def test_table_of_only_empty_tensors():
    dev = torch.device("cuda")
    shapes = [(W.BACKBONE, (0, 16)), (W.EXPERT, (8, 0)), (W.ROUTER, (0,)), (W.EXPERT, (0, 4, 4))]
    ws = [torch.zeros(s, dtype=torch.bfloat16, device=dev) for _, s in shapes]
    gs = [torch.zeros(s, dtype=torch.bfloat16, device=dev) for _, s in shapes]
    opt = SkewAdam([(t, ws[k], gs[k], k) for k, (t, _) in enumerate(shapes)])
    assert opt.state_nbytes == 0
    for t in (1, 2):
        opt.step(t, max_grad_norm=1.0 if t == 2 else 0.0)
    torch.cuda.synchronize()
    kk, route = opt.clip_info()
    assert list(kk) == [0.0] * len(shapes) and list(route) == [0] * len(shapes)


@pytest.mark.parametrize("hp", [oracle.DEFAULTS, dict(oracle.DEFAULTS, weight_decay=0.05, max_grad_norm=1.0)],
                         ids=["plain", "gnorm+decay"])
def test_nonfinite_gradients_propagate_as_in_the_oracle(hp):
    """Non-finite gradients propagate (no skipping): a NaN element makes its tensor's clip
    factor, and so every weight of that tensor, NaN; an infinite one gives infinite second
    moments. Each tier gets a NaN at step 2 and an infinity at step 3; the other tensors and
    every state array must still match the oracle. With the gradient-norm scaling the norm
    itself is NaN, and so is every tensor."""
    from parity_util import ParityRun
    shapes = [("bb", W.BACKBONE, (64, 512)), ("bb.vec", W.BACKBONE, (300,)), ("ex", W.EXPERT, (128, 520)),
              ("ex.b", W.EXPERT, (64, 64)), ("rt", W.ROUTER, (64, 8)), ("bb.clean", W.BACKBONE, (64, 64)),
              ("ex.clean", W.EXPERT, (96, 1024))]
    wl = W.Workload("nonfinite", [W.Spec(n, t, s, k) for k, (n, t, s) in enumerate(shapes)], 4)

    def mutate(t, G):
        if t == 2:
            for k in (0, 2, 4):
                G[k].view(-1)[7] = float("nan")
        if t == 3:
            for k in (1, 3):
                G[k].view(-1)[5] = float("inf")

    pr = ParityRun(wl, hp=hp)
    for t in range(1, 5):
        pr.step(t, mutate=mutate)
    log(f"  total: {pr.stats}")
    assert pr.stats.ok(), pr.stats
    kk, _ = pr.opt.clip_info()
    assert all(kk[k] != kk[k] for k in (0, 2, 4))              # NaN clip factors
    for k in (0, 2, 4):
        assert torch.isnan(pr.W[k].float()).all()
    clean_nan = [bool(torch.isnan(pr.W[k].float()).any()) for k in (5, 6)]
    assert clean_nan == ([True, True] if hp.get("max_grad_norm", 0.0) > 0 else [False, False])


def test_experts_zero_from_step_6_decay_as_in_the_oracle():
    """Two experts draw gradients at steps 1-5 and none from step 6 on (zero-gradient steps
    after real ones: R and C decay by beta2 from nonzero values); every tensor compared."""
    wl = W.get("tiny_late_zero")
    log("[parity] tiny, two experts zero from step 6: 21 tensors, 10 steps, all compared")
    st = run(wl)
    assert st.ok(), st


def test_expert_rows_always_zero():
    """Experts with 90% of their rows zero at every step: R_i = 0 on those rows beside
    nonzero rows (their elements sit on the eps floor with U = 0); every tensor compared."""
    wl = W.get("zero_rows")
    log("[parity] experts with 90% zero rows, 19 tensors, 8 steps, all compared")
    st = run(wl)
    assert st.ok(), st


@pytest.mark.parametrize("hp", [oracle.DEFAULTS, dict(oracle.DEFAULTS, weight_decay=0.05, max_grad_norm=1.0)],
                         ids=["plain", "gnorm+decay"])
def test_row_band_widths_with_partial_chunks(hp):
    """Row-band matrices whose rows end inside a 512-column chunk, with and without momentum:
    the block loads mask the lanes past the row (for M, each of its two 1 KiB halves on its
    own) and the last block of a band holds rows past the band's end. Widths of 2, 4, 9 and
    17 chunks take one to four chunks per wave (17: the general load loop); every tensor
    compared. Also the widest row-band rows: 11008 columns (22 chunks, the ragged mix's
    experts) and 16384 columns (32 chunks, the row-band limit), with and without momentum,
    and 16392 columns, the first width past it (pass 1 by tiles instead)."""
    shapes = [("bb.w1000", W.BACKBONE, (300, 1000)), ("bb.w1544", W.BACKBONE, (70, 1544)),
              ("bb.w4104", W.BACKBONE, (33, 4104)), ("bb.w8200", W.BACKBONE, (40, 8200)),
              ("ex.w1544", W.EXPERT, (96, 1544)), ("ex.w8200", W.EXPERT, (24, 8200)),
              ("ex.w11008", W.EXPERT, (37, 11008)), ("bb.w11008", W.BACKBONE, (19, 11008)),
              ("ex.w16384", W.EXPERT, (21, 16384)), ("bb.w16384", W.BACKBONE, (9, 16384)),
              ("ex.w16392", W.EXPERT, (11, 16392)),
              ("rt", W.ROUTER, (256, 8))]
    specs = [W.Spec(name, tier, shape, k) for k, (name, tier, shape) in enumerate(shapes)]
    wl = W.Workload("partial_chunks", specs, 4)
    log(f"[parity] {len(specs)} row-band widths with partial chunks, 4 steps, {hp}; all compared")
    st = run(wl, hp=hp)
    assert st.ok(), st
    assert st.compared > 0


def test_row_strides_past_a_32_bit_block_span():
    """Aligned expert rows whose stride makes one block of rows span 2^31 bytes or more: the
    row-band pass addresses a block by 32-bit offsets in its aligned variant, so such a tensor
    takes the element-load variant. Beside it, a large stride below that limit keeps the
    aligned one. Both against the oracle (the last block of each band is partial), and the
    memory between the rows stays untouched."""
    dev = torch.device("cuda")
    specs = [W.Spec("ex.far", W.EXPERT, (5, 8192), 0), W.Spec("ex.near", W.EXPERT, (6, 8192), 1)]
    wl = W.Workload("row_strides", specs, 3)
    strides = ((1 << 28) + 8, (1 << 20) + 8)
    log("[parity] expert rows at strides 2^28 + 8 and 2^20 + 8, 3 steps")
    bases, Ws, Gs = [], [], []
    for s, ld in zip(specs, strides):
        n, m = s.shape
        wb = torch.zeros((n - 1) * ld + m, dtype=torch.bfloat16, device=dev)
        gb = torch.zeros_like(wb)
        w = wb.as_strided((n, m), (ld, 1))
        w.copy_(W.init_weight(s, wl, dev))
        bases.append((wb, gb))
        Ws.append(w)
        Gs.append(gb.as_strided((n, m), (ld, 1)))
    pr = ParityRun(wl, weights=Ws, grads=Gs)
    for t in range(1, 4):
        pr.step(t)
    assert pr.stats.ok(), pr.stats
    assert pr.stats.compared == 3 * sum(s.numel for s in wl.specs)
    for (wb, gb), w, g in zip(bases, Ws, Gs):
        assert torch.count_nonzero(wb) == torch.count_nonzero(w)
        assert torch.count_nonzero(gb) == torch.count_nonzero(g)
    del bases, Ws, Gs, pr
    torch.cuda.empty_cache()


def test_overlapping_row_views_are_refused_before_any_launch():
    """A view whose rows overlap (an expanded row, or an unfold window: row stride below the
    row length) would make the in-place update write past the view; the binding refuses it
    and the C ABI refuses a stride below the width as well."""
    from paper_2607_19058_amd import TensorDesc, lib, make_desc
    import ctypes
    dev = torch.device("cuda")
    base = torch.zeros((1, 1024), dtype=torch.bfloat16, device=dev)
    w = base.expand(256, 1024)
    g = torch.zeros((1, 1024), dtype=torch.bfloat16, device=dev).expand(256, 1024)
    for tier in (W.BACKBONE, W.EXPERT, W.ROUTER):
        with pytest.raises(ValueError, match="overlapping rows"):
            SkewAdam([(tier, w, g, 0)])
    flat = torch.zeros(4096, dtype=torch.bfloat16, device=dev)
    win = flat.unfold(0, 1024, 512)          # rows of 1024 at a stride of 512
    gwin = torch.zeros_like(flat).unfold(0, 1024, 512)
    with pytest.raises(ValueError, match="overlapping rows"):
        SkewAdam([(W.EXPERT, win, gwin, 0)])
    stk = torch.zeros((1, 1, 1024), dtype=torch.bfloat16, device=dev).expand(2, 64, 1024)
    with pytest.raises(ValueError, match="overlapping rows"):
        SkewAdam([(W.EXPERT, stk, stk, 0)])
    d = make_desc(W.EXPERT, 2, 256, 1024, 512, 0, base.data_ptr(), base.data_ptr())
    arr = (TensorDesc * 1)(d)
    ctx = ctypes.c_void_p()
    st = torch.empty(1 << 20, dtype=torch.uint8, device=dev)
    assert lib().skew_state_init(ctypes.byref(ctx), arr, 1, st.data_ptr(), st.numel(), st.data_ptr(), st.numel(),
                                 None) == -1
    torch.cuda.synchronize()
    assert torch.count_nonzero(base) == 0



def test_structured_gradients_clip_factor_matches_the_oracle():
    """Gradients whose R_i or C_j repeat (a constant gradient; a rank-one gradient of two
    magnitudes per row and per column): the roundings of R_i c'_j and of the square root then
    repeat and do not average out, so the clip stage must not trust a statistical spread. With
    clipping active (threshold 0.5), every clip factor (skew_clip_info) equals the oracle's
    float bit for bit, and weights and state meet the parity bar. Row-band tensors with and
    without momentum, a wide tensor (pass 1 by tiles) and a stacked tensor."""
    import numpy as np
    shapes = [("ex.const", W.EXPERT, (256, 1024)), ("ex.rank1", W.EXPERT, (512, 512)),
              ("bb.const", W.BACKBONE, (128, 2048)), ("bb.rank1", W.BACKBONE, (96, 1536)),
              ("ex.wide_const", W.EXPERT, (16, 16392)), ("ex.stack_const", W.EXPERT, (4, 64, 512)),
              ("rt", W.ROUTER, (64, 8))]
    specs = [W.Spec(name, tier, shape, k) for k, (name, tier, shape) in enumerate(shapes)]
    wl = W.Workload("structured", specs, 5)
    hp = dict(oracle.DEFAULTS, clip_threshold=0.5)

    def structured(t, G):
        for k, s in enumerate(specs):
            if s.tier == W.ROUTER:
                continue
            if "rank1" in s.name:
                n, m = s.shape
                a = torch.where(torch.arange(n, device=G[k].device) % 3 == 0, 1.5, 1.0)
                b = torch.where(torch.arange(m, device=G[k].device) % 5 == 0, 1.5, 1.0)
                sign = torch.where((torch.arange(n * m, device=G[k].device).view(n, m) * 7 + t) % 11 < 5, -1.0, 1.0)
                G[k].copy_(sign * (2e-3 * (1 + 0.25 * t)) * a[:, None] * b[None, :])
            else:
                G[k].fill_(2e-3 * (1 + 0.25 * t))

    pr = ParityRun(wl, hp=hp)
    routes_seen = set()
    for t in range(1, 6):
        pr.step(t, mutate=structured)
        kk, route = pr.opt.clip_info()
        for k, s in enumerate(specs):
            o = pr.O[k]
            k_oracle = np.float32(1.0 / max(1.0, o.rms / hp["clip_threshold"]))
            assert np.float32(kk[k]).view(np.uint32) == k_oracle.view(np.uint32), (s.name, t, kk[k], k_oracle)
            routes_seen.add(route[k] & 0xF)
    log(f"  total: {pr.stats}; clip routes seen {sorted(routes_seen)}")
    assert pr.stats.ok(), pr.stats


def test_two_contexts_on_two_streams_match_serial_runs():
    """Two contexts stepped at the same time on two streams, each with its own state and
    workspace, end with the weights, state and clip factors, bit for bit, of the same two
    contexts stepped one after the other on one stream: no device memory is shared between
    contexts. One context takes the gradient-norm scaling and the decay, the other the plain
    step; the second holds row-band, wide (pass 1 by tiles), stacked, vector and router
    tensors large enough for the two steps' kernels to overlap."""
    dev = torch.device("cuda", 0)
    shapes_b = [("ex.a", W.EXPERT, (1024, 4096)), ("ex.b", W.EXPERT, (4096, 1024)),
                ("ex.stack", W.EXPERT, (2, 512, 2048)), ("bb", W.BACKBONE, (1024, 2048)),
                ("bb.wide", W.BACKBONE, (64, 20000)), ("bb.vec", W.BACKBONE, (2048,)), ("rt", W.ROUTER, (2048, 64))]
    wl_b = W.Workload("two_streams", [W.Spec(n, tier, shape, k) for k, (n, tier, shape) in enumerate(shapes_b)], 3)
    hps = [dict(weight_decay=0.05, max_grad_norm=1e-2), dict()]
    runs = []   # per workload: gradients, weights of the concurrent and of the serial run, contexts
    for wl in (W.get("tiny"), wl_b):
        G = [torch.empty(s.shape, dtype=torch.bfloat16, device=dev) for s in wl.specs]
        Wc = [W.init_weight(s, wl, dev) for s in wl.specs]
        Ws = [w.clone() for w in Wc]

        def make(Wt, wl=wl, G=G):
            return SkewAdam([(s.tier, Wt[k], G[k], s.tensor_id, s.state_flags) for k, s in enumerate(wl.specs)])
        runs.append((wl, G, Wc, Ws, make(Wc), make(Ws)))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    main = torch.cuda.current_stream()
    for t in (1, 2, 3):
        for wl, G, *_ in runs:
            sc = W.expert_scales(wl, t)
            for k, s in enumerate(wl.specs):
                W.fill_grad(s, wl, t, G[k], sc)
        torch.cuda.synchronize()
        ready = torch.cuda.Event()
        ready.record(main)
        for j, run_j in enumerate(runs):
            streams[j].wait_event(ready)
            run_j[4].step(t, stream=streams[j], **hps[j])
        torch.cuda.synchronize()
        for j, run_j in enumerate(runs):
            run_j[5].step(t, stream=main, **hps[j])
        torch.cuda.synchronize()
    for wl, G, Wc, Ws, oc, osr in runs:
        log(f"two streams: {wl.name}, {len(wl.specs)} tensors compared bit for bit")
        for k, s in enumerate(wl.specs):
            assert torch.equal(Wc[k].view(torch.uint8), Ws[k].view(torch.uint8)), (wl.name, s.name, "w")
            vc, vs = oc.state_views(k), osr.state_views(k)
            assert vc.keys() == vs.keys()
            for name in vc:
                assert torch.equal(vc[name].view(torch.uint8), vs[name].view(torch.uint8)), (wl.name, s.name, name)
        assert oc.clip_info() == osr.clip_info()
        oc.close()
        osr.close()


@pytest.mark.parametrize("hp", [
    dict(beta1=0.0, beta2=0.0),
    dict(beta1=0.5, beta2=0.5),
    dict(beta1=0.99, beta2=0.9999, lr=1e-2),
    dict(eps=1e-30),
    dict(eps=1e-3),
    dict(clip_threshold=float("inf")),
    dict(clip_threshold=1e-3, lr=0.0),
], ids=["no_memory", "short_memory", "long_memory_high_lr", "floor_1e-30", "floor_1e-3", "no_clipping",
        "clip_everywhere_lr0"])
def test_hyper_parameter_extremes_tiny_every_tensor(hp):
    """The tiny one-layer set (21 tensors in every tier) under hyper-parameters at the edges
    the step allows: EMAs with no memory (beta = 0: R, C, M and V are this step's), short and
    very long memories, an eps floor far below or above the second moments, no clipping
    (threshold +inf), and clipping everywhere with lr = 0 (only the dither acts, and it never
    moves a weight by itself); 4 steps, every tensor against the oracle."""
    log(f"[parity] tiny, hyper-parameters {hp}, 4 steps, all compared")
    st = run(W.get("tiny"), steps=4, hp=dict(oracle.DEFAULTS, **hp))
    assert st.ok(), st
