"""GPU parity of the step's two optional terms against the CPU oracle: the decoupled weight
decay fused ahead of the dithered cast (Sec. 3 footnote, Sec. 6; router exempt) and the
global gradient-norm scaling (the trainer's clipping at 1.0, Sec. 4), alone and together,
on the tiny workload (every tensor), the unit shapes, and sampled tensors of the one-layer,
ragged and 6.78B workloads. The gradient-norm mode runs the row-band pass twice (sums, then
the update sums with R folded under the scale), so these tests also cover that path."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_19058_amd import SkewAdam
from paper_2607_19058_amd import workloads as W

from parity_util import log, run

pytestmark = pytest.mark.gpu

DECAY = dict(oracle.DEFAULTS, weight_decay=0.05)
STRONG_DECAY = dict(oracle.DEFAULTS, weight_decay=10.0)     # lr*lambda = 3e-3: visible in bf16
GNORM = dict(oracle.DEFAULTS, max_grad_norm=1.0)
BOTH = dict(oracle.DEFAULTS, weight_decay=0.05, max_grad_norm=1.0)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    torch.cuda.init()


@pytest.mark.parametrize("hp", [DECAY, STRONG_DECAY], ids=["lambda0.05", "lambda10"])
def test_decay_tiny_every_tensor(hp):
    log(f"[parity] tiny, weight decay {hp['weight_decay']}: 21 tensors, 10 steps, all compared")
    st = run(W.get("tiny"), hp=hp)
    assert st.ok(), st


@pytest.mark.parametrize("hp", [GNORM, BOTH], ids=["gnorm", "gnorm+decay"])
def test_gradnorm_tiny_every_tensor(hp):
    log(f"[parity] tiny, gradient norm {hp}: 21 tensors, 10 steps, all compared")
    st = run(W.get("tiny"), hp=hp)
    assert st.ok(), st


def test_gradnorm_tiny_exact_clip_everywhere():
    from paper_2607_19058_amd.skewadam import FLAG_EXACT_CLIP
    log("[parity] tiny, gradient norm and decay, exact clip re-check forced")
    st = run(W.get("tiny"), hp=BOTH, flags=FLAG_EXACT_CLIP)
    assert st.ok(), st


def _unit_workload():
    specs = []
    shapes = [(1, 1), (1, 7), (7, 1), (3, 5), (13, 17), (256, 8), (64, 520), (33, 1031), (5,), (1,), (4097,),
              (2, 2048), (300, 2056)]
    for tier in (W.BACKBONE, W.EXPERT, W.ROUTER):
        for sh in shapes:
            specs.append(W.Spec(f"t{tier}_{'x'.join(map(str, sh))}", tier, sh, len(specs)))
    return W.Workload("unit", specs, 3)


def test_gradnorm_unit_shapes_all_tiers():
    log("[parity] unit shapes, gradient norm 0.05 and strong decay, 3 steps")
    st = run(_unit_workload(), hp=dict(oracle.DEFAULTS, lr=1e-2, weight_decay=2.0, max_grad_norm=0.05))
    assert st.ok(), st


def test_gradnorm_scale_above_the_norm_is_the_plain_step():
    """A max_grad_norm above ||G|| gives scale 1 and the same bits as the step without it
    (the two-pass path against the one-pass path)."""
    dev = torch.device("cuda")
    wl = W.get("tiny")
    G = [torch.empty(s.shape, dtype=torch.bfloat16, device=dev) for s in wl.specs]
    outs = []
    for mgn in (0.0, 1e4):
        Wt = [W.init_weight(s, wl, dev) for s in wl.specs]
        opt = SkewAdam([(s.tier, Wt[k], G[k], s.tensor_id) for k, s in enumerate(wl.specs)])
        for t in range(1, 6):
            sc = W.expert_scales(wl, t)
            for k, s in enumerate(wl.specs):
                W.fill_grad(s, wl, t, G[k], sc)
            opt.step(t, max_grad_norm=mgn)
        torch.cuda.synchronize()
        outs.append(([w.clone() for w in Wt], opt.state.clone()))
        opt.close()
    for a, b in zip(outs[0][0], outs[1][0]):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(outs[0][1], outs[1][1])


def test_gradnorm_layer_sampled():
    wl = W.get("layer")
    names = {s.name: s.tensor_id for s in wl.specs}
    sc = W.expert_scales(wl, 1)[0]
    zero_e = int(np.flatnonzero(sc == 0)[0])
    big_e = int(np.argmax(sc))
    sample = [names["attn.0"], names["ffn.down"], names[f"ex{zero_e}.up"], names[f"ex{big_e}.up"],
              names["ex7.down"], names["router"]]
    log(f"[parity] layer, gradient norm and decay: 263 tensors, 5 steps, sampled {sample}")
    st = run(wl, sample=sample, hp=BOTH)
    assert st.ok(), st


def test_gradnorm_ragged_sampled():
    wl = W.get("ragged")
    names = {s.name: s.tensor_id for s in wl.specs}
    sample = [names["norm.1"], names["bias.2"], names["attn.0"], names["exA3.up"], names["exB40.down"],
              names["router"]]
    log(f"[parity] ragged, gradient norm and decay: 269 tensors, 8 steps, sampled {sample}")
    st = run(wl, steps=8, sample=sample, hp=BOTH)
    assert st.ok(), st


def test_gradnorm_full_6p78b_sampled():
    wl = W.get("full")
    names = {s.name: s.tensor_id for s in wl.specs}
    sample = [names["norm.3"], names["attn.7"], names["lm_head"], names["ex5.gate"], names["ex77.down"],
              names["router.1"]]
    log(f"[parity] full 6.78B, gradient norm and decay: 432 tensors, 4 steps, sampled {sample}")
    st = run(wl, steps=4, sample=sample, hp=BOTH)
    assert st.ok(), st


def test_new_hparam_errors_launch_nothing():
    dev = torch.device("cuda")
    w = torch.ones((4, 8), dtype=torch.bfloat16, device=dev)
    g = torch.ones_like(w)
    opt = SkewAdam([(W.EXPERT, w, g, 0)])
    from paper_2607_19058_amd import SkewError
    for bad in (dict(weight_decay=-0.1), dict(weight_decay=float("nan")), dict(weight_decay=float("inf")),
                dict(max_grad_norm=-1.0), dict(max_grad_norm=float("nan")), dict(max_grad_norm=float("inf"))):
        with pytest.raises(SkewError):
            opt.step(1, **bad)
    torch.cuda.synchronize()
    assert torch.equal(w, torch.ones_like(w))


# ----------------------------------------------------------------------------- tier variants
def _with_flags(wl, flags_by_tier):
    import dataclasses
    specs = [dataclasses.replace(s, state_flags=flags_by_tier.get(s.tier, 0)) for s in wl.specs]
    return W.Workload(wl.name, specs, wl.steps, grad_kind=wl.grad_kind, seed=wl.seed, banks=wl.banks,
                      zero_per_step=wl.zero_per_step, fixed_zero=wl.fixed_zero,
                      expert_sparsity=wl.expert_sparsity, outlier_rate=wl.outlier_rate,
                      outlier_scale=wl.outlier_scale, redraw_shares=wl.redraw_shares)


VARIANTS = {
    "expert_momentum": {W.EXPERT: oracle.STATE_MOMENTUM},
    "factored_router": {W.ROUTER: oracle.STATE_FACTORED},
    "uniform": {t: oracle.STATE_MOMENTUM | oracle.STATE_FACTORED for t in (W.BACKBONE, W.EXPERT, W.ROUTER)},
}


@pytest.mark.parametrize("variant", sorted(VARIANTS))
def test_variants_tiny_every_tensor(variant):
    log(f"[parity] tiny, tier variant {variant}: 21 tensors, 6 steps, all compared")
    st = run(_with_flags(W.get("tiny"), VARIANTS[variant]), steps=6)
    assert st.ok(), st


def test_variants_unit_shapes_with_gradnorm():
    log("[parity] unit shapes, uniform variant, gradient norm and decay, 3 steps")
    st = run(_with_flags(_unit_workload(), VARIANTS["uniform"]),
             hp=dict(oracle.DEFAULTS, lr=1e-2, weight_decay=2.0, max_grad_norm=0.05))
    assert st.ok(), st


def test_variant_expert_momentum_layer_sampled():
    wl = _with_flags(W.get("layer"), VARIANTS["expert_momentum"])
    names = {s.name: s.tensor_id for s in wl.specs}
    sample = [names["attn.0"], names["ex3.up"], names["ex100.down"], names["router"]]
    log(f"[parity] layer, momentum on experts: 263 tensors, 3 steps, sampled {sample}")
    st = run(wl, steps=3, sample=sample)
    assert st.ok(), st


# ----------------------------------------------------------------------------- stacked tensors
@pytest.mark.parametrize("hp", [oracle.DEFAULTS, BOTH], ids=["plain", "gnorm+decay"])
def test_stacked_tiny_every_tensor(hp):
    log(f"[parity] tiny with stacked (8, 256, 1024) expert tensors, {hp}, 8 steps, all compared")
    st = run(W.get("tiny_stacked"), hp=hp)
    assert st.ok(), st


def test_stacked_exact_clip_everywhere():
    from paper_2607_19058_amd.skewadam import FLAG_EXACT_CLIP
    log("[parity] tiny stacked with the exact clip re-check forced")
    st = run(W.get("tiny_stacked"), steps=4, flags=FLAG_EXACT_CLIP)
    assert st.ok(), st


def test_stacked_clip_factor_is_shared():
    """skew_clip_info reports one clip factor per descriptor: a stacked tensor's slices
    share it (their parity with the oracle, whose clip runs over the whole tensor, is
    checked above)."""
    dev = torch.device("cuda")
    wl = W.get("tiny_stacked")
    Wt = [W.init_weight(s, wl, dev) for s in wl.specs]
    G = [torch.empty(s.shape, dtype=torch.bfloat16, device=dev) for s in wl.specs]
    opt = SkewAdam([(s.tier, Wt[k], G[k], s.tensor_id) for k, s in enumerate(wl.specs)])
    sc = W.expert_scales(wl, 1)
    for k, s in enumerate(wl.specs):
        W.fill_grad(s, wl, 1, G[k], sc)
    opt.step(1)
    kk, route = opt.clip_info()
    assert len(kk) == len(wl.specs)
    assert all(0.0 < x <= 1.0 for x in kk)


def test_stacked_more_than_2p31_elements():
    """A stacked expert tensor of 129 x 4096 x 4096 = 2,164,260,864 elements (> 2^31, the
    size at which 8-bit optimizer kernels stop, Sec. 3 footnote), every element compared."""
    wl = W.Workload("stacked_big", [W.Spec("ex", W.EXPERT, (129, 4096, 4096), 0)], 2)
    log("[parity] stacked 129x4096x4096 expert tensor, 2 steps")
    st = run(wl)
    assert st.ok(), st
    assert st.compared >= 2 * 129 * 4096 * 4096


# ----------------------------------------------------------------------------- exact ulp, fp32 masters
def test_exact_ulp_dither_tiny_every_tensor():
    from paper_2607_19058_amd.skewadam import FLAG_EXACT_ULP
    log("[parity] tiny with the exact-ulp dither, 10 steps, all compared")
    st = run(W.get("tiny"), flags=FLAG_EXACT_ULP)
    assert st.ok(), st


def test_exact_ulp_dither_unit_shapes_with_decay():
    from paper_2607_19058_amd.skewadam import FLAG_EXACT_ULP
    log("[parity] unit shapes, exact-ulp dither and strong decay, 3 steps")
    st = run(_unit_workload(), hp=dict(oracle.DEFAULTS, lr=1e-2, weight_decay=2.0), flags=FLAG_EXACT_ULP)
    assert st.ok(), st


@pytest.mark.parametrize("flags,decay", [(0, 0.0), (2, 0.0), (2, 0.05)], ids=["plain", "exact_ulp", "exact_ulp+decay"])
def test_weights_of_every_finite_bf16_value(flags, decay):
    """Weights that take every finite bf16 value (both signs, every mantissa, biased exponents
    0 to 254: zero, the subnormals and the largest binade) in a factored expert matrix, a
    factored backbone matrix with momentum, an exact-V backbone vector and an exact-V router
    matrix, 3 steps, every element against the oracle. The dither's width comes from |w| or,
    in the exact-ulp mode, from w's exponent (clamped to the smallest normal binade for zero
    and the subnormals)."""
    from parity_util import ParityRun
    dev = torch.device("cuda", 0)
    e = np.arange(255, dtype=np.uint16)[:, None]              # biased exponent: one row each
    c = np.arange(256, dtype=np.uint16)[None, :]              # sign and mantissa: one column each
    pat = ((c >> 7) << 15) | (e << 7) | (c & 0x7F)            # (255, 256) bf16 bit patterns
    shapes = [("ex", W.EXPERT, (255, 256)), ("bb", W.BACKBONE, (255, 256)), ("bb.vec", W.BACKBONE, (255 * 256,)),
              ("rt", W.ROUTER, (255, 256))]
    specs = [W.Spec(n, tier, shape, k) for k, (n, tier, shape) in enumerate(shapes)]
    wl = W.Workload("every_bf16", specs, 3)
    weights = [torch.from_numpy(pat.reshape(shape).astype(np.int16)).view(torch.bfloat16).to(dev).contiguous()
               for _, _, shape in shapes]
    log(f"[parity] every finite bf16 weight value, flags {flags}, decay {decay}, 3 steps, all compared")
    pr = ParityRun(wl, weights=weights, flags=flags, hp=dict(oracle.DEFAULTS, weight_decay=decay))
    for t in (1, 2, 3):
        pr.step(t)
    assert pr.stats.ok(), pr.stats


@pytest.mark.parametrize("width", [256, 2048, 8192])
def test_gradients_spanning_the_bf16_exponent_range(width):
    """Gradients that take every bf16 value of biased exponent 0 to 140 (zero, the subnormals,
    both signs, every mantissa; |g| < 2^14, so no sum of squares overflows a float), one
    exponent per row (the 256 sign-and-mantissa patterns repeated along rows of `width`), in a
    factored expert matrix, a factored backbone matrix with momentum, an exact-V vector and
    an exact-V router matrix, rows shuffled differently at each of 3 steps; every element
    against the oracle. Rows of subnormal gradients have R_i = 0 in float beside nonzero
    elements; every other row spans the eps floor. The widths take the row-band pass with one
    wave per row, two, and eight."""
    from parity_util import ParityRun
    e = np.arange(141, dtype=np.uint16)[:, None]
    c = np.arange(width, dtype=np.uint16)[None, :] & 0xFF
    pat = ((c >> 7) << 15) | (e << 7) | (c & 0x7F)            # (141, width) bf16 bit patterns
    shapes = [("ex", W.EXPERT, (141, width)), ("bb", W.BACKBONE, (141, width)), ("bb.vec", W.BACKBONE, (141 * width,)),
              ("rt", W.ROUTER, (141, width))]
    specs = [W.Spec(n, tier, shape, k) for k, (n, tier, shape) in enumerate(shapes)]
    wl = W.Workload("bf16_range_grads", specs, 3)

    def spread(t, G):
        rng = np.random.default_rng(1000 + t)
        for k, (_, _, shape) in enumerate(shapes):
            g = pat[rng.permutation(141)].reshape(shape)
            G[k].copy_(torch.from_numpy(g.astype(np.int16)).view(torch.bfloat16).to(G[k].device))

    log("[parity] gradients over bf16 exponents 0..140, 3 steps, all compared")
    pr = ParityRun(wl)
    for t in (1, 2, 3):
        pr.step(t, mutate=spread)
    assert pr.stats.ok(), pr.stats


def test_fp32_masters_router_and_norms():
    """Float32 master weights for the router and the vectors (the paper's fp32 router and
    norms, Table 5): updated in float32 with no cast, bit for bit with the oracle, beside
    bf16 tensors, with decay and the gradient-norm scaling."""
    import dataclasses
    base = _unit_workload()
    specs = [dataclasses.replace(s, state_flags=oracle.STATE_FP32)
             if (s.tier == W.ROUTER or len(s.shape) == 1) else s for s in base.specs]
    wl = W.Workload("unit_fp32", specs, 3)
    log("[parity] unit shapes with float32 router and vectors, decay and gradient norm, 3 steps")
    st = run(wl, hp=dict(oracle.DEFAULTS, lr=1e-2, weight_decay=0.5, max_grad_norm=0.05))
    assert st.ok(), st


def test_fp32_master_refused_on_factored_tensors():
    dev = torch.device("cuda")
    w = torch.zeros((4, 8), dtype=torch.float32, device=dev)
    from paper_2607_19058_amd import SkewError
    with pytest.raises(SkewError):
        SkewAdam([(W.EXPERT, w, w.clone(), 0, oracle.STATE_FP32)])
