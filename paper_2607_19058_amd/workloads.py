"""Seeded synthetic workloads for the SkewAdam step: tensor inventories and inputs.

This module holds no arithmetic of the method. It lists the parameter tensors of
each workload (tier, shape, id) and draws bf16 weights and gradients with seeded
torch generators, on any device. The paper trains on OpenWebText; that dataset
and its trained weights are not used here. Synthetic gradients stand in for
them, with the paper model's tier sizes (App. B, Table 6) and the routing skew of
top-2-of-128 experts (Sec. 3 "The tiers": each expert sees about 1/64 of tokens).

Workloads (rows x cols, row-major):
  tiny    4 x 256x256 backbone; 8 experts x 2 x 256x1024; router 256x8; 2 of 8
          experts always receive zero gradients. 10 steps.
  layer   one MoE layer at width 2048: backbone 4 x 2048x2048 + 2048x8192 + 8192x2048;
          128 experts x {2048x8192, 8192x2048}; router 2048x128. 5 steps.
  full    the 6,784,327,680-parameter set at width 2048 that reproduces the paper's
          tier counts exactly (backbone 341,352,448 / experts 6,442,450,944 /
          router 524,288): token embedding 50304x2048 and untied head 2048x50304,
          positions 512x2048, 20 x 2048x2048 attention, dense SwiGLU 2x 2048x8192 +
          8192x2048, 20 norm vectors of 2048; 128 experts x {2048x8192, 2048x8192,
          8192x2048}; two routers 2048x128. 20 steps.
  stress  layer shapes; Student-t(2) gradients x 1e-3, 0.1% of entries x 100, expert
          entries zero with probability 0.9. 5 steps.
  ragged  backbone 4 x 4096x4096 + 8 vectors of 4096; experts 64 x {1536x6144, 6144x1536}
          + 64 x {4096x11008, 11008x4096}; router 4096x64. 50 steps.

Gradients: N(0, sigma^2) with sigma = 1e-3, bf16 round-to-nearest. Expert e's sigma is
scaled by rho_e = 64 pi_e with pi = 2 x Dirichlet(1) over the experts of a bank (top-2
routing: shares sum to 2, mean share 1/64, mean rho 1), redrawn each step, and about
5% of experts (6 of 128, 3 of 64) get all-zero gradients each step. Weights:
N(0, 0.02^2), bf16 round-to-nearest, drawn once.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

BACKBONE, EXPERT, ROUTER = 0, 1, 2
STATE_FP32 = 4   # the tier-variant flag of float32 master weights and gradients
SIGMA_G, SIGMA_W = 1e-3, 0.02


@dataclass
class Spec:
    name: str
    tier: int
    shape: tuple
    tensor_id: int
    bank: int = -1       # expert bank (routing group) or -1
    expert: int = -1     # expert index within its bank (a stacked tensor: its first) or -1
    state_flags: int = 0 # tier variant of the ablation (momentum / factored router)

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape))


@dataclass
class Workload:
    name: str
    specs: List[Spec]
    steps: int
    grad_kind: str = "normal"          # "normal" | "student_t"
    seed: int = 0
    banks: Dict[int, int] = field(default_factory=dict)   # bank -> number of experts
    zero_per_step: Dict[int, int] = field(default_factory=dict)
    fixed_zero: Optional[Dict[int, List[int]]] = None      # bank -> experts zero at every step
    fixed_zero_from: int = 1           # ... from this step on (earlier steps draw them as usual)
    expert_zero_rows: float = 0.0      # share of each expert matrix's rows that are always zero
    expert_sparsity: float = 0.0       # i.i.d. zero probability of expert entries
    outlier_rate: float = 0.0
    outlier_scale: float = 1.0
    redraw_shares: bool = True

    @property
    def numel(self) -> int:
        return sum(s.numel for s in self.specs)

    def tier_numel(self, tier: int, ndim: Optional[int] = None) -> int:
        return sum(s.numel for s in self.specs if s.tier == tier and (ndim is None or len(s.shape) == ndim))


def _builder():
    specs: List[Spec] = []

    def add(name, tier, shape, count=1, bank=-1, expert=-1):
        for k in range(count):
            specs.append(Spec(f"{name}{'' if count == 1 else '.' + str(k)}", tier, tuple(shape), len(specs),
                              bank, expert))
    return specs, add


def tiny() -> Workload:
    specs, add = _builder()
    add("bb", BACKBONE, (256, 256), 4)
    for e in range(8):
        add(f"ex{e}.w", EXPERT, (256, 1024), 2, bank=0, expert=e)
    add("router", ROUTER, (256, 8))
    rng = np.random.default_rng(0)
    zero = sorted(rng.choice(8, 2, replace=False).tolist())
    return Workload("tiny", specs, 10, banks={0: 8}, fixed_zero={0: zero}, redraw_shares=False)


def _layer_specs(add):
    add("attn", BACKBONE, (2048, 2048), 4)
    add("ffn.up", BACKBONE, (2048, 8192))
    add("ffn.down", BACKBONE, (8192, 2048))
    for e in range(128):
        add(f"ex{e}.up", EXPERT, (2048, 8192), bank=0, expert=e)
        add(f"ex{e}.down", EXPERT, (8192, 2048), bank=0, expert=e)
    add("router", ROUTER, (2048, 128))


def layer() -> Workload:
    specs, add = _builder()
    _layer_specs(add)
    return Workload("layer", specs, 5, banks={0: 128}, zero_per_step={0: 6})


def stress() -> Workload:
    specs, add = _builder()
    _layer_specs(add)
    return Workload("stress", specs, 5, grad_kind="student_t", banks={0: 128}, zero_per_step={0: 6},
                    expert_sparsity=0.9, outlier_rate=1e-3, outlier_scale=100.0)


def full() -> Workload:
    specs, add = _builder()
    add("tok_embed", BACKBONE, (50304, 2048))
    add("lm_head", BACKBONE, (2048, 50304))
    add("pos_embed", BACKBONE, (512, 2048))
    add("attn", BACKBONE, (2048, 2048), 20)
    add("ffn.gate", BACKBONE, (2048, 8192))
    add("ffn.up", BACKBONE, (2048, 8192))
    add("ffn.down", BACKBONE, (8192, 2048))
    add("norm", BACKBONE, (2048,), 20)
    for e in range(128):
        add(f"ex{e}.gate", EXPERT, (2048, 8192), bank=0, expert=e)
        add(f"ex{e}.up", EXPERT, (2048, 8192), bank=0, expert=e)
        add(f"ex{e}.down", EXPERT, (8192, 2048), bank=0, expert=e)
    add("router", ROUTER, (2048, 128), 2)
    return Workload("full", specs, 20, banks={0: 128}, zero_per_step={0: 6})


def ragged() -> Workload:
    specs, add = _builder()
    add("attn", BACKBONE, (4096, 4096), 4)
    add("norm", BACKBONE, (4096,), 4)
    add("bias", BACKBONE, (4096,), 4)
    for e in range(64):
        add(f"exA{e}.up", EXPERT, (1536, 6144), bank=0, expert=e)
        add(f"exA{e}.down", EXPERT, (6144, 1536), bank=0, expert=e)
    for e in range(64):
        add(f"exB{e}.up", EXPERT, (4096, 11008), bank=1, expert=e)
        add(f"exB{e}.down", EXPERT, (11008, 4096), bank=1, expert=e)
    add("router", ROUTER, (4096, 64))
    return Workload("ragged", specs, 50, banks={0: 64, 1: 64}, zero_per_step={0: 3, 1: 3})


def stacked(wl: Workload) -> Workload:
    """The same parameters with each expert projection of a bank stacked into one
    (E, n, m) tensor (slice e = expert e), in place of E separate matrices."""
    import dataclasses
    groups: Dict[tuple, List[Spec]] = {}
    order: List[object] = []
    for s in wl.specs:
        if s.tier == EXPERT and s.bank >= 0 and len(s.shape) == 2:
            key = (s.bank, s.name.split(".", 1)[-1], s.shape)
            if key not in groups:
                groups[key] = []
                order.append(key)
            groups[key].append(s)
        else:
            order.append(s)
    specs: List[Spec] = []
    for item in order:
        if isinstance(item, Spec):
            specs.append(dataclasses.replace(item, tensor_id=len(specs)))
            continue
        members = sorted(groups[item], key=lambda x: x.expert)
        bank, proj, shape = item
        assert [m.expert for m in members] == list(range(len(members))), "experts 0..E-1 of the bank"
        specs.append(Spec(f"ex.{proj}", EXPERT, (len(members),) + shape, len(specs), bank=bank, expert=0))
    return dataclasses.replace(wl, name=wl.name + "_stacked", specs=specs)


VARIANTS = {   # tier variants of the ablation (Table 3): state flags by tier
    "skewadam": {},
    "expert_momentum": {EXPERT: 1},
    "factored_router": {ROUTER: 2},
    "uniform": {BACKBONE: 3, EXPERT: 3, ROUTER: 3},
}


def with_variant(wl: Workload, variant: str) -> Workload:
    import dataclasses
    flags = VARIANTS[variant]
    specs = [dataclasses.replace(s, state_flags=flags.get(s.tier, 0)) for s in wl.specs]
    return dataclasses.replace(wl, name=f"{wl.name}_{variant}" if flags else wl.name, specs=specs)


def tiny_stacked() -> Workload:
    """The tiny workload with each expert bank projection stacked into one (8, n, m) tensor."""
    base = tiny()
    specs = [s for s in base.specs if s.bank < 0]
    nid = max(s.tensor_id for s in base.specs) + 1
    for proj, shape in (("up", (8, 256, 1024)), ("down", (8, 256, 1024))):
        specs.append(Spec(f"ex.{proj}", EXPERT, shape, nid, bank=0, expert=0))
        nid += 1
    return Workload("tiny_stacked", specs, 8, banks={0: 8}, fixed_zero=base.fixed_zero, redraw_shares=True,
                    zero_per_step={0: 1})


def tiny_late_zero() -> Workload:
    """The tiny workload whose two zero experts draw gradients at steps 1-5 and none from
    step 6 on: their R and C then decay by beta2 from real values."""
    import dataclasses
    return dataclasses.replace(tiny(), name="tiny_late_zero", fixed_zero_from=6)


def zero_rows() -> Workload:
    """Experts with 90% of their rows entirely zero at every step (R_i = 0 there), beside a
    backbone and a router: 8 experts x {512x2048, 2048x512}."""
    specs, add = _builder()
    add("bb", BACKBONE, (512, 512), 2)
    for e in range(8):
        add(f"ex{e}.up", EXPERT, (512, 2048), bank=0, expert=e)
        add(f"ex{e}.down", EXPERT, (2048, 512), bank=0, expert=e)
    add("router", ROUTER, (512, 8))
    return Workload("zero_rows", specs, 8, banks={0: 8}, expert_zero_rows=0.9, zero_per_step={0: 1})


CONFIGS = {"tiny": tiny, "layer": layer, "full": full, "stress": stress, "ragged": ragged,
           "tiny_stacked": tiny_stacked, "tiny_late_zero": tiny_late_zero, "zero_rows": zero_rows}


def get(name: str) -> Workload:
    return CONFIGS[name]()


# ----------------------------------------------------------------------------------------------
# seeded draws
# ----------------------------------------------------------------------------------------------
def _seed(*parts: int) -> int:
    """Deterministic 63-bit seed from integers (no relation to the dither hash)."""
    ss = np.random.SeedSequence([int(p) & 0xFFFFFFFF for p in parts])
    lo, hi = (int(x) for x in ss.generate_state(2, np.uint32))
    return (lo | (hi << 32)) & ((1 << 63) - 1)


def expert_scales(wl: Workload, step: int) -> Dict[int, np.ndarray]:
    """Per bank, the gradient scale rho_e of each expert at `step` (0 = no gradient)."""
    out = {}
    for bank, ne in wl.banks.items():
        rng = np.random.default_rng(_seed(wl.seed, 7, bank, step if wl.redraw_shares else 0))
        if wl.redraw_shares:
            pi = 2.0 * rng.dirichlet(np.ones(ne))      # token shares under top-2 routing (sum 2)
            rho = (ne / 2.0) * pi                      # mean 1
        else:
            rho = np.ones(ne)
        if wl.fixed_zero is not None and step >= wl.fixed_zero_from:
            rho[wl.fixed_zero.get(bank, [])] = 0.0
        nz = wl.zero_per_step.get(bank, 0)
        if nz:
            rho[rng.choice(ne, nz, replace=False)] = 0.0
        out[bank] = rho
    return out


def init_weight(spec: Spec, wl: Workload, device, out=None):
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(_seed(wl.seed, 1, spec.tensor_id))
    w = torch.randn(spec.shape, generator=gen, device=device, dtype=torch.float32).mul_(SIGMA_W)
    if out is None:
        return w if spec.state_flags & STATE_FP32 else w.to(torch.bfloat16)   # float32 masters stay float32
    out.copy_(w)
    return out


def fill_grad(spec: Spec, wl: Workload, step: int, out, scales: Optional[Dict[int, np.ndarray]] = None):
    """Draw tensor `spec`'s gradient for `step` into the bf16 tensor `out`."""
    import torch
    if scales is None:
        scales = expert_scales(wl, step)
    stacked = len(spec.shape) == 3 and spec.bank >= 0   # slice e is expert `expert + e`
    if stacked:
        rho = scales[spec.bank][spec.expert:spec.expert + spec.shape[0]]
        if not np.any(rho):
            out.zero_()
            return out
    else:
        rho = 1.0 if spec.bank < 0 else float(scales[spec.bank][spec.expert])
        if rho == 0.0:
            out.zero_()
            return out
    dev = out.device
    gen = torch.Generator(device=dev)
    gen.manual_seed(_seed(wl.seed, 2, step, spec.tensor_id))
    z = torch.randn(spec.shape, generator=gen, device=dev, dtype=torch.float32)
    if wl.grad_kind == "student_t":
        # t with 2 degrees of freedom: Z / sqrt(chi2_2 / 2) and chi2_2 / 2 = -ln U
        u = torch.rand(spec.shape, generator=gen, device=dev, dtype=torch.float32).clamp_(min=1e-30)
        z.div_(torch.sqrt(-torch.log(u)))
        del u
    if wl.outlier_rate > 0:
        hit = torch.rand(spec.shape, generator=gen, device=dev) < wl.outlier_rate
        z.mul_(torch.where(hit, wl.outlier_scale, 1.0))
        del hit
    if wl.expert_sparsity > 0 and spec.tier == EXPERT:
        keep = torch.rand(spec.shape, generator=gen, device=dev) >= wl.expert_sparsity
        z.mul_(keep)
        del keep
    if wl.expert_zero_rows > 0 and spec.tier == EXPERT and len(spec.shape) == 2:
        # the same rows at every step (R_i stays exactly 0 there, beside nonzero rows)
        rows = np.random.default_rng(_seed(wl.seed, 3, spec.tensor_id)).random(spec.shape[0])
        z[torch.as_tensor(rows < wl.expert_zero_rows, device=dev)] = 0.0
    if stacked:
        z.mul_(torch.as_tensor(SIGMA_G * rho, dtype=torch.float32, device=dev)[:, None, None])
    else:
        z.mul_(SIGMA_G * rho)
    out.copy_(z)
    return out
