"""Pins the closed-form state model (Eq. 2 plus the exact-v term of the vector
parameters) to every state and parameter figure the paper prints (Table 1,
Table 3, Table 6, Fig. 1, Sec. 3) for its 6.78B MoE."""
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")
UNIT = {"GiB": 2.0**30, "MiB": 2.0**20, "KiB": 2.0**10, "MB_dec": 1e6, "Mparams": 1e6}


def _values():
    out = {}
    for line in open(os.path.join(GOLD, "paper_state_memory.txt")):
        line = line.split("|")[0].strip()
        if not line or line.startswith("#"):
            continue
        key, val, unit, dec = line.split()
        out[key] = (float(val), unit, int(dec))
    return out


def _inventory():
    tensors = []
    for line in open(os.path.join(GOLD, "paper_model_inventory.txt")):
        line = line.split("|")[0].strip()
        if not line or line.startswith("#"):
            continue
        tier, count, shape = line.split()
        dims = tuple(int(s) for s in shape.split("x"))
        tensors += [(oracle.TIER_NAMES[tier], dims)] * int(count)
    return tensors


VALUES = _values()
INV = _inventory()


def _check(key, amount):
    val, unit, dec = VALUES[key]
    got = round(amount / UNIT[unit], dec)
    assert got == pytest.approx(val, abs=0.5 * 10.0**-dec), (key, amount / UNIT[unit], val)


def _parts(policy="skewadam", tier=None, kind=None, ndim=None):
    tot = 0
    for t, s in INV:
        if tier is not None and t != tier:
            continue
        if ndim is not None and len(s) != ndim:
            continue
        p = oracle.tensor_state_parts(t, s, policy)
        tot += p[kind] if kind else sum(p.values())
    return 4 * tot


def _count(tier=None, ndim=None):
    return sum(int(np.prod(s)) for t, s in INV if (tier is None or t == tier) and (ndim is None or len(s) == ndim))


def test_parameter_counts():
    _check("params_backbone", _count(oracle.BACKBONE))
    _check("params_expert", _count(oracle.EXPERT))
    _check("params_router", _count(oracle.ROUTER))
    _check("params_norms", _count(oracle.BACKBONE, ndim=1))
    _check("params_total", _count())
    _check("weights_bf16_gib", 2 * _count())
    # exact tier sizes of the App. B architecture (its layer inventory counted out)
    assert _count(oracle.BACKBONE) == 341_352_448
    assert _count(oracle.EXPERT) == 6_442_450_944
    assert _count(oracle.ROUTER) == 524_288


def test_table6_components():
    B, E, R = oracle.BACKBONE, oracle.EXPERT, oracle.ROUTER
    _check("backbone_momentum_mib", _parts(tier=B, kind="m"))
    _check("backbone_momentum_gib", _parts(tier=B, kind="m"))
    _check("backbone_factored_mib", _parts(tier=B, kind="rc"))
    _check("backbone_vectors_mib", _parts(tier=B, kind="v"))
    _check("expert_factored_mib", _parts(tier=E, kind="rc"))
    _check("router_v_mib", _parts(tier=R, kind="v"))
    # Fig. 1 prints the same byte counts in decimal MB
    _check("fig1_backbone_v_mbdec", _parts(tier=B, kind="rc") + _parts(tier=B, kind="v"))
    _check("fig1_expert_v_mbdec", _parts(tier=E, kind="rc"))
    _check("fig1_router_v_mbdec", _parts(tier=R, kind="v"))


def test_totals_and_adamw():
    total = oracle.state_bytes(INV)
    assert total == _parts()
    assert total == 1_380_800_000
    _check("state_total_skewadam", total)
    _check("state_adamw", oracle.adamw_state_bytes(INV))
    _check("state_one_fp32_buffer", 4 * _count())
    # Eq. 2's approximation S ~ 4 N_bb holds to better than 1.2%
    assert abs(total / (4 * _count(oracle.BACKBONE)) - 1) < 0.012


def test_table3_ablation_states():
    _check("ablation_expert_momentum", oracle.state_bytes(INV, "expert_momentum"))
    _check("ablation_factored_router", oracle.state_bytes(INV, "factored_router"))
    _check("ablation_uniform", oracle.state_bytes(INV, "uniform"))
    _check("expert_momentum_cost_gib",
           oracle.state_bytes(INV, "expert_momentum") - oracle.state_bytes(INV))


def test_factored_vs_full_single_matrix():
    _check("factored_4096_kib", 4 * oracle.tensor_state_parts(oracle.EXPERT, (4096, 4096))["rc"])
    _check("full_4096_mib", 4 * 4096 * 4096)


def test_tier_rules():
    B, E, R = oracle.BACKBONE, oracle.EXPERT, oracle.ROUTER
    assert oracle.tensor_state_parts(B, (3, 5)) == {"m": 15, "v": 0, "rc": 8}
    assert oracle.tensor_state_parts(B, (7,)) == {"m": 7, "v": 7, "rc": 0}
    assert oracle.tensor_state_parts(E, (3, 5)) == {"m": 0, "v": 0, "rc": 8}
    assert oracle.tensor_state_parts(E, (7,)) == {"m": 0, "v": 7, "rc": 0}
    assert oracle.tensor_state_parts(R, (3, 5)) == {"m": 0, "v": 15, "rc": 0}
    assert oracle.tensor_state_parts(E, (4, 3, 5)) == {"m": 0, "v": 0, "rc": 32}   # stacked (E, n, m)
    assert oracle.tensor_state_parts(E, (0, 5)) == {"m": 0, "v": 0, "rc": 0}
