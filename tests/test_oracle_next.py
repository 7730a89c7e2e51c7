"""Pins of the oracle's two optional terms of the step.

Decoupled weight decay (Sec. 3 footnote and Sec. 6: fused into the float32 update ahead of
the dithered cast; Table 5: lambda = 0.05, none on the router) and the global gradient-norm
scaling the trainer applies before every step (Sec. 4: clipping at 1.0), both against
torch's own routines in float64: torch.optim.AdamW for the decay, and
torch.nn.utils.clip_grad_norm_ followed by torch.optim.Adam for the scaling.
"""
import numpy as np
import pytest
import torch

import oracle

B, E, R = oracle.BACKBONE, oracle.EXPERT, oracle.ROUTER
LR, B1, B2, EPS = (float(np.float32(v)) for v in (3e-4, 0.9, 0.999, 1e-8))


def bf16(x) -> np.ndarray:
    t = torch.as_tensor(np.asarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def f32(b) -> np.ndarray:
    return oracle.bf16_to_f32(b)


def make(tier, w, tid=0, flags=0):
    w = np.ascontiguousarray(w, np.uint16)
    return oracle.Tensor(tier=tier, w=w.copy(), g=np.zeros_like(w), tensor_id=tid, state_flags=flags).init_state()


def rank1_grads(rng, n, m, steps):
    a = rng.choice([1.0, 1.5], n) * 2.0 ** rng.integers(-3, 1, n)
    b = rng.choice([1.0, 1.5], m) * 2.0 ** rng.integers(-3, 1, m)
    out = []
    for _ in range(steps):
        lt = rng.choice([1.0, 1.25, 1.5]) * 2.0 ** -2
        g = rng.choice([-1.0, 1.0], (n, m)) * np.outer(a, b) * lt
        out.append(bf16(g))
    return out


# ----------------------------------------------------------------------------- weight decay
def _adamw_reference(tier, shape, grads, beta1, lam, decayed=True):
    """torch.optim.AdamW in float64 beside the oracle (eps -> 0, no update clip): the
    weight the oracle hands to the dither equals AdamW's updated weight."""
    rng = np.random.default_rng(11)
    T = make(tier, bf16(rng.normal(0, 0.02, shape)), 3)
    p = torch.zeros(shape, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=LR, betas=(beta1, B2), eps=0.0, weight_decay=lam if decayed else 0.0,
                            foreach=False)
    for t, g in enumerate(grads, start=1):
        T.g = g
        w_before = f32(T.w).astype(np.float64)
        with torch.no_grad():
            p.copy_(torch.from_numpy(w_before))
        p.grad = torch.from_numpy(f32(g).astype(np.float64))
        opt.step()
        oracle.step([T], t, eps=1e-30, clip_threshold=float("inf"), want_x=True, weight_decay=lam)
        ref = p.detach().numpy()
        # two float32 roundings of a value ~|w| (the decayed weight, then the update)
        np.testing.assert_allclose(T.x_out, ref, rtol=2.5e-7, atol=2e-9)


@pytest.mark.parametrize("lam", [0.05, 10.0])
def test_decay_backbone_vector_is_adamw(lam):
    rng = np.random.default_rng(12)
    grads = [bf16(rng.normal(0, 1e-2, (33,)) + 1e-4) for _ in range(6)]
    _adamw_reference(B, (33,), grads, beta1=B1, lam=lam)


@pytest.mark.parametrize("lam", [0.05, 10.0])
def test_decay_rank_one_expert_is_adamw_without_momentum(lam):
    rng = np.random.default_rng(13)
    _adamw_reference(E, (6, 11), rank1_grads(rng, 6, 11, 6), beta1=0.0, lam=lam)


def test_router_takes_no_decay():
    rng = np.random.default_rng(14)
    grads = [bf16(rng.normal(0, 1e-2, (9, 13)) + 1e-4) for _ in range(4)]
    _adamw_reference(R, (9, 13), grads, beta1=0.0, lam=10.0, decayed=False)


def test_decay_with_zero_update_is_one_rounding():
    """With U = 0 the weight handed to the dither is RN(w - (lr lambda) w): within half a
    float ulp of the float64 product, and the router keeps w exactly."""
    rng = np.random.default_rng(15)
    w0 = bf16(rng.normal(0, 0.02, (8, 16)))
    lam = 0.05
    wd = np.float32(LR * lam)
    for tier in (B, E, R):
        T = make(tier, w0)      # zero gradients: R = C = 0, D = sqrt(eps), U = 0
        oracle.step([T], 1, want_x=True, want_u=True, weight_decay=lam)
        assert not np.any(T.u_out)
        w = f32(w0).astype(np.float64)
        if tier == R:
            assert np.array_equal(T.x_out, f32(w0))
        else:
            exact = w - float(wd) * w
            ulp = np.spacing(np.abs(exact).astype(np.float32)).astype(np.float64)
            assert np.all(np.abs(T.x_out.astype(np.float64) - exact) <= 0.5 * ulp)
            assert np.any(T.x_out != f32(w0))


def test_zero_decay_is_bit_identical_to_no_decay():
    rng = np.random.default_rng(16)
    w0 = bf16(rng.normal(0, 0.02, (7, 9)))
    g = bf16(rng.normal(0, 1e-3, (7, 9)))
    outs = []
    for lam in (None, 0.0):
        T = make(B, w0)
        T.g = g
        if lam is None:
            oracle.step([T], 1)
        else:
            oracle.step([T], 1, weight_decay=lam)
        outs.append(T.w.copy())
    assert np.array_equal(outs[0], outs[1])


# ----------------------------------------------------------------------------- gradient norm
def _clip_adam_reference(specs, steps, max_norm, seed=21):
    """torch.nn.utils.clip_grad_norm_ over all tensors, then torch.optim.Adam (beta1 = 0 for
    tiers without momentum), in float64, beside one oracle step over the same tensors."""
    rng = np.random.default_rng(seed)
    Ts, ps, opts = [], [], []
    for k, (tier, shape, grad_fn) in enumerate(specs):
        Ts.append(make(tier, bf16(rng.normal(0, 0.02, shape)), k))
        ps.append(torch.zeros(shape, dtype=torch.float64, requires_grad=True))
        opts.append(torch.optim.Adam([ps[-1]], lr=LR, betas=(B1 if tier == B else 0.0, B2), eps=0.0,
                                     foreach=False))
    for t in range(1, steps + 1):
        for (tier, shape, grad_fn), T, p in zip(specs, Ts, ps):
            T.g = grad_fn(rng)
            with torch.no_grad():
                p.copy_(torch.from_numpy(f32(T.w).astype(np.float64)))
            p.grad = torch.from_numpy(f32(T.g).astype(np.float64))
        total = torch.nn.utils.clip_grad_norm_(ps, max_norm)
        for opt in opts:
            opt.step()
        oracle.step(Ts, t, eps=1e-30, clip_threshold=float("inf"), want_x=True, max_grad_norm=max_norm)
        coef = min(1.0, max_norm / (float(total) + 1e-6))
        assert abs(oracle.last_gcoef() - coef) <= 1e-7 * coef
        for T, p in zip(Ts, ps):
            np.testing.assert_allclose(T.x_out, p.detach().numpy(), rtol=2e-7, atol=4e-9)
    return Ts


def test_gradnorm_is_global_over_tensors_backbone_vectors():
    specs = [(B, (33,), lambda r: bf16(r.normal(0, 0.3, (33,)) + 1e-3)),
             (B, (17,), lambda r: bf16(r.normal(0, 0.05, (17,)) + 1e-3))]
    _clip_adam_reference(specs, 5, max_norm=1.0)


def test_gradnorm_router_and_rank_one_matrices():
    rng = np.random.default_rng(22)
    g_bb = iter(rank1_grads(rng, 12, 5, 4))
    specs = [(R, (9, 13), lambda r: bf16(r.normal(0, 0.2, (9, 13)) + 1e-3)),
             (B, (12, 5), lambda r: next(g_bb))]
    _clip_adam_reference(specs, 4, max_norm=0.5)


def test_gradnorm_above_the_norm_is_bit_identical_to_off():
    rng = np.random.default_rng(23)
    shapes = [(8, 24), (40,), (5, 3)]
    w0 = [bf16(rng.normal(0, 0.02, s)) for s in shapes]
    g = [bf16(rng.normal(0, 1e-3, s)) for s in shapes]
    res = []
    for mgn in (0.0, 1e3):
        Ts = [make(tier, w) for tier, w in zip((E, B, R), w0)]
        for T, gg in zip(Ts, g):
            T.g = gg
        oracle.step(Ts, 1, max_grad_norm=mgn)
        assert oracle.last_gcoef() == 1.0
        res.append([T.w.copy() for T in Ts] + [T.r for T in Ts if T.r is not None])
    for a, b in zip(*res):
        assert np.array_equal(a, b)


def test_gradnorm_factored_rank_one_equals_exact_tier():
    """I1 with the scaling on: for rank-one G*G the factored statistics (c^2 times the exact
    sums) and the exact second moment of the scaled gradient give the same update."""
    rng = np.random.default_rng(24)
    n, m = 6, 10
    w0 = bf16(rng.normal(0, 0.02, (n, m)))
    Tf, Tx = make(E, w0, 5), make(R, w0, 5)
    for t, g in enumerate(rank1_grads(rng, n, m, 5), start=1):
        Tf.g = Tx.g = g
        oracle.step([Tf], t, want_u=True, max_grad_norm=0.3, gsq_total=float(np.sum(f32(g).astype(np.float64) ** 2)))
        cf = oracle.last_gcoef()
        oracle.step([Tx], t, want_u=True, max_grad_norm=0.3)
        assert oracle.last_gcoef() == cf < 1.0
        np.testing.assert_allclose(Tf.u_out, Tx.u_out, rtol=2e-6, atol=1e-7)


def test_gradnorm_sample_with_the_set_sum_equals_the_full_set():
    """A step over a sample of the tensors, given the whole set's sum of squares, updates the
    sample exactly as the step over the whole set does."""
    rng = np.random.default_rng(25)
    shapes = [(8, 24), (40,), (5, 3), (16, 16)]
    tiers = (E, B, R, B)
    w0 = [bf16(rng.normal(0, 0.02, s)) for s in shapes]
    g = [bf16(rng.normal(0, 0.1, s)) for s in shapes]
    full = [make(tier, w) for tier, w in zip(tiers, w0)]
    for T, gg in zip(full, g):
        T.g = gg
    oracle.step(full, 1, max_grad_norm=1.0)
    c_full = oracle.last_gcoef()
    assert c_full < 1.0
    total = sum(float(np.sum(f32(gg).astype(np.float64) ** 2)) for gg in g)
    part = [make(tiers[i], w0[i]) for i in (0, 3)]
    for T, i in zip(part, (0, 3)):
        T.g = g[i]
    oracle.step(part, 1, max_grad_norm=1.0, gsq_total=total)
    assert oracle.last_gcoef() == c_full
    for T, i in zip(part, (0, 3)):
        assert np.array_equal(T.w, full[i].w)


def test_gradnorm_nonfinite_norm_propagates():
    T = make(E, bf16(np.full((3, 4), 0.01)))
    g = np.zeros((3, 4), np.float32)
    g[1, 2] = np.inf
    T.g = bf16(g)
    oracle.step([T], 1, max_grad_norm=1.0)
    # inf norm: the scale is 0 and inf * 0 is NaN
    assert oracle.last_gcoef() == 0.0
    assert np.isnan(f32(T.w)).any()


# ----------------------------------------------------------------------------- tier variants
def _variant_adam(tier, flags, shape, grads, beta1):
    rng = np.random.default_rng(31)
    T = make(tier, bf16(rng.normal(0, 0.02, shape)), 7, flags)
    p = torch.zeros(shape, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([p], lr=LR, betas=(beta1, B2), eps=0.0, foreach=False)
    for t, g in enumerate(grads, start=1):
        T.g = g
        w_before = f32(T.w).astype(np.float64)
        with torch.no_grad():
            p.copy_(torch.from_numpy(w_before))
        p.grad = torch.from_numpy(f32(g).astype(np.float64))
        opt.step()
        oracle.step([T], t, eps=1e-30, clip_threshold=float("inf"), want_u=True, want_x=True)
        np.testing.assert_allclose(T.u_out, (w_before - p.detach().numpy()) / LR, rtol=3e-6, atol=3e-6)
        np.testing.assert_allclose(T.x_out, p.detach().numpy(), rtol=1e-7, atol=2e-9)
    return T


def test_variant_expert_momentum_is_adam():
    """Table 3 '+ momentum on experts': a rank-one expert matrix with momentum is Adam."""
    rng = np.random.default_rng(32)
    T = _variant_adam(E, oracle.STATE_MOMENTUM, (6, 11), rank1_grads(rng, 6, 11, 6), beta1=B1)
    assert T.m is not None and T.r is not None and T.v is None


def test_variant_factored_router_is_adam_without_momentum():
    """Table 3 'factored router': a rank-one router matrix, factored, is Adam(beta1 = 0)."""
    rng = np.random.default_rng(33)
    T = _variant_adam(R, oracle.STATE_FACTORED, (9, 8), rank1_grads(rng, 9, 8, 6), beta1=0.0)
    assert T.v is None and T.r is not None and T.m is None


def test_variant_uniform_router_is_adam():
    """Table 3 'uniform (momentum + factored)': the router with both is Adam(beta1, beta2)."""
    rng = np.random.default_rng(34)
    _variant_adam(R, oracle.STATE_MOMENTUM | oracle.STATE_FACTORED, (7, 12), rank1_grads(rng, 7, 12, 6),
                  beta1=B1)


def test_variant_router_vector_stays_exact():
    T = make(R, bf16(np.full(16, 0.01)), 0, oracle.STATE_FACTORED)
    assert T.v is not None and T.r is None      # vectors keep the exact second moment (Alg. 1)


# ----------------------------------------------------------------------------- stacked tensors
@pytest.mark.parametrize("tier", [E, B])
def test_stacked_equals_separate_slices(tier):
    """A stacked (E, n, m) tensor factors per slice (Sec. 3 footnote): without the clip
    binding, each slice's R, C, M, update and pre-dither weight equal those of the slice
    stepped alone; the clip's RMS runs over the whole tensor."""
    rng = np.random.default_rng(41)
    Eb, n, m = 4, 6, 10
    w0 = bf16(rng.normal(0, 0.02, (Eb, n, m)))
    S = make(tier, w0, 9)
    parts = [make(tier, w0[e], 100 + e) for e in range(Eb)]
    for t in range(1, 4):
        scale = 10.0 ** rng.uniform(-4, -1, Eb)
        g = bf16(rng.normal(0, 1, (Eb, n, m)) * scale[:, None, None])
        S.g = g
        oracle.step([S], t, clip_threshold=float("inf"), want_u=True, want_x=True)
        ss = 0.0
        for e, P in enumerate(parts):
            P.g = g[e].copy()
            oracle.step([P], t, clip_threshold=float("inf"), want_u=True, want_x=True)
            assert np.array_equal(S.r[e], P.r) and np.array_equal(S.c[e], P.c)
            if tier == B:
                assert np.array_equal(S.m[e], P.m)
            assert np.array_equal(S.u_out[e], P.u_out)
            ss += P.rms ** 2 * n * m
        assert abs(S.rms ** 2 * Eb * n * m - ss) <= 1e-12 * ss
        # keep the slices' weights equal to the stacked ones (the dither differs by index)
        for e, P in enumerate(parts):
            P.w = S.w[e].copy()


def test_stacked_clip_runs_over_the_whole_tensor():
    rng = np.random.default_rng(42)
    Eb, n, m = 3, 5, 8
    S = make(E, bf16(rng.normal(0, 0.02, (Eb, n, m))), 1)
    g = rng.normal(0, 1e-3, (Eb, n, m))
    g[1] *= 30.0                       # one slice dominates the update's RMS
    S.g = bf16(g)
    oracle.step([S], 1, clip_threshold=0.5, want_u=True)
    rms_after = float(np.sqrt(np.mean(S.u_out.astype(np.float64) ** 2)))
    assert S.rms > 0.5 and abs(rms_after - 0.5) <= 1e-6     # one factor k for all slices


# ----------------------------------------------------------------------------- exact-ulp dither
def _bf16_next(bits):
    return bits + 1   # positive finite bf16: the next value up


def test_exact_ulp_dither_keeps_grid_points():
    """With the exact ulp the noise stays strictly inside +-ulp(w)/2, so a weight with a zero
    update rounds back to itself (off powers of two, where the spacing below is half)."""
    rng = np.random.default_rng(51)
    w0 = bf16(rng.normal(0, 0.02, (64, 64)))
    pow2 = (w0 & 0x7F) == 0
    assert pow2.any()
    w0[pow2] += 1                                          # off exact powers of two
    T = make(E, w0)
    oracle.step([T], 1, exact_ulp=True)                    # zero gradients: U = 0
    assert np.array_equal(T.w, w0)
    T2 = make(E, w0)
    oracle.step([T2], 1)                                   # the approximate width moves some
    assert not np.array_equal(T2.w, w0)


@pytest.mark.parametrize("frac", [0.1, 0.37, 0.5, 0.83])
def test_exact_ulp_dither_is_unbiased_stochastic_rounding(frac):
    """Unbiased stochastic rounding (Sec. 3): with the exact ulp, a pre-cast value at
    fraction f of the way between two bf16 neighbours rounds up with probability f."""
    n = 1 << 15
    lo_bits = np.full(n, 0x3C81, np.uint16)                # 2^-6 (1 + 2^-7): spacing 2^-13 either side
    lo = float(f32(lo_bits[:1])[0])
    ulp = 2.0 ** -13
    # backbone vector (exact V), t = 1: U = sign(g); choose lr so that x = w + frac * ulp
    T = make(B, lo_bits + np.uint16(1))                    # w one step up, x lands below it
    T.g = bf16(np.full(n, 1e-2))
    lr = (1.0 - frac) * ulp
    oracle.step([T], 1, lr=lr, clip_threshold=float("inf"), want_x=True, exact_ulp=True)
    x = T.x_out.astype(np.float64)
    f_emp = float(np.mean((x - lo) / ulp))
    assert abs(f_emp - frac) < 2e-3
    up = np.mean(T.w == lo_bits + np.uint16(1))
    assert np.all((T.w == lo_bits) | (T.w == lo_bits + np.uint16(1)))
    assert abs(up - f_emp) < 4.0 * np.sqrt(f_emp * (1 - f_emp) / n) + 1e-3


# ----------------------------------------------------------------------------- float32 masters
def test_fp32_master_vector_is_adamw():
    """Float32 master weights (the paper's fp32 norms and router, Table 5) are updated in
    float32 with no cast: a backbone vector follows AdamW to float32 accuracy."""
    rng = np.random.default_rng(61)
    shape = (48,)
    w0 = rng.normal(0, 0.02, shape).astype(np.float32)
    T = oracle.Tensor(tier=B, w=w0.copy(), g=np.zeros(shape, np.float32), tensor_id=2,
                      state_flags=oracle.STATE_FP32).init_state()
    p = torch.tensor(w0.astype(np.float64), requires_grad=True)
    opt = torch.optim.AdamW([p], lr=LR, betas=(B1, B2), eps=0.0, weight_decay=0.05, foreach=False)
    for t in range(1, 7):
        g = rng.normal(0, 1e-2, shape).astype(np.float32) + 1e-4
        T.g = g
        with torch.no_grad():
            p.copy_(torch.from_numpy(T.w.astype(np.float64)))
        p.grad = torch.from_numpy(g.astype(np.float64))
        opt.step()
        oracle.step([T], t, eps=1e-30, clip_threshold=float("inf"), weight_decay=0.05)
        np.testing.assert_allclose(T.w, p.detach().numpy(), rtol=3e-7, atol=1e-10)


def test_fp32_master_router_matrix_and_factored_refusal():
    rng = np.random.default_rng(62)
    T = oracle.Tensor(tier=R, w=rng.normal(0, 0.02, (8, 4)).astype(np.float32), g=np.zeros((8, 4), np.float32),
                      tensor_id=3, state_flags=oracle.STATE_FP32).init_state()
    T.g = rng.normal(0, 1e-2, (8, 4)).astype(np.float32)
    w_before = T.w.copy()
    assert oracle.step([T], 1) == 0 and not np.array_equal(T.w, w_before)
    F = oracle.Tensor(tier=E, w=np.zeros((8, 4), np.float32), g=np.zeros((8, 4), np.float32), tensor_id=4,
                      state_flags=oracle.STATE_FP32).init_state()
    assert oracle.step([F], 1) == -2


def test_exact_ulp_of_subnormal_weights():
    """bf16 subnormals (biased exponent 0) are spaced 2^-133 apart, like the smallest normal
    binade. With the exact ulp and U = 0 such a weight stays on its grid point; an update of
    a fraction f of that spacing rounds up with probability f, which pins the spacing the
    dither takes among the subnormals (half of it would round up never for f < 1/4, twice it
    would round up 3/8 of the time at f = 1/4)."""
    sub = np.arange(1, 128, dtype=np.uint16)                     # positive subnormal bf16 values
    w0 = np.concatenate([sub, sub | np.uint16(0x8000)]).reshape(2, 127)
    T = make(E, w0)
    oracle.step([T], 1, exact_ulp=True)                          # zero gradients: U = 0
    assert np.array_equal(T.w, w0)
    n = 1 << 15
    spacing = 2.0 ** -133
    for frac in (0.25, 0.75):
        base = np.full(n, 0x0040, np.uint16)                     # 64 * 2^-133
        V = make(B, base + np.uint16(1))                          # backbone vector, exact V
        V.g = bf16(np.full(n, 1e-2))                              # t = 1: U = sign(g) = 1
        lr = float(np.float32((1.0 - frac) * spacing))           # exact in float32 (subnormal)
        oracle.step([V], 1, lr=lr, clip_threshold=float("inf"), want_x=True, exact_ulp=True)
        x = V.x_out.astype(np.float64)
        assert np.allclose((x - 64 * spacing) / spacing, frac)
        assert np.all((V.w == base) | (V.w == base + np.uint16(1)))
        up = float(np.mean(V.w == base + np.uint16(1)))
        assert abs(up - frac) < 4.0 * np.sqrt(frac * (1 - frac) / n) + 2e-3, (frac, up)
