"""Pins the oracle's step to what the paper and the mathematics fix.

I1  rank-one exactness of the factored estimator (Sec. 3 "Factored second moments")
I2  a zero-gradient step is a pure EMA decay of R and C and leaves U = 0 (Eq. 1)
I3  update clipping bounds RMS(U) by d, with equality when it clips (Sec. 3; Alg. 1)
I4  at t = 1 the bias-corrected update of an unfloored element is sign(g) (Alg. 1)
I5  special cases equal torch.optim.Adam: the router tier is Adam(beta1=0), a backbone
    vector is Adam(beta1, beta2), and rank-one factored tensors match both (Alg. 1)
I6  the dither has half-width 2^-8 |w| (ulp(w) ~ 2^-7 |w|, Sec. 3), checked against the
    analytic rounding probabilities
plus a float64 dense brute force on tiny shapes.
"""
import numpy as np
import pytest
import torch

import oracle

B, E, R = oracle.BACKBONE, oracle.EXPERT, oracle.ROUTER
# the step's hyper-parameters are float32 values; references use the same rounded numbers
LR, B1, B2, EPS = (float(np.float32(v)) for v in (3e-4, 0.9, 0.999, 1e-8))


def bf16(x) -> np.ndarray:
    """float -> bf16 bits via torch (round to nearest even)."""
    t = torch.as_tensor(np.asarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def f32(b) -> np.ndarray:
    return oracle.bf16_to_f32(b)


def make(tier, w, tid=0):
    w = np.ascontiguousarray(w, np.uint16)
    return oracle.Tensor(tier=tier, w=w.copy(), g=np.zeros_like(w), tensor_id=tid).init_state()


def rank1_grads(rng, n, m, steps):
    """bf16-exact gradients whose elementwise square is rank one at every step:
    g_ij = s_ij * a_i * b_j * l_t with 2-bit factors times powers of two."""
    a = rng.choice([1.0, 1.5], n) * 2.0 ** rng.integers(-3, 1, n)
    b = rng.choice([1.0, 1.5], m) * 2.0 ** rng.integers(-3, 1, m)
    out = []
    for _ in range(steps):
        lt = rng.choice([1.0, 1.25, 1.5]) * 2.0 ** -2
        s = rng.choice([-1.0, 1.0], (n, m))
        g = s * np.outer(a, b) * lt
        gb = bf16(g)
        assert np.array_equal(f32(gb).astype(np.float64), g)       # exactly representable
        out.append(gb)
    return out


# ----------------------------------------------------------------------------- I1
@pytest.mark.parametrize("shape", [(5, 7), (16, 3), (1, 9), (9, 1)])
def test_I1_rank_one_factored_equals_exact(shape):
    rng = np.random.default_rng(1)
    n, m = shape
    w0 = bf16(rng.normal(0, 0.02, shape))
    fac, ex = make(E, w0, 3), make(R, w0, 3)       # same id -> same dither
    for t, g in enumerate(rank1_grads(rng, n, m, 6), start=1):
        for T in (fac, ex):
            T.g = g
            T.w = w0.copy()
        oracle.step([fac, ex], t, want_u=True)
        assert fac.r.mean() >= EPS     # the clamp max(mean R, eps) is inactive: the estimate is exact
        np.testing.assert_allclose(fac.u_out, ex.u_out, rtol=2e-6, atol=0)
        vhat = np.outer(fac.r, fac.c) / max(fac.r.mean(), EPS)
        np.testing.assert_allclose(vhat, ex.v.reshape(n, m), rtol=4e-6)


# ----------------------------------------------------------------------------- I2
@pytest.mark.parametrize("tier", [E, B])
@pytest.mark.parametrize("scale", [1e-3, 1e-1])
def test_I2_zero_gradient_step_is_pure_decay(tier, scale):
    rng = np.random.default_rng(2)
    shape = (6, 10)
    T = make(tier, bf16(rng.normal(0, 0.02, shape)), 5)
    for t in (1, 2, 3):
        T.g = bf16(rng.normal(0, scale, shape))
        oracle.step([T], t)
    r0, c0, w0 = T.r.copy(), T.c.copy(), T.w.copy()
    m0 = None if T.m is None else T.m.copy()
    vhat0 = np.outer(r0, c0) / max(float(r0.mean()), EPS)
    T.g = np.zeros(shape, np.uint16)
    oracle.step([T], 4, want_u=True, want_x=True)
    assert np.array_equal(T.r, (np.float32(B2) * r0).astype(np.float32))
    assert np.array_equal(T.c, (np.float32(B2) * c0).astype(np.float32))
    vhat1 = np.outer(T.r, T.c) / max(float(T.r.mean()), EPS)
    # R C^T / mean(R) decays by beta2; once mean(R) sits on its eps clamp, R C^T / eps decays by beta2^2
    clamped = r0.mean() < EPS
    assert clamped == (scale == 1e-3)
    np.testing.assert_allclose(vhat1, (B2 * B2 if clamped else B2) * vhat0, rtol=1e-6)
    if tier == E:
        assert np.all(T.u_out == 0) and np.array_equal(T.x_out, f32(w0))
    else:  # momentum keeps moving the backbone; M decays exactly by beta1
        assert np.array_equal(T.m, (np.float32(B1) * m0).astype(np.float32))


def test_I2_never_routed_expert_stays_finite():
    T = make(E, bf16(np.full((4, 8), 0.5)), 9)
    for t in range(1, 4):
        w_before = f32(T.w).copy()
        oracle.step([T], t, want_u=True, want_x=True)
        assert np.all(T.r == 0) and np.all(T.c == 0)
        assert np.all(T.u_out == 0) and np.array_equal(T.x_out, w_before)
        assert np.all(np.isfinite(f32(T.w)))


# ----------------------------------------------------------------------------- I3
@pytest.mark.parametrize("tier,shape,scale", [(E, (32, 48), 1e-3), (B, (32, 48), 1e-3), (R, (16, 8), 1e-3),
                                              (E, (32, 48), 1e-1), (B, (40,), 1e-2)])
@pytest.mark.parametrize("d", [1.0, 0.5, 3.0])
def test_I3_clip_bounds_rms(tier, shape, scale, d):
    rng = np.random.default_rng(3)
    T = make(tier, bf16(rng.normal(0, 0.02, shape)), 1)
    saw_clip = saw_free = False
    for t in range(1, 13):
        g = rng.normal(0, scale, shape) * (1 + 20 * (rng.random(shape) < 0.01))
        T.g = bf16(g)
        oracle.step([T], t, clip_threshold=d, want_u=True)
        rms_u = float(np.sqrt(np.mean(T.u_out.astype(np.float64) ** 2)))
        assert rms_u <= d * (1 + 1e-6)
        if T.rms / d > 1:
            saw_clip = True
            assert rms_u == pytest.approx(d, rel=1e-6)
        else:
            saw_free = True
            assert rms_u == pytest.approx(T.rms, rel=1e-6)
    assert saw_clip or saw_free


# ----------------------------------------------------------------------------- I4
@pytest.mark.parametrize("tier,shape,rank1", [(R, (8, 12), False), (B, (50,), False),
                                              (E, (7, 5), True), (B, (7, 5), True)])
def test_I4_first_step_is_sign(tier, shape, rank1):
    rng = np.random.default_rng(4)
    if rank1:
        g = rank1_grads(rng, *shape, 1)[0]   # |g| >= 2^-8 > sqrt(eps / (1 - beta2)) ~ 3.2e-3
    else:   # exact-v tensors: every element with |g| > 3.2e-3 is unfloored
        g = bf16(rng.choice([-1, 1], shape) * rng.uniform(1e-2, 1, shape))
    T = make(tier, bf16(rng.normal(0, 0.02, shape)), 2)
    T.g = g
    oracle.step([T], 1, want_u=True)
    np.testing.assert_allclose(T.u_out, np.sign(f32(g)), rtol=0, atol=6e-7)
    assert T.rms == pytest.approx(1.0, abs=1e-6)


# ----------------------------------------------------------------------------- I5
def _adam_reference(tier, shape, grads, beta1, rank1=False):
    """Run torch.optim.Adam in float64 next to the oracle (eps -> 0, no clip) and
    compare the update the oracle applies with Adam's, step by step."""
    rng = np.random.default_rng(5)
    T = make(tier, bf16(rng.normal(0, 0.02, shape)), 4)
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
        adam_u = (w_before - p.detach().numpy()) / LR
        # |U| <= ~1; fp32 momentum loses relative accuracy only where it cancels to ~0
        np.testing.assert_allclose(T.u_out, adam_u, rtol=3e-6, atol=3e-6)
        np.testing.assert_allclose(T.x_out, p.detach().numpy(), rtol=1e-7, atol=2e-9)


def test_I5_router_is_adam_without_momentum():
    rng = np.random.default_rng(6)
    grads = [bf16(rng.normal(0, 1e-2, (9, 13)) + 1e-4) for _ in range(8)]
    _adam_reference(R, (9, 13), grads, beta1=0.0)


def test_I5_backbone_vector_is_adam():
    rng = np.random.default_rng(7)
    grads = [bf16(rng.normal(0, 1e-2, (33,)) + 1e-4) for _ in range(8)]
    _adam_reference(B, (33,), grads, beta1=B1)


def test_I5_rank_one_expert_is_adam_without_momentum():
    rng = np.random.default_rng(8)
    _adam_reference(E, (6, 11), rank1_grads(rng, 6, 11, 8), beta1=0.0)


def test_I5_rank_one_backbone_matrix_is_adam():
    rng = np.random.default_rng(9)
    _adam_reference(B, (12, 5), rank1_grads(rng, 12, 5, 8), beta1=B1)


# ----------------------------------------------------------------------------- brute force
def _dense_reference(tier, g_list, w0, d=1.0):
    """float64 dense reference of the whole step (factored V rebuilt as a full matrix)."""
    shape = w0.shape
    n, m = (1, shape[0]) if len(shape) == 1 else shape
    exact = tier == R or len(shape) == 1
    M = np.zeros((n, m)); V = np.zeros((n, m)); Rr = np.zeros(n); Cc = np.zeros(m)
    xs, us = [], []
    w = f32(w0).astype(np.float64).reshape(n, m)
    for t, gb in enumerate(g_list, start=1):
        g = f32(gb).astype(np.float64).reshape(n, m)
        if exact:
            V = B2 * V + (1 - B2) * g * g
            Vh = V
        else:
            Rr = B2 * Rr + (1 - B2) * (g * g).mean(axis=1)
            Cc = B2 * Cc + (1 - B2) * (g * g).mean(axis=0)
            Vh = np.outer(Rr, Cc) / max(Rr.mean(), EPS)
        D = np.sqrt(np.maximum(Vh, EPS))
        if tier == B:
            M = B1 * M + (1 - B1) * g
            Uh = np.sqrt(1 - B2**t) / (1 - B1**t) * M / D
        else:
            Uh = np.sqrt(1 - B2**t) * g / D
        U = Uh / max(1.0, np.sqrt(np.mean(Uh**2)) / d)
        xs.append(w - LR * U)
        us.append(U)
    return us, xs


@pytest.mark.parametrize("shape", [(1, 1), (1, 7), (7, 1), (3, 5), (13, 17), (256, 8), (5,), (1,), (64,)])
@pytest.mark.parametrize("tier", [B, E, R])
def test_bruteforce_tiny(shape, tier):
    rng = np.random.default_rng(hash((shape, tier)) & 0xFFFF)
    w0 = bf16(rng.normal(0, 0.02, shape))
    grads = [bf16(rng.normal(0, 10.0 ** rng.uniform(-4, -1), shape)) for _ in range(3)]
    us, xs = _dense_reference(tier, grads, w0)
    T = make(tier, w0, 1)
    for t, g in enumerate(grads, start=1):
        T.g = g
        T.w = w0.copy()             # keep w fixed so the float64 reference sees the same w
        oracle.step([T], t, want_u=True, want_x=True)
        np.testing.assert_allclose(T.u_out.reshape(us[t - 1].shape), us[t - 1], rtol=3e-6, atol=1e-7)
        np.testing.assert_allclose(T.x_out.reshape(xs[t - 1].shape), xs[t - 1], rtol=2e-7, atol=1e-10)


def test_empty_tensor_is_a_no_op():
    T = oracle.Tensor(tier=E, w=np.zeros((0, 5), np.uint16), g=np.zeros((0, 5), np.uint16), tensor_id=0)
    T.r, T.c = np.zeros(0, np.float32), np.zeros(5, np.float32)
    assert oracle.step([T], 1) == 0
    assert np.all(T.c == 0)


def test_step_zero_is_rejected():
    T = make(E, bf16(np.ones((2, 2))))
    assert oracle.step([T], 0) != 0


def test_nonfinite_gradients_propagate():
    rng = np.random.default_rng(10)
    for tier, shape in [(E, (4, 6)), (R, (4, 6)), (B, (4, 6)), (B, (9,))]:
        T = make(tier, bf16(rng.normal(0, 0.02, shape)), 1)
        g = rng.normal(0, 1e-3, shape)
        g.flat[3] = np.nan
        T.g = bf16(g)
        oracle.step([T], 1)
        assert np.all(np.isnan(f32(T.w)))     # NaN reaches the clip factor and so every weight


# ----------------------------------------------------------------------------- I6
def _bf16_value(bits):
    return float(np.array([(int(bits) & 0xFFFF) << 16], np.uint32).view(np.float32)[0])


def _rounding_distribution(x, h):
    """Analytic P(bf16_rne(x + xi) = v) for xi uniform on (-h, h): the share of
    (x - h, x + h) that lies between the midpoints around each bf16 value v."""
    b = int(np.float32(x).view(np.uint32)) >> 16
    cands = [_bf16_value(k) for k in range(b - 3, b + 4)] if x >= 0 else \
        [_bf16_value(k) for k in range(b + 3, b - 4, -1)]
    cands = sorted(set(cands))
    probs = {}
    for i in range(1, len(cands) - 1):
        lo_edge = 0.5 * (cands[i - 1] + cands[i])
        hi_edge = 0.5 * (cands[i] + cands[i + 1])
        overlap = max(0.0, min(hi_edge, x + h) - max(lo_edge, x - h))
        if overlap > 0:
            probs[cands[i]] = overlap / (2 * h)
    assert abs(sum(probs.values()) - 1) < 1e-9
    return probs


def _check_distribution(out, probs, tol=0.01):
    vals, counts = np.unique(out, return_counts=True)
    emp = dict(zip(vals.tolist(), (counts / out.size).tolist()))
    assert set(emp) <= set(probs), (emp, probs)
    for v, pr in probs.items():
        assert emp.get(v, 0.0) == pytest.approx(pr, abs=tol), (v, emp, probs)


@pytest.mark.parametrize("wval", [1.0, 1.25, 1.5, 1.875, -0.75, 3.0e-3])
def test_I6_dither_moves_zero_update_weights_as_analysed(wval):
    """A weight with U = 0 sits on the bf16 grid; noise of half-width h = 2^-8 |w|
    (ulp(w) taken as 2^-7 |w|, Sec. 3) carries it across a neighbouring midpoint
    with the probability the interval geometry gives."""
    n = 1 << 16
    w = float(f32(bf16([wval]))[0])
    T = make(E, bf16(np.full((1, n), w)), 17)
    oracle.step([T], 1, want_x=True)
    assert np.all(T.x_out == w)
    _check_distribution(f32(T.w).astype(np.float64).ravel(), _rounding_distribution(w, 2.0**-8 * abs(w)))


@pytest.mark.parametrize("wval,sign", [(1.0, 1), (0.8125, -1), (-0.40625, 1), (0.0234375, -1)])
def test_I6_dither_rounding_probability_off_grid(wval, sign):
    """Constant router gradients give U = sign(g) at t = 1 (I4), so every element
    ends at the same x = w - lr*sign(g) between two bf16 values; the shares rounded
    to each neighbour must follow the uniform noise of half-width 2^-8 |w|."""
    n = 1 << 16
    w = float(f32(bf16([wval]))[0])
    T = make(R, bf16(np.full((1, n), w)), 23)
    T.g = bf16(np.full((1, n), 0.5 * sign))
    oracle.step([T], 1, want_x=True)
    x = float(T.x_out[0, 0])
    assert np.all(T.x_out == x) and x == pytest.approx(w - LR * sign, rel=1e-6)
    _check_distribution(f32(T.w).astype(np.float64).ravel(), _rounding_distribution(x, 2.0**-8 * abs(w)))
