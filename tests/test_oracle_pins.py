"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Each test fixes one part of the method by a closed form, an invariant, brute force on a tiny input
or an independent library routine, so that a dropped term, a wrong sign or index, a transposed
operand or a wrong learning-rate factor in the oracle fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from synth import NS_COEFFS, f32_to_bf16_bits, bf16_bits_to_f32

A, B, C = NS_COEFFS
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _p(s):
    # the quintic written in Horner form, independently of the oracle's scalar helper
    s2 = s * s
    return s * (A + s2 * (B + s2 * C))


def _pk(s, k):
    for _ in range(k):
        s = _p(s)
    return s


def _rand(rng, m, n):
    return rng.standard_normal((m, n))


def _orth(rng, n):
    q, r = np.linalg.qr(rng.standard_normal((n, n)))
    return q * np.sign(np.diag(r))


# ---------------------------------------------------------------- momentum (a1)

@pytest.mark.parametrize("beta", [0.5, 0.95])
def test_momentum_zero_buffer_closed_form(beta):
    rng = np.random.default_rng(0)
    g = _rand(rng, 7, 11)
    buf, u = oracle.momentum_update(g, np.zeros_like(g), beta, nesterov=True)
    np.testing.assert_allclose(buf, (1 - beta) * g, rtol=0, atol=1e-15)
    np.testing.assert_allclose(u, (1 - beta * beta) * g, rtol=0, atol=1e-15)
    buf2, u2 = oracle.momentum_update(g, np.zeros_like(g), beta, nesterov=False)
    np.testing.assert_allclose(u2, (1 - beta) * g, rtol=0, atol=1e-15)


@pytest.mark.parametrize("beta", [0.5, 0.95])
def test_momentum_zero_grad_closed_form(beta):
    rng = np.random.default_rng(1)
    m0 = _rand(rng, 5, 9)
    buf, u = oracle.momentum_update(np.zeros_like(m0), m0, beta, nesterov=True)
    np.testing.assert_allclose(buf, beta * m0, rtol=0, atol=1e-15)
    np.testing.assert_allclose(u, beta * beta * m0, rtol=0, atol=1e-15)


def test_momentum_two_steps_unrolled():
    # EMA unrolled by hand over two steps: buf2 = beta^2 m0 + beta (1-beta) g1 + (1-beta) g2
    rng = np.random.default_rng(2)
    beta = 0.9
    m0, g1, g2 = (_rand(rng, 4, 6) for _ in range(3))
    b1, _ = oracle.momentum_update(g1, m0, beta)
    b2, u2 = oracle.momentum_update(g2, b1, beta)
    exp = beta ** 2 * m0 + beta * (1 - beta) * g1 + (1 - beta) * g2
    np.testing.assert_allclose(b2, exp, rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(u2, (1 - beta) * g2 + beta * exp, rtol=1e-14, atol=1e-14)


# ---------------------------------------------------------------- normalisation (a2)

def test_normalize_unit_frobenius_and_zero():
    rng = np.random.default_rng(3)
    x = _rand(rng, 13, 17) * 123.0
    x0 = oracle.frobenius_normalize(x, 1e-7)
    assert abs(math.sqrt((x0 ** 2).sum()) - 1.0) < 1e-14
    z = oracle.frobenius_normalize(np.zeros((3, 4)), 1e-7)
    assert not z.any()
    tiny = np.full((2, 2), 1e-9)  # norm 2e-9 < eps: divided by eps (clamp)
    np.testing.assert_allclose(oracle.frobenius_normalize(tiny, 1e-7), tiny / 1e-7, rtol=1e-15)


def test_zero_input_gives_zero_update():
    o = oracle.newton_schulz(np.zeros((6, 10)), A, B, C, 5)
    assert o.shape == (6, 10) and not o.any()


# ---------------------------------------------------------------- Newton-Schulz (a3, a4)

@pytest.mark.parametrize("shape", [(6, 6), (5, 9), (9, 5), (1, 4)])
@pytest.mark.parametrize("steps", [1, 2, 5])
def test_ns_diagonal_reduces_to_scalar_polynomial(shape, steps):
    m, n = shape
    rng = np.random.default_rng(4)
    k = min(m, n)
    d = rng.uniform(0.2, 3.0, size=k) * rng.choice([-1.0, 1.0], size=k)
    x = np.zeros((m, n))
    x[np.arange(k), np.arange(k)] = d
    o = oracle.newton_schulz(x, A, B, C, steps)
    nrm = math.sqrt(float((d ** 2).sum()))
    exp = np.zeros((m, n))
    exp[np.arange(k), np.arange(k)] = [_pk(v / nrm, steps) for v in d]
    np.testing.assert_allclose(o, exp, rtol=0, atol=1e-14)


def test_ns_orthogonal_equivariance():
    rng = np.random.default_rng(5)
    for (m, n) in [(24, 40), (40, 24), (16, 16)]:
        x = _rand(rng, m, n)
        U, V = _orth(rng, m), _orth(rng, n)
        lhs = oracle.newton_schulz(U @ x @ V.T, A, B, C, 5)
        rhs = U @ oracle.newton_schulz(x, A, B, C, 5) @ V.T
        np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-12)


@pytest.mark.parametrize("shape", [(1, 7), (5, 3), (8, 8), (64, 96), (96, 64)])
@pytest.mark.parametrize("steps", [0, 1, 5])
def test_ns_matches_svd_brute_force(shape, steps):
    rng = np.random.default_rng(6)
    x = _rand(rng, *shape)
    Uu, s, Vt = np.linalg.svd(x, full_matrices=False)
    s0 = s / math.sqrt(float((s ** 2).sum()))
    exp = (Uu * np.array([_pk(v, steps) for v in s0])) @ Vt
    o = oracle.newton_schulz(x, A, B, C, steps)
    np.testing.assert_allclose(o, exp, rtol=0, atol=1e-13)


def test_ns_transpose_consistency():
    rng = np.random.default_rng(7)
    for (m, n) in [(12, 30), (30, 12), (17, 17)]:
        x = _rand(rng, m, n)
        np.testing.assert_allclose(oracle.newton_schulz(x.T, A, B, C, 5),
                                   oracle.newton_schulz(x, A, B, C, 5).T, rtol=0, atol=1e-13)


def _band():
    # critical points of p: p'(s) = A + 3 B s^2 + 5 C s^4 = 0 (a quadratic in s^2)
    disc = math.sqrt(9 * B * B - 20 * A * C)
    lo_sq, hi_sq = (-3 * B - disc) / (10 * C), (-3 * B + disc) / (10 * C)
    s_max, s_min = math.sqrt(lo_sq), math.sqrt(hi_sq)     # local max, local min of p
    return _p(s_min), _p(s_max)


def test_ns_singular_values_stay_in_band():
    lo, hi = _band()
    assert abs(hi - 1.2023686) < 1e-6 and abs(lo - 0.6818315) < 1e-6
    rng = np.random.default_rng(8)
    for steps in (1, 2, 5):
        o = oracle.newton_schulz(_rand(rng, 64, 96), A, B, C, steps)
        sv = np.linalg.svd(o, compute_uv=False)
        assert sv.max() <= hi + 1e-12
        if steps == 5:  # every input sigma is well above 0.0015 here
            assert sv.min() >= lo - 1e-12


def test_ns_rank_one_closed_form():
    rng = np.random.default_rng(9)
    x, y = rng.standard_normal(10), rng.standard_normal(25)
    # p^5(1) evaluated in exact rational arithmetic from the decimal coefficients
    a, b, c = (Fraction(str(v)) for v in NS_COEFFS)
    s = Fraction(1)
    for _ in range(5):
        s = a * s + b * s ** 3 + c * s ** 5
    o = oracle.newton_schulz(np.outer(x, y), A, B, C, 5)
    exp = float(s) * np.outer(x / np.linalg.norm(x), y / np.linalg.norm(y))
    np.testing.assert_allclose(o, exp, rtol=0, atol=1e-13)
    assert abs(float(s) - 0.69643640946975) < 1e-13


def test_ns_one_step_expanded():
    rng = np.random.default_rng(10)
    x = _rand(rng, 9, 14)
    x0 = x / np.linalg.norm(x)
    G = x0 @ x0.T
    exp = A * x0 + B * (G @ x0) + C * (G @ (G @ x0))
    np.testing.assert_allclose(oracle.newton_schulz(x, A, B, C, 1), exp, rtol=0, atol=1e-14)
    np.testing.assert_allclose(oracle.newton_schulz(x, A, B, C, 0), x0, rtol=0, atol=1e-15)


def test_ns_step_bounds():
    with pytest.raises(ValueError):
        oracle.newton_schulz(np.ones((2, 2)), A, B, C, 100)


# ---------------------------------------------------------------- apply (a5)

def test_lr_factor_closed_forms():
    assert oracle.lr_factor(256, 512, "original") == 1.0
    assert oracle.lr_factor(512, 256, "original") == math.sqrt(2.0)
    assert oracle.lr_factor(384, 128, "match_rms_adamw") == 0.2 * math.sqrt(384)
    assert oracle.lr_factor(128, 384, "match_rms_adamw") == 0.2 * math.sqrt(384)
    assert oracle.lr_factor(9, 3, "none") == 1.0


def test_apply_special_cases():
    rng = np.random.default_rng(11)
    p, O = _rand(rng, 4, 5), _rand(rng, 4, 5)
    np.testing.assert_array_equal(oracle.apply_update(p, O, 0.0, 0.3, 1.7), p)
    np.testing.assert_allclose(oracle.apply_update(p, O, 0.02, 0.0, 1.5) - p, -0.03 * O,
                               rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.apply_update(p, np.zeros_like(O), 0.1, 0.5, 2.0), 0.95 * p,
                               rtol=1e-15)


def test_bf16_widening_exact():
    x = np.array([1.0, -2.5, 3.140625, 1e-3, 65504.0], dtype=np.float32)
    bits = f32_to_bf16_bits(x)
    np.testing.assert_array_equal(oracle.bf16_widen(bits), bf16_bits_to_f32(bits).astype(np.float64))
    assert oracle.bf16_widen(np.array([0x3F80], dtype=np.uint16))[0] == 1.0
    assert oracle.bf16_widen(np.array([0xC020], dtype=np.uint16))[0] == -2.5


# ---------------------------------------------------------------- AdamW (a6)

def test_adamw_first_step_closed_form():
    rng = np.random.default_rng(12)
    p, g = rng.standard_normal(1000), rng.standard_normal(1000)
    z = np.zeros_like(p)
    lr, wd, eps = 1e-3, 1e-2, 1e-8
    p1, m1, v1 = oracle.adamw_step(p, g, z, z, lr=lr, beta1=0.9, beta2=0.999, eps=eps,
                                   weight_decay=wd, step=1)
    np.testing.assert_allclose(p1, p * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-13)
    np.testing.assert_allclose(m1, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v1, 0.001 * g * g, rtol=1e-13)


def test_adamw_matches_torch_optim_adamw():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(13)
    p0 = rng.standard_normal(257)
    grads = [rng.standard_normal(257) for _ in range(4)]
    kw = dict(lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=1e-2)
    tp = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([tp], foreach=False, **kw)
    p, m, v = p0, np.zeros(257), np.zeros(257)
    for t, g in enumerate(grads, start=1):
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        p, m, v = oracle.adamw_step(p, g, m, v, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                                    weight_decay=1e-2, step=t)
    st = opt.state[tp]
    np.testing.assert_allclose(p, tp.detach().numpy(), rtol=0, atol=1e-15)
    np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-14, atol=1e-18)
    np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-14, atol=1e-18)


# ---------------------------------------------------------------- whole Muon step vs torch.optim.Muon

def _torch_muon(p0, grads, **kw):
    torch = pytest.importorskip("torch")
    if not hasattr(torch.optim, "Muon"):
        pytest.skip("torch.optim.Muon not available")
    tp = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Muon([tp], **kw)
    for g in grads:
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    return tp.detach().numpy(), opt.state[tp]["momentum_buffer"].numpy()


@pytest.mark.parametrize("shape,mode", [((64, 128), "original"), ((128, 64), "original"),
                                        ((96, 32), "match_rms_adamw")])
def test_muon_step_matches_torch_optim_muon(shape, mode):
    # torch.optim.Muon always runs NS in bf16: the update is compared at bf16 level, the
    # momentum buffer (pure fp64 arithmetic in both) tightly.
    rng = np.random.default_rng(14)
    p0 = rng.standard_normal(shape) * 0.02
    g1, g2 = rng.standard_normal(shape), rng.standard_normal(shape)
    hp = dict(lr=0.02, weight_decay=0.0, momentum=0.95, nesterov=True, ns_steps=5)
    tp, tbuf = _torch_muon(p0, [g1, g2], ns_coefficients=NS_COEFFS, adjust_lr_fn=mode, **hp)
    p, buf = p0, np.zeros(shape)
    for g in (g1, g2):
        p, buf, _ = oracle.muon_step(p, g, buf, lr=0.02, weight_decay=0.0, momentum=0.95,
                                     nesterov=True, a=A, b=B, c=C, ns_steps=5, lr_adjust=mode)
    np.testing.assert_allclose(buf, tbuf, rtol=1e-13, atol=1e-15)
    d_or, d_t = p - p0, tp - p0
    assert np.linalg.norm(d_or - d_t) / np.linalg.norm(d_or) < 3e-2


def test_muon_weight_decay_uses_unadjusted_lr():
    # large decay makes the decay term dominate the step: a decay scaled by the shape factor,
    # or a missing decay, is far outside the bf16-level tolerance
    rng = np.random.default_rng(15)
    shape = (128, 32)  # original factor = 2
    p0 = rng.standard_normal(shape)
    g = rng.standard_normal(shape)
    tp, _ = _torch_muon(p0, [g], lr=0.02, weight_decay=0.5, momentum=0.95, nesterov=True,
                        ns_steps=5, ns_coefficients=NS_COEFFS, adjust_lr_fn="original")
    p, _, _ = oracle.muon_step(p0, g, np.zeros(shape), lr=0.02, weight_decay=0.5, momentum=0.95,
                               nesterov=True, a=A, b=B, c=C, ns_steps=5, lr_adjust="original")
    d_or, d_t = p - p0, tp - p0
    assert np.linalg.norm(d_or - d_t) / np.linalg.norm(d_or) < 1e-2


def test_paper_setup_matches_torch_optim_muon():
    # the paper's own latency setting (Section 5.1): 2 NS steps, momentum 0.5, match_rms_adamw
    cfg = json.load(open(os.path.join(GOLDEN, "paper_setup_hparams.json")))["muon"]
    rng = np.random.default_rng(16)
    shape = (48, 80)
    p0 = rng.standard_normal(shape) * 0.02
    g = rng.standard_normal(shape)
    tp, tbuf = _torch_muon(p0, [g], lr=cfg["lr"], weight_decay=cfg["weight_decay"],
                           momentum=cfg["momentum"], nesterov=True, ns_steps=cfg["ns_steps"],
                           ns_coefficients=NS_COEFFS, adjust_lr_fn=cfg["lr_adjust"])
    p, buf, _ = oracle.muon_step(p0, g, np.zeros(shape), lr=cfg["lr"],
                                 weight_decay=cfg["weight_decay"], momentum=cfg["momentum"],
                                 nesterov=True, a=A, b=B, c=C, ns_steps=cfg["ns_steps"],
                                 lr_adjust=cfg["lr_adjust"])
    np.testing.assert_allclose(buf, tbuf, rtol=1e-13)
    d_or, d_t = p - p0, tp - p0
    assert np.linalg.norm(d_or - d_t) / np.linalg.norm(d_or) < 3e-2


# ---------------------------------------------------------------- per-step coefficient schedules

def _p_coef(s, a, b, c):
    s2 = s * s
    return s * (a + s2 * (b + s2 * c))


def _random_schedule(rng, k):
    # perturbations of the fixed triple: every step different
    base = np.array([A, B, C])
    return [tuple(base * (1.0 + 0.05 * rng.standard_normal(3))) for _ in range(k)]


def test_schedule_constant_equals_fixed_triple():
    rng = np.random.default_rng(40)
    x = _rand(rng, 24, 56)
    o1 = oracle.newton_schulz(x, A, B, C, 5)
    o2 = oracle.newton_schulz(x, 0.0, 0.0, 0.0, 5, schedule=[(A, B, C)] * 5)
    assert np.array_equal(o1, o2)


@pytest.mark.parametrize("shape", [(6, 6), (4, 9), (9, 4)])
def test_schedule_diagonal_composes_step_polynomials(shape):
    # NS of a diagonal matrix acts entrywise; step k applies its own polynomial p_k
    m, n = shape
    rng = np.random.default_rng(41)
    sched = _random_schedule(rng, 4)
    k = min(m, n)
    d = rng.uniform(0.2, 2.0, size=k) * rng.choice([-1.0, 1.0], size=k)
    x = np.zeros((m, n))
    x[np.arange(k), np.arange(k)] = d
    nrm = math.sqrt(float((d ** 2).sum()))
    vals = []
    for v in d:
        s = v / nrm
        for (a, b, c) in sched:
            s = _p_coef(s, a, b, c)
        vals.append(s)
    exp = np.zeros((m, n))
    exp[np.arange(k), np.arange(k)] = vals
    np.testing.assert_allclose(oracle.newton_schulz(x, A, B, C, 4, schedule=sched), exp, rtol=0, atol=1e-12)


def test_schedule_one_step_expanded():
    # K = 1 with triple (a0, b0, c0): a0 X + b0 X X^T X + c0 (X X^T)^2 X, X = x / ||x||_F
    rng = np.random.default_rng(42)
    x = _rand(rng, 12, 20)
    a0, b0, c0 = 2.0, -1.25, 0.375
    X = x / np.linalg.norm(x)
    G = X @ X.T
    exp = a0 * X + b0 * G @ X + c0 * G @ G @ X
    np.testing.assert_allclose(oracle.newton_schulz(x, A, B, C, 1, schedule=[(a0, b0, c0)]), exp,
                               rtol=0, atol=1e-14)


def test_schedule_cubic_newton_schulz_converges_to_polar_factor():
    # the textbook cubic Newton-Schulz iteration X <- 1.5 X - 0.5 X X^T X (a schedule with c = 0)
    # converges to the orthogonal polar factor U V^T for singular values in (0, sqrt(3))
    # (full rank: zero singular values would only be amplified by rounding)
    rng = np.random.default_rng(43)
    U = _orth(rng, 8)
    V = _orth(rng, 10)[:, :8]
    s = np.linspace(0.3, 1.0, 8)
    x = (U * s) @ V.T
    o = oracle.newton_schulz(x, A, B, C, 20, schedule=[(1.5, -0.5, 0.0)] * 20)
    np.testing.assert_allclose(o, U @ V.T, rtol=0, atol=1e-13)


@pytest.mark.parametrize("shape", [(5, 3), (8, 8), (16, 24)])
def test_schedule_matches_svd_brute_force(shape):
    rng = np.random.default_rng(44)
    sched = _random_schedule(rng, 3)
    x = _rand(rng, *shape)
    Uu, s, Vt = np.linalg.svd(x, full_matrices=False)
    s0 = s / math.sqrt(float((s ** 2).sum()))
    mapped = []
    for v in s0:
        for (a, b, c) in sched:
            v = _p_coef(v, a, b, c)
        mapped.append(v)
    exp = (Uu * np.array(mapped)) @ Vt
    np.testing.assert_allclose(oracle.newton_schulz(x, A, B, C, 3, schedule=sched), exp, rtol=0, atol=1e-12)


def test_schedule_length_must_match_steps():
    with pytest.raises(ValueError):
        oracle.newton_schulz(np.ones((3, 4)), A, B, C, 2, schedule=[(A, B, C)])


# ---------------------------------------------------------------- owner-side gradient reduction

def test_reduce_single_part_is_identity():
    rng = np.random.default_rng(50)
    g = f32_to_bf16_bits(rng.standard_normal((7, 9)).astype(np.float32))
    assert np.array_equal(oracle.reduce_gradients([g]), bf16_bits_to_f32(g).astype(np.float64))


def test_reduce_identical_parts_and_mean():
    rng = np.random.default_rng(51)
    g = rng.standard_normal((5, 6)).astype(np.float32)
    W = 8
    s = oracle.reduce_gradients([g] * W)
    np.testing.assert_array_equal(s, W * g.astype(np.float64))  # exact: W is a power of two
    np.testing.assert_array_equal(oracle.reduce_gradients([g] * W, 1.0 / W), g.astype(np.float64))


def test_reduce_is_the_plain_sum_on_integers():
    # integer-valued parts: every partial sum is exact, so the result must equal the integer sum in
    # any order
    rng = np.random.default_rng(52)
    parts = [rng.integers(-100, 100, size=(4, 5)).astype(np.float32) for _ in range(6)]
    want = sum(p.astype(np.int64) for p in parts).astype(np.float64) * 0.5
    np.testing.assert_array_equal(oracle.reduce_gradients(parts, 0.5), want)
    np.testing.assert_array_equal(oracle.reduce_gradients(parts[::-1], 0.5), want)


def test_reduce_then_muon_equals_muon_of_the_sum():
    rng = np.random.default_rng(53)
    parts = [rng.standard_normal((12, 20)) * 1e-3 for _ in range(3)]
    p0 = rng.standard_normal((12, 20)) * 0.02
    m0 = np.zeros((12, 20))
    g = parts[0] + parts[1] + parts[2]
    kw = dict(lr=0.02, weight_decay=0.01, momentum=0.95, nesterov=True, a=A, b=B, c=C, ns_steps=5)
    r1 = oracle.muon_step(p0, oracle.reduce_gradients(parts), m0, **kw)
    r2 = oracle.muon_step(p0, g, m0, **kw)
    for x, y in zip(r1, r2):
        np.testing.assert_allclose(x, y, rtol=0, atol=1e-15)
