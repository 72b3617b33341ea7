"""Pins of the fp64 Shampoo oracle (Section 5.7; Gupta et al. 2018, matrix case) against closed forms,
library routines, SVD brute force and invariants that a dropped term, a wrong exponent, a swapped
side or a transposed operand would break."""
import numpy as np
import pytest

from oracle import shampoo as S


def _orth(rng, d):
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    return q * np.sign(np.diag(r))


def _spd(rng, d, rank=None, scale=1.0):
    A = rng.standard_normal((d, rank or d)) * scale
    return A @ A.T


@pytest.mark.parametrize("p", [1, 2, 4])
def test_root_of_diagonal_is_elementwise(p):
    d = np.array([4.0, 0.5, 9.0, 1e-3, 0.0])
    eps, rel = 1e-4, 1e-3
    rho = eps + rel * np.linalg.norm(d)
    X = S.inverse_root(np.diag(d), p, eps, rel)
    np.testing.assert_allclose(X, np.diag((d + rho) ** (-1.0 / p)), rtol=1e-13, atol=0)


def test_root_p1_is_the_inverse():
    rng = np.random.default_rng(1)
    A = _spd(rng, 12)
    np.testing.assert_allclose(S.inverse_root(A, 1, 0.3, 0.0), np.linalg.inv(A + 0.3 * np.eye(12)),
                               rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("p", [2, 4])
def test_root_power_times_matrix_is_identity(p):
    rng = np.random.default_rng(2)
    A = _spd(rng, 10, rank=6)       # rank deficient: the ridge makes it definite
    X = S.inverse_root(A, p, 1e-2, 1e-3)
    rho = 1e-2 + 1e-3 * np.linalg.norm(A)
    np.testing.assert_allclose(np.linalg.matrix_power(X, p) @ (A + rho * np.eye(10)), np.eye(10),
                               atol=1e-9)
    np.testing.assert_allclose(X, X.T, atol=1e-12)
    assert np.linalg.eigvalsh(X).min() > 0


def test_root_orthogonal_equivariance_and_scaling():
    rng = np.random.default_rng(3)
    A = _spd(rng, 9)
    Q = _orth(rng, 9)
    X = S.inverse_root(A, 4, 0.05, 0.0)
    np.testing.assert_allclose(S.inverse_root(Q @ A @ Q.T, 4, 0.05, 0.0), Q @ X @ Q.T, atol=1e-11)
    # a purely relative ridge scales: (cA + rel |cA| I)^{-1/4} = c^{-1/4} (A + rel |A| I)^{-1/4}
    c = 37.0
    np.testing.assert_allclose(S.inverse_root(c * A, 4, 0.0, 1e-3),
                               c ** -0.25 * S.inverse_root(A, 4, 0.0, 1e-3), rtol=1e-11)


@pytest.mark.parametrize("m,n", [(5, 8), (8, 5), (6, 6), (1, 7)])
def test_first_step_from_zero_state_is_svd_closed_form(m, n):
    # L = U S^2 U^T, R = V S^2 V^T  =>  L^-1/4 G R^-1/4 = U diag(s (s^2+rho_L)^-1/4 (s^2+rho_R)^-1/4) V^T
    rng = np.random.default_rng(10 * m + n)
    G = rng.standard_normal((m, n))
    hp = S.ShampooHParams(lr=0.1, eps=1e-3, eps_rel=1e-4)
    p, L, R, PL, PR, U = S.shampoo_step(np.zeros((m, n)), G, np.zeros((m, m)), np.zeros((n, n)),
                                        None, None, hp)
    u, s, vt = np.linalg.svd(G, full_matrices=False)
    rho_l = 1e-3 + 1e-4 * np.sqrt(np.sum(s ** 4))
    rho_r = rho_l     # ||G G^T||_F = ||G^T G||_F = sqrt(sum s^4)
    f = s * (s ** 2 + rho_l) ** -0.25 * (s ** 2 + rho_r) ** -0.25
    np.testing.assert_allclose(U, (u * f) @ vt, atol=1e-11)
    np.testing.assert_allclose(p, -0.1 * U, atol=1e-12)
    np.testing.assert_allclose(L, G @ G.T, atol=1e-12)
    np.testing.assert_allclose(R, G.T @ G, atol=1e-12)


def test_rank_one_accumulation_over_two_steps():
    # G_k = s_k x y^T: L = (s1^2 + s2^2) x x^T, so U_2 = s2 (s1^2 + s2^2 + rho)^-1/2 x y^T (eps only)
    rng = np.random.default_rng(5)
    x = rng.standard_normal(7); x /= np.linalg.norm(x)
    y = rng.standard_normal(4); y /= np.linalg.norm(y)
    hp = S.ShampooHParams(lr=1.0, eps=1e-2, eps_rel=0.0)
    L, R = np.zeros((7, 7)), np.zeros((4, 4))
    p = np.zeros((7, 4))
    p, L, R, _, _, U1 = S.shampoo_step(p, 3.0 * np.outer(x, y), L, R, None, None, hp)
    np.testing.assert_allclose(U1, 3.0 / np.sqrt(9.0 + 1e-2) * np.outer(x, y), atol=1e-13)
    p, L, R, _, _, U2 = S.shampoo_step(p, -2.0 * np.outer(x, y), L, R, None, None, hp)
    np.testing.assert_allclose(U2, -2.0 / np.sqrt(13.0 + 1e-2) * np.outer(x, y), atol=1e-13)
    np.testing.assert_allclose(p, -(U1 + U2), atol=1e-13)


def test_ema_statistics_and_side_assignment():
    # a wide gradient: L is m x m from G G^T, R is n x n from G^T G; EMA weights as given
    rng = np.random.default_rng(6)
    G1, G2 = rng.standard_normal((3, 5)), rng.standard_normal((3, 5))
    L, R = S.update_statistics(np.zeros((3, 3)), np.zeros((5, 5)), G1, 0.9, 0.1)
    L, R = S.update_statistics(L, R, G2, 0.9, 0.1)
    assert L.shape == (3, 3) and R.shape == (5, 5)
    # trace(L) = trace(R) = weighted sum of squared Frobenius norms
    t = 0.9 * 0.1 * np.sum(G1 ** 2) + 0.1 * np.sum(G2 ** 2)
    assert abs(np.trace(L) - t) < 1e-12 and abs(np.trace(R) - t) < 1e-12
    # the first statistic decays once: L - weight G2 G2^T = beta weight G1 G1^T
    np.testing.assert_allclose(L - 0.1 * G2 @ G2.T, 0.09 * G1 @ G1.T, atol=1e-13)


def test_stale_preconditioners_and_identity_reduce_to_sgd():
    rng = np.random.default_rng(7)
    G = rng.standard_normal((4, 6)); P0 = rng.standard_normal((4, 6))
    hp = S.ShampooHParams(lr=0.05, weight_decay=0.1, refresh=False)
    p, L, R, PL, PR, U = S.shampoo_step(P0, G, np.zeros((4, 4)), np.zeros((6, 6)), np.eye(4), np.eye(6), hp)
    np.testing.assert_allclose(U, G, atol=0)
    np.testing.assert_allclose(p, P0 * (1 - 0.05 * 0.1) - 0.05 * G, atol=1e-15)
    # the statistics still accumulate when the preconditioners are stale
    np.testing.assert_allclose(L, G @ G.T, atol=1e-13)


def test_whole_step_orthogonal_equivariance():
    # with a purely relative ridge and zero state: step(Q1 G Q2^T) = Q1 step(G) Q2^T
    rng = np.random.default_rng(8)
    G = rng.standard_normal((6, 9))
    Q1, Q2 = _orth(rng, 6), _orth(rng, 9)
    hp = S.ShampooHParams(lr=1.0, eps=0.0, eps_rel=1e-3)
    z = lambda d: np.zeros((d, d))
    U = S.shampoo_step(np.zeros((6, 9)), G, z(6), z(9), None, None, hp)[5]
    Uq = S.shampoo_step(np.zeros((6, 9)), Q1 @ G @ Q2.T, z(6), z(9), None, None, hp)[5]
    np.testing.assert_allclose(Uq, Q1 @ U @ Q2.T, atol=1e-10)


def test_bf16_gradient_is_widened_exactly():
    import synth
    rng = np.random.default_rng(9)
    g = rng.standard_normal((3, 4)).astype(np.float32)
    bits = synth.f32_to_bf16_bits(g)
    hp = S.ShampooHParams(lr=1.0, eps=1e-2, eps_rel=0.0)
    a = S.shampoo_step(np.zeros((3, 4)), bits, np.zeros((3, 3)), np.zeros((4, 4)), None, None, hp)[5]
    b = S.shampoo_step(np.zeros((3, 4)), synth.bf16_bits_to_f32(bits).astype(np.float64),
                       np.zeros((3, 3)), np.zeros((4, 4)), None, None, hp)[5]
    np.testing.assert_array_equal(a, b)
