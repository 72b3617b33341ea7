"""Pins of the fp64 SOAP oracle (Section 5.7; Vyas et al. 2024, matrix case) against PyTorch AdamW,
closed forms, hand-worked Householder factors, eigenvectors from a symmetric eigensolver and
invariants that a dropped term, a wrong bias correction, a swapped side or a transposed basis
would break."""
import numpy as np
import pytest
import torch

from oracle import soap as S
import synth


def _orth(rng, d):
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    return q * np.sign(np.diag(r))


def _state(rng, m, n, basis=True):
    st = dict(param=rng.standard_normal((m, n)) * 0.02, grad=rng.standard_normal((m, n)) * 1e-3,
              exp_avg=rng.standard_normal((m, n)) * 1e-4, exp_avg_sq=rng.random((m, n)) * 1e-7)
    A = rng.standard_normal((m, m + 3))
    B = rng.standard_normal((n, n + 3))
    st["L"], st["R"] = A @ A.T * 1e-6, B @ B.T * 1e-6
    st["QL"] = _orth(rng, m) if basis else np.eye(m)
    st["QR"] = _orth(rng, n) if basis else np.eye(n)
    return st


def _run(st, step, hp):
    return S.soap_step(st["param"], st["grad"], st["exp_avg"], st["exp_avg_sq"], st["L"], st["R"],
                       st["QL"], st["QR"], step, hp)


def test_identity_basis_is_torch_adamw():
    """With Q_L = Q_R = I (and no refresh) three SOAP steps are three torch.optim.AdamW steps."""
    rng = np.random.default_rng(0)
    m, n = 7, 5
    hp = S.SoapHParams(lr=0.01, weight_decay=0.1, beta1=0.9, beta2=0.99, eps=1e-6)
    p = rng.standard_normal((m, n))
    M, V = np.zeros((m, n)), np.zeros((m, n))
    L, R = np.zeros((m, m)), np.zeros((n, n))
    tp = torch.tensor(p, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([tp], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=hp.weight_decay)
    for t in range(1, 4):
        g = rng.standard_normal((m, n))
        p, M, V, L, R, QL, QR, _ = S.soap_step(p, g, M, V, L, R, np.eye(m), np.eye(n), t, hp)
        np.testing.assert_array_equal(QL, np.eye(m))
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        st = opt.state[tp]
        np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-15)
        np.testing.assert_allclose(M, st["exp_avg"].numpy(), rtol=1e-13, atol=0)
        np.testing.assert_allclose(V, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=0)


@pytest.mark.parametrize("step", [1, 4])
def test_aligned_gradient_closed_form(step):
    """G = Q_L D Q_R^T with zero moments at t = 1: G' = D, the bias corrections cancel the (1 - beta)
    factors, N' = D / (|D| + eps) on the diagonal and 0 elsewhere, N = Q_L N' Q_R^T (a
    polar-factor-like update). At t = 4 from zero moments the bias corrections no longer cancel."""
    rng = np.random.default_rng(1)
    m, n = 6, 9
    QL, QR = _orth(rng, m), _orth(rng, n)
    d = np.array([3.0, -1.0, 0.5, -2e-3, 7.0, 1e-6])
    D = np.zeros((m, n))
    D[np.arange(m), np.arange(m)] = d
    G = QL @ D @ QR.T
    hp = S.SoapHParams(lr=0.5, weight_decay=0.0, beta1=0.8, beta2=0.9, eps=1e-3)
    out = S.soap_step(np.zeros((m, n)), G, np.zeros((m, n)), np.zeros((m, n)), np.zeros((m, m)),
                      np.zeros((n, n)), QL, QR, step, hp)
    b1, b2 = hp.beta1, hp.beta2
    mp = (1 - b1) * d / (1 - b1 ** step)
    vp = np.sqrt((1 - b2) * d * d) / np.sqrt(1 - b2 ** step)
    Np = np.zeros((m, n))
    Np[np.arange(m), np.arange(m)] = mp / (vp + hp.eps)
    np.testing.assert_allclose(out[7], QL @ Np @ QR.T, atol=1e-13)
    np.testing.assert_allclose(out[0], -hp.lr * (QL @ Np @ QR.T), atol=1e-13)
    # V lives in the eigenbasis coordinates: only the diagonal is non-zero
    Vd = np.zeros((m, n))
    Vd[np.arange(m), np.arange(m)] = (1 - b2) * d * d
    np.testing.assert_allclose(out[2], Vd, atol=1e-15)


def test_basis_column_signs_do_not_matter():
    rng = np.random.default_rng(2)
    st = _state(rng, 5, 8)
    hp = S.SoapHParams(lr=0.02, weight_decay=0.01)
    ref = _run(st, 3, hp)
    st2 = dict(st)
    st2["QL"] = st["QL"] * np.array([1, -1, -1, 1, -1])
    st2["QR"] = st["QR"] * np.where(np.arange(8) % 3 == 0, -1.0, 1.0)
    got = _run(st2, 3, hp)
    for a, b in zip(ref[:5], got[:5]):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(ref[7], got[7], rtol=1e-12, atol=1e-18)


def test_orthogonal_equivariance_of_the_whole_step():
    """Rotating G, M, p by U (.) W^T, the statistics by U (.) U^T / W (.) W^T and the bases by U / W
    rotates N, p', M' the same way, leaves V unchanged and rotates the refreshed bases (up to
    column signs)."""
    rng = np.random.default_rng(3)
    m, n = 6, 4
    st = _state(rng, m, n)
    U, W = _orth(rng, m), _orth(rng, n)
    hp = S.SoapHParams(lr=0.05, weight_decay=0.1, refresh=True, refresh_iters=2)
    ref = _run(st, 2, hp)
    rot = dict(param=U @ st["param"] @ W.T, grad=U @ st["grad"] @ W.T, exp_avg=U @ st["exp_avg"] @ W.T,
               exp_avg_sq=st["exp_avg_sq"], L=U @ st["L"] @ U.T, R=W @ st["R"] @ W.T,
               QL=U @ st["QL"], QR=W @ st["QR"])
    got = _run(rot, 2, hp)
    np.testing.assert_allclose(got[0], U @ ref[0] @ W.T, atol=1e-13)
    np.testing.assert_allclose(got[1], U @ ref[1] @ W.T, atol=1e-15)
    np.testing.assert_allclose(got[2], ref[2], rtol=1e-10, atol=1e-20)
    np.testing.assert_allclose(got[3], U @ ref[3] @ U.T, atol=1e-15)
    np.testing.assert_allclose(got[7], U @ ref[7] @ W.T, atol=1e-11)
    for q_got, q_ref, X in ((got[5], ref[5], U), (got[6], ref[6], W)):
        a = X @ q_ref
        s = np.sign(np.sum(a * q_got, axis=0))
        np.testing.assert_allclose(q_got, a * s, atol=1e-10)


def test_householder_factor_by_hand():
    """2 x 2 Householder QR worked by hand with LAPACK's convention (R_11 = -sign(a_11) |a_1|):
    v = (1, c / (a - beta)), tau = (beta - a) / beta, beta = -5 for the column (3, 4); the last
    column's reflector is the identity, so Q = I - tau v v^T."""
    Q = S.orthonormal_factor(np.array([[3.0, 1.0], [4.0, 2.0]]))
    np.testing.assert_allclose(Q, np.array([[-0.6, -0.8], [-0.8, 0.6]]), atol=1e-15)
    assert S.orthonormal_factor(np.array([[2.5]]))[0, 0] == 1.0  # a 1 x 1 factor is the identity


@pytest.mark.parametrize("d", [1, 5, 24])
def test_refresh_is_a_qr_of_the_power_step(d):
    """The refreshed basis is orthogonal and Q'^T (S Q) is upper triangular (the QR definition)."""
    rng = np.random.default_rng(4)
    A = rng.standard_normal((d, d + 2))
    Sm = A @ A.T
    Q0 = _orth(rng, d)
    Q1 = S.refresh_basis(Sm, Q0)
    np.testing.assert_allclose(Q1.T @ Q1, np.eye(d), atol=1e-13)
    Rm = Q1.T @ (Sm @ Q0)
    np.testing.assert_allclose(np.tril(Rm, -1), 0.0, atol=1e-12 * np.abs(Rm).max())


def test_orthogonal_iteration_reaches_the_eigenvectors():
    """Repeated refreshes with frozen statistics converge to the eigenvectors of S (from
    numpy.linalg.eigh), ordered by decreasing eigenvalue, up to signs."""
    rng = np.random.default_rng(5)
    d = 8
    E = _orth(rng, d)
    lam = 2.0 ** -np.arange(d)       # well separated: ratio 1/2 per step
    Sm = (E * lam) @ E.T
    Q = S.refresh_basis(Sm, np.eye(d), iters=80)
    w, Ev = np.linalg.eigh(Sm)
    Ev = Ev[:, ::-1]
    np.testing.assert_allclose(np.abs(Q.T @ Ev), np.eye(d), atol=1e-9)


def test_refresh_uses_the_updated_statistics_and_leaves_v():
    rng = np.random.default_rng(6)
    st = _state(rng, 4, 6)
    hp = S.SoapHParams(refresh=True, shampoo_beta=0.7, shampoo_weight=0.3)
    out = _run(st, 5, hp)
    L2 = 0.7 * st["L"] + 0.3 * st["grad"] @ st["grad"].T
    R2 = 0.7 * st["R"] + 0.3 * st["grad"].T @ st["grad"]
    np.testing.assert_allclose(out[3], L2, rtol=1e-13)
    np.testing.assert_allclose(out[4], R2, rtol=1e-13)
    np.testing.assert_allclose(out[5], S.refresh_basis(L2, st["QL"]), atol=1e-13)
    np.testing.assert_allclose(out[6], S.refresh_basis(R2, st["QR"]), atol=1e-13)
    no = _run(st, 5, S.SoapHParams(refresh=False, shampoo_beta=0.7, shampoo_weight=0.3))
    for k in (0, 1, 2, 7):  # the update uses the bases of the previous refresh either way
        np.testing.assert_array_equal(out[k], no[k])


def test_zero_gradient_and_state_only_decays():
    hp = S.SoapHParams(lr=0.1, weight_decay=0.2)
    p = np.full((3, 4), 2.0)
    out = S.soap_step(p, np.zeros((3, 4)), np.zeros((3, 4)), np.zeros((3, 4)), np.zeros((3, 3)),
                      np.zeros((4, 4)), np.eye(3), np.eye(4), 1, hp)
    np.testing.assert_array_equal(out[7], 0.0)
    np.testing.assert_allclose(out[0], p * (1 - 0.1 * 0.2), rtol=0)


def test_bf16_gradient_widens_exactly():
    rng = np.random.default_rng(7)
    st = _state(rng, 4, 5)
    bits = synth.f32_to_bf16_bits(rng.standard_normal((4, 5)).astype(np.float32))
    st["grad"] = bits
    hp = S.SoapHParams()
    got = _run(st, 1, hp)
    st["grad"] = synth.bf16_bits_to_f32(bits).astype(np.float64)
    ref = _run(st, 1, hp)
    np.testing.assert_array_equal(got[7], ref[7])


# ------------------------------------------------------------------ one-sided preconditioning

def test_both_sides_beyond_the_limit_is_adamw():
    """Both sides longer than max_precond_dim: no basis on either side, the step is AdamW
    (torch.optim.AdamW on the CPU in float64, three steps)."""
    import torch
    rng = np.random.default_rng(300)
    m, n = 9, 7
    hp = S.SoapHParams(lr=1e-2, weight_decay=0.1, beta1=0.9, beta2=0.99, eps=1e-8, max_precond_dim=6)
    p = rng.standard_normal((m, n))
    M = np.zeros((m, n))
    V = np.zeros((m, n))
    tp = torch.tensor(p.copy(), requires_grad=True)
    opt = torch.optim.AdamW([tp], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps, weight_decay=hp.weight_decay)
    for t in range(1, 4):
        g = rng.standard_normal((m, n))
        p, M, V, L2, R2, QL, QR, N = S.soap_step(p, g, M, V, None, None, None, None, t, hp)
        assert L2 is None and R2 is None and QL is None and QR is None
        tp.grad = torch.tensor(g)
        opt.step()
        np.testing.assert_allclose(p, tp.detach().numpy(), rtol=0, atol=1e-14)
        np.testing.assert_allclose(M, opt.state[tp]["exp_avg"].numpy(), rtol=0, atol=1e-15)
        np.testing.assert_allclose(V, opt.state[tp]["exp_avg_sq"].numpy(), rtol=0, atol=1e-15)


def test_one_sided_step_is_transpose_consistent():
    """A left side beyond the limit on G (m x n) is the right side beyond it on G^T: every output
    is the transpose, with the roles of the two bases and statistics swapped (three steps with a
    refresh after each)."""
    rng = np.random.default_rng(301)
    m, n = 12, 5
    hp = S.SoapHParams(lr=3e-3, weight_decay=0.01, refresh=True, max_precond_dim=8)
    p = rng.standard_normal((m, n))
    M, V, R, QR = np.zeros((m, n)), np.zeros((m, n)), np.zeros((n, n)), np.eye(n)
    pt, Mt, Vt, Lt, QLt = p.T.copy(), np.zeros((n, m)), np.zeros((n, m)), np.zeros((n, n)), np.eye(n)
    for t in range(1, 4):
        g = rng.standard_normal((m, n))
        p, M, V, L2, R, QL2, QR, N = S.soap_step(p, g, M, V, None, R, None, QR, t, hp)
        pt, Mt, Vt, Lt, R2t, QLt, QR2t, Nt = S.soap_step(pt, g.T, Mt, Vt, Lt, None, QLt, None, t, hp)
        assert L2 is None and QL2 is None and R2t is None and QR2t is None
        for a, b in ((p, pt), (M, Mt), (V, Vt), (N, Nt)):
            np.testing.assert_allclose(a, b.T, rtol=0, atol=1e-13)
        np.testing.assert_allclose(R, Lt, rtol=0, atol=1e-13)
        np.testing.assert_allclose(QR, QLt, rtol=0, atol=1e-12)


def test_right_only_closed_form_on_an_aligned_gradient():
    """Left side beyond the limit, right basis Q_R: a gradient G = A Q_R^T has G' = A, so at t = 1
    from zero moments N = (A / (|A| + eps)) Q_R^T exactly (bias corrections cancel)."""
    rng = np.random.default_rng(302)
    m, n = 11, 4
    q, r = np.linalg.qr(rng.standard_normal((n, n)))
    QR = q * np.sign(np.diag(r))
    A = rng.standard_normal((m, n))
    G = A @ QR.T
    hp = S.SoapHParams(lr=1e-2, eps=1e-8, max_precond_dim=n)
    _, _, V, L2, R2, QL2, QR2, N = S.soap_step(np.zeros((m, n)), G, np.zeros((m, n)), np.zeros((m, n)),
                                               None, np.zeros((n, n)), None, QR, 1, hp)
    np.testing.assert_allclose(N, (A / (np.abs(A) + hp.eps)) @ QR.T, rtol=0, atol=1e-13)
    np.testing.assert_allclose(V, (1 - hp.beta2) * A * A, rtol=1e-13, atol=0)
    assert L2 is None and QL2 is None
    np.testing.assert_allclose(R2, hp.shampoo_weight * G.T @ G, rtol=1e-13, atol=1e-15)
    np.testing.assert_array_equal(QR2, QR)   # no refresh: the basis is returned as it was
