"""GPU parity of the SOAP owner step and of its orthonormal factor (through the C ABI) against the
fp64 oracle (numpy.linalg.qr for the refresh) on the same seeded inputs.

Tolerances, from a float32 emulation of the same arithmetic on these inputs (fp32 products and
a float32 blocked Householder QR):
* the direction N (and the parameter through it): emulation <= 7e-7 relative; bar 1e-4 (the
  paper's own SOAP check matches a gathered reference to 1.3e-4). The Adam division amplifies the
  products' rounding by |M'| / sqrt(V): the seeded second moments are positive and bounded away
  from zero, V = s^2 (0.5 + U(0, 1)), as an EMA over many squared gradients is. (With V drawn as
  an independent squared Gaussian, entries with sqrt(V) ~ 1e-7 against |M'| ~ 1e-3 put N' at ~1e4
  and the float32 emulation itself 3e-4 away from the exact result.)
* M 1e-6 (one fp32 fma per element; emulation 4e-8), V and the statistics 1e-5 (fp32 products
  squared or summed; emulation 5e-8).
* refreshed bases (compared up to column signs, which do not change N): emulation <= 1.5e-6 for
  the full-rank statistics used here (condition ~ 20-30); bar 1e-4. For rank-deficient statistics
  the basis of the null space is not unique: there only orthogonality and the triangular form of
  Q^T S are checked.
* the standalone factor against numpy.linalg.qr: 1e-4 for condition <= 1e3 (emulation 2.5e-6 at
  condition 600).
"""
import sys

import numpy as np
import pytest
import scipy.linalg

import synth
from oracle import soap as OS
from tests.helpers import check_bf16_param, from_dev, rel_fro, to_dev

pytestmark = pytest.mark.gpu

N_TOL = 1e-4
Q_TOL = 1e-4


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def native():
    import torch
    from paper_2607_05895_amd import native as nat
    nat.lib()
    assert torch.cuda.is_available()
    return nat


def _sync():
    import torch
    torch.cuda.synchronize()


def _orth(rng, d):
    q, r = scipy.linalg.qr(rng.standard_normal((d, d)), check_finite=False)
    return q * np.sign(np.diag(r))


def _f32(x):
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def _sign_aligned_err(q, q_ref):
    s = np.sign(np.sum(q * q_ref, axis=0))
    s[s == 0] = 1.0
    return rel_fro(q * s, q_ref)


# ------------------------------------------------------------------ orthonormal factor

@pytest.mark.parametrize("d", [1, 2, 15, 16, 17, 100, 127, 128, 129, 255, 256, 257, 300, 640])
def test_orthonormal_factor_matches_numpy_qr(native, d):
    """Against LAPACK's QR: one-panel and ragged sizes, and sizes at and around the 128-column blocks
    whose updates run on the GEMM (127 .. 129, 255 .. 257)."""
    import torch
    _say(f"orthonormal factor d={d}")
    rng = np.random.default_rng(100 + d)
    A = rng.standard_normal((d, d + 8))
    a = (A @ A.T @ _orth(rng, d)).astype(np.float32)     # condition ~ 10-50
    q = torch.empty((d, d), dtype=torch.float32, device="cuda")
    native.orthonormal_factor_t(to_dev(a, synth.F32), q)
    _sync()
    qg = from_dev(q)
    ref = OS.orthonormal_factor(a.astype(np.float64))
    assert _sign_aligned_err(qg, ref) <= Q_TOL
    np.testing.assert_allclose(qg.T @ qg, np.eye(d), atol=2e-5)


@pytest.mark.parametrize("d", sorted(int(x) for x in np.random.default_rng(77).integers(2, 1000, 8)))
def test_orthonormal_factor_random_sizes(native, d):
    """Seeded random sizes: ragged last panels (d mod 16) and row counts that are not multiples of
    the 512 panel threads."""
    import torch
    _say(f"orthonormal factor random d={d}")
    rng = np.random.default_rng(200 + d)
    a = (rng.standard_normal((d, d)) + 0.5 * d ** 0.5 * np.eye(d)).astype(np.float32)
    q = torch.empty((d, d), dtype=torch.float32, device="cuda")
    native.orthonormal_factor_t(to_dev(a, synth.F32), q)
    _sync()
    qg = from_dev(q)
    assert _sign_aligned_err(qg, OS.orthonormal_factor(a.astype(np.float64))) <= Q_TOL
    np.testing.assert_allclose(qg.T @ qg, np.eye(d), atol=2e-5)


def test_orthonormal_factor_rank_deficient_and_signs(native):
    """A rank-deficient input still gives an orthogonal factor with Q^T A upper triangular; on a
    full-rank input LAPACK's signs are reproduced (no column flips)."""
    import torch
    _say("orthonormal factor rank deficient")
    rng = np.random.default_rng(7)
    for d, r in ((200, 37), (300, 1)):
        B = rng.standard_normal((d, r))
        a = (B @ B.T).astype(np.float32)
        q = torch.empty((d, d), dtype=torch.float32, device="cuda")
        native.orthonormal_factor_t(to_dev(a, synth.F32), q)
        _sync()
        qg = from_dev(q)
        np.testing.assert_allclose(qg.T @ qg, np.eye(d), atol=2e-5)
        Rm = qg.T @ a.astype(np.float64)
        assert np.abs(np.tril(Rm, -1)).max() <= 1e-5 * np.abs(Rm).max()
    a = rng.standard_normal((64, 64)).astype(np.float32) + 8 * np.eye(64, dtype=np.float32)
    q = torch.empty((64, 64), dtype=torch.float32, device="cuda")
    native.orthonormal_factor_t(to_dev(a, synth.F32), q)
    _sync()
    assert rel_fro(from_dev(q), OS.orthonormal_factor(a.astype(np.float64))) <= Q_TOL


def test_orthonormal_factor_at_the_largest_side(native):
    """d = 4096, the largest side: every thread of the panel kernel holds 8 rows of the first panel."""
    import torch
    _say("orthonormal factor d=4096")
    d = 4096
    rng = np.random.default_rng(4096)
    A = rng.standard_normal((d, d)) + 0.5 * d ** 0.5 * np.eye(d)   # well conditioned
    a = A.astype(np.float32)
    q = torch.empty((d, d), dtype=torch.float32, device="cuda")
    native.orthonormal_factor_t(to_dev(a, synth.F32), q)
    _sync()
    qg = from_dev(q)
    ref = OS.orthonormal_factor(a.astype(np.float64))
    assert _sign_aligned_err(qg, ref) <= Q_TOL
    d_orth = np.abs(qg.T @ qg - np.eye(d)).max()
    assert d_orth <= 2e-5, d_orth


# ------------------------------------------------------------------ SOAP step

SHAPES = [(1, 50), (65, 129), (200, 96), (256, 512), (300, 300), (640, 1152)]
TINY = [(1, 1), (2, 3), (3, 2)]  # far below one tile: padding and 1x1 / 2x2 / 3x3 statistics


class _Mat:
    """One matrix with full-rank statistics and random orthogonal bases (host fp64 copies of the
    fp32 values the device holds)."""

    def __init__(self, rng, m, n, pdt, gdt, g_std=1e-3, bases=True, maxd=4096):
        t = synth.random_muon_tensors(rng, m, n, pdt, gdt, g_std=g_std, p_std=0.02)
        self.m, self.n, self.pdt, self.gdt = m, n, pdt, gdt
        self.p, self.g = t.param, t.grad
        self.M = _f32(rng.standard_normal((m, n)) * g_std)
        self.V = _f32(g_std ** 2 * (0.5 + rng.random((m, n))))
        # a side longer than maxd has no statistic and no basis
        self.L = self.QL = self.R = self.QR = None
        if m <= maxd:
            A = rng.standard_normal((m, 2 * m)) * g_std
            self.L = _f32(A @ A.T)
            self.QL = _f32(_orth(rng, m)) if bases else np.eye(m)
        if n <= maxd:
            B = rng.standard_normal((n, 2 * n)) * g_std
            self.R = _f32(B @ B.T)
            self.QR = _f32(_orth(rng, n)) if bases else np.eye(n)

    def device(self):
        import torch
        self.dp = to_dev(self.p, self.pdt)
        self.dg = to_dev(self.g, self.gdt)
        f = lambda x: to_dev(x.astype(np.float32), synth.F32) if x is not None else None  # noqa: E731
        self.dM, self.dV, self.dL, self.dR = f(self.M), f(self.V), f(self.L), f(self.R)
        self.dQL, self.dQR = f(self.QL), f(self.QR)
        self.dN = torch.zeros((self.m, self.n), dtype=torch.float32, device="cuda")
        return self

    def entry(self, native):
        return native.soap_entry_t(self.dp, self.dg, self.dM, self.dV, self.dL, self.dR, self.dQL, self.dQR,
                                   self.dN)


def _oracle_step(mat, step, hp):
    p_in = getattr(mat, "p_in", mat.p)
    out = OS.soap_step(p_in, mat.g, mat.M, mat.V, mat.L, mat.R, mat.QL, mat.QR, step, hp)
    mat.p_or, mat.M, mat.V, mat.L, mat.R, QL, QR, mat.N_or = out
    mat.QL_prev, mat.QR_prev = mat.QL, mat.QR
    mat.QL, mat.QR = QL, QR
    p32 = mat.p_or.astype(np.float32)
    mat.p_in = synth.f32_to_bf16_bits(p32) if mat.pdt == synth.BF16 else p32


def _check(mat, hp, full_rank=True):
    en = rel_fro(from_dev(mat.dN), mat.N_or)
    assert en <= N_TOL, ("N", en)
    assert rel_fro(from_dev(mat.dM), mat.M) <= 1e-6, ("M", rel_fro(from_dev(mat.dM), mat.M))
    assert rel_fro(from_dev(mat.dV), mat.V) <= 1e-5, ("V", rel_fro(from_dev(mat.dV), mat.V))
    for dS, S_ref in ((mat.dL, mat.L), (mat.dR, mat.R)):
        assert (dS is None) == (S_ref is None)
        if dS is not None:
            assert rel_fro(from_dev(dS), S_ref) <= 1e-5
    if hp.refresh:
        for dq, q_ref, S_stat, q_prev in ((mat.dQL, mat.QL, mat.L, mat.QL_prev),
                                          (mat.dQR, mat.QR, mat.R, mat.QR_prev)):
            if dq is None:   # a side without a basis
                continue
            qg = from_dev(dq)
            d = qg.shape[0]
            np.testing.assert_allclose(qg.T @ qg, np.eye(d), atol=2e-5)
            if full_rank:
                assert _sign_aligned_err(qg, q_ref) <= Q_TOL, ("Q", _sign_aligned_err(qg, q_ref))
            else:
                Rm = qg.T @ (S_stat @ q_prev)
                assert np.abs(np.tril(Rm, -1)).max() <= 1e-5 * np.abs(Rm).max()
    pg = from_dev(mat.dp)
    un = hp.lr * np.linalg.norm(mat.N_or)
    if mat.pdt == synth.BF16:
        assert check_bf16_param(pg, mat.p_or, un, N_TOL) <= 1.0
    else:
        assert np.linalg.norm(pg - mat.p_or) <= N_TOL * un + 1e-6 * np.linalg.norm(mat.p_or)


def _hp(native, **kw):
    d = dict(lr=3e-3, weight_decay=0.01, beta1=0.95, beta2=0.95, eps=1e-8, shampoo_beta=0.95,
             shampoo_weight=0.05, refresh=True, refresh_iters=1)
    d.update(kw)
    step = d.pop("step", 3)
    return (native.soap_hparams(step=step, **d), OS.SoapHParams(**d), step)


@pytest.mark.parametrize("shape", SHAPES + TINY)
@pytest.mark.parametrize("dts", [(synth.BF16, synth.BF16), (synth.F32, synth.F32)])
def test_soap_step_matches_oracle(native, shape, dts):
    m, n = shape
    _say(f"soap {m}x{n} {dts}")
    rng = np.random.default_rng(9000 + m + 7 * n + (dts[0] == synth.F32))
    mat = _Mat(rng, m, n, *dts).device()
    hpn, hpo, step = _hp(native)
    ws = native.soap_workspace_t([mat.entry(native)], hpn)
    native.soap_step_t([mat.entry(native)], hpn, ws)
    _sync()
    _oracle_step(mat, step, hpo)
    _check(mat, hpo)


def test_soap_grouped_three_steps_with_refresh_iterations(native):
    """All shapes in one call, mixed dtypes, three consecutive steps on one workspace: step 1
    without refresh, steps 2 and 3 with refresh (the second with 3 power-QR repetitions), the
    gradient redrawn every step; the library's refreshed bases feed its next step."""
    _say("soap grouped three steps")
    rng = np.random.default_rng(9100)
    mats = [_Mat(rng, m, n, synth.BF16 if i % 2 == 0 else synth.F32,
                 synth.BF16 if i % 3 else synth.F32).device() for i, (m, n) in enumerate(SHAPES)]
    ents = [x.entry(native) for x in mats]
    plan = [dict(refresh=False, step=1), dict(refresh=True, step=2), dict(refresh=True, refresh_iters=3, step=3)]
    hp_big = _hp(native, refresh=True, refresh_iters=3)[0]
    ws = native.soap_workspace_t(ents, hp_big)
    for k, kw in enumerate(plan):
        if k > 0:
            for x in mats:
                x.g = synth.random_muon_tensors(rng, x.m, x.n, x.pdt, x.gdt).grad
                x.dg.copy_(to_dev(x.g, x.gdt))
        hpn, hpo, step = _hp(native, **kw)
        native.soap_step_t(ents, hpn, ws)
        _sync()
        for x in mats:
            _oracle_step(x, step, hpo)
            _check(x, hpo)


def test_soap_many_entries_in_one_call(native):
    """24 seeded random shapes (sides 1 .. 300, mixed dtypes) in one call with the refresh: the
    grouped launches' tile prefixes and the sides' different panel counts."""
    _say("soap 24 entries")
    rng = np.random.default_rng(9700)
    dts = (synth.BF16, synth.F32)
    mats = [_Mat(rng, int(rng.integers(1, 301)), int(rng.integers(1, 301)), dts[i % 2], dts[(i // 2) % 2]).device()
            for i in range(24)]
    hpn, hpo, step = _hp(native)
    ents = [x.entry(native) for x in mats]
    native.soap_step_t(ents, hpn, native.soap_workspace_t(ents, hpn))
    _sync()
    for x in mats:
        _oracle_step(x, step, hpo)
        _check(x, hpo)


def test_soap_identity_bases_is_adamw(native):
    """Bases at the identity, no refresh: one SOAP step equals one step of the library's AdamW
    kernel on the same tensors (the reduction the oracle is pinned to), bases left unchanged."""
    import torch
    _say("soap identity bases vs adamw")
    rng = np.random.default_rng(9200)
    m, n = 96, 200
    mat = _Mat(rng, m, n, synth.F32, synth.F32, bases=False).device()
    hpn, hpo, step = _hp(native, refresh=False, step=2)
    keep = (mat.dQL.clone(), mat.dQR.clone())
    p2, g2 = mat.dp.clone(), mat.dg.clone()
    ea, eas = to_dev(mat.M.astype(np.float32), synth.F32), to_dev(mat.V.astype(np.float32), synth.F32)
    native.soap_step_t([mat.entry(native)], hpn, native.soap_workspace_t([mat.entry(native)], hpn))
    native.adamw_step_t([native.adamw_entry_t(p2, g2, ea, eas)], lr=hpo.lr, beta1=hpo.beta1,
                        beta2=hpo.beta2, eps=hpo.eps, weight_decay=hpo.weight_decay, step=step)
    _sync()
    assert bool((mat.dQL == keep[0]).all()) and bool((mat.dQR == keep[1]).all())
    assert rel_fro(from_dev(mat.dp), from_dev(p2)) <= 1e-6
    assert rel_fro(from_dev(mat.dM), from_dev(ea)) <= 1e-6
    assert rel_fro(from_dev(mat.dV), from_dev(eas)) <= 1e-5
    _oracle_step(mat, step, hpo)
    _check(mat, hpo)


def test_soap_rank_deficient_statistics_from_zero(native):
    """Statistics from zero (rank <= min(m, n) after one gradient) and identity bases: the update
    matches; the refreshed bases are orthogonal with Q^T (S Q_prev) upper triangular (the basis of
    the null space is not unique)."""
    _say("soap rank deficient statistics")
    rng = np.random.default_rng(9300)
    mats = []
    for (m, n) in [(65, 129), (256, 512)]:
        x = _Mat(rng, m, n, synth.BF16, synth.BF16, bases=False)
        x.L, x.R = np.zeros((m, m)), np.zeros((n, n))
        x.M, x.V = np.zeros((m, n)), np.zeros((m, n))
        mats.append(x.device())
    hpn, hpo, step = _hp(native, step=1)
    ents = [x.entry(native) for x in mats]
    native.soap_step_t(ents, hpn, native.soap_workspace_t(ents, hpn))
    _sync()
    for x in mats:
        _oracle_step(x, step, hpo)
        _check(x, hpo, full_rank=False)


def test_soap_lr_zero_and_determinism(native):
    import torch
    _say("soap lr=0 and determinism")
    rng = np.random.default_rng(9400)
    mats = [_Mat(rng, m, n, synth.BF16, synth.BF16).device() for (m, n) in [(200, 96), (256, 512)]]
    hpn, _, _ = _hp(native, lr=0.0, weight_decay=0.0)
    ents = [x.entry(native) for x in mats]
    ws = native.soap_workspace_t(ents, hpn)
    state0 = [[t.clone() for t in (x.dM, x.dV, x.dL, x.dR, x.dQL, x.dQR)] for x in mats]
    p0 = [x.dp.clone() for x in mats]
    native.soap_step_t(ents, hpn, ws)
    _sync()
    out1 = [[t.clone() for t in (x.dN, x.dQL, x.dQR)] for x in mats]
    for x, p, st in zip(mats, p0, state0):
        assert bool((x.dp.view(torch.int16) == p.view(torch.int16)).all())
        for dst, src in zip((x.dM, x.dV, x.dL, x.dR, x.dQL, x.dQR), st):
            dst.copy_(src)
    native.soap_step_t(ents, hpn, ws)
    _sync()
    for x, o in zip(mats, out1):
        for a, b in zip((x.dN, x.dQL, x.dQR), o):
            assert bool((a == b).all())


def test_soap_step_with_a_4096_side(native):
    """A 64 x 4096 matrix: the right basis is 4096 x 4096 (the largest side), refreshed by the QR."""
    _say("soap 64x4096")
    rng = np.random.default_rng(9600)
    mat = _Mat(rng, 64, 4096, synth.BF16, synth.BF16).device()
    hpn, hpo, step = _hp(native)
    ents = [mat.entry(native)]
    native.soap_step_t(ents, hpn, native.soap_workspace_t(ents, hpn))
    _sync()
    _oracle_step(mat, step, hpo)
    _check(mat, hpo)


def _offset_view(t):
    """The same values in a buffer that starts 4 bytes past a 16-byte boundary (a view into a larger
    allocation)."""
    import torch
    big = torch.zeros(t.numel() + 1, dtype=t.dtype, device=t.device)
    v = big[1:].view(t.shape)
    v.copy_(t)
    assert v.data_ptr() % 16 == 4
    return v


@pytest.mark.parametrize("refresh", [True, False])
def test_soap_unaligned_caller_buffers_take_the_copy_path(native, refresh):
    """Tile-multiple sides use 16-byte aligned caller statistics and bases where they lie and copy
    the others: the same step on the same values through both paths gives the same bits."""
    import torch
    _say(f"soap in place vs copied buffers, refresh {refresh}")
    runs = []
    for offset in (False, True):
        x = _Mat(np.random.default_rng(9900 + refresh), 256, 384, synth.BF16, synth.BF16).device()
        if offset:
            x.dL, x.dR, x.dQL, x.dQR = (_offset_view(t) for t in (x.dL, x.dR, x.dQL, x.dQR))
        hpn, _, _ = _hp(native, refresh=refresh)
        ents = [x.entry(native)]
        native.soap_step_t(ents, hpn, native.soap_workspace_t(ents, hpn))
        _sync()
        runs.append([t.clone() for t in (x.dN, x.dp, x.dM, x.dV, x.dL, x.dR, x.dQL, x.dQR)])
    for a, b in zip(*runs):
        assert torch.equal(a, b)


def test_soap_benchmark_configuration_full_size(native):
    """The configuration bench.py times: the GPT-2-small share's 12 matrices in one call, bf16
    parameters and gradients, full-rank statistics and random orthogonal bases, refresh on; every
    matrix against the oracle. Then a step without refresh on a new gradient (also timed): the
    bases, read where they lie, stay unchanged."""
    import torch
    _say("soap benchmark configuration")
    wl = synth.workload(2)
    rng = np.random.default_rng(9500)
    mats = [_Mat(rng, e.m, e.n, synth.BF16, synth.BF16, g_std=0.02).device() for e in wl.muon]
    hpn, hpo, step = _hp(native, lr=3e-3, weight_decay=0.01, step=5)
    ents = [x.entry(native) for x in mats]
    ws = native.soap_workspace_t(ents, hpn)
    native.soap_step_t(ents, hpn, ws)
    _sync()
    for x in mats:
        _oracle_step(x, step, hpo)
        _check(x, hpo)
    hpn2, hpo2, step2 = _hp(native, lr=3e-3, weight_decay=0.01, step=6, refresh=False)
    keep = []
    for x in mats:
        x.g = synth.random_muon_tensors(rng, x.m, x.n, x.pdt, x.gdt, g_std=0.02).grad
        x.dg.copy_(to_dev(x.g, x.gdt))
        x.QL = from_dev(x.dQL).astype(np.float64)   # the refreshed bases as the device stores them
        x.QR = from_dev(x.dQR).astype(np.float64)
        keep.append((x.dQL.clone(), x.dQR.clone()))
    native.soap_step_t(ents, hpn2, ws)
    _sync()
    for x, (kl, kr) in zip(mats, keep):
        _oracle_step(x, step2, hpo2)
        _check(x, hpo2)
        assert torch.equal(kl, x.dQL) and torch.equal(kr, x.dQR)


# ------------------------------------------------------------------ one-sided preconditioning

ONE_SIDED = [(100, 50), (50, 100), (100, 200), (40, 50), (64, 64), (65, 30), (129, 64)]


def test_soap_one_sided_grouped_three_steps(native):
    """max_precond_dim = 64: sides longer than 64 have no basis. One call groups matrices with a
    basis on the left only, the right only, both and neither (each side at the boundary 64 / 65
    too), mixed dtypes, over three steps (no refresh, refresh, refresh with 3 repetitions), the
    gradient redrawn every step."""
    _say("soap one-sided grouped three steps")
    rng = np.random.default_rng(9700)
    mats = [_Mat(rng, m, n, synth.BF16 if i % 2 == 0 else synth.F32, synth.BF16 if i % 3 else synth.F32,
                 maxd=64).device() for i, (m, n) in enumerate(ONE_SIDED)]
    ents = [x.entry(native) for x in mats]
    plan = [dict(refresh=False, step=1), dict(refresh=True, step=2), dict(refresh=True, refresh_iters=3, step=3)]
    ws = native.soap_workspace_t(ents, _hp(native, refresh=True, refresh_iters=3, max_precond_dim=64)[0])
    for k, kw in enumerate(plan):
        if k > 0:
            for x in mats:
                x.g = synth.random_muon_tensors(rng, x.m, x.n, x.pdt, x.gdt).grad
                x.dg.copy_(to_dev(x.g, x.gdt))
        hpn, hpo, step = _hp(native, max_precond_dim=64, **kw)
        native.soap_step_t(ents, hpn, ws)
        _sync()
        for x in mats:
            _oracle_step(x, step, hpo)
            _check(x, hpo)


@pytest.mark.parametrize("shape", [(14336, 4096), (4096, 14336)])
def test_soap_llama_ffn_shapes_one_sided(native, shape):
    """The Llama-3-8B FFN shapes with the default limit (4096): the 14336 side has no basis, the
    4096 side a 4096 x 4096 basis refreshed by the QR (a 4096 x 4096 full-rank statistic)."""
    m, n = shape
    _say(f"soap one-sided {m}x{n}")
    rng = np.random.default_rng(9800 + m)
    mat = _Mat(rng, m, n, synth.BF16, synth.BF16).device()
    assert (mat.L is None) == (m > 4096) and (mat.R is None) == (n > 4096)
    hpn, hpo, step = _hp(native)
    ents = [mat.entry(native)]
    native.soap_step_t(ents, hpn, native.soap_workspace_t(ents, hpn))
    _sync()
    _oracle_step(mat, step, hpo)
    _check(mat, hpo)
