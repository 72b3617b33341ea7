"""GPU parity of the Shampoo owner step and the inverse root (through the C ABI) against the fp64
oracle (eigendecomposition roots) on the same seeded inputs.

Tolerances, from a float32 emulation of the coupled Newton iteration on these inputs (20
iterations, ridge 1e-6 ||S||_F), which the GPU reproduces to two digits:
* U = P_L G P_R: for a Gaussian gradient with min(m, n) <= 0.75 max(m, n) the statistics' nonzero
  spectrum stays away from zero (Marchenko-Pastur edge (sqrt(max) - sqrt(min))^2 sigma^2) and the
  emulation is within 3.5e-5 of the exact update: bar 1e-4. A square gradient has singular values
  far below the ridge (sigma_min^2 ~ 1e-12 against rho ~ 7e-9 at 300 x 300), which float32
  resolves only coarsely: emulation 2.4e-4, bar 5e-4.
* P restricted to the gradient's range (P_L G, G P_R): 1e-4 (emulation <= 1.3e-5).
* The whole P: 1e-4 for the well-conditioned side (the shorter side of a rectangular gradient);
  else the ridge bar 2e-8 / eps_rel. On a rank-deficient side the null directions of S carry
  rho^(-1/4), the largest eigenvalues of P, and dominate ||P||_F. The coupled iteration works on
  M = z (S + rho I), whose eigenvalue there starts at z rho ~ eps_rel, so float32 rounding of M
  (absolute, ~2^-24 ||M||) perturbs it by ~2^-24 / eps_rel relative: the condition number of
  S + rho I is ~1 / eps_rel. A float32 emulation of the iteration gives a relative error of
  (6.0-7.3e-9) / eps_rel in P there, independent of d from 256 to 1536 (6.7e-3 at eps_rel 1e-6,
  6.6e-4 at 1e-5, 7e-5 at 1e-4); the GPU measured 1.4e-2 at d = 3072 and eps_rel 1e-6. The exact root
  of the same float32-stored statistic is within 2-4e-4, so the limit is the iteration's float32
  arithmetic at that condition number, not the statistic's storage. Those directions never enter
  U of the same statistics; a stale step on a new gradient with components outside the statistic's
  range does take them into U: its bar is the same ridge bar (emulation: the U error equals the
  P error in those directions).
* Statistics 1e-5 (fp32 sums). Parameters: bf16 rounding-aware (half an ulp plus the U bar times
  lr ||U||); fp32 parameters the U bar times lr ||U|| + 1e-6 ||p||.
"""
import sys

import numpy as np
import pytest

import synth
from oracle import shampoo as OS
from tests.helpers import check_bf16_param, from_dev, rel_fro, to_dev

pytestmark = pytest.mark.gpu

U_TOL = 1e-4
STAT_TOL = 1e-5


def _u_tol(m, n):
    return U_TOL if min(m, n) <= 0.75 * max(m, n) else 5e-4


def _ridge_tol(eps_rel):
    """Relative accuracy of P in the null directions of a rank-deficient statistic (float32
    iteration at condition number ~1 / eps_rel; see the module docstring)."""
    return max(U_TOL, 2e-8 / eps_rel)


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


def _spd(rng, d, cond):
    """Symmetric positive definite d x d with eigenvalues log-spaced over [1/cond, 1]."""
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    q = q * np.sign(np.diag(r))
    w = np.logspace(0, -np.log10(cond), d) if d > 1 else np.ones(1)
    return (q * w) @ q.T


# ------------------------------------------------------------------ inverse root

@pytest.mark.parametrize("d", [1, 7, 100, 128, 129, 257, 640])
@pytest.mark.parametrize("p", [1, 2, 4])
def test_inverse_root_matches_oracle(native, d, p):
    import torch
    _say(f"inverse root d={d} p={p}")
    rng = np.random.default_rng(1000 + 10 * d + p)
    a = _spd(rng, d, 1e3).astype(np.float32)
    ad = to_dev(a, synth.F32)
    out = torch.empty((d, d), dtype=torch.float32, device="cuda")
    native.inverse_root_t(ad, out, p=p, eps=1e-9, eps_rel=1e-6, iters=30)
    _sync()
    ref = OS.inverse_root(a.astype(np.float64), p, 1e-9, 1e-6)
    err = rel_fro(from_dev(out), ref)
    assert err <= 1e-4, err
    # a tile-multiple d is read where it lies: still read only
    np.testing.assert_array_equal(from_dev(ad), a)


def test_inverse_root_input_read_in_place_or_copied(native):
    """A tile-multiple d whose input is 16-byte aligned is read where it lies; the same values at a
    4-byte offset take the copy path. Same bits either way."""
    import torch
    _say("inverse root: aligned vs offset input")
    d = 256
    a = _spd(np.random.default_rng(1300), d, 1e3).astype(np.float32)
    outs = []
    for offset in (False, True):
        ad = to_dev(a, synth.F32)
        if offset:
            big = torch.zeros(d * d + 1, dtype=torch.float32, device="cuda")
            ad = big[1:].view(d, d)
            ad.copy_(to_dev(a, synth.F32))
            assert ad.data_ptr() % 16 == 4
        out = torch.empty((d, d), dtype=torch.float32, device="cuda")
        native.inverse_root_t(ad, out, p=4, eps=1e-9, eps_rel=1e-6, iters=30)
        _sync()
        outs.append(out.clone())
        np.testing.assert_array_equal(from_dev(ad), a)
    assert torch.equal(outs[0], outs[1])


def test_inverse_root_of_diagonal_and_scaled_identity(native):
    import torch
    _say("inverse root diagonal")
    d = 300
    w = np.logspace(0, -3, d).astype(np.float32)
    for a in (np.diag(w), 2.5 * np.eye(d, dtype=np.float32)):
        out = torch.empty((d, d), dtype=torch.float32, device="cuda")
        native.inverse_root_t(to_dev(a, synth.F32), out, p=4, eps=1e-6, eps_rel=0.0, iters=30)
        _sync()
        got = from_dev(out)
        rho = 1e-6
        np.testing.assert_allclose(np.diag(got), (np.diag(a).astype(np.float64) + rho) ** -0.25, rtol=2e-5)
        off = got - np.diag(np.diag(got))
        assert np.abs(off).max() == 0.0   # products of diagonal matrices stay exactly diagonal


# ------------------------------------------------------------------ Shampoo step

SHAPES = [(1, 50), (65, 129), (200, 96), (256, 512), (300, 300), (640, 1152)]
TINY = [(1, 1), (2, 3), (3, 2)]  # far below one tile: padding and 1x1 / 2x2 / 3x3 statistics


class _Mat:
    """One matrix: host copies (oracle side) and device tensors (library side)."""

    def __init__(self, rng, m, n, pdt, gdt, p_std=0.02, g_std=1e-3):
        t = synth.random_muon_tensors(rng, m, n, pdt, gdt, g_std=g_std, p_std=p_std)
        self.m, self.n, self.pdt, self.gdt = m, n, pdt, gdt
        self.p, self.g = t.param, t.grad
        self.L = np.zeros((m, m))
        self.R = np.zeros((n, n))
        self.PL = self.PR = None

    def device(self):
        import torch
        self.dp = to_dev(self.p, self.pdt)
        self.dg = to_dev(self.g, self.gdt)
        self.dL = torch.zeros((self.m, self.m), dtype=torch.float32, device="cuda")
        self.dR = torch.zeros((self.n, self.n), dtype=torch.float32, device="cuda")
        self.dPL = torch.zeros((self.m, self.m), dtype=torch.float32, device="cuda")
        self.dPR = torch.zeros((self.n, self.n), dtype=torch.float32, device="cuda")
        self.dU = torch.zeros((self.m, self.n), dtype=torch.float32, device="cuda")
        return self

    def entry(self, native):
        return native.shampoo_entry_t(self.dp, self.dg, self.dL, self.dR, self.dPL, self.dPR, self.dU)


def _oracle_step(mat, hp):
    """The oracle's step from the stored state; the parameter it starts from is the stored one
    (rounded to the parameter dtype after every step, as the library stores it)."""
    p_in = getattr(mat, "p_in", mat.p)
    p, L, R, PL, PR, U = OS.shampoo_step(p_in, mat.g, mat.L, mat.R, mat.PL, mat.PR, hp)
    mat.p_or, mat.L, mat.R, mat.PL, mat.PR, mat.U_or = p, L, R, PL, PR, U
    p32 = p.astype(np.float32)
    mat.p_in = synth.f32_to_bf16_bits(p32) if mat.pdt == synth.BF16 else p32


def _check(mat, hp, check_p=True):
    G = OS._f64(mat.g)
    U = from_dev(mat.dU)
    ut = _u_tol(mat.m, mat.n)
    eu = rel_fro(U, mat.U_or)
    assert eu <= ut, ("U", eu)
    assert rel_fro(from_dev(mat.dL), mat.L) <= STAT_TOL
    assert rel_fro(from_dev(mat.dR), mat.R) <= STAT_TOL
    if hp.refresh:
        PL, PR = from_dev(mat.dPL), from_dev(mat.dPR)
        assert rel_fro(PL @ G, mat.PL @ G) <= U_TOL, ("PL G", rel_fro(PL @ G, mat.PL @ G))
        assert rel_fro(G @ PR, G @ mat.PR) <= U_TOL, ("G PR", rel_fro(G @ PR, G @ mat.PR))
        tol_l = 1e-4 if mat.m <= 0.75 * mat.n else _ridge_tol(hp.eps_rel)
        tol_r = 1e-4 if mat.n <= 0.75 * mat.m else _ridge_tol(hp.eps_rel)
        assert rel_fro(PL, mat.PL) <= tol_l, ("PL", rel_fro(PL, mat.PL))
        assert rel_fro(PR, mat.PR) <= tol_r, ("PR", rel_fro(PR, mat.PR))
    if check_p:
        pg = from_dev(mat.dp)
        un = hp.lr * np.linalg.norm(mat.U_or)
        if mat.pdt == synth.BF16:
            assert check_bf16_param(pg, mat.p_or, un, ut) <= 1.0
        else:
            assert np.linalg.norm(pg - mat.p_or) <= ut * un + 1e-6 * np.linalg.norm(mat.p_or)


def _hp(native, **kw):
    d = dict(lr=0.05, weight_decay=0.01, beta=1.0, weight=1.0, eps=1e-12, eps_rel=1e-6, refresh=True,
             root_iters=20)
    d.update(kw)
    return native.shampoo_hparams(**d), OS.ShampooHParams(lr=d["lr"], weight_decay=d["weight_decay"],
                                                         beta=d["beta"], weight=d["weight"], eps=d["eps"],
                                                         eps_rel=d["eps_rel"], refresh=d["refresh"])


@pytest.mark.parametrize("shape", SHAPES + TINY)
@pytest.mark.parametrize("dts", [(synth.BF16, synth.BF16), (synth.F32, synth.F32)])
def test_shampoo_step_matches_oracle(native, shape, dts):
    m, n = shape
    _say(f"shampoo {m}x{n} {dts}")
    rng = np.random.default_rng(2000 + m + 7 * n + (dts[0] == synth.F32))
    mat = _Mat(rng, m, n, *dts).device()
    hpn, hpo = _hp(native)
    ws = native.shampoo_workspace_t([mat.entry(native)], hpn)
    native.shampoo_step_t([mat.entry(native)], hpn, ws)
    _sync()
    _oracle_step(mat, hpo)
    _check(mat, hpo)


def test_shampoo_grouped_mixed_shapes_two_steps_ema(native):
    """All shapes in one call, mixed dtypes, two consecutive steps with EMA statistics (the second
    gradient redrawn), one shared workspace."""
    _say("shampoo grouped two steps")
    rng = np.random.default_rng(3000)
    mats = [_Mat(rng, m, n, synth.BF16 if i % 2 == 0 else synth.F32,
                 synth.BF16 if i % 3 else synth.F32).device() for i, (m, n) in enumerate(SHAPES)]
    hpn, hpo = _hp(native, beta=0.9, weight=0.1, weight_decay=0.1)
    ents = [x.entry(native) for x in mats]
    ws = native.shampoo_workspace_t(ents, hpn)
    for step in range(2):
        if step == 1:
            for x in mats:
                x.g = synth.random_muon_tensors(rng, x.m, x.n, x.pdt, x.gdt).grad
                x.dg.copy_(to_dev(x.g, x.gdt))
        native.shampoo_step_t(ents, hpn, ws)
        _sync()
        for x in mats:
            _oracle_step(x, hpo)
    for x in mats:
        _check(x, hpo)


def test_shampoo_stale_preconditioners(native):
    """refresh = 0: the stored P_L, P_R (seeded SPD inputs, not computed by the library) are used
    as given and left unchanged, while the statistics still accumulate. Sides whose dimension is a
    multiple of 128 (read in place) and others (copied) in one call, bf16 and fp32 gradients."""
    _say("shampoo stale preconditioners")
    rng = np.random.default_rng(4000)
    mats = []
    for i, (m, n) in enumerate([(65, 129), (256, 512), (300, 300), (384, 200), (130, 256)]):
        x = _Mat(rng, m, n, synth.BF16, synth.F32 if i >= 3 else synth.BF16).device()
        x.PL = _spd(rng, m, 10.0)
        x.PR = _spd(rng, n, 10.0)
        x.dPL.copy_(to_dev(x.PL.astype(np.float32), synth.F32))
        x.dPR.copy_(to_dev(x.PR.astype(np.float32), synth.F32))
        x.PL = x.PL.astype(np.float32).astype(np.float64)
        x.PR = x.PR.astype(np.float32).astype(np.float64)
        mats.append(x)
    hpn, hpo = _hp(native, refresh=False)
    ents = [x.entry(native) for x in mats]
    ws = native.shampoo_workspace_t(ents, hpn)
    keep = [(x.dPL.clone(), x.dPR.clone()) for x in mats]
    native.shampoo_step_t(ents, hpn, ws)
    _sync()
    for x, (kl, kr) in zip(mats, keep):
        _oracle_step(x, hpo)
        assert rel_fro(from_dev(x.dU), x.U_or) <= 1e-5
        assert bool((x.dPL == kl).all()) and bool((x.dPR == kr).all())
        _check(x, hpo)


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
def test_shampoo_unaligned_caller_buffers_take_the_copy_path(native, refresh):
    """Tile-multiple sides use 16-byte aligned caller statistics and preconditioners where they lie
    and copy the others: the same step on the same values through both paths gives the same bits
    (the copies are exact and the arithmetic is the same)."""
    import torch
    _say(f"shampoo in place vs copied buffers, refresh {refresh}")
    m, n = 256, 384
    runs = []
    for offset in (False, True):
        x = _Mat(np.random.default_rng(4200 + refresh), m, n, synth.BF16, synth.BF16).device()
        S = _spd(np.random.default_rng(77), m, 10.0).astype(np.float32)
        T = _spd(np.random.default_rng(78), n, 10.0).astype(np.float32)
        x.dL.copy_(to_dev(S * 1e-3, synth.F32))
        x.dR.copy_(to_dev(T * 1e-3, synth.F32))
        x.dPL.copy_(to_dev(S, synth.F32))
        x.dPR.copy_(to_dev(T, synth.F32))
        if offset:
            x.dL, x.dR, x.dPL, x.dPR = (_offset_view(t) for t in (x.dL, x.dR, x.dPL, x.dPR))
        hpn, _ = _hp(native, refresh=refresh, beta=0.9, weight=0.1)
        ents = [x.entry(native)]
        native.shampoo_step_t(ents, hpn, native.shampoo_workspace_t(ents, hpn))
        _sync()
        runs.append([t.clone() for t in (x.dU, x.dL, x.dR, x.dPL, x.dPR, x.dp)])
    for a, b in zip(*runs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("eps_rel", [1e-6, 1e-4])
@pytest.mark.parametrize("dts", [(synth.BF16, synth.BF16), (synth.F32, synth.F32)])
def test_shampoo_stale_step_on_new_gradient_after_rank_deficient_refresh(native, eps_rel, dts):
    """Refresh from a rank-deficient left statistic (768 x 768 of rank 192), then a stale step
    (refresh = 0) on a new gradient whose columns lie mostly outside that statistic's range, so
    that P_L's null directions (eigenvalue rho^(-1/4)) dominate U. Compared with the oracle's stale
    step from its own fp64 preconditioners; U within the ridge bar."""
    import torch
    m, n = 768, 192
    _say(f"shampoo stale step on a new gradient, eps_rel {eps_rel:g}, {dts}")
    rng = np.random.default_rng(4100 + int(-np.log10(eps_rel)) + 10 * (dts[0] == synth.F32))
    mat = _Mat(rng, m, n, *dts).device()
    hpn, hpo = _hp(native, eps_rel=eps_rel, beta=0.95, weight=0.05)
    ws = native.shampoo_workspace_t([mat.entry(native)], hpn)
    native.shampoo_step_t([mat.entry(native)], hpn, ws)
    _sync()
    _oracle_step(mat, hpo)
    _check(mat, hpo)
    # the new gradient: its share of U that comes from outside the first statistic's range
    g2 = synth.random_muon_tensors(rng, m, n, dts[0], dts[1]).grad
    G1, G2 = OS._f64(mat.g), OS._f64(g2)
    Q, _ = np.linalg.qr(G1)
    outside = G2 - Q @ (Q.T @ G2)
    share = np.linalg.norm(mat.PL @ outside @ mat.PR) / np.linalg.norm(mat.PL @ G2 @ mat.PR)
    assert share > 0.9, share
    mat.g = g2
    mat.dg.copy_(to_dev(g2, mat.gdt))
    hpn2, hpo2 = _hp(native, eps_rel=eps_rel, beta=0.95, weight=0.05, refresh=False)
    pl0, pr0 = mat.dPL.clone(), mat.dPR.clone()
    native.shampoo_step_t([mat.entry(native)], hpn2, ws)
    _sync()
    _oracle_step(mat, hpo2)
    eu = rel_fro(from_dev(mat.dU), mat.U_or)
    bar = _ridge_tol(eps_rel)
    _say(f"  stale U rel err {eu:.3e} (bar {bar:.1e}; share of U outside the old range {share:.3f})")
    assert eu <= bar, eu
    assert torch.equal(pl0, mat.dPL) and torch.equal(pr0, mat.dPR)   # read, not written
    assert rel_fro(from_dev(mat.dL), mat.L) <= STAT_TOL
    assert rel_fro(from_dev(mat.dR), mat.R) <= STAT_TOL
    pg, un = from_dev(mat.dp), hpo2.lr * np.linalg.norm(mat.U_or)
    if mat.pdt == synth.BF16:
        assert check_bf16_param(pg, mat.p_or, un, bar) <= 1.0
    else:
        assert np.linalg.norm(pg - mat.p_or) <= bar * un + 1e-6 * np.linalg.norm(mat.p_or)


def test_shampoo_lr_zero_and_determinism(native):
    import torch
    _say("shampoo lr=0 and determinism")
    rng = np.random.default_rng(5000)
    mats = [_Mat(rng, m, n, synth.BF16, synth.BF16).device() for (m, n) in [(200, 96), (256, 512)]]
    hpn, _ = _hp(native, lr=0.0, weight_decay=0.0)
    ents = [x.entry(native) for x in mats]
    ws = native.shampoo_workspace_t(ents, hpn)
    p0 = [x.dp.clone() for x in mats]
    native.shampoo_step_t(ents, hpn, ws)
    _sync()
    u1 = [x.dU.clone() for x in mats]
    for x, p in zip(mats, p0):
        assert bool((x.dp.view(torch.int16) == p.view(torch.int16)).all())
        x.dL.zero_()
        x.dR.zero_()
    native.shampoo_step_t(ents, hpn, ws)
    _sync()
    for x, u in zip(mats, u1):
        assert bool((x.dU == u).all())


@pytest.mark.parametrize("p", [1, 2, 4])
def test_inverse_root_iteration_cap_beyond_convergence(native, p):
    """Iterations after convergence are skipped (the iterate is copied): a cap of 100 gives the
    result of 30 to within the convergence threshold's effect (2.5e-6 relative), and both match
    the oracle."""
    import torch
    _say(f"inverse root cap p={p}")
    d = 257
    rng = np.random.default_rng(7000 + p)
    a = _spd(rng, d, 1e4).astype(np.float32)
    ad = to_dev(a, synth.F32)
    outs = []
    for iters in (30, 100):
        out = torch.empty((d, d), dtype=torch.float32, device="cuda")
        native.inverse_root_t(ad, out, p=p, eps=1e-9, eps_rel=1e-6, iters=iters)
        _sync()
        outs.append(from_dev(out))
    ref = OS.inverse_root(a.astype(np.float64), p, 1e-9, 1e-6)
    assert rel_fro(outs[1], outs[0]) <= 5e-6
    assert rel_fro(outs[1], ref) <= 1e-4
    np.testing.assert_array_equal(outs[1], outs[1].T)   # stored exactly symmetric


def test_shampoo_benchmark_configuration_full_size(native):
    """The configuration bench.py --shampoo times: the GPT-2-small share's 12 matrices in one call,
    EMA statistics (beta 0.95, weight 0.05), ridge 1e-12 + 1e-6 ||S||_F, 20 root iterations, bf16
    parameters and gradients; every matrix against the oracle (two refresh steps, so the second sees
    EMA statistics, then a stale step on a third gradient, as timed too)."""
    import torch
    _say("shampoo benchmark configuration")
    wl = synth.workload(2)
    rng = np.random.default_rng(8000)
    mats = [_Mat(rng, e.m, e.n, synth.BF16, synth.BF16, g_std=0.02).device() for e in wl.muon]
    hpn, hpo = _hp(native, lr=1e-3, weight_decay=0.01, beta=0.95, weight=0.05)
    ents = [x.entry(native) for x in mats]
    ws = native.shampoo_workspace_t(ents, hpn)
    for step in range(2):
        if step == 1:
            for x in mats:
                x.g = synth.random_muon_tensors(rng, x.m, x.n, x.pdt, x.gdt, g_std=0.02).grad
                x.dg.copy_(to_dev(x.g, x.gdt))
        native.shampoo_step_t(ents, hpn, ws)
        _sync()
        for x in mats:
            _oracle_step(x, hpo)
    for x in mats:
        _check(x, hpo)
    # the stale step: the preconditioners are the oracle's fp32-rounded ones as stored on the device
    hpn2, hpo2 = _hp(native, lr=1e-3, weight_decay=0.01, beta=0.95, weight=0.05, refresh=False)
    keep = []
    for x in mats:
        x.g = synth.random_muon_tensors(rng, x.m, x.n, x.pdt, x.gdt, g_std=0.02).grad
        x.dg.copy_(to_dev(x.g, x.gdt))
        x.PL = from_dev(x.dPL).astype(np.float64)
        x.PR = from_dev(x.dPR).astype(np.float64)
        keep.append((x.dPL.clone(), x.dPR.clone()))
    native.shampoo_step_t(ents, hpn2, ws)
    _sync()
    for x, (kl, kr) in zip(mats, keep):
        _oracle_step(x, hpo2)
        assert rel_fro(from_dev(x.dU), x.U_or) <= 1e-5
        assert torch.equal(kl, x.dPL) and torch.equal(kr, x.dPR)
        _check(x, hpo2)
