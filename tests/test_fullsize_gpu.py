"""Full-size parity: whole owner shares through the C ABI in the launch configuration the benchmark
times (every matrix of the share in one mfsdp_muon_step call), checked against the fp64 oracle.

* Momentum: sampled elements of every matrix, recomputed one by one by the oracle (<= 1e-6).
* Update and parameters: the full oracle on one matrix of each distinct shape of the Llama shares
  (up to 28672 x 8192 and 8192 x 28672, about a minute of fp64 oracle each) and on the uneven
  plan's largest tall, largest wide, square and three smallest matrices (<= 2e-2 relative
  Frobenius over the matrix and <= 5e-2 on every 256 x 256 block of the update, so that a
  mis-addressed, transposed or stale block fails; rounding-aware for bf16 parameters).
* Every matrix, whatever its size: properties of the NS output that hold at any size. For any
  input every output singular value is at most p(s-) = 1.2024 (s- the local maximum of the
  quintic), so the largest singular value (power iteration on O O^T) and the mean squared singular
  value ||O||_F^2 / r are bounded by it. For Gaussian inputs with aspect ratio s / r >= 2 the
  smallest normalised singular value is about (1 - sqrt(r / s)) / sqrt(r) > 0.003 at these sizes,
  so after 5 steps every singular value is also at least p(s+) = 0.6818 and the mean squared
  singular value is bounded below by it. Bounds are widened by the bf16 tolerance.
* AdamW: sampled elements of the 128256 x 4096 embedding, the small tensors in full.
"""
import math
import sys

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import check_bf16_param, from_dev, rel_fro, tile_rel_errors, to_dev

pytestmark = pytest.mark.gpu

A, B, C = synth.NS_COEFFS
BAND_LO, BAND_HI = 0.6818315, 1.2023686
TOL = 2e-2
TILE_TOL = 5e-2   # per 256 x 256 block of the update


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run_share(wl, idx_muon, with_adamw, keep_host):
    """Run the listed Muon entries of a share (and its AdamW tensors) in one call each."""
    import torch
    from paper_2607_05895_amd import native
    pool = synth.thread_pool()
    host, dev, ents = {}, {}, []
    for i in idx_muon:
        e = wl.muon[i]
        t = synth.muon_entry(wl, i, pool)
        p = to_dev(t.param, e.param_dtype)
        g = to_dev(t.grad, e.grad_dtype)
        mo = to_dev(t.momentum, synth.F32)
        uo = torch.empty((e.m, e.n), dtype=torch.float32, device="cuda")
        dev[i] = (p, g, mo, uo)
        ents.append(native.muon_entry_t(p, g, mo, uo))
        host[i] = t if i in keep_host else synth.MuonTensors(None, t.grad, t.momentum)
    hp = wl.hp
    h = native.muon_hparams(lr=hp.lr, weight_decay=hp.weight_decay, momentum=hp.momentum,
                            nesterov=hp.nesterov, a=hp.a, b=hp.b, c=hp.c, ns_steps=hp.ns_steps,
                            eps=hp.eps, lr_adjust=hp.lr_adjust, ns_dtype=hp.ns_dtype)
    ws = native.muon_workspace_t(ents, h)
    native.muon_step_t(ents, h, ws)
    adam = {}
    if with_adamw and wl.adamw:
        aents = []
        for j, e in enumerate(wl.adamw):
            t = synth.adamw_entry(wl, j, pool)
            tens = (to_dev(t.param, e.param_dtype), to_dev(t.grad, e.grad_dtype),
                    to_dev(t.exp_avg, synth.F32), to_dev(t.exp_avg_sq, synth.F32))
            adam[j] = (t, tens)
            aents.append(native.adamw_entry_t(*tens))
        ah = wl.adamw_hp
        native.adamw_step_t(aents, lr=ah.lr, beta1=ah.beta1, beta2=ah.beta2, eps=ah.eps,
                            weight_decay=ah.weight_decay, step=ah.step)
    torch.cuda.synchronize()
    del ws
    return host, dev, adam


def _check_momentum_sampled(wl, host, dev, nsamp=8192):
    import torch
    rng = np.random.default_rng(123)
    for i, t in host.items():
        e = wl.muon[i]
        numel = e.m * e.n
        idx = rng.integers(0, numel, size=min(nsamp, numel))
        g = t.grad.reshape(-1)[idx]
        m0 = t.momentum.reshape(-1)[idx]
        buf, _ = oracle.momentum_update(g, m0, wl.hp.momentum, wl.hp.nesterov)
        got = from_dev(dev[i][2].reshape(-1)[torch.from_numpy(idx).cuda()])
        assert rel_fro(got, buf) <= 1e-6, (e.name, "momentum")


def _check_full(wl, i, host, dev):
    e = wl.muon[i]
    t = host[i]
    hp = wl.hp
    p_or, buf_or, O = oracle.muon_step(t.param, t.grad, t.momentum, lr=hp.lr,
                                       weight_decay=hp.weight_decay, momentum=hp.momentum,
                                       nesterov=hp.nesterov, a=hp.a, b=hp.b, c=hp.c,
                                       ns_steps=hp.ns_steps, eps=hp.eps, lr_adjust=hp.lr_adjust)
    p, _, mo, uo = dev[i]
    assert rel_fro(from_dev(mo), buf_or) <= 1e-6
    og = from_dev(uo)
    err = rel_fro(og, O)
    tiles = tile_rel_errors(og, O)
    worst = np.unravel_index(int(np.argmax(tiles)), tiles.shape)
    _say(f"  {e.name} {e.m}x{e.n}: update rel err {err:.3e}, worst 256-block {tiles.max():.3e} at {worst}")
    assert err <= TOL, (e.name, err)
    assert tiles.max() <= TILE_TOL, (e.name, worst, float(tiles.max()))
    f = oracle.lr_factor(e.m, e.n, hp.lr_adjust)
    ratio = check_bf16_param(from_dev(p), p_or, hp.lr * f * np.linalg.norm(O), TOL)
    assert ratio <= 1.0, (e.name, "param", ratio)


def _check_band(wl, i, dev, iters=30):
    import torch
    e = wl.muon[i]
    uo = dev[i][3]
    r = min(e.m, e.n)
    O = uo if e.m <= e.n else uo.t()
    msq = float((O.double() ** 2).sum()) / r
    assert msq <= (BAND_HI * (1 + TOL)) ** 2, (e.name, msq)
    if max(e.m, e.n) >= 2 * r:
        assert msq >= (BAND_LO * (1 - TOL)) ** 2, (e.name, msq)
    # largest singular value: power iteration on O O^T (fp32 products of the test's own)
    v = torch.randn(r, device="cuda", generator=torch.Generator("cuda").manual_seed(7))
    v /= v.norm()
    lam = 0.0
    for _ in range(iters):
        w = O @ (O.t() @ v)
        lam = float(w.norm())
        v = w / lam
    smax = math.sqrt(lam)
    assert smax <= BAND_HI * (1 + TOL), (e.name, smax)


# --------------------------------------------------------------------- Llama-3-8B share (bench)

@pytest.fixture(scope="module")
def llama8b():
    wl = synth.workload(3)
    first = {}
    for i, e in enumerate(wl.muon):
        first.setdefault((e.m, e.n), i)
    keep = set(first.values())
    _say(f"running {wl.name}: {len(wl.muon)} matrices in one call")
    host, dev, adam = _run_share(wl, list(range(len(wl.muon))), True, keep)
    yield wl, host, dev, adam, first
    dev.clear()
    import torch
    torch.cuda.empty_cache()


def test_llama8b_momentum_sampled(llama8b):
    wl, host, dev, _, _ = llama8b
    _check_momentum_sampled(wl, host, dev)


@pytest.mark.parametrize("shape", [(1024, 4096), (4096, 4096), (14336, 4096), (4096, 14336)])
def test_llama8b_full_oracle(llama8b, shape):
    wl, host, dev, _, first = llama8b
    _check_full(wl, first[shape], host, dev)


def test_llama8b_band_every_matrix(llama8b):
    wl, _, dev, _, _ = llama8b
    for i in range(len(wl.muon)):
        _check_band(wl, i, dev)


def test_llama8b_adamw(llama8b):
    wl, _, _, adam, _ = llama8b
    ah = wl.adamw_hp
    for j, (t, tens) in adam.items():
        p_or, m_or, v_or = oracle.adamw_step(t.param, t.grad, t.exp_avg, t.exp_avg_sq, lr=ah.lr,
                                             beta1=ah.beta1, beta2=ah.beta2, eps=ah.eps,
                                             weight_decay=ah.weight_decay, step=ah.step)
        assert rel_fro(from_dev(tens[2]), m_or) <= 1e-6
        assert rel_fro(from_dev(tens[3]), v_or) <= 1e-6


# --------------------------------------------------------------------- Llama-3-70B heavy share

@pytest.fixture(scope="module")
def llama70b():
    wl = synth.workload(5)
    first = {}
    for i, e in enumerate(wl.muon):
        first.setdefault((e.m, e.n), i)
    idx = sorted(first.values())
    _say(f"running {wl.name}: its {len(idx)} distinct shapes in one call")
    host, dev, _ = _run_share(wl, idx, False, set(idx))
    yield wl, host, dev, first
    dev.clear()
    import torch
    torch.cuda.empty_cache()


def test_llama70b_momentum_sampled(llama70b):
    wl, host, dev, _ = llama70b
    _check_momentum_sampled(wl, host, dev)


@pytest.mark.parametrize("shape", [(1024, 8192), (8192, 8192), (28672, 8192), (8192, 28672)])
def test_llama70b_full_oracle(llama70b, shape):
    wl, host, dev, first = llama70b
    _check_full(wl, first[shape], host, dev)


def test_llama70b_band(llama70b):
    wl, _, dev, _ = llama70b
    for i in dev:
        _check_band(wl, i, dev)


# --------------------------------------------------------------------- uneven owner plan + embedding

@pytest.fixture(scope="module")
def uneven():
    wl = synth.workload(4)
    def cost(i):
        m, n = wl.muon[i].m, wl.muon[i].n
        return (min(m, n), min(m, n) ** 2 * max(m, n))
    order = sorted(range(len(wl.muon)), key=cost)
    small = order[:3]
    tall = max((i for i in order if wl.muon[i].m > wl.muon[i].n), key=cost)
    wide = max((i for i in order if wl.muon[i].m < wl.muon[i].n), key=cost)
    square = [i for i in order if wl.muon[i].m == wl.muon[i].n]
    picked = {"smallest": small, "largest_tall": [tall], "largest_wide": [wide], "square": square}
    _say(f"running {wl.name}: {len(wl.muon)} matrices in one call + AdamW")
    keep = {i for v in picked.values() for i in v}
    host, dev, adam = _run_share(wl, list(range(len(wl.muon))), True, keep)
    yield wl, host, dev, adam, picked
    dev.clear()
    adam.clear()
    import torch
    torch.cuda.empty_cache()


def test_uneven_momentum_sampled(uneven):
    wl, host, dev, _, _ = uneven
    _check_momentum_sampled(wl, host, dev)


@pytest.mark.parametrize("which", ["smallest", "largest_tall", "largest_wide", "square"])
def test_uneven_full_oracle(uneven, which):
    wl, host, dev, _, picked = uneven
    assert picked[which], which
    for i in picked[which]:
        _check_full(wl, i, host, dev)


def test_uneven_band_every_matrix(uneven):
    wl, _, dev, _, _ = uneven
    for i in range(len(wl.muon)):
        _check_band(wl, i, dev, iters=20)


def test_uneven_adamw_embedding_sampled(uneven):
    import torch
    wl, _, _, adam, _ = uneven
    ah = wl.adamw_hp
    rng = np.random.default_rng(5)
    for j, (t, tens) in adam.items():
        numel = t.param.size
        idx = rng.integers(0, numel, size=min(1 << 16, numel)) if numel > (1 << 20) else np.arange(numel)
        p_or, m_or, v_or = oracle.adamw_step(t.param[idx], t.grad[idx], t.exp_avg[idx],
                                             t.exp_avg_sq[idx], lr=ah.lr, beta1=ah.beta1,
                                             beta2=ah.beta2, eps=ah.eps,
                                             weight_decay=ah.weight_decay, step=ah.step)
        ti = torch.from_numpy(idx).cuda()
        assert rel_fro(from_dev(tens[2][ti]), m_or) <= 1e-6
        assert rel_fro(from_dev(tens[3][ti]), v_or) <= 1e-6
        p0 = oracle.bf16_widen(t.param[idx]) if t.param.dtype == np.uint16 else t.param[idx]
        pg = from_dev(tens[0][ti])
        half = 0.5 * 2.0 ** (np.floor(np.log2(np.abs(p_or))) - 7)
        bound = half + 1e-6 * np.abs(p_or - p0) + 4 * 2.0 ** -24 * np.abs(p_or)
        assert np.all(np.abs(pg - p_or) <= bound)
