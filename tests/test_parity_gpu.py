"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the same seeded inputs.

Tolerances (relative Frobenius unless stated):
  NS output / update  <= 1e-4 on the fp32 NS path (shapes with short side <= 768),
                      <= 2e-2 on the bf16-MFMA path;
  Muon momentum       <= 1e-6;
  bf16 parameters     rounding-aware: ||P - P_or|| <= 2e-2 lr f ||O_or|| + ||half-ulp(P_or)||;
  AdamW               m, v <= 1e-6; p elementwise <= half-ulp(p_or) + 1e-6 |dp_or| + 4 ulp_f32.
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


# ------------------------------------------------------------------ standalone Newton-Schulz

NS_SHAPES_BF16 = [(256, 512), (512, 256), (100, 300), (300, 100), (257, 513), (768, 768),
                  (1, 300), (640, 1152), (1024, 4096), (513, 257)]


@pytest.mark.parametrize("shape", NS_SHAPES_BF16)
@pytest.mark.parametrize("steps", [1, 5])
def test_ns_bf16_matches_oracle(native, shape, steps):
    import torch
    m, n = shape
    _say(f"ns bf16 {m}x{n} steps={steps}")
    rng = np.random.default_rng(100 + m + 3 * n + steps)
    x = rng.standard_normal((m, n), dtype=np.float32)
    xb = synth.f32_to_bf16_bits(x)
    xd = to_dev(xb, synth.BF16)
    out = torch.empty((m, n), dtype=torch.float32, device="cuda")
    native.newton_schulz_t(xd, out, A, B, C, steps, 1e-7, "bf16")
    _sync()
    ref = oracle.newton_schulz(xb, A, B, C, steps)
    og = from_dev(out)
    err = rel_fro(og, ref)
    assert err <= 2e-2, err
    assert float(tile_rel_errors(og, ref).max()) <= 5e-2


@pytest.mark.parametrize("shape", [(256, 512), (512, 256), (100, 300), (65, 129), (768, 768), (3, 5)])
@pytest.mark.parametrize("steps", [0, 1, 5])
def test_ns_f32_matches_oracle(native, shape, steps):
    import torch
    m, n = shape
    _say(f"ns f32 {m}x{n} steps={steps}")
    rng = np.random.default_rng(200 + m + n + steps)
    x = rng.standard_normal((m, n), dtype=np.float32)
    xd = to_dev(x, synth.F32)
    out = torch.empty((m, n), dtype=torch.float32, device="cuda")
    native.newton_schulz_t(xd, out, A, B, C, steps, 1e-7, "f32")
    _sync()
    ref = oracle.newton_schulz(x, A, B, C, steps)
    err = rel_fro(from_dev(out), ref)
    assert err <= 1e-4, err


def test_ns_bf16_single_step_exact_products(native):
    # one NS step is a fixed polynomial of X0: checks the MFMA fragment/output layout and the
    # symmetric-tile mirroring on a matrix with several tiles per side
    import torch
    m, n = 768, 1280
    rng = np.random.default_rng(7)
    xb = synth.f32_to_bf16_bits(rng.standard_normal((m, n), dtype=np.float32))
    out = torch.empty((m, n), dtype=torch.float32, device="cuda")
    native.newton_schulz_t(to_dev(xb, synth.BF16), out, A, B, C, 1, 1e-7, "bf16")
    _sync()
    ref = oracle.newton_schulz(xb, A, B, C, 1)
    assert rel_fro(from_dev(out), ref) <= 1e-2


def test_ns_zero_input_gives_zero(native):
    import torch
    x = torch.zeros((300, 200), dtype=torch.bfloat16, device="cuda")
    out = torch.full((300, 200), 7.0, dtype=torch.float32, device="cuda")
    native.newton_schulz_t(x, out, A, B, C, 5, 1e-7, "bf16")
    _sync()
    assert float(out.abs().max()) == 0.0


def test_ns_bf16_output_dtype(native):
    import torch
    m, n = 200, 333
    rng = np.random.default_rng(8)
    x = rng.standard_normal((m, n), dtype=np.float32)
    out = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
    native.newton_schulz_t(to_dev(x, synth.F32), out, A, B, C, 5, 1e-7, "bf16")
    _sync()
    assert rel_fro(from_dev(out), oracle.newton_schulz(x, A, B, C, 5)) <= 2e-2


# ------------------------------------------------------------------ the Muon step

def _run_muon(native, tensors, specs, hp, with_update=True):
    import torch
    dev = []
    ents = []
    for t, e in zip(tensors, specs):
        p = to_dev(t.param, e.param_dtype)
        g = to_dev(t.grad, e.grad_dtype)
        mo = to_dev(t.momentum, synth.F32)
        uo = torch.empty((e.m, e.n), dtype=torch.float32, device="cuda") if with_update else None
        dev.append((p, g, mo, uo))
        ents.append(native.muon_entry_t(p, g, mo, uo))
    h = native.muon_hparams(lr=hp.lr, weight_decay=hp.weight_decay, momentum=hp.momentum,
                            nesterov=hp.nesterov, a=hp.a, b=hp.b, c=hp.c, ns_steps=hp.ns_steps,
                            eps=hp.eps, lr_adjust=hp.lr_adjust, ns_dtype=hp.ns_dtype,
                            ns_schedule=hp.ns_schedule)
    ws = native.muon_workspace_t(ents, h)
    native.muon_step_t(ents, h, ws)
    _sync()
    return dev


def _check_muon(tensors, specs, dev, hp, upd_tol):
    worst = 0.0
    for t, e, (p, g, mo, uo) in zip(tensors, specs, dev):
        p_or, buf_or, O = oracle.muon_step(
            t.param, t.grad, t.momentum, lr=hp.lr, weight_decay=hp.weight_decay,
            momentum=hp.momentum, nesterov=hp.nesterov, a=hp.a, b=hp.b, c=hp.c,
            ns_steps=hp.ns_steps, eps=hp.eps, lr_adjust=hp.lr_adjust, ns_schedule=hp.ns_schedule)
        assert rel_fro(from_dev(mo), buf_or) <= 1e-6, (e.name, "momentum")
        if uo is not None:
            og = from_dev(uo)
            err = rel_fro(og, O)
            worst = max(worst, err)
            assert err <= upd_tol, (e.name, e.m, e.n, err)
            # and on every 256 x 256 block, so that an error confined to one block shows
            tmax = float(tile_rel_errors(og, O).max())
            assert tmax <= 2.5 * upd_tol, (e.name, e.m, e.n, "worst block", tmax)
        f = oracle.lr_factor(e.m, e.n, hp.lr_adjust)
        pg = from_dev(p)
        if e.param_dtype == synth.BF16:
            ratio = check_bf16_param(pg, p_or, hp.lr * f * np.linalg.norm(O), upd_tol)
            assert ratio <= 1.0, (e.name, "param", ratio)
        else:
            # fp32 parameters: the step lr f O is compared through the parameter delta
            p0 = t.param.astype(np.float64)
            d_or, d_g = p_or - p0, pg - p0
            assert rel_fro(d_g, d_or) <= max(upd_tol, 1e-4) * 1.5, (e.name, "param delta")
    return worst


def test_muon_fp32_single_matrix_256x512(native):
    wl = synth.workload(1)
    _say(f"muon {wl.name}")
    tensors = [synth.muon_entry(wl, 0)]
    dev = _run_muon(native, tensors, wl.muon, wl.hp)
    _check_muon(tensors, wl.muon, dev, wl.hp, 1e-4)


def test_muon_gpt2_small_share(native):
    wl = synth.workload(2)
    _say(f"muon {wl.name}")
    tensors = [synth.muon_entry(wl, i) for i in range(len(wl.muon))]
    dev = _run_muon(native, tensors, wl.muon, wl.hp)
    _check_muon(tensors, wl.muon, dev, wl.hp, 2e-2)


@pytest.mark.parametrize("shape", [(2048, 4096), (4096, 2048), (1024, 4096), (2048, 2048)])
def test_muon_single_matrix_few_tiles(native, shape):
    """One matrix alone in a call, so that each launch has fewer 256 x 256 tiles than the GPU has
    CUs (2048 x 4096: 36 / 36 / 128, wide and tall, the last update with the fused parameter update);
    the Gram and square launches run on 128 x 128 tiles (136 upper ones; the Gram's K = 4096 in 2
    ranges). Matches the oracle and is bitwise reproducible."""
    import torch
    m, n = shape
    _say(f"muon single matrix {m}x{n}")
    rng = np.random.default_rng(5000 + m + n)
    specs = [synth.MuonSpec(m, n, f"s{m}x{n}")]
    tensors = [synth.random_muon_tensors(rng, m, n)]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)
    dev2 = _run_muon(native, tensors, specs, hp)
    for a, b in zip(dev[0], dev2[0]):
        assert torch.equal(a, b)


def test_muon_split_gram_contraction(native):
    """Two 1024 x 8192 matrices (wide and tall) alone in a call: their Gram launch runs on 128 x 128
    tiles (72 upper ones, K = 8192), so the contraction is split into K ranges (4 of 2048, within the
    partial-tile budget of a quarter of the per-matrix buffers); each range's fp32 partial tile is
    added in order by the second pass. Matches the oracle and is bitwise reproducible."""
    import torch
    _say("muon split Gram contraction: 1024x8192, 8192x1024")
    rng = np.random.default_rng(5100)
    specs = [synth.MuonSpec(1024, 8192, "wide"), synth.MuonSpec(8192, 1024, "tall")]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in specs]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)
    dev2 = _run_muon(native, tensors, specs, hp)
    for a, b in zip(dev[0], dev2[0]):
        assert torch.equal(a, b)


def test_muon_split_gram_contraction_full_size_tiles(native):
    """A 4096 x 4096 and a 1024 x 8192 matrix in one call: too many 128 x 128 tiles for one round
    (528 + 36), so every launch runs on 256 x 256 tiles, and the Gram launch (146 tiles) splits the
    1024 x 8192 matrix's K = 8192 into 2 ranges, summed by the 256 x 256 second pass. Matches the
    oracle and is bitwise reproducible."""
    import torch
    _say("muon split Gram contraction on 256 x 256 tiles: 4096x4096, 1024x8192")
    rng = np.random.default_rng(5200)
    specs = [synth.MuonSpec(4096, 4096, "square"), synth.MuonSpec(1024, 8192, "wide")]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in specs]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)
    dev2 = _run_muon(native, tensors, specs, hp)
    for a, b in zip(dev[0], dev2[0]):
        assert torch.equal(a, b)


def test_muon_small_and_full_size_tiles_give_the_same_bits(native):
    """Two 768 x 768 matrices stepped alone (their Gram and square launches run on 128 x 128 tiles)
    and again next to a 4096 x 4096 matrix (too many 128 x 128 tiles: every launch on 256 x 256
    tiles). Neither call splits a contraction, and each output element is accumulated over K in the
    same order on either tile, so the 768 x 768 matrices' parameters, momenta and updates agree
    bit for bit."""
    import torch
    _say("muon 128 x 128 vs 256 x 256 tiles: 2 x 768x768 alone and next to 4096x4096")
    rng = np.random.default_rng(5300)
    small = [synth.MuonSpec(768, 768, "a"), synth.MuonSpec(768, 768, "b")]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in small]
    big = synth.MuonSpec(4096, 4096, "big")
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    alone = _run_muon(native, tensors, small, hp)
    mixed = _run_muon(native, tensors + [synth.random_muon_tensors(rng, big.m, big.n)], small + [big], hp)
    for a, b in zip(alone, mixed[:2]):
        for x, y in zip(a[:1] + a[2:], b[:1] + b[2:]):  # param, momentum, update
            assert torch.equal(x, y)


MIXED = [(256, 512), (512, 256), (384, 384), (100, 700), (700, 100), (130, 1000), (1, 50),
         (50, 1), (768, 3072), (3072, 768)]


@pytest.mark.parametrize("mode", ["original", "match_rms_adamw", "none"])
def test_muon_mixed_shapes_and_lr_modes(native, mode):
    _say(f"muon mixed lr_adjust={mode}")
    rng = np.random.default_rng({"original": 1, "match_rms_adamw": 2, "none": 3}[mode])
    specs = [synth.MuonSpec(m, n, f"e{m}x{n}") for (m, n) in MIXED]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in specs]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.05, lr_adjust=mode)
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)


def test_muon_mixed_dtypes_fp32_grads_and_params(native):
    _say("muon mixed dtypes")
    rng = np.random.default_rng(11)
    specs = [synth.MuonSpec(300, 500, "a", synth.F32, synth.F32),
             synth.MuonSpec(500, 300, "b", synth.BF16, synth.F32),
             synth.MuonSpec(256, 256, "c", synth.F32, synth.BF16)]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n, e.param_dtype, e.grad_dtype) for e in specs]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)


def test_muon_paper_setting_two_steps(native):
    # Section 5.1: 2 NS steps, momentum 0.5, match_rms_adamw, lr 1e-3, wd 1e-2
    _say("muon paper setting")
    rng = np.random.default_rng(12)
    specs = [synth.MuonSpec(512, 1024, "w"), synth.MuonSpec(1024, 512, "t")]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in specs]
    hp = synth.MuonHParams(lr=1e-3, weight_decay=1e-2, momentum=0.5, ns_steps=2,
                           lr_adjust="match_rms_adamw")
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)


@pytest.mark.parametrize("case", ["k0", "no_nesterov", "zero_grad", "lr0"])
def test_muon_edge_cases(native, case):
    _say(f"muon edge {case}")
    rng = np.random.default_rng(13)
    specs = [synth.MuonSpec(320, 200, "x"), synth.MuonSpec(200, 320, "y")]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in specs]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    if case == "k0":
        hp.ns_steps = 0
    elif case == "no_nesterov":
        hp.nesterov = False
    elif case == "zero_grad":
        for t in tensors:
            t.grad[:] = 0
    elif case == "lr0":
        hp.lr = 0.0
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)
    if case == "lr0":
        for t, (p, *_rest) in zip(tensors, dev):
            import torch
            assert np.array_equal(p.view(torch.int16).cpu().numpy().view(np.uint16), t.param)


def test_muon_update_out_optional_and_deterministic(native):
    import torch
    _say("muon determinism")
    rng = np.random.default_rng(14)
    specs = [synth.MuonSpec(640, 896, "a"), synth.MuonSpec(896, 640, "b")]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in specs]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    d1 = _run_muon(native, tensors, specs, hp, with_update=False)
    d2 = _run_muon(native, tensors, specs, hp, with_update=True)
    for (p1, _, m1, _), (p2, _, m2, _) in zip(d1, d2):
        assert torch.equal(p1.view(torch.int16), p2.view(torch.int16))
        assert torch.equal(m1, m2)


@pytest.mark.parametrize("ns_dtype", ["bf16", "f32"])
def test_muon_tiny_degenerate_shapes(native, ns_dtype):
    """Matrices far below one tile (1x1, single rows and columns, 2x2, 3x3, 16x16) grouped in one
    call: zero padding must leave their NS iterates exact on the padded tiles. A 1x1 or single-row
    matrix has one normalised singular value, 1, so its update is the scalar quintic iterated on 1."""
    _say(f"muon tiny shapes {ns_dtype}")
    rng = np.random.default_rng(16)
    shapes = [(1, 1), (1, 2), (2, 1), (2, 2), (3, 3), (1, 257), (257, 1), (16, 16)]
    specs = [synth.MuonSpec(m, n, f"t{m}x{n}", synth.BF16, synth.BF16) for (m, n) in shapes]
    tensors = [synth.random_muon_tensors(rng, m, n) for (m, n) in shapes]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01, ns_dtype=ns_dtype)
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2 if ns_dtype == "bf16" else 1e-4)


def test_muon_two_consecutive_steps(native):
    # state carried across calls on the same workspace
    import torch
    _say("muon two steps")
    rng = np.random.default_rng(15)
    specs = [synth.MuonSpec(384, 512, "a")]
    t = synth.random_muon_tensors(rng, 384, 512)
    g2 = synth.f32_to_bf16_bits(rng.standard_normal((384, 512), dtype=np.float32) * np.float32(1e-3))
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    p = to_dev(t.param, synth.BF16); g = to_dev(t.grad, synth.BF16); mo = to_dev(t.momentum, synth.F32)
    uo = torch.empty((384, 512), dtype=torch.float32, device="cuda")
    ents = [native.muon_entry_t(p, g, mo, uo)]
    h = native.muon_hparams(lr=0.02, weight_decay=0.01)
    ws = native.muon_workspace_t(ents, h)
    native.muon_step_t(ents, h, ws)
    g.copy_(to_dev(g2, synth.BF16))
    native.muon_step_t(ents, h, ws)
    _sync()
    _, buf1, _ = oracle.muon_step(t.param, t.grad, t.momentum, lr=0.02, weight_decay=0.01,
                                  momentum=0.95, nesterov=True, a=A, b=B, c=C, ns_steps=5)
    _, buf2, O2 = oracle.muon_step(t.param, g2, buf1, lr=0.02, weight_decay=0.01, momentum=0.95,
                                   nesterov=True, a=A, b=B, c=C, ns_steps=5)
    assert rel_fro(from_dev(mo), buf2) <= 1e-6
    assert rel_fro(from_dev(uo), O2) <= 2e-2


# ------------------------------------------------------------------ AdamW

@pytest.mark.parametrize("step", [1, 7])
def test_adamw_matches_oracle(native, step):
    import torch
    _say(f"adamw step={step}")
    rng = np.random.default_rng(20 + step)
    cases = [(768, synth.BF16, synth.BF16), (1001, synth.F32, synth.F32), (4096 * 3 + 5, synth.BF16, synth.F32),
             (3, synth.F32, synth.BF16), (70000, synth.BF16, synth.BF16)]
    host, ents, devs = [], [], []
    for (numel, pdt, gdt) in cases:
        p32 = (1 + 0.02 * rng.standard_normal(numel)).astype(np.float32)
        g32 = (0.02 * rng.standard_normal(numel)).astype(np.float32)
        pa = synth.f32_to_bf16_bits(p32) if pdt == synth.BF16 else p32
        ga = synth.f32_to_bf16_bits(g32) if gdt == synth.BF16 else g32
        if step == 1:
            m0 = np.zeros(numel, np.float32); v0 = np.zeros(numel, np.float32)
        else:
            m0 = (0.01 * rng.standard_normal(numel)).astype(np.float32)
            v0 = (1e-4 * rng.random(numel)).astype(np.float32)
        pd, gd = to_dev(pa, pdt), to_dev(ga, gdt)
        md, vd = to_dev(m0, synth.F32), to_dev(v0, synth.F32)
        ents.append(native.adamw_entry_t(pd, gd, md, vd))
        devs.append((pd, md, vd, gd))  # every buffer stays alive until the kernel has run
        host.append((pa, ga, m0, v0, pdt))
    kw = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2)
    native.adamw_step_t(ents, step=step, **kw)
    _sync()
    for (pa, ga, m0, v0, pdt), (pd, md, vd, _gd) in zip(host, devs):
        p_or, m_or, v_or = oracle.adamw_step(pa, ga, m0, v0, step=step, **kw)
        assert rel_fro(from_dev(md), m_or) <= 1e-6
        assert rel_fro(from_dev(vd), v_or) <= 1e-6
        p0 = oracle.bf16_widen(pa) if pa.dtype == np.uint16 else pa.astype(np.float64)
        pg = from_dev(pd)
        half = (0.5 * 2.0 ** (np.floor(np.log2(np.abs(p_or))) - 7) if pdt == synth.BF16
                else np.zeros_like(p_or))
        bound = half + 1e-6 * np.abs(p_or - p0) + 4 * 2.0 ** -24 * np.abs(p_or)
        assert np.all(np.abs(pg - p_or) <= bound), float(np.max(np.abs(pg - p_or) - bound))


# ------------------------------------------------------------------ per-step NS coefficient schedules

# Schedules that keep every singular value bounded (a schedule that lets them grow, e.g. random
# perturbations of the triple, amplifies bf16 rounding beyond the tolerance on the bf16 path, in the
# kernel and in a CPU emulation of its rounding alike):
# two steps of the fixed triple, then three of the quintic p(s) = (15 s - 10 s^3 + 3 s^5) / 8
# (p(1) = 1, p'(1) = p''(1) = 0)
PADE_SCHEDULE = [(A, B, C)] * 2 + [(1.875, -1.25, 0.375)] * 3
# three quintic steps then the textbook cubic iteration (a, b, c) = (1.5, -0.5, 0)
MIXED_SCHEDULE = [(A, B, C)] * 3 + [(1.5, -0.5, 0.0)] * 3


@pytest.mark.parametrize("ns_dtype,tol", [("bf16", 2e-2), ("f32", 1e-4)])
@pytest.mark.parametrize("shape", [(256, 512), (513, 257), (100, 700)])
@pytest.mark.parametrize("which", ["pade", "mixed"])
def test_ns_schedule_matches_oracle(native, ns_dtype, tol, shape, which):
    import torch
    m, n = shape
    sched = PADE_SCHEDULE if which == "pade" else MIXED_SCHEDULE
    _say(f"ns schedule {which} {ns_dtype} {m}x{n}")
    rng = np.random.default_rng(310 + m + n)
    x = rng.standard_normal((m, n), dtype=np.float32)
    xd = to_dev(x, synth.F32)
    out = torch.empty((m, n), dtype=torch.float32, device="cuda")
    native.newton_schulz_schedule_t(xd, out, sched, 1e-7, ns_dtype)
    _sync()
    ref = oracle.newton_schulz(x, A, B, C, len(sched), schedule=sched)
    err = rel_fro(from_dev(out), ref)
    assert err <= tol, err


@pytest.mark.parametrize("ns_dtype", ["bf16", "f32"])
def test_ns_constant_schedule_is_bitwise_the_fixed_triple(native, ns_dtype):
    import torch
    m, n = 384, 640
    rng = np.random.default_rng(320)
    xd = to_dev(rng.standard_normal((m, n), dtype=np.float32), synth.F32)
    o1 = torch.empty((m, n), dtype=torch.float32, device="cuda")
    o2 = torch.empty_like(o1)
    native.newton_schulz_t(xd, o1, A, B, C, 5, 1e-7, ns_dtype)
    native.newton_schulz_schedule_t(xd, o2, [(A, B, C)] * 5, 1e-7, ns_dtype)
    _sync()
    assert torch.equal(o1, o2)


def test_muon_with_schedule_matches_oracle(native):
    _say("muon schedule")
    rng = np.random.default_rng(330)
    shapes = [(256, 512), (512, 256), (100, 700), (700, 100), (384, 384)]
    specs = [synth.MuonSpec(m, n, f"s{m}x{n}") for (m, n) in shapes]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n) for e in specs]
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01, ns_steps=5, ns_schedule=tuple(PADE_SCHEDULE))
    dev = _run_muon(native, tensors, specs, hp)
    _check_muon(tensors, specs, dev, hp, 2e-2)


# ------------------------------------------------------------------ owner-side gradient reduction

def _parts(rng, W, m, n, dtype):
    return [synth.f32_to_bf16_bits((rng.standard_normal((m, n)) * 1e-3).astype(np.float32))
            if dtype == synth.BF16 else (rng.standard_normal((m, n)) * 1e-3).astype(np.float32)
            for _ in range(W)]


@pytest.mark.parametrize("W", [1, 3, 8, 64])
@pytest.mark.parametrize("gdt", [synth.BF16, synth.F32])
def test_muon_reduce_matches_oracle(native, W, gdt):
    import torch
    _say(f"muon reduce W={W} grad={gdt}")
    rng = np.random.default_rng(400 + W)
    shapes = [(256, 512), (512, 256), (100, 700), (300, 101), (1, 50)]
    specs = [synth.MuonSpec(m, n, f"r{m}x{n}", synth.BF16, gdt) for (m, n) in shapes]
    tensors = [synth.random_muon_tensors(rng, e.m, e.n, e.param_dtype, gdt) for e in specs]
    parts = [_parts(rng, W, e.m, e.n, gdt) for e in specs]
    scale = 1.0 / W
    hp = synth.MuonHParams(lr=0.02, weight_decay=0.01)
    dev, ents, dparts, outs = [], [], [], []
    for i, (t, e) in enumerate(zip(tensors, specs)):
        p = to_dev(t.param, e.param_dtype)
        mo = to_dev(t.momentum, synth.F32)
        uo = torch.empty((e.m, e.n), dtype=torch.float32, device="cuda")
        dev.append((p, None, mo, uo))
        dparts.append([to_dev(x, gdt) for x in parts[i]])
        # the entry's grad is not read by the reduce step; its dtype names the parts' dtype
        ents.append(native.muon_entry_t(p, dparts[-1][0], mo, uo))
        outs.append(torch.empty((e.m, e.n), dtype=torch.bfloat16 if gdt == synth.BF16 else torch.float32,
                                device="cuda") if i % 2 == 0 else None)
    h = native.muon_hparams(lr=hp.lr, weight_decay=hp.weight_decay, momentum=hp.momentum,
                            nesterov=hp.nesterov, ns_steps=hp.ns_steps, eps=hp.eps,
                            lr_adjust=hp.lr_adjust, ns_dtype=hp.ns_dtype)
    ws = native.muon_workspace_t(ents, h)
    native.muon_step_reduce_t(ents, dparts, scale, h, ws, reduced_out=outs)
    _sync()
    for i, (t, e) in enumerate(zip(tensors, specs)):
        g = oracle.reduce_gradients(parts[i], scale)
        if outs[i] is not None:
            got = from_dev(outs[i])
            if gdt == synth.BF16:
                half = 0.5 * 2.0 ** (np.floor(np.log2(np.maximum(np.abs(g), 1e-30))) - 7)
                assert np.all(np.abs(got - g) <= half + 1e-6 * np.abs(g)), (e.name, "reduced bf16")
            else:
                assert rel_fro(got, g) <= 1e-6, (e.name, "reduced f32")
        tt = synth.MuonTensors(t.param, g, t.momentum)
        _check_muon([tt], [e], [dev[i]], hp, 2e-2)


def test_muon_reduce_single_part_is_bitwise_the_plain_step(native):
    import torch
    rng = np.random.default_rng(410)
    m, n = 384, 640
    t = synth.random_muon_tensors(rng, m, n)
    h = native.muon_hparams(lr=0.02, weight_decay=0.01)
    res = []
    for mode in ("plain", "reduce"):
        p = to_dev(t.param, synth.BF16)
        g = to_dev(t.grad, synth.BF16)
        mo = to_dev(t.momentum, synth.F32)
        e = native.muon_entry_t(p, g, mo)
        ws = native.muon_workspace_t([e], h)
        if mode == "plain":
            native.muon_step_t([e], h, ws)
        else:
            native.muon_step_reduce_t([e], [[g]], 1.0, h, ws)
        _sync()
        res.append((p.clone(), mo.clone()))
    assert torch.equal(res[0][0], res[1][0]) and torch.equal(res[0][1], res[1][1])
