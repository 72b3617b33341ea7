"""GPU test of mfsdp_muon_step_noalloc (the Muon step for callers that cannot allocate) through the C
ABI: on two calls in a row, the second with a smaller input, its outputs (parameters, momentum and
the NS output) equal bitwise those of mfsdp_muon_step with a caller workspace on copies of the same
inputs, and both match the fp64 oracle at the bars of the other parity tests (update <= 2e-2
relative Frobenius on the bf16 path, 1e-4 on the fp32 path; momentum <= 1e-6; bf16 parameters
rounding-aware)."""
import sys

import numpy as np
import pytest

import oracle
import synth
from tests.helpers import check_bf16_param, from_dev, rel_fro, to_dev

pytestmark = pytest.mark.gpu

A, B, C = synth.NS_COEFFS


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _make(rng, shapes, pdt, gdt):
    """Host tensors and two device copies of each (one per entry point)."""
    import torch
    out = []
    for (m, n) in shapes:
        t = synth.random_muon_tensors(rng, m, n, pdt, gdt)
        copies = []
        for _ in range(2):
            copies.append((to_dev(t.param, pdt), to_dev(t.grad, gdt), to_dev(t.momentum, synth.F32),
                           torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")))
        out.append((m, n, t, copies))
    return out


def _compare(native, items, hp_kw, update_tol):
    import torch
    h = native.muon_hparams(**hp_kw)
    ents = [[native.muon_entry_t(*c[k]) for (_, _, _, c) in items] for k in range(2)]
    ws = native.muon_workspace_t(ents[0], h)
    assert ws.numel() <= native.NOALLOC_SCRATCH_BYTES
    native.muon_step_t(ents[0], h, ws)
    native.muon_step_noalloc_t(ents[1], h)
    torch.cuda.synchronize()
    for (m, n, t, c) in items:
        for a, b, what in zip(c[0], c[1], ("param", "grad", "momentum", "update_out")):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32)), \
                (m, n, what)
        p_or, buf_or, O = oracle.muon_step(t.param, t.grad, t.momentum, lr=hp_kw["lr"],
                                           weight_decay=hp_kw["weight_decay"], momentum=0.95,
                                           nesterov=True, a=A, b=B, c=C, ns_steps=5)
        p, _, mo, uo = c[1]
        err = rel_fro(from_dev(uo), O)
        _say(f"  noalloc {m}x{n}: update rel err {err:.3e}")
        assert err <= update_tol, (m, n, err)
        assert rel_fro(from_dev(mo), buf_or) <= 1e-6, (m, n)
        f = oracle.lr_factor(m, n, "original")
        ratio = check_bf16_param(from_dev(p), p_or, hp_kw["lr"] * f * np.linalg.norm(O), update_tol)
        assert ratio <= 1.0, (m, n, ratio)


def test_noalloc_matches_workspace_step_twice():
    import torch
    from paper_2607_05895_amd import native
    native.lib()
    assert torch.cuda.is_available()
    rng = np.random.default_rng(77)
    # first call: several bf16 matrices (tall, wide, ragged) in one call
    _say("noalloc call 1: 384x640, 640x384, 257x513, 1x300 (bf16)")
    first = _make(rng, [(384, 640), (640, 384), (257, 513), (1, 300)], synth.BF16, synth.BF16)
    _compare(native, first, dict(lr=0.02, weight_decay=0.01), 2e-2)
    # second call, smaller input: one matrix, on the same scratch array (which still holds the
    # first call's contents)
    _say("noalloc call 2: 200x96 (bf16)")
    second = _make(rng, [(200, 96)], synth.BF16, synth.BF16)
    _compare(native, second, dict(lr=0.02, weight_decay=0.01), 2e-2)


def test_noalloc_fp32_path_after_bf16():
    import torch
    from paper_2607_05895_amd import native
    rng = np.random.default_rng(78)
    items = _make(rng, [(256, 512)], synth.F32, synth.F32)
    h = dict(lr=0.02, weight_decay=0.0, ns_dtype="f32")
    hp = native.muon_hparams(**h)
    ents = [[native.muon_entry_t(*c[k]) for (_, _, _, c) in items] for k in range(2)]
    ws = native.muon_workspace_t(ents[0], hp)
    native.muon_step_t(ents[0], hp, ws)
    native.muon_step_noalloc_t(ents[1], hp)
    torch.cuda.synchronize()
    (m, n, t, c) = items[0]
    for a, b in zip(c[0], c[1]):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    _, buf_or, O = oracle.muon_step(t.param, t.grad, t.momentum, lr=0.02, weight_decay=0.0,
                                    momentum=0.95, nesterov=True, a=A, b=B, c=C, ns_steps=5)
    assert rel_fro(from_dev(c[1][3]), O) <= 1e-4
    assert rel_fro(from_dev(c[1][2]), buf_or) <= 1e-6


def test_noalloc_split_gram_contraction_matches_workspace_step():
    """One 768 x 3072 matrix alone: its Gram launch has 6 tiles with K = 3072, so both entry points
    split that contraction into K ranges (within the partial-tile budget of the plan they share);
    the outputs equal bitwise and match the oracle."""
    from paper_2607_05895_amd import native
    rng = np.random.default_rng(79)
    _say("noalloc call: 768x3072 (bf16, split Gram contraction)")
    items = _make(rng, [(768, 3072)], synth.BF16, synth.BF16)
    _compare(native, items, dict(lr=0.02, weight_decay=0.01), 2e-2)


def test_noalloc_rejects_entries_beyond_the_scratch():
    import torch
    from paper_2607_05895_amd import native
    m = n = 4096  # needs 192 MiB of workspace
    p = torch.zeros((m, n), dtype=torch.bfloat16, device="cuda")
    g = torch.ones((m, n), dtype=torch.bfloat16, device="cuda")
    mo = torch.zeros((m, n), dtype=torch.float32, device="cuda")
    with pytest.raises(native.MfsdpError) as ei:
        native.muon_step_noalloc_t([native.muon_entry_t(p, g, mo)], native.muon_hparams())
    assert ei.value.status == native.E_INVALID
    assert "MFSDP_NOALLOC_SCRATCH_BYTES" in str(ei.value)
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(mo)) == 0 and int(torch.count_nonzero(p)) == 0
