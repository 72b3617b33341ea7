"""The torch.optim front ends (paper_2607_05895_amd.optim) against the fp64 oracle: two steps of a
small owner share (2D weights on Muon, Shampoo or SOAP, vectors on AdamW) with state carried by
the optimizer, and a state_dict round trip. Tolerances as in the kernel parity tests."""
import numpy as np
import pytest

import oracle
import synth
from oracle import shampoo as OS
from oracle import soap as OSP
from tests.helpers import check_bf16_param, from_dev, rel_fro, to_dev

pytestmark = pytest.mark.gpu


def _model(rng):
    """(name, param bits/array, dtype) of a tiny decoder block: 3 matrices and 3 vectors."""
    out = []
    for name, shape in (("q", (256, 256)), ("up", (512, 256)), ("down", (256, 512))):
        t = synth.random_muon_tensors(rng, *shape, synth.BF16, synth.BF16, g_std=1e-3)
        out.append((name, t.param, [t.grad, synth.random_muon_tensors(rng, *shape).grad], synth.BF16))
    for name, n in (("ln.w", 256), ("ln.b", 256), ("bias", 512)):
        p = rng.standard_normal(n).astype(np.float32)
        out.append((name, p, [(rng.standard_normal(n) * 1e-2).astype(np.float32) for _ in range(2)],
                    synth.F32))
    return out


def _torch_params(model):
    import torch
    ps, grads = [], []
    for name, p, gs, dt in model:
        t = to_dev(p, dt).clone()
        t.requires_grad_(True)
        ps.append(t)
        grads.append([to_dev(g, dt) for g in gs])
    return ps, grads


def test_owner_muon_two_steps_match_oracle():
    from paper_2607_05895_amd.optim import OwnerMuon
    rng = np.random.default_rng(11)
    model = _model(rng)
    ps, grads = _torch_params(model)
    opt = OwnerMuon(ps, lr=0.02, weight_decay=0.01, momentum=0.95, adamw_lr=1e-3, adamw_weight_decay=0.01)
    for step in range(2):
        for p, g in zip(ps, grads):
            p.grad = g[step]
        opt.step()
    import torch
    torch.cuda.synchronize()
    for (name, p0, gs, dt), p in zip(model, ps):
        if p.dim() == 2:
            buf = np.zeros(p0.shape)
            pin = p0
            for step in range(2):
                pout, buf, O = oracle.muon_step(pin, gs[step], buf, lr=0.02, weight_decay=0.01, momentum=0.95,
                                                nesterov=True, a=3.4445, b=-4.7750, c=2.0315, ns_steps=5)
                pin = synth.f32_to_bf16_bits(pout.astype(np.float32))
            assert rel_fro(from_dev(opt.state[p]["momentum_buffer"]), buf) <= 1e-6, name
            f = max(1.0, p0.shape[0] / p0.shape[1]) ** 0.5
            assert check_bf16_param(from_dev(p.detach()), pout, 0.02 * f * np.linalg.norm(O), 2e-2) <= 1.0, name
        else:
            pin, m, v = p0.astype(np.float64), np.zeros(p0.shape), np.zeros(p0.shape)
            for step in range(2):
                pin, m, v = oracle.adamw_step(pin.astype(np.float32), gs[step], m, v, lr=1e-3, beta1=0.9,
                                              beta2=0.999, eps=1e-8, weight_decay=0.01, step=step + 1)
            assert opt.state[p]["step"] == 2
            assert rel_fro(from_dev(opt.state[p]["exp_avg"]), m) <= 1e-6, name
            assert rel_fro(from_dev(opt.state[p]["exp_avg_sq"]), v) <= 1e-6, name
            assert np.abs(from_dev(p.detach()) - pin).max() <= 1e-6 * np.abs(pin).max() + 1e-7, name


def test_owner_shampoo_refresh_then_stale_matches_oracle():
    from paper_2607_05895_amd.optim import OwnerShampoo
    import torch
    rng = np.random.default_rng(12)
    # the same gradient at both steps: it stays in the range of the step-0 statistics, where the
    # stale preconditioners are accurate; recomputing them at step 1 (from twice the statistic)
    # would scale U by 2^(-1/2), so the refresh schedule is checked
    model = [(n, p, [gs[0], gs[0]], dt) for n, p, gs, dt in _model(rng) if dt == synth.BF16]
    ps, grads = _torch_params(model)
    opt = OwnerShampoo(ps, lr=0.05, weight_decay=0.01, beta=1.0, weight=1.0, precondition_frequency=2)
    for step in range(2):
        for p, g in zip(ps, grads):
            p.grad = g[step]
        opt.step()
    torch.cuda.synchronize()
    for (name, p0, gs, dt), p in zip(model, ps):
        m, n = p0.shape
        L, R, PL, PR, pin = np.zeros((m, m)), np.zeros((n, n)), None, None, p0
        for step in range(2):
            hp = OS.ShampooHParams(lr=0.05, weight_decay=0.01, beta=1.0, weight=1.0, eps=1e-12, eps_rel=1e-6,
                                   refresh=step == 0)
            pout, L, R, PL, PR, U = OS.shampoo_step(pin, gs[step], L, R, PL, PR, hp)
            pin = synth.f32_to_bf16_bits(pout.astype(np.float32))
        st = opt.state[p]
        assert rel_fro(from_dev(st["L"]), L) <= 1e-5 and rel_fro(from_dev(st["R"]), R) <= 1e-5, name
        tol = 1e-4 if min(m, n) <= 0.75 * max(m, n) else 5e-4
        assert check_bf16_param(from_dev(p.detach()), pout, 0.05 * np.linalg.norm(U), tol) <= 1.0, name


def _well_conditioned_grads(rng, d, k):
    """k gradients U diag(s) V^T with s in [0.5, 1] 1e-3: square and well conditioned, so every
    statistic and every refreshed basis is fully determined (float32 resolves it to ~1e-6)."""
    out = []
    for _ in range(k):
        U, _r = np.linalg.qr(rng.standard_normal((d, d)))
        V, _r = np.linalg.qr(rng.standard_normal((d, d)))
        g = (U * (1e-3 * rng.uniform(0.5, 1.0, d))) @ V.T
        out.append(g.astype(np.float32))
    return out


def test_owner_soap_three_steps_match_oracle():
    """Refresh after step 1 and step 3 (precondition_frequency 3), AdamW on the vectors."""
    from paper_2607_05895_amd.optim import OwnerSOAP
    import torch
    rng = np.random.default_rng(14)
    model = []
    for name, d in (("q", 256), ("o", 128)):
        p = synth.random_muon_tensors(rng, d, d, synth.BF16, synth.BF16).param
        model.append((name, p, [synth.f32_to_bf16_bits(g) for g in _well_conditioned_grads(rng, d, 3)],
                      synth.BF16))
    for name, n in (("ln.w", 256), ("bias", 128)):
        p = rng.standard_normal(n).astype(np.float32)
        model.append((name, p, [(rng.standard_normal(n) * 1e-2).astype(np.float32) for _ in range(3)],
                      synth.F32))
    ps, grads = _torch_params(model)
    opt = OwnerSOAP(ps, lr=3e-3, weight_decay=0.01, precondition_frequency=3)
    for step in range(3):
        for p, g in zip(ps, grads):
            p.grad = g[step]
        opt.step()
    torch.cuda.synchronize()
    for (name, p0, gs, dt), p in zip(model, ps):
        if p0.ndim == 1:
            pin, m_, v_ = p0, np.zeros_like(p0), np.zeros_like(p0)
            for step in range(3):
                pin, m_, v_ = oracle.adamw_step(pin, gs[step], m_, v_, lr=1e-3, beta1=0.9, beta2=0.999,
                                                eps=1e-8, weight_decay=0.01, step=step + 1)
                pin = pin.astype(np.float32)
            assert np.abs(from_dev(p.detach()) - pin).max() <= 1e-6, name
            continue
        d = p0.shape[0]
        M, V, L, R = np.zeros((d, d)), np.zeros((d, d)), np.zeros((d, d)), np.zeros((d, d))
        QL, QR, pin = np.eye(d), np.eye(d), p0
        for step in range(3):
            hp = OSP.SoapHParams(lr=3e-3, weight_decay=0.01, refresh=step in (0, 2))
            pout, M, V, L, R, QL, QR, N = OSP.soap_step(pin, gs[step], M, V, L, R, QL, QR, step + 1, hp)
            pin = synth.f32_to_bf16_bits(pout.astype(np.float32))
        st = opt.state[p]
        assert st["step"] == 3
        assert rel_fro(from_dev(st["exp_avg"]), M) <= 1e-5, name
        assert rel_fro(from_dev(st["L"]), L) <= 1e-5 and rel_fro(from_dev(st["R"]), R) <= 1e-5, name
        for q, qo in ((from_dev(st["QL"]), QL), (from_dev(st["QR"]), QR)):
            s_ = np.sign(np.sum(q * qo, axis=0))
            assert rel_fro(q * s_, qo) <= 1e-4, name
        assert check_bf16_param(from_dev(p.detach()), pout, 3e-3 * np.linalg.norm(N), 1e-4) <= 1.0, name


def test_owner_soap_on_llama_layer_shapes():
    """OwnerSOAP on Llama-3-8B layer shapes over two steps (refresh after the first): the FFN
    matrices 14336 x 4096 and 4096 x 14336 keep a 4096 x 4096 basis on their short side only (the
    long side is beyond max_precond_dim = 4096), a 4096 x 4096 matrix has both; against the oracle.
    Gradients with a well-conditioned spectrum on the square matrix, so that its refreshed bases are
    unique up to column signs."""
    from paper_2607_05895_amd.optim import OwnerSOAP
    import torch
    rng = np.random.default_rng(15)
    model = []
    for name, (m, n) in (("gate", (14336, 4096)), ("down", (4096, 14336))):
        p = synth.random_muon_tensors(rng, m, n, synth.BF16, synth.BF16).param
        gs = [synth.random_muon_tensors(rng, m, n, synth.BF16, synth.BF16).grad for _ in range(2)]
        model.append((name, p, gs, synth.BF16))
    p = synth.random_muon_tensors(rng, 4096, 4096, synth.BF16, synth.BF16).param
    model.append(("wq", p, [synth.f32_to_bf16_bits(g) for g in _well_conditioned_grads(rng, 4096, 2)], synth.BF16))
    ps, grads = _torch_params(model)
    opt = OwnerSOAP(ps, lr=3e-3, weight_decay=0.01, precondition_frequency=10)
    for step in range(2):
        for p_, g in zip(ps, grads):
            p_.grad = g[step]
        opt.step()
    torch.cuda.synchronize()
    for (name, p0, gs, dt), p_ in zip(model, ps):
        m, n = p0.shape
        st = opt.state[p_]
        assert ("L" in st) == (m <= 4096) and ("R" in st) == (n <= 4096), name
        M, V = np.zeros((m, n)), np.zeros((m, n))
        L = np.zeros((m, m)) if m <= 4096 else None
        R = np.zeros((n, n)) if n <= 4096 else None
        QL = np.eye(m) if m <= 4096 else None
        QR = np.eye(n) if n <= 4096 else None
        pin = p0
        for step in range(2):
            hp = OSP.SoapHParams(lr=3e-3, weight_decay=0.01, refresh=step == 0)
            pout, M, V, L, R, QL, QR, N = OSP.soap_step(pin, gs[step], M, V, L, R, QL, QR, step + 1, hp)
            pin = synth.f32_to_bf16_bits(pout.astype(np.float32))
        assert rel_fro(from_dev(st["exp_avg"]), M) <= 1e-5, name
        assert rel_fro(from_dev(st["exp_avg_sq"]), V) <= 1e-5, name
        for key, S_ref, Q_ref in (("L", L, QL), ("R", R, QR)):
            if S_ref is None:
                continue
            assert rel_fro(from_dev(st[key]), S_ref) <= 1e-5, (name, key)
            q = from_dev(st["Q" + key])
            s_ = np.sign(np.sum(q * Q_ref, axis=0))
            assert rel_fro(q * s_, Q_ref) <= 1e-4, (name, "Q" + key)
        assert check_bf16_param(from_dev(p_.detach()), pout, 3e-3 * np.linalg.norm(N), 1e-4) <= 1.0, name


@pytest.mark.parametrize("which", ["muon", "shampoo", "soap"])
def test_state_dict_round_trip_continues_identically(which):
    """Three steps, the optimizer rebuilt from its state_dict after the first: the parameters end
    bitwise the same. With precondition_frequency 2 the Shampoo steps after the resume are a stale
    one (it needs the saved preconditioners) and a refresh; the SOAP ones a refresh and a stale one."""
    from paper_2607_05895_amd.optim import OwnerMuon, OwnerShampoo, OwnerSOAP
    import torch
    rng = np.random.default_rng(13)
    model = _model(rng)
    cls, kw = {"muon": (OwnerMuon, dict(lr=0.02)),
               "shampoo": (OwnerShampoo, dict(precondition_frequency=2)),
               "soap": (OwnerSOAP, dict(precondition_frequency=2))}[which]
    runs = []
    for resume in (False, True):
        ps, grads = _torch_params(model)
        opt = cls(ps, **kw)
        for k in range(3):
            for p, g in zip(ps, grads):
                p.grad = g[k % len(g)]
            opt.step()
            if resume and k == 0:
                sd = opt.state_dict()
                opt = cls(ps, **kw)
                opt.load_state_dict(sd)
        torch.cuda.synchronize()
        runs.append([p.detach().clone() for p in ps])
    for a, b in zip(*runs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("which", ["muon", "shampoo", "soap"])
def test_empty_parameters_change_nothing(which):
    """An empty matrix and an empty vector in the group (nothing to update) leave the other
    parameters' updates bitwise as without them, and get no state."""
    from paper_2607_05895_amd.optim import OwnerMuon, OwnerShampoo, OwnerSOAP
    import torch
    rng = np.random.default_rng(17)
    model = _model(rng)
    cls = {"muon": OwnerMuon, "shampoo": OwnerShampoo, "soap": OwnerSOAP}[which]
    runs = []
    for with_empty in (False, True):
        ps, grads = _torch_params(model)
        extra = []
        if with_empty:
            for shape in ((0, 256), (0,)):
                e = torch.zeros(shape, dtype=torch.bfloat16, device="cuda", requires_grad=True)
                e.grad = torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
                extra.append(e)
        opt = cls(extra + ps)
        for k in range(2):
            for p, g in zip(ps, grads):
                p.grad = g[k]
            opt.step()
        torch.cuda.synchronize()
        assert all(e not in opt.state for e in extra)
        runs.append([p.detach().clone() for p in ps])
    for a, b in zip(*runs):
        assert torch.equal(a, b)
