"""Host-side tests of the C ABI that need no GPU: the library loads, exports every symbol the header
declares, and rejects invalid arguments before anything is enqueued."""
import ctypes
import os
import re

import pytest

from paper_2607_05895_amd import native

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    text = open(os.path.join(ROOT, "include", "mfsdp.h")).read()
    return sorted(set(re.findall(r"\b(mfsdp_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = native.lib()
    decl = _declared_symbols()
    assert set(decl) == set(native.EXPORTS)
    for name in decl:
        assert hasattr(L, name), name


def test_abi_version_and_status_strings():
    assert native.mfsdp_abi_version() == native.ABI_VERSION == 6
    assert native.mfsdp_status_string(0) == "MFSDP_OK"
    assert native.mfsdp_status_string(-1) == "MFSDP_E_INVALID"
    assert native.mfsdp_status_string(-2) == "MFSDP_E_WORKSPACE"
    assert native.mfsdp_status_string(-3) == "MFSDP_E_HIP"


FAKE = 1 << 20  # a 16-byte aligned non-NULL address; never dereferenced (validation fails first)


def _entry(**kw):
    d = dict(param=FAKE, grad=FAKE * 2, momentum=FAKE * 3, m=64, n=128, param_dtype=1,
             grad_dtype=1, update_out=None)
    d.update(kw)
    return native.MuonEntry(**d)


@pytest.mark.parametrize("bad", [
    dict(m=0), dict(n=-1), dict(param=None), dict(grad=None), dict(momentum=None),
    dict(param_dtype=7), dict(grad_dtype=-1), dict(param=FAKE + 8), dict(update_out=FAKE + 4),
])
def test_muon_rejects_bad_entries(bad):
    hp = native.muon_hparams()
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step([_entry(), _entry(**bad)], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


@pytest.mark.parametrize("bad", [
    dict(ns_steps=100), dict(ns_steps=-1), dict(lr=-1.0), dict(weight_decay=-0.1),
    dict(momentum=1.0), dict(momentum=-0.5), dict(eps=0.0), dict(lr_adjust=3), dict(ns_dtype=5),
    dict(a=float("inf")),
])
def test_muon_rejects_bad_hparams(bad):
    hp = native.muon_hparams(**bad)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step([_entry()], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


@pytest.mark.parametrize("sched", [[(3.4, -4.7, float("nan"))] * 5, [(float("inf"), 0.0, 0.0)] * 5])
def test_muon_rejects_non_finite_schedule(sched):
    hp = native.muon_hparams(ns_schedule=sched)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step([_entry()], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


def test_schedule_replaces_the_fixed_triple_in_validation():
    # with a schedule the (a, b, c) fields are not used, so they may be anything
    hp = native.muon_hparams(a=float("nan"), ns_schedule=[(3.4445, -4.775, 2.0315)] * 5)
    assert native.mfsdp_muon_workspace_size([_entry()], hp) > 0


def test_newton_schulz_schedule_argument_checks():
    ws = native.mfsdp_ns_workspace_size(64, 64, native.BF16)
    good = [(3.4445, -4.775, 2.0315)] * 3
    for sched, kw in [([(1.0, float("nan"), 0.0)] * 3, {}), (good, dict(m=0)), (good, dict(x_dtype=3)),
                      ([(1.0, 0.0, 0.0)] * 100, {})]:
        args = dict(x=FAKE, x_dtype=1, out=FAKE * 2, out_dtype=1, m=64, n=64, schedule=sched,
                    eps=1e-7, ns_dtype=1, workspace=FAKE * 16, workspace_bytes=ws, stream=0)
        args.update(kw)
        with pytest.raises(native.MfsdpError) as ei:
            native.mfsdp_newton_schulz_schedule(**args)
        assert ei.value.status == native.E_INVALID
    # NULL coefficients with steps > 0
    L = native.lib()
    assert L.mfsdp_newton_schulz_schedule(FAKE, 1, FAKE * 2, 1, 64, 64, None, 3, 1e-7, 1, FAKE * 16,
                                          ws, None) == native.E_INVALID


def test_muon_step_reduce_argument_checks():
    hp = native.muon_hparams()
    ents = [_entry(grad=None), _entry(grad=None)]
    parts = [[FAKE * 4, FAKE * 5], [FAKE * 6, FAKE * 7]]
    for kw in [dict(grad_parts=[[FAKE * 4, None], [FAKE * 6, FAKE * 7]]),
               dict(grad_parts=[[FAKE * 4 + 8, FAKE * 5], [FAKE * 6, FAKE * 7]]),
               dict(grad_parts=[[FAKE] * 65, [FAKE] * 65]),
               dict(grad_scale=float("nan")),
               dict(reduced_out=[None, FAKE + 4])]:
        args = dict(entries=ents, grad_parts=parts, grad_scale=0.5, reduced_out=None, hp=hp,
                    workspace=FAKE * 16, workspace_bytes=1 << 40, stream=0)
        args.update(kw)
        with pytest.raises(native.MfsdpError) as ei:
            native.mfsdp_muon_step_reduce(**args)
        assert ei.value.status == native.E_INVALID
    # zero parts
    L = native.lib()
    arr = (native.MuonEntry * 1)(_entry(grad=None))
    assert L.mfsdp_muon_step_reduce(arr, 1, None, 0, 1.0, None, ctypes.byref(hp), FAKE * 16,
                                    1 << 40, None) == native.E_INVALID
    # the plain step still needs the entry gradient
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step([_entry(grad=None)], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


def test_muon_workspace_checks():
    hp = native.muon_hparams()
    need = native.mfsdp_muon_workspace_size([_entry()], hp)
    assert need > 0
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step([_entry()], hp, FAKE * 16, need - 1, 0)
    assert ei.value.status == native.E_WORKSPACE
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step([_entry()], hp, FAKE * 16 + 16, need, 0)  # not 256-aligned
    assert ei.value.status == native.E_WORKSPACE
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step([_entry()], hp, None, need, 0)
    assert ei.value.status == native.E_WORKSPACE


def test_workspace_size_scales_with_padding():
    hp = native.muon_hparams()
    small = native.mfsdp_muon_workspace_size([_entry(m=100, n=300)], hp)
    exact = native.mfsdp_muon_workspace_size([_entry(m=256, n=512)], hp)
    assert small == exact  # both pad to 256 x 512 tiles
    f32 = native.muon_hparams(ns_dtype="f32")
    assert native.mfsdp_muon_workspace_size([_entry(m=100, n=300)], f32) < 2 * small
    # the sum over entries: two entries need more than one
    assert native.mfsdp_muon_workspace_size([_entry(), _entry()], hp) > \
        native.mfsdp_muon_workspace_size([_entry()], hp)


def test_zero_count_is_noop():
    hp = native.muon_hparams()
    native.mfsdp_muon_step([], hp, None, 0, 0)
    assert native.lib().mfsdp_muon_workspace_size(None, 0, ctypes.byref(hp)) == 0
    native.mfsdp_adamw_step([], 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 0)


def test_newton_schulz_argument_checks():
    ws = native.mfsdp_ns_workspace_size(64, 64, native.BF16)
    for kw in [dict(steps=100), dict(m=0), dict(x_dtype=3), dict(eps=-1.0), dict(out=FAKE)]:
        args = dict(x=FAKE, x_dtype=1, out=FAKE * 2, out_dtype=1, m=64, n=64, a=3.4445, b=-4.775,
                    c=2.0315, steps=5, eps=1e-7, ns_dtype=1, workspace=FAKE * 16,
                    workspace_bytes=ws, stream=0)
        args.update(kw)
        with pytest.raises(native.MfsdpError) as ei:
            native.mfsdp_newton_schulz(**args)
        assert ei.value.status == native.E_INVALID
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_newton_schulz(FAKE, 1, FAKE * 2, 1, 64, 64, 3.4, -4.7, 2.0, 5, 1e-7, 1,
                                   FAKE * 16, ws - 256, 0)
    assert ei.value.status == native.E_WORKSPACE


@pytest.mark.parametrize("kw", [dict(step=0), dict(lr=-1.0), dict(beta1=1.0), dict(beta2=-0.1),
                                dict(eps=0.0), dict(weight_decay=-1.0)])
def test_adamw_rejects_bad_hparams(kw):
    args = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1)
    args.update(kw)
    e = native.AdamWEntry(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, 100, 1, 1)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_adamw_step([e], **args)
    assert ei.value.status == native.E_INVALID


@pytest.mark.parametrize("bad", [dict(numel=0), dict(param=None), dict(exp_avg=FAKE + 4),
                                 dict(grad_dtype=2)])
def test_adamw_rejects_bad_entries(bad):
    d = dict(param=FAKE, grad=FAKE * 2, exp_avg=FAKE * 3, exp_avg_sq=FAKE * 4, numel=100,
             param_dtype=1, grad_dtype=1)
    d.update(bad)
    good = native.AdamWEntry(FAKE, FAKE * 2, FAKE * 3, FAKE * 4, 100, 1, 1)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_adamw_step([good, native.AdamWEntry(**d)], 1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 0)
    assert ei.value.status == native.E_INVALID


# ---------------------------------------------------------------------------------------------
# Shampoo and the inverse root

def _sh_entry(**kw):
    d = dict(param=FAKE, grad=FAKE * 2, L=FAKE * 3, R=FAKE * 4, PL=FAKE * 5, PR=FAKE * 6, m=96,
             n=200, param_dtype=1, grad_dtype=1, update_out=None)
    d.update(kw)
    return native.ShampooEntry(**d)


@pytest.mark.parametrize("bad", [
    dict(m=0), dict(n=70000), dict(param=None), dict(grad=None), dict(L=None), dict(R=None),
    dict(PL=None), dict(PR=None), dict(param_dtype=3), dict(grad_dtype=-1), dict(L=FAKE * 3 + 2),
    dict(param=FAKE + 1), dict(update_out=FAKE + 2),
])
def test_shampoo_rejects_bad_entries(bad):
    hp = native.shampoo_hparams()
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_shampoo_step([_sh_entry(), _sh_entry(**bad)], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


@pytest.mark.parametrize("bad", [
    dict(lr=-1.0), dict(weight_decay=-1.0), dict(beta=-0.1), dict(weight=float("nan")), dict(eps=0.0),
    dict(eps_rel=-1e-6), dict(root_iters=0), dict(root_iters=101), dict(lr=float("inf")),
])
def test_shampoo_rejects_bad_hparams(bad):
    hp = native.shampoo_hparams(**bad)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_shampoo_step([_sh_entry()], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID
    assert native.mfsdp_shampoo_workspace_size([_sh_entry()], hp) == 0


def test_shampoo_refresh_flag_and_workspace_checks():
    hp = native.shampoo_hparams()
    hp.refresh = 2
    with pytest.raises(native.MfsdpError):
        native.mfsdp_shampoo_step([_sh_entry()], hp, FAKE * 16, 1 << 40, 0)
    hp = native.shampoo_hparams()
    need = native.mfsdp_shampoo_workspace_size([_sh_entry()], hp)
    # padded to 128: G, G^T and P_L G (3 x 128 x 256) plus 5 matrices per side (128^2 + 256^2)
    assert need >= 4 * (3 * 128 * 256 + 5 * (128 ** 2 + 256 ** 2))
    for ws, nb in ((None, need), (FAKE * 16 + 8, need), (FAKE * 16, need - 1)):
        with pytest.raises(native.MfsdpError) as ei:
            native.mfsdp_shampoo_step([_sh_entry()], hp, ws, nb, 0)
        assert ei.value.status == native.E_WORKSPACE
    # the size query does not depend on the data pointers, and count == 0 is a no-op
    assert native.mfsdp_shampoo_workspace_size([_sh_entry(param=None, L=None)], hp) == need
    assert native.mfsdp_shampoo_workspace_size([], hp) == 0
    native.mfsdp_shampoo_step([], hp, None, 0, 0)


@pytest.mark.parametrize("bad", [
    dict(d=0), dict(d=70000), dict(p=3), dict(p=0), dict(eps=0.0), dict(eps_rel=-1.0), dict(iters=0),
    dict(iters=101), dict(a=None), dict(out=None), dict(a=FAKE + 2),
])
def test_inverse_root_rejects_bad_arguments(bad):
    args = dict(a=FAKE, out=FAKE * 2, d=100, p=4, eps=1e-9, eps_rel=1e-6, iters=20)
    args.update(bad)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_inverse_root(args["a"], args["out"], args["d"], args["p"], args["eps"],
                                  args["eps_rel"], args["iters"], FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


def test_inverse_root_workspace_query():
    assert native.mfsdp_inverse_root_workspace_size(100, 4, 20) >= 5 * 128 * 128 * 4
    assert native.mfsdp_inverse_root_workspace_size(100, 3, 20) == 0
    assert native.mfsdp_inverse_root_workspace_size(0, 4, 20) == 0
    need = native.mfsdp_inverse_root_workspace_size(300, 2, 7)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_inverse_root(FAKE, FAKE * 2, 300, 2, 1e-9, 0.0, 7, FAKE * 16, need - 1, 0)
    assert ei.value.status == native.E_WORKSPACE


def _needed_bytes(fn):
    with pytest.raises(native.MfsdpError) as ei:
        fn()
    assert ei.value.status == native.E_WORKSPACE
    return int(re.search(r"\((\d+) bytes\)", str(ei.value)).group(1))


@pytest.mark.parametrize("refresh", [0, 1])
def test_shampoo_size_query_equals_what_the_call_needs(refresh):
    ents = [_sh_entry(), _sh_entry(m=1, n=50, param_dtype=0), _sh_entry(m=300, n=129)]
    hp = native.shampoo_hparams(refresh=bool(refresh), root_iters=7)
    q = native.mfsdp_shampoo_workspace_size([native.ShampooEntry(m=e.m, n=e.n, param_dtype=e.param_dtype,
                                                                 grad_dtype=e.grad_dtype) for e in ents], hp)
    assert q > 0
    assert _needed_bytes(lambda: native.mfsdp_shampoo_step(ents, hp, FAKE * 16, 0, 0)) == q


@pytest.mark.parametrize("p,iters", [(1, 1), (2, 8), (4, 20)])
def test_inverse_root_size_query_equals_what_the_call_needs(p, iters):
    q = native.mfsdp_inverse_root_workspace_size(257, p, iters)
    assert _needed_bytes(lambda: native.mfsdp_inverse_root(FAKE, FAKE * 2, 257, p, 1e-9, 1e-6, iters,
                                                           FAKE * 16, 0, 0)) == q


def test_shampoo_rejects_calls_beyond_the_launch_size_limit():
    big = [_sh_entry(m=65536, n=65536) for _ in range(300)]
    with pytest.raises(native.MfsdpError, match="2\\^30 tiles"):
        native.mfsdp_shampoo_step(big, native.shampoo_hparams(), FAKE * 16, 1 << 62, 0)
    assert native.mfsdp_shampoo_workspace_size(big, native.shampoo_hparams()) == 0


def test_muon_rejects_calls_beyond_the_launch_size_limit():
    big = [_entry(m=65536, n=65536) for _ in range(1100)]
    with pytest.raises(native.MfsdpError, match="2\\^30 tiles"):
        native.mfsdp_muon_step(big, native.muon_hparams(), FAKE * 16, 1 << 62, 0)


# ---------------------------------------------------------------------------------------------
# SOAP and the orthonormal factor

def _soap_entry(**kw):
    d = dict(param=FAKE, grad=FAKE * 2, exp_avg=FAKE * 3, exp_avg_sq=FAKE * 4, L=FAKE * 5, R=FAKE * 6,
             QL=FAKE * 7, QR=FAKE * 8, m=96, n=200, param_dtype=1, grad_dtype=1, update_out=None)
    d.update(kw)
    return native.SoapEntry(**d)


@pytest.mark.parametrize("bad", [
    dict(m=0), dict(n=65537), dict(m=70000), dict(param=None), dict(grad=None), dict(exp_avg=None),
    dict(exp_avg_sq=None), dict(L=None), dict(R=None), dict(QL=None), dict(QR=None), dict(param_dtype=3),
    dict(grad_dtype=-1), dict(QL=FAKE * 7 + 2), dict(exp_avg_sq=FAKE * 4 + 1), dict(update_out=FAKE + 2),
])
def test_soap_rejects_bad_entries(bad):
    hp = native.soap_hparams()
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_soap_step([_soap_entry(), _soap_entry(**bad)], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


@pytest.mark.parametrize("bad", [
    dict(lr=-1.0), dict(weight_decay=-1.0), dict(beta1=1.0), dict(beta2=-0.1), dict(beta1=float("nan")),
    dict(eps=0.0), dict(shampoo_beta=-1.0), dict(shampoo_weight=float("inf")), dict(step=0),
    dict(refresh_iters=0), dict(refresh_iters=101), dict(lr=float("inf")), dict(max_precond_dim=-1),
    dict(max_precond_dim=4097),
])
def test_soap_rejects_bad_hparams(bad):
    hp = native.soap_hparams(**bad)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_soap_step([_soap_entry()], hp, FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID
    assert native.mfsdp_soap_workspace_size([_soap_entry()], hp) == 0


def test_soap_refresh_flag_and_workspace_checks():
    hp = native.soap_hparams()
    hp.refresh = 2
    with pytest.raises(native.MfsdpError):
        native.mfsdp_soap_step([_soap_entry()], hp, FAKE * 16, 1 << 40, 0)
    hp = native.soap_hparams(refresh=True)
    need = native.mfsdp_soap_workspace_size([_soap_entry()], hp)
    # padded to 128: 8 mp np + 3 (mp^2 + np^2) floats, plus the QR panels 16 (m + n) + 512 floats
    assert need >= 4 * (8 * 128 * 256 + 3 * (128 ** 2 + 256 ** 2) + 16 * (96 + 200) + 512)
    for ws, nb in ((None, need), (FAKE * 16 + 8, need), (FAKE * 16, need - 1)):
        with pytest.raises(native.MfsdpError) as ei:
            native.mfsdp_soap_step([_soap_entry()], hp, ws, nb, 0)
        assert ei.value.status == native.E_WORKSPACE
    assert native.mfsdp_soap_workspace_size([_soap_entry(param=None, QL=None)], hp) == need
    assert native.mfsdp_soap_workspace_size([], hp) == 0
    native.mfsdp_soap_step([], hp, None, 0, 0)


@pytest.mark.parametrize("refresh,iters", [(0, 1), (1, 1), (1, 4)])
def test_soap_size_query_equals_what_the_call_needs(refresh, iters):
    ents = [_soap_entry(), _soap_entry(m=1, n=50, param_dtype=0), _soap_entry(m=300, n=129)]
    hp = native.soap_hparams(refresh=bool(refresh), refresh_iters=iters, step=4)
    q = native.mfsdp_soap_workspace_size([native.SoapEntry(m=e.m, n=e.n, param_dtype=e.param_dtype,
                                                           grad_dtype=e.grad_dtype) for e in ents], hp)
    assert q > 0
    assert _needed_bytes(lambda: native.mfsdp_soap_step(ents, hp, FAKE * 16, 0, 0)) == q


@pytest.mark.parametrize("bad", [dict(d=0), dict(d=4097), dict(a=None), dict(q=None), dict(a=FAKE + 2)])
def test_orthonormal_factor_rejects_bad_arguments(bad):
    args = dict(a=FAKE, q=FAKE * 2, d=100)
    args.update(bad)
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_orthonormal_factor(args["a"], args["q"], args["d"], FAKE * 16, 1 << 40, 0)
    assert ei.value.status == native.E_INVALID


def test_orthonormal_factor_workspace_query():
    assert native.mfsdp_orthonormal_factor_workspace_size(0) == 0
    assert native.mfsdp_orthonormal_factor_workspace_size(4097) == 0
    for d in (1, 100, 4096):
        q = native.mfsdp_orthonormal_factor_workspace_size(d)
        dp = -(-d // 128) * 128
        assert q >= 4 * (2 * dp * dp + 16 * d + 256)
        assert _needed_bytes(lambda: native.mfsdp_orthonormal_factor(FAKE, FAKE * 2, d, FAKE * 16, 0, 0)) == q


def test_library_build_id_matches_the_sources():
    from paper_2607_05895_amd import build_lib
    assert native.mfsdp_build_id() == build_lib.source_id()
    assert re.fullmatch(r"[0-9a-f]{16}", native.mfsdp_build_id())


def test_stale_library_is_refused(monkeypatch):
    """A library built from other sources than the tree's is not loaded (no silent stale binary)."""
    from paper_2607_05895_amd import build_lib
    native.lib()
    monkeypatch.setattr(native, "_lib", None)
    monkeypatch.setattr(build_lib, "source_id", lambda: "0" * 16)
    with pytest.raises(ImportError, match="other sources"):
        native.lib()
    monkeypatch.undo()
    assert native.lib() is not None


def test_noalloc_rejects_entries_beyond_the_scratch_before_any_gpu_work():
    """A list that needs more workspace than the allocation-free step's static array is refused by
    the argument checks (no device is touched: the pointers here are never dereferenced)."""
    hp = native.muon_hparams()
    big = [_entry(m=4096, n=4096)]
    need = native.mfsdp_muon_workspace_size(big, hp)
    assert need > native.NOALLOC_SCRATCH_BYTES
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step_noalloc(big, hp, 0)
    assert ei.value.status == native.E_INVALID
    assert "MFSDP_NOALLOC_SCRATCH_BYTES" in native.mfsdp_last_error()
    with pytest.raises(native.MfsdpError) as ei:
        native.mfsdp_muon_step_noalloc([_entry(m=0)], hp, 0)
    assert ei.value.status == native.E_INVALID
    native.mfsdp_muon_step_noalloc([], hp, 0)  # count == 0 is a no-op


def test_soap_sides_beyond_the_preconditioned_limit():
    """A side longer than max_precond_dim has no basis: its statistic and basis pointers are not
    required, and its d x d buffers drop out of the workspace (size queries only: no GPU work)."""
    two = native.mfsdp_soap_workspace_size([_soap_entry(m=3000, n=200)], native.soap_hparams())
    one = native.mfsdp_soap_workspace_size([_soap_entry(m=3000, n=200)], native.soap_hparams(max_precond_dim=2048))
    mp = 3072
    assert two - one >= 3 * mp * mp * 4   # Q_L, Q_L^T / the power step, and L of the left side
    assert native.mfsdp_soap_workspace_size([_soap_entry(m=20000, n=4096, L=None, QL=None)],
                                            native.soap_hparams()) > 0
    assert native.mfsdp_soap_workspace_size([_soap_entry(m=5000, n=6000, L=None, QL=None, R=None, QR=None)],
                                            native.soap_hparams()) > 0
    # a side within the limit still needs its pointers
    with pytest.raises(native.MfsdpError, match="NULL"):
        native.mfsdp_soap_step([_soap_entry(m=20000, n=200, R=None)], native.soap_hparams(), FAKE * 16, 1 << 40, 0)
