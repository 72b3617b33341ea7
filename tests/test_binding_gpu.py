"""The torch helpers refuse, before any launch, tensors whose shape, dtype or layout differs from
what the call reads and writes (a smaller buffer would be written past its end)."""
import pytest

from paper_2607_05895_amd import native

pytestmark = pytest.mark.gpu


def _t(shape, dtype="f32"):
    import torch
    return torch.zeros(shape, dtype=torch.float32 if dtype == "f32" else torch.bfloat16, device="cuda")


def test_muon_entry_checks():
    m, n = 64, 96
    p, g, mo = _t((m, n), "bf16"), _t((m, n), "bf16"), _t((m, n))
    native.muon_entry_t(p, g, mo)  # well formed
    with pytest.raises(TypeError, match="dtype"):
        native.muon_entry_t(p, g, _t((m, n), "bf16"))          # bf16 momentum: half the bytes
    with pytest.raises(ValueError, match="shape"):
        native.muon_entry_t(p, g, _t((m, n - 1)))
    with pytest.raises(ValueError, match="shape"):
        native.muon_entry_t(p, _t((n, m), "bf16"), mo)
    with pytest.raises(ValueError, match="contiguous"):
        native.muon_entry_t(p, _t((n, m), "bf16").t(), mo)
    with pytest.raises(TypeError, match="dtype"):
        native.muon_entry_t(p, g, mo, update_out=_t((m, n), "bf16"))


def test_reduce_parts_checks():
    m, n = 64, 96
    p, g, mo = _t((m, n), "bf16"), _t((m, n), "bf16"), _t((m, n))
    e = native.muon_entry_t(p, g, mo)
    h = native.muon_hparams()
    ws = native.muon_workspace_t([e], h)
    with pytest.raises(TypeError, match="dtype"):
        native.muon_step_reduce_t([e], [[g, _t((m, n))]], 0.5, h, ws)  # fp32 part, bf16 entry
    with pytest.raises(ValueError, match="shape"):
        native.muon_step_reduce_t([e], [[g, _t((m, n + 1), "bf16")]], 0.5, h, ws)
    with pytest.raises(ValueError, match="one item per entry"):
        native.muon_step_reduce_t([e], [], 0.5, h, ws)


def test_shampoo_soap_and_factor_checks():
    m, n = 32, 48
    p, g = _t((m, n), "bf16"), _t((m, n), "bf16")
    L, R = _t((m, m)), _t((n, n))
    native.shampoo_entry_t(p, g, L, R, _t((m, m)), _t((n, n)))
    with pytest.raises(ValueError, match="shape"):
        native.shampoo_entry_t(p, g, L, R, _t((n, n)), _t((n, n)))
    with pytest.raises(ValueError, match="shape"):
        native.soap_entry_t(p, g, _t((m, n)), _t((m, n)), L, R, _t((m, m)), _t((m, m)))
    with pytest.raises(TypeError, match="dtype"):
        native.soap_entry_t(p, g, _t((m, n), "bf16"), _t((m, n)), L, R, _t((m, m)), _t((n, n)))
    with pytest.raises(ValueError, match="shape"):
        native.orthonormal_factor_t(_t((m, m)), _t((m, m + 1)))
    with pytest.raises(TypeError, match="dtype"):
        native.inverse_root_t(_t((m, m), "bf16"), _t((m, m)))
    with pytest.raises(ValueError, match="shape"):
        native.newton_schulz_t(_t((m, n), "bf16"), _t((n, m)))
    with pytest.raises(TypeError, match="dtype"):
        native.muon_step_t([native.muon_entry_t(p, g, _t((m, n)))], native.muon_hparams(), _t((1024,)))
