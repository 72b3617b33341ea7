"""The torch helpers of the binding check the tensors they pass to the library (the C ABI takes plain
pointers and cannot): CPU tensors are refused before any library call."""
import pytest
import torch

from paper_2607_05895_amd import native


def test_cpu_tensors_are_refused_by_every_entry_helper():
    p = torch.zeros(8, 8, dtype=torch.bfloat16)
    f = torch.zeros(8, 8)
    with pytest.raises(ValueError, match="CUDA"):
        native.muon_entry_t(p, p, f)
    with pytest.raises(ValueError, match="CUDA"):
        native.adamw_entry_t(p, p, f, f)
    with pytest.raises(ValueError, match="CUDA"):
        native.shampoo_entry_t(p, p, f, f, f, f)
    with pytest.raises(ValueError, match="CUDA"):
        native.soap_entry_t(p, p, f, f, f, f, f, f)


def test_entries_must_be_matrices():
    v = torch.zeros(8)
    for fn, args in ((native.muon_entry_t, (v, v, v)), (native.shampoo_entry_t, (v,) * 6),
                     (native.soap_entry_t, (v,) * 8)):
        with pytest.raises(ValueError, match="2D"):
            fn(*args)


def test_non_tensors_are_refused():
    with pytest.raises(TypeError, match="torch.Tensor"):
        native._ptr(12345, "param")
