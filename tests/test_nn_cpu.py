"""Host-side checks of the torch modules: shapes, argument validation, and that
CPU tensors are refused (the modules have no torch fallback)."""
import pytest
import torch

from paper_2312_06881_amd.nn import DyadFF, DyadLinear


def test_parameter_shapes_and_init_bound():
    mod = DyadLinear(64, 256, 4, "DT")
    assert mod.w1.shape == mod.w2.shape == (4, 64, 16)
    assert mod.bias.shape == (256,)
    assert mod.w1.dtype == torch.bfloat16
    bound = 1.0 / (2 * 64 / 4) ** 0.5
    for p in (mod.w1, mod.w2, mod.bias):
        assert float(p.detach().abs().max()) <= bound
    assert "n_dyad=4" in repr(mod) and "variant=DT" in repr(mod)
    ff = DyadFF(64, 256, 4, "OT", bias=False)
    assert ff.fc1.w1.shape == (4, 64, 16) and ff.fc2.w1.shape == (4, 16, 64)
    assert ff.fc1.bias is None and ff.fc2.bias is None


def test_invalid_arguments():
    with pytest.raises(ValueError):
        DyadLinear(64, 250, 4)
    with pytest.raises(ValueError):
        DyadLinear(64, 256, 4, "XT")


def test_cpu_tensors_refused():
    mod = DyadLinear(64, 256, 4)
    with pytest.raises(ValueError, match="device tensors"):
        mod(torch.zeros(5, 64, dtype=torch.bfloat16))
    ff = DyadFF(64, 256, 4)
    with pytest.raises(ValueError, match="device tensors"):
        ff(torch.zeros(5, 64, dtype=torch.bfloat16))
