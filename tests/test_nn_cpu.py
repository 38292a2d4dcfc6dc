"""Host-side checks of the PyTorch modules (no kernel runs): shapes, dtypes and
the layout the ABI needs are validated before any call reaches the library."""
import pytest

torch = pytest.importorskip("torch")
cnn = pytest.importorskip("paper_2410_15352_amd.nn")


def test_module_validation():
    with pytest.raises(ValueError):
        cnn.CompActGroup(64, [32, 16], [8, 8], device="cpu", weight=torch.zeros(64, 40, dtype=torch.bfloat16))
    with pytest.raises(ValueError):
        cnn.CompActLinear(64, 32, 8, device="cpu", weight=torch.zeros(64, 32))          # fp32 weight
    lin = cnn.CompActLinear(64, 32, 8, device="cpu")
    assert lin.weight.dtype == torch.bfloat16 and tuple(lin.weight.shape) == (64, 32)
    assert [tuple(g.shape) for g in lin.ghat] == [(8, 32)] and lin.seeds == [1 << 32]
    with pytest.raises(TypeError):
        lin(torch.zeros(4, 64))                                                          # fp32 input
    with pytest.raises(ValueError):
        lin(torch.zeros(4, 48, dtype=torch.bfloat16))                                    # wrong width


def test_group_slices_and_default_seeds():
    g = cnn.CompActGroup(64, [32, 16, 24], [8, 8, 4], device="cpu")
    assert g.msum == 72 and g.rsum == 20
    assert g.seeds == [1 << 32, 2 << 32, 3 << 32]
    w = g.weight_slice(1)
    assert tuple(w.shape) == (64, 16) and w.data_ptr() == g.weight.data_ptr() + 32 * 2


def test_abi_layout_of_padded_buffers():
    t = cnn._empty2d(5, 13, torch.bfloat16, "cpu")
    assert tuple(t.shape) == (5, 13) and t.stride() == (16, 1)
    # a view with an odd leading dimension is copied into a padded buffer
    odd = torch.zeros(6, 13, dtype=torch.bfloat16)[:5]
    assert cnn._as_abi(odd).stride(0) == 16
    ok = torch.zeros(5, 16, dtype=torch.bfloat16)
    assert cnn._as_abi(ok) is ok
