"""Host-side logic of Pi_Sec-Linear (no GPU): the rotation block length and
the activation window."""
import pytest

from oracle.quant import max_qx
from paper_2607_29221_amd.secure_linear import activation_window, rotation_block


@pytest.mark.parametrize("K,block", [(8192, 8192), (28672, 4096), (4096, 4096), (65536, 32768), (96, 32)])
def test_rotation_block(K, block):
    assert rotation_block(K) == block


def test_rotation_block_rejects_odd_widths():
    with pytest.raises(ValueError):
        rotation_block(24)


@pytest.mark.parametrize("K,q_x", [(8192, 1997), (28672, 567)])
def test_activation_window_values(K, q_x):
    """Largest q_x with K (127 + 4)(q_x + 4) <= 2^31 - 1 (int8 weights,
    |e| <= 4): 1997 at K = 8192 and 567 at K = 28672."""
    assert activation_window(K, 127, 4) == q_x == max_qx(K, 127, margin=4)
    assert K * 131 * (q_x + 4) <= 2 ** 31 - 1 < K * 131 * (q_x + 5)


def test_activation_window_without_noise():
    assert activation_window(8192, 127, 0) == (2 ** 31 - 1) // (8192 * 127)


def test_binding_rejects_undersized_tensors():
    """The binding checks tensor sizes against the sizes it passes, before
    any call reaches the library (no GPU needed: the checks raise first)."""
    import pytest
    import torch

    from paper_2607_29221_amd import mosaic as m

    class FakeCuda(torch.Tensor):
        @property
        def is_cuda(self):
            return True

    small = torch.zeros((4, 8), dtype=torch.int32).as_subclass(FakeCuda)
    r = m.rng(1, 2, 3, m.DIST_UNIFORM)
    with pytest.raises(ValueError):
        m.mosaic_sample(r, 5, 8, out=small)
    with pytest.raises(ValueError):
        m.mosaic_sample(r, 4, 9, out=small)
    dig = m.Digits(torch.zeros((4, 256), dtype=torch.int8).as_subclass(FakeCuda), 64)
    with pytest.raises(ValueError):
        m.mosaic_masked_matmul(dig, dig, 4, 4, 65, small)          # K beyond the digit buffer
    with pytest.raises(ValueError):
        m.mosaic_masked_matmul(dig, dig, 5, 4, 64, small)          # M beyond the rows
    with pytest.raises(ValueError):
        m.mosaic_unmask(small, None, dig, dig, 4, 9, 64, y=small)  # N beyond ym
    cpu = torch.zeros((4, 8), dtype=torch.int32)
    with pytest.raises(ValueError):
        m.mosaic_sample(r, 4, 8, out=cpu)                           # host memory
