"""Helpers for the GPU tests: moving ring matrices between torch and numpy."""
import numpy as np
import torch


def to_np_u32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint32)


def to_dev_ring(x: np.ndarray) -> torch.Tensor:
    """uint32 numpy matrix -> int32 device tensor holding the same bits."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.uint32).view(np.int32)).cuda()


def digits_np(d) -> np.ndarray:
    """Raw bytes of a Digits view's buffer (whole rows)."""
    return d.buf.detach().cpu().numpy()


def unpack_digits(d, rows=None):
    """Ring matrix held by a Digits view (columns col0 .. col0+cols)."""
    from oracle.ring import digit_layout_unpack, padded_k
    raw = digits_np(d)
    r = raw.shape[0] if rows is None else rows
    sub = raw[:r, 4 * d.col0: 4 * d.col0 + 4 * padded_k(d.cols)]
    return digit_layout_unpack(np.ascontiguousarray(sub), r, d.cols)


def pad_is_zero(d) -> bool:
    from oracle.ring import digit_layout_pad_is_zero, padded_k
    raw = digits_np(d)
    sub = raw[:, 4 * d.col0: 4 * d.col0 + 4 * padded_k(d.cols)]
    return digit_layout_pad_is_zero(np.ascontiguousarray(sub), raw.shape[0], d.cols)
