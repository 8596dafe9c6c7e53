"""Packing of 4-bit weight codes (the W4A8 setting) into the library's layout.

Codes are signed values in [-7, 7] (per-output-channel symmetric, as the
8-bit ones).  Row o of the packed weight holds K / 2 bytes; its 32-bit word g
(bytes 4 g .. 4 g + 3) carries codes 8 g .. 8 g + 7: byte b of the word has
code 8 g + b in its low nibble and code 8 g + b + 4 in its high nibble, both
as 4-bit two's complement.  So masking a word with 0x0F0F0F0F gives codes
8 g .. 8 g + 3 in consecutive bytes, and shifting it right by 4 first gives
8 g + 4 .. 8 g + 7: the unpacked bytes come out in k order.
"""
import numpy as np


def pack(codes: np.ndarray) -> np.ndarray:
    """int8 codes [N][K] in [-8, 7], K % 8 == 0 -> uint8 [N][K / 2]."""
    c = np.asarray(codes)
    if c.ndim != 2 or c.shape[1] % 8 != 0:
        raise ValueError("codes must be [N][K] with K % 8 == 0")
    if c.size and (c.min() < -8 or c.max() > 7):
        raise ValueError("codes must lie in [-8, 7]")
    n, k = c.shape
    nib = (c.astype(np.int16) & 0xF).astype(np.uint8).reshape(n, k // 8, 2, 4)
    packed = nib[:, :, 0, :] | (nib[:, :, 1, :] << 4)          # [N][K/8][4]
    return np.ascontiguousarray(packed.reshape(n, k // 2))
