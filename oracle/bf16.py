"""bfloat16 <-> float32 conversions at the bit level (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

bfloat16 is the upper half of an IEEE binary32 word.  Widening is exact (shift
left by 16); narrowing rounds to nearest, ties to even, on the 16 dropped bits.
Pinned exhaustively against torch's CPU casts in the test suite.
"""
import numpy as np


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even narrowing; NaN inputs map to a quiet NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) & np.uint64(0xFFFF)
    nan = np.isnan(x)
    if nan.any():
        r = np.where(nan, (u >> np.uint64(16)) | np.uint64(0x40), r)
    return r.astype(np.uint16)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 value -> nearest bf16 value, returned as fp32."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))
