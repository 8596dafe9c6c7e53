"""Layout of the packed 4-bit weight (W4A8): host-side packing only, no GPU."""
import numpy as np
import pytest

from paper_2603_04800_amd import int4


def _unpack(packed: np.ndarray, k: int) -> np.ndarray:
    """Independent reading of the documented layout, one nibble at a time."""
    n = packed.shape[0]
    out = np.zeros((n, k), np.int8)
    for o in range(n):
        for g in range(k // 8):
            for b in range(4):
                byte = int(packed[o, 4 * g + b])
                for half, kk in ((byte & 0xF, 8 * g + b), (byte >> 4, 8 * g + b + 4)):
                    out[o, kk] = half - 16 if half >= 8 else half
    return out


def test_pack_known_bytes():
    codes = np.array([[0, 1, 2, 3, 4, 5, 6, 7], [-1, -2, -3, -4, -5, -6, -7, 0]], np.int8)
    p = int4.pack(codes)
    assert p.dtype == np.uint8 and p.shape == (2, 4)
    assert p[0].tolist() == [0x40, 0x51, 0x62, 0x73]
    assert p[1].tolist() == [0xBF, 0xAE, 0x9D, 0x0C]


def test_pack_round_trip():
    rng = np.random.default_rng(3)
    codes = rng.integers(-7, 8, (5, 48)).astype(np.int8)
    assert np.array_equal(_unpack(int4.pack(codes), 48), codes)


def test_pack_rejects_bad_input():
    with pytest.raises(ValueError):
        int4.pack(np.zeros((2, 12), np.int8))
    with pytest.raises(ValueError):
        int4.pack(np.full((1, 8), 9, np.int8))
