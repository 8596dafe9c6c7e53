"""Pins of the comparator oracle (oracle/comparators.py): SmoothQuant with the
unified factor (Sec. 4.1), MAS with per-modality weights (Sec. 4.2) and the
SQNR diagnostic (eq. sqnr); and the product-side comparator calibration
against it.  Each pin checks against something other than the code under
test: a closed form, an identity between methods, or Theorem 2's ordering."""
import numpy as np
import pytest

from oracle import calibration as cal
from oracle import comparators as cmp
from oracle import inference as inf
from paper_2603_04800_amd import calibrate as pcal


def _layer(seed, T=(96, 80, 72), K=32, N=24, scales=(1.0, 30.0, 2.0)):
    rng = np.random.default_rng(seed)
    mod = np.concatenate([np.full(c, m, np.int32) for m, c in enumerate(T)])
    x = rng.standard_normal((mod.size, K)).astype(np.float32)
    for m, s in enumerate(scales[:len(T)]):
        x[mod == m] *= np.float32(s)
    x[:, :2] *= 20                       # outlier channels shared by all modalities
    if len(T) > 2:
        x[mod == 2, 5:7] *= 10           # and two of the third modality's own
    w = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    return x, mod, w


def test_sqnr_closed_form():
    """eq. sqnr: an output off by a relative eps on every element has
    SQNR = -20 log10(eps); an exact output is +inf; the ratio is scale free."""
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((5, 40))
    for eps in (1e-1, 1e-3, 2.5e-5):
        s = cmp.sqnr_db(ref, ref * (1 + eps))
        assert np.allclose(s, -20 * np.log10(eps), atol=1e-6)
        assert np.allclose(cmp.sqnr_db(7.0 * ref, 7.0 * ref * (1 + eps)), s, atol=1e-9)
    assert np.all(np.isinf(cmp.sqnr_db(ref, ref)))
    # error orthogonal to the signal, energy ratio 100 -> 20 dB
    y = ref.copy()
    y[:, 0] = 0.0
    e = ref - y
    expect = 10 * np.log10((ref ** 2).sum(1) / (e ** 2).sum(1))
    assert np.allclose(cmp.sqnr_db(ref, y), expect)


def test_unified_factor_is_the_dominant_modality_factor():
    """Sec. 4.1: s^uni is proportional to the range of the dominant modality,
    so with beta = 1/2 it equals, channel by channel, the largest of the
    per-modality MAS factors (exactly: sqrt and fl are monotone)."""
    x, mod, w = _layer(3)
    wmax = cal.weight_range(w)
    per_mod = np.stack([cal.smoothing_factor(cal.channel_range(x, mod, m), wmax)[0]
                        for m in range(3)])
    s_uni, inv = cmp.unified_factor(x, w)
    assert np.array_equal(s_uni, per_mod.max(axis=0))
    assert np.array_equal(inv, (np.float32(1) / s_uni).astype(np.float32))


def test_mas_only_text_rows_equal_the_shared_weight_layer():
    """Text rows see Q(x S_t^-1) Q(S_t W) under both MAS-only and MASQuant."""
    x, mod, w = _layer(4)
    art = cal.calibrate(x, mod, w, 3, rank=8)
    y_mq = inf.linear(x, mod, art["inv_smooth"], art["wq"], art["w_scale"], art["l_down"],
                      art["r_up"])
    y_mas = cmp.mas_only_linear(x, mod, w, 3)
    text = mod == 0
    assert np.array_equal(y_mq[text], y_mas[text])
    assert not np.array_equal(y_mq[~text], y_mas[~text])


def test_mas_only_with_one_factor_is_smoothquant():
    """Given the unified factor for every modality, the per-modality weights
    are all Q(S^uni W): MAS-only then equals the SmoothQuant comparator bit
    for bit."""
    x, mod, w = _layer(5)
    sq = cmp.smoothquant_artifacts(x, w, 3)
    y_sq = inf.linear(x, mod, sq["inv_smooth"], sq["wq"], sq["w_scale"], sq["l_down"],
                      sq["r_up"])
    y_mas = cmp.mas_only_linear(x, mod, w, 3, smoothing=sq["s32"])
    assert np.array_equal(y_sq, y_mas)


def test_compensation_sqnr_grows_with_rank():
    """Sec. 4.3 / Theorem 2: a larger rank leaves a smaller whitened residual,
    so the non-text SQNR of the layer rises with r; at full rank the weight
    seen by those rows is S_m W unquantized, at least as good as MAS-only."""
    x, mod, w = _layer(6, T=(128, 128), K=32, N=24, scales=(1.0, 30.0))
    y_fp = x.astype(np.float64) @ w.astype(np.float64)
    vis = mod == 1
    got = []
    for r in (0, 4, 12, 24):
        art = cal.calibrate(x, mod, w, 2, rank=r)
        y = inf.linear(x, mod, art["inv_smooth"], art["wq"], art["w_scale"], art["l_down"],
                       art["r_up"])
        got.append(np.mean(cmp.sqnr_db(y_fp, y)[vis]))
    assert all(a < b for a, b in zip(got, got[1:])), got
    mas = np.mean(cmp.sqnr_db(y_fp, cmp.mas_only_linear(x, mod, w, 2))[vis])
    assert got[-1] >= mas, (got, mas)


@pytest.mark.parametrize("n_mod", [2, 3])
def test_product_smoothquant_calibration_matches_oracle(n_mod):
    """The comparator's artifacts for the GPU (paper_2603_04800_amd.calibrate)
    equal the oracle's bit for bit."""
    x, mod, w = _layer(7, T=(64, 64, 64)[:n_mod])
    ref = cmp.smoothquant_artifacts(x, w, n_mod)
    got = pcal.calibrate_smoothquant(x, w, n_mod, lr_dtype="f32")
    assert np.array_equal(got["inv_smooth"], ref["inv_smooth"])
    assert np.array_equal(got["wq"], ref["wq"])
    assert np.array_equal(got["w_scale"], ref["w_scale"])
    assert got["l_down"].shape == ref["l_down"].shape and got["r_up"].shape == ref["r_up"].shape


def test_product_mas_only_calibration_matches_oracle():
    """The MAS-only comparator's artifacts for the GPU: per-modality factors
    and one weight Q(S_m W) per modality, equal to the oracle's bit for bit."""
    x, mod, w = _layer(8)
    got = pcal.calibrate_mas_only(x, mod, w, 3, lr_dtype="f32")
    wmax = cal.weight_range(w)
    for m in range(3):
        s32, inv = cal.smoothing_factor(cal.channel_range(x, mod, m), wmax)
        wq, w_scale, _ = cal.quantize_weight(w, s32)
        assert np.array_equal(got["inv_smooth"][m], inv)
        assert np.array_equal(got["wq"][m], wq)
        assert np.array_equal(got["w_scale"][m], w_scale)
    # and the per-modality composition is the oracle's MAS-only layer
    y = np.zeros((x.shape[0], w.shape[1]), np.float32)
    for m in range(3):
        rows = mod == m
        y[rows] = inf.linear(x[rows], np.zeros(rows.sum(), np.int32), got["inv_smooth"][m][None],
                             got["wq"][m], got["w_scale"][m])
    assert np.array_equal(y, cmp.mas_only_linear(x, mod, w, 3))
