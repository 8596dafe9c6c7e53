"""Oracle for the comparison methods and the SQNR diagnostic.

TEST INFRASTRUCTURE ONLY (see the package docstring).

  * SmoothQuant with the unified factor (Sec. 4.1): one smoothing vector for
    every token, s^uni_i = (max_t |x_ti|)^beta / (max_j |w_ji|)^(1 - beta)
    over the tokens of all modalities (beta = 1/2), the shared weight
    Q(S^uni W), no compensation.  It runs on the same inference rule as the
    layer (inference.linear with rank 0).
  * MAS only (Sec. 4.2, the inference equation closing it): every modality
    has its own quantized weight, y_t = Q(x_t S_m^-1) Q(S_m W), no
    compensation.
  * SQNR (eq. sqnr): 10 log10(||y_t||^2 / ||y_t - y^_t||^2) per token, here
    between the unquantized layer output X W and a method's output.
"""
import numpy as np

from . import calibration as cal
from . import inference as inf


def unified_factor(x, w):
    """(s32, inv_s32) of the unified factor: the range taken over all tokens."""
    return cal.smoothing_factor(np.max(np.abs(np.asarray(x, np.float64)), axis=0),
                                cal.weight_range(w))


def smoothquant_artifacts(x, w, n_mod: int, weight_bits: int = 8) -> dict:
    """The SmoothQuant comparator in the layer's layouts: the unified factor
    for every modality, Q(S^uni W) per output channel, rank 0."""
    s32, inv = unified_factor(x, w)
    wq, w_scale, wdq = cal.quantize_weight(w, s32, weight_bits)
    k, n = np.asarray(x).shape[1], wq.shape[0]
    return dict(s32=np.tile(s32, (n_mod, 1)), inv_smooth=np.tile(inv, (n_mod, 1)), wq=wq,
                w_scale=w_scale, wdq=wdq, l_down=np.zeros((max(n_mod - 1, 0), 0, k), np.float32),
                r_up=np.zeros((max(n_mod - 1, 0), n, 0), np.float32))


def mas_only_linear(x, modality, w, n_mod: int, weight_bits: int = 8, smoothing=None):
    """y [T][N] float32 with per-modality weights Q(S_m W) (MAS without the
    shared weight and without compensation).  ``smoothing`` optionally gives
    the factors s32 [M][K]; by default the MAS initial factors."""
    x = np.asarray(x, np.float32)
    modality = np.asarray(modality)
    wmax = cal.weight_range(w)
    y = np.zeros((x.shape[0], np.asarray(w).shape[1]), np.float32)
    for m in range(n_mod):
        rows = np.nonzero(modality == m)[0]
        if rows.size == 0:
            continue
        if smoothing is None:
            s32, inv = cal.smoothing_factor(cal.channel_range(x, modality, m), wmax)
        else:
            s32 = np.asarray(smoothing[m], np.float32)
            inv = (np.float32(1) / s32).astype(np.float32)
        wq, w_scale, _ = cal.quantize_weight(w, s32, weight_bits)
        sub = np.zeros(rows.size, np.int32)
        y[rows] = inf.linear(x[rows], sub, inv[None, :], wq, w_scale)
    return y


def sqnr_db(y_ref, y) -> np.ndarray:
    """Per-token SQNR in dB (eq. sqnr); +inf where the token is reproduced exactly."""
    r = np.asarray(y_ref, np.float64)
    e = r - np.asarray(y, np.float64)
    sig = np.sum(r * r, axis=1)
    err = np.sum(e * e, axis=1)
    with np.errstate(divide="ignore"):
        return np.where(err > 0, 10.0 * np.log10(sig / np.where(err > 0, err, 1.0)), np.inf)
