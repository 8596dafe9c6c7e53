"""Oracle for the offline factors the modality-aware linear consumes.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Written from the paper's definitions, in its order and notation, with dense
fp64 linear algebra (no thin or randomized shortcuts), so it is meant for
C_in up to a few thousand:

  G1  R^m_i = max_t |x^m_{t,i}|                       (Sec. 4.1, range R^m)
  G2  w_i = max_j |w_{j,i}| over the output channels of input channel i
  G3  s^m_i = sqrt(R^m_i / w_i)                       (Sec. 4.2, MAS initial factors)
  G4  Q(S_t W): per-output-channel symmetric int8 (or 4-bit for W4A8)
                                                      (eq. PTQ, Sec. 4.3; Tables 1-2)
  G5  dW = S_m W - Q(S_t W)                           (Sec. 4.3, residual)
  G6  P Lambda P^T = SVD((X_m S_m^-1)^T (X_m S_m^-1)), T = (P Lambda^1/2)^T
  G7  SVD(T dW) = U Sigma V^T, truncated to rank r
  G8  L1 = T^-1 U_r, L2 = Sigma_r V_r^T               (eq. l1l2)

Readings (listed in the design notes): the covariance gets a ridge
eps * tr(C) / K * I so that T is invertible when a modality has fewer
calibration rows than channels; R and w are floored at 1e-5; the smoothing
factor is stored as s32 = fl(s) and applied as inv_s = fl(1 / s32); the
"fp" difference base (S_m - S_t) W is available beside the paper-literal
quantized base.
"""
import numpy as np

from .bf16 import bf16_round

QMAX = 127
FLOOR = 1e-5


def channel_range(x: np.ndarray, modality: np.ndarray, m: int) -> np.ndarray:
    """G1: R^m_i over the rows of modality m (zeros if it has none)."""
    rows = np.asarray(x, np.float64)[np.asarray(modality) == m]
    if rows.shape[0] == 0:
        return np.zeros(np.asarray(x).shape[1])
    return np.max(np.abs(rows), axis=0)


def weight_range(w: np.ndarray) -> np.ndarray:
    """G2: for W in [C_in][C_out], the max magnitude along each input channel."""
    return np.max(np.abs(np.asarray(w, np.float64)), axis=1)


def smoothing_factor(r: np.ndarray, wmax: np.ndarray):
    """G3 (alpha = 1/2): returns (s32, inv_s32) as float32."""
    s = np.sqrt(np.maximum(r, FLOOR) / np.maximum(wmax, FLOOR))
    s32 = s.astype(np.float32)
    inv = (np.float32(1.0) / s32).astype(np.float32)
    return s32, inv


def quantize_weight(w: np.ndarray, s32_text: np.ndarray, bits: int = 8):
    """G4: Q(S_t W) with one symmetric scale per output channel, b-bit codes
    in [-(2^(b-1) - 1), 2^(b-1) - 1] (b = 8: W8A8; b = 4: the W4A8 setting).

    Returns codes wq [N][K] int8, scales w_scale [N] float32 and the
    dequantized weight wdq [K][N] fp64 (codes times the stored fp32 scale)."""
    qmax = (1 << (bits - 1)) - 1
    ws = np.asarray(s32_text, np.float64)[:, None] * np.asarray(w, np.float64)   # [K][N]
    n = ws.shape[1]
    wq = np.zeros((n, ws.shape[0]), np.int8)
    scale = np.zeros(n, np.float32)
    for o in range(n):
        col = ws[:, o]
        delta = np.max(np.abs(col)) / qmax
        if delta > 0:
            wq[o] = np.clip(np.rint(col / delta), -qmax, qmax).astype(np.int8)
        scale[o] = np.float32(delta)
    wdq = wq.T.astype(np.float64) * scale.astype(np.float64)[None, :]
    return wq, scale, wdq


def weight_difference(w, s32_m, s32_t, wdq, base: str = "quantized") -> np.ndarray:
    """G5: dW for modality m.  'quantized': S_m W - Q(S_t W) as printed in
    Sec. 4.3; 'fp': (S_m - S_t) W, the float cross-modal difference."""
    w = np.asarray(w, np.float64)
    sm = np.asarray(s32_m, np.float64)[:, None]
    if base == "quantized":
        return sm * w - wdq
    if base == "fp":
        return (sm - np.asarray(s32_t, np.float64)[:, None]) * w
    raise ValueError(base)


def whitening(z: np.ndarray, ridge: float = 1e-6):
    """G6: T = (P Lambda^1/2)^T from the eigen-decomposition (the SVD of a
    symmetric PSD matrix) of the smoothed activations' covariance.
    Returns (T, T^-1)."""
    z = np.asarray(z, np.float64)
    c = z.T @ z
    k = c.shape[0]
    if ridge > 0:
        c = c + ridge * (np.trace(c) / k) * np.eye(k)
    lam, p = np.linalg.eigh(c)
    lam = np.maximum(lam, 0.0)
    t = (p * np.sqrt(lam)[None, :]).T
    with np.errstate(divide="ignore"):
        inv_sqrt = np.where(lam > 0, 1.0 / np.sqrt(np.where(lam > 0, lam, 1.0)), 0.0)
    t_inv = p * inv_sqrt[None, :]
    return t, t_inv


def cmc_factors(z: np.ndarray, dw: np.ndarray, rank: int, ridge: float = 1e-6):
    """G7-G8: L1 [K][r] and L2 [r][N] such that dW ~ L1 L2 (eq. l1l2)."""
    k, n = np.asarray(dw).shape
    if rank == 0:
        return np.zeros((k, 0)), np.zeros((0, n))
    t, t_inv = whitening(z, ridge)
    u, sig, vt = np.linalg.svd(t @ np.asarray(dw, np.float64), full_matrices=False)
    r = min(rank, sig.shape[0])
    l1 = np.zeros((k, rank))
    l2 = np.zeros((rank, n))
    l1[:, :r] = t_inv @ u[:, :r]
    l2[:r] = sig[:r, None] * vt[:r]
    return l1, l2


def calibrate(x, modality, w, n_mod: int, rank: int, lr_dtype: str = "f32",
              base: str = "quantized", ridge: float = 1e-6, smoothing=None,
              weight_bits: int = 8) -> dict:
    """All artifacts of one layer in the C library's layouts.

    ``smoothing`` optionally overrides the per-modality factors s32 [M][K];
    ``weight_bits`` = 4 gives the W4A8 setting (the residual dW and the CMC
    factors are then taken against the 4-bit shared weight)."""
    x = np.asarray(x, np.float32)
    modality = np.asarray(modality)
    wmax = weight_range(w)
    if smoothing is None:
        s32 = np.zeros((n_mod, x.shape[1]), np.float32)
        for m in range(n_mod):
            s32[m], _ = smoothing_factor(channel_range(x, modality, m), wmax)
    else:
        s32 = np.asarray(smoothing, np.float32)
    inv = (np.float32(1.0) / s32).astype(np.float32)
    wq, w_scale, wdq = quantize_weight(w, s32[0], weight_bits)
    k, n = x.shape[1], wq.shape[0]
    l_down = np.zeros((max(n_mod - 1, 0), rank, k))
    r_up = np.zeros((max(n_mod - 1, 0), n, rank))
    l1s, l2s = [], []
    for m in range(1, n_mod):
        rows = x[modality == m].astype(np.float64)
        dw = weight_difference(w, s32[m], s32[0], wdq, base)
        if rows.shape[0] == 0:
            l1, l2 = np.zeros((k, rank)), np.zeros((rank, n))
        else:
            z = rows / s32[m].astype(np.float64)[None, :]
            l1, l2 = cmc_factors(z, dw, rank, ridge)
        l1s.append(l1)
        l2s.append(l2)
        l_down[m - 1] = l1.T
        r_up[m - 1] = l2.T
    if lr_dtype == "bf16":
        l_down = bf16_round(l_down.astype(np.float32))
        r_up = bf16_round(r_up.astype(np.float32))
    elif lr_dtype == "f64":        # unrounded factors, for the exactness pins
        pass
    else:
        l_down = l_down.astype(np.float32)
        r_up = r_up.astype(np.float32)
    return dict(s32=s32, inv_smooth=inv, wq=wq, w_scale=w_scale, wdq=wdq,
                l_down=l_down, r_up=r_up, l1=l1s, l2=l2s)
