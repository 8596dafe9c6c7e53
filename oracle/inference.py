"""Oracle for the inference of one modality-aware quantized linear.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The layer (Sec. 4.3, the final case equation): every token row x_t of modality
m is smoothed by S_m^-1 and quantized; all rows multiply the single shared
quantized weight Q(S_t W) (text smoothing, Sec. 4.3 "store only one quantized
weight"); rows of a non-text modality additionally receive the unquantized
low-rank term (x_t S_m^-1) L1^m L2^m.

Readings where the paper is silent (each listed in the design notes):
  * quantizer (eq. PTQ): symmetric, z = 0, [q_min, q_max] = [-127, 127],
    round half to even; activations per token, Delta_t = amax_t / 127, and the
    codes use a multiply by fl(127 / amax_t);
  * S_m^-1 is applied as a multiply by inv_s = fl(1 / s_m);
  * dequantization order: (float(acc) * Delta_t) * Delta_w[o];
  * the compensation is computed in fp64 from the fp32 smoothed row and the
    stored factor values, then added once to the fp32 dequantized product;
  * bf16 outputs: one round-to-nearest-even of the fp32 result.

Array conventions (the C library's layouts):
  x            float32 [T][K]  (bf16 inputs already widened, which is exact)
  modality     int32   [T], 0 = text
  inv_smooth   float32 [M][K]
  wq           int8    [N][K]   = Q(S_t W) transposed (K contiguous)
  w_scale      float32 [N]
  l_down       float   [M-1][r][K] = (L1^m)^T for m = 1..M-1
  r_up         float   [M-1][N][r] = (L2^m)^T
"""
import numpy as np

from .bf16 import bf16_round

QMAX = 127


# O2: smoothing (Sec. 3.1 computational invariance; Sec. 4.3 uses X_m S_m^-1)
def smooth(x: np.ndarray, modality: np.ndarray, inv_smooth: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32)
    inv = np.asarray(inv_smooth, dtype=np.float32)[np.asarray(modality)]
    return (x * inv).astype(np.float32)          # one fp32 multiply per element


# O3-O4: per-token symmetric int8 quantization (eq. PTQ with z = 0)
def quantize_per_token(xs: np.ndarray):
    xs = np.asarray(xs, dtype=np.float32)
    amax = np.max(np.abs(xs), axis=1) if xs.shape[1] else np.zeros(xs.shape[0], np.float32)
    amax = amax.astype(np.float32)
    nz = amax > 0
    safe = np.where(nz, amax, np.float32(1))
    delta = np.where(nz, safe / np.float32(QMAX), np.float32(0)).astype(np.float32)
    rq = np.where(nz, np.float32(QMAX) / safe, np.float32(0)).astype(np.float32)
    scaled = (xs * rq[:, None]).astype(np.float32)
    q = np.clip(np.rint(scaled), -QMAX, QMAX).astype(np.int8)
    return q, delta


def smooth_quant(x, modality, inv_smooth):
    """Codes q [T][K] int8 and per-token scales Delta [T] float32."""
    return quantize_per_token(smooth(x, modality, inv_smooth))


# O5: exact integer product of the codes with the shared weight codes.
def int_gemm(q: np.ndarray, wq: np.ndarray) -> np.ndarray:
    """acc[t, o] = sum_i q[t, i] * wq[o, i] as int32.

    Every partial sum is an integer of magnitude < 2^53, so the fp64 BLAS
    product is exact whatever its blocking or summation order."""
    acc = np.asarray(q, np.float64) @ np.asarray(wq, np.float64).T
    assert np.all(np.abs(acc) < 2.0 ** 31), "int32 accumulator overflow"
    return acc.astype(np.int64).astype(np.int32)


# O6: dequantization of the shared-weight product.
def dequant(acc: np.ndarray, x_scale: np.ndarray, w_scale: np.ndarray) -> np.ndarray:
    a = np.asarray(acc, np.int32).astype(np.float32)            # RNE for |acc| > 2^24
    y = (a * np.asarray(x_scale, np.float32)[:, None]).astype(np.float32)
    return (y * np.asarray(w_scale, np.float32)[None, :]).astype(np.float32)


def w8a8_gemm(q, x_scale, wq, w_scale):
    """int32 accumulators and their dequantized fp32 product (no compensation)."""
    acc = int_gemm(q, wq)
    return acc, dequant(acc, x_scale, w_scale)


# O7: Cross-Modal Compensation term (Sec. 4.3, final case equation).
def compensation(xs: np.ndarray, modality: np.ndarray, l_down, r_up, n_out=None) -> np.ndarray:
    """c[t] = (xs_t L1^m) L2^m for rows with modality m != text, 0 otherwise (fp64)."""
    xs = np.asarray(xs, np.float32)
    modality = np.asarray(modality)
    T = xs.shape[0]
    if n_out is None:
        n_out = np.asarray(r_up).shape[1]
    c = np.zeros((T, n_out), np.float64)
    if l_down is None or len(l_down) == 0:
        return c
    for m in range(1, len(l_down) + 1):
        rows = np.nonzero(modality == m)[0]
        if rows.size == 0:
            continue
        l1 = np.asarray(l_down[m - 1], np.float64).T          # [K][r]
        l2 = np.asarray(r_up[m - 1], np.float64).T            # [r][N]
        u = xs[rows].astype(np.float64) @ l1                  # [rows][r]
        c[rows] = u @ l2
    return c


def dequantized_weight(wq, w_scale) -> np.ndarray:
    """Q(S_t W) in the paper's layout [K][N], fp64."""
    return np.asarray(wq, np.float64).T * np.asarray(w_scale, np.float32).astype(np.float64)[None, :]


def linear(x, modality, inv_smooth, wq, w_scale, l_down=None, r_up=None,
           quantize_activations: bool = True) -> np.ndarray:
    """The layer output Y [T][N] in float32.

    With ``quantize_activations=False`` the activation quantizer is replaced by
    the identity and the product with the (dequantized) shared weight is taken
    in fp64 and returned in fp64 -- the diagnostic used for the
    computational-invariance pins."""
    modality = np.asarray(modality)
    xs = smooth(x, modality, inv_smooth)
    c = compensation(xs, modality, l_down, r_up, n_out=np.asarray(wq).shape[0])
    if quantize_activations:
        q, dx = quantize_per_token(xs)
        _, y0 = w8a8_gemm(q, dx, wq, w_scale)
        y = y0.astype(np.float64) + c
        nontext = modality != 0
        out = y0.copy()
        out[nontext] = y[nontext].astype(np.float32)
        return out
    return xs.astype(np.float64) @ dequantized_weight(wq, w_scale) + c


def lowrank_comp(x, modality, inv_smooth, l_down, r_up, y_in) -> np.ndarray:
    """y_out = y_in + (x S_m^-1 L1^m) L2^m on non-text rows, rounded once to fp32."""
    modality = np.asarray(modality)
    xs = smooth(x, modality, inv_smooth)
    c = compensation(xs, modality, l_down, r_up)
    y_in = np.asarray(y_in, np.float32)
    out = y_in.copy()
    nt = modality != 0
    out[nt] = (y_in[nt].astype(np.float64) + c[nt]).astype(np.float32)
    return out


# O8: output cast.
def to_output(y: np.ndarray, dtype: str) -> np.ndarray:
    y = np.asarray(y, np.float32)
    return bf16_round(y) if dtype == "bf16" else y


def relerr(y: np.ndarray, y_ref: np.ndarray) -> float:
    """max |y - y_ref| / max(|y_ref|, rms of the reference row): a per-element
    relative error that stays meaningful at outputs near zero."""
    y = np.asarray(y, np.float64)
    r = np.asarray(y_ref, np.float64)
    if r.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(r * r, axis=1, keepdims=True))
    den = np.maximum(np.abs(r), rms)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(y - r) / den))
