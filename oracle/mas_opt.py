"""Oracle for the MAS factor optimisation (Sec. 4.2: the per-modality MAE
objective, eq. mas_quant; the loss weights lambda_m and the two epochs of
the ablation in Sec. 5).

TEST INFRASTRUCTURE ONLY (see the package docstring).

For one modality m with calibration rows X_m [T][K] and the float weight
W [K][N] (paper layout):

  L(S_m) = mean_{t,o} | Q(X_m S_m^-1) Q(S_m W) - X_m W |_{t,o}

with the inference quantizers: per-token symmetric int8 on the fp32
smoothed row (eq. PTQ) and per-output-channel symmetric b-bit on S_m W
(Sec. 4.3).  Readings (listed in the design notes):

* MAE is the mean of the absolute errors over the T x N outputs;
* the straight-through estimator passes each quantizer's gradient as if it
  were the identity, so with Xq = Q(X S^-1) and Wq = Q(S W) dequantized,
  dL/ds_i = sum_{t,o} G_to (-(x_ti / s_i^2) Wq_io + Xq_ti w_io),
  G = sign(Q(X S^-1) Q(S W) - X W) / (T N);
* the factors are optimised in log space, s = exp(theta), with Adam
  (beta1 0.9, beta2 0.999, eps 1e-8, step lr on theta), one step per
  batch of calibration rows, lambda_m multiplying the modality's gradient;
  the factor used in each step is s32 = fl32(exp(theta)), applied as
  fl32(1 / s32) to the activations, exactly as at inference.
"""
import numpy as np

from .calibration import quantize_weight
from .inference import quantize_per_token, smooth


def forward(x, s32, w, bits: int = 8):
    """(Xq [T][K], Wq [K][N], R [T][N]) in fp64: the dequantized operands of
    the quantized product and its residual against X W."""
    x = np.asarray(x, np.float32)
    s32 = np.asarray(s32, np.float32)
    inv = (np.float32(1.0) / s32).astype(np.float32)
    q, delta = quantize_per_token(smooth(x, np.zeros(x.shape[0], np.int64), inv[None, :]))
    xq = q.astype(np.float64) * delta.astype(np.float64)[:, None]
    _, _, wq = quantize_weight(w, s32, bits)                   # [K][N] dequantized
    r = xq @ wq - x.astype(np.float64) @ np.asarray(w, np.float64)
    return xq, wq, r


def mae_loss(x, s32, w, bits: int = 8) -> float:
    """eq. mas_quant as a mean absolute error."""
    return float(np.mean(np.abs(forward(x, s32, w, bits)[2])))


def ste_gradient(x, s32, w, bits: int = 8):
    """(loss, dL/ds [K]) under the straight-through estimator."""
    xq, wq, r = forward(x, s32, w, bits)
    g_out = np.sign(r) / r.size
    a = g_out @ wq.T                                           # [T][K]
    b = xq.T @ g_out                                           # [K][N]
    s = np.asarray(s32, np.float64)
    x64 = np.asarray(x, np.float64)
    grad = -np.sum(x64 * a, axis=0) / (s * s) + np.sum(np.asarray(w, np.float64) * b, axis=1)
    return float(np.mean(np.abs(r))), grad


def adam_step(theta, m1, m2, g, step: int, lr: float, b1=0.9, b2=0.999, eps=1e-8):
    """One Adam update (step counts from 1); returns (theta, m1, m2)."""
    m1 = b1 * m1 + (1 - b1) * g
    m2 = b2 * m2 + (1 - b2) * g * g
    mh = m1 / (1 - b1 ** step)
    vh = m2 / (1 - b2 ** step)
    return theta - lr * mh / (np.sqrt(vh) + eps), m1, m2


def optimise(x, modality, w, s_init, lam=None, epochs: int = 2, batch: int = 256,
             lr: float = 1e-2, bits: int = 8):
    """Optimised factors s32 [M][K] and the per-step losses of each modality:
    for every modality, `epochs` passes over its calibration rows in order,
    in batches of `batch` rows, one Adam step on theta = ln s per batch."""
    x = np.asarray(x, np.float32)
    modality = np.asarray(modality)
    s_init = np.asarray(s_init, np.float32)
    n_mod = s_init.shape[0]
    lam = np.ones(n_mod) if lam is None else np.asarray(lam, np.float64)
    out = s_init.copy()
    losses = []
    for m in range(n_mod):
        rows = x[modality == m]
        hist = []
        if rows.shape[0] == 0 or lam[m] == 0:
            losses.append(hist)
            continue
        theta = np.log(s_init[m].astype(np.float64))
        m1 = np.zeros_like(theta)
        m2 = np.zeros_like(theta)
        step = 0
        for _ in range(epochs):
            for b0 in range(0, rows.shape[0], batch):
                s32 = np.exp(theta).astype(np.float32)
                loss, g = ste_gradient(rows[b0:b0 + batch], s32, w, bits)
                hist.append(loss)
                step += 1
                theta, m1, m2 = adam_step(theta, m1, m2, lam[m] * s32.astype(np.float64) * g,
                                          step, lr)
        out[m] = np.exp(theta).astype(np.float32)
        losses.append(hist)
    return out, losses
