"""MAS factor optimisation on the GPU (Sec. 4.2, eq. mas_quant).

For each modality m, starting from the MAS initial factors, minimise

    L(S_m) = mean | Q(X_m S_m^-1) Q(S_m W) - X_m W |

over the calibration rows of m, with the inference quantizers in the
forward pass (masq_smooth_quant: per-token int8 of the fp32 smoothed row;
masq_quantize_weight: per-output-channel b-bit Q(S_m W)) and the
straight-through estimator in the backward pass.  The factors are optimised
in log space (s = exp(theta)) with Adam, one step per batch of rows, for
`epochs` passes (2, as in the paper's ablation), each modality's gradient
scaled by its loss weight lambda_m (1, as in the paper).  Every product,
quantizer, reduction and the Adam update of theta runs in the library's
kernels (masq_adam_log_step keeps theta, the moments and the next factors on
the device); the losses of the steps are device scalars read once at the
end.
"""
from __future__ import annotations

import numpy as np


class _Step:
    """One modality's forward and straight-through backward pass on a batch."""

    def __init__(self, xb, w64, wt, bits):
        import torch

        from . import ops
        self.ops, self.torch = ops, torch
        self.xb, self.wt, self.w64, self.bits = xb, wt, w64, bits
        dev = xb.device
        ones = torch.ones(xb.shape[1], dtype=torch.float32, device=dev)
        self.x64 = ops.gather_smoothed(xb, torch.arange(xb.shape[0], dtype=torch.int32,
                                                        device=dev), ones)
        self.ref = ops.dgemm(self.x64, w64)                  # X W, fp64
        self.mod0 = torch.zeros(xb.shape[0], dtype=torch.int32, device=dev)

    def device_step(self, s_t, inv_t, loss_out=None):
        """dL/ds [K] fp64 (device) at the factors s_t [K] f32 with inv_t =
        fl32(1 / s_t); the loss goes to the device scalar loss_out."""
        ops = self.ops
        q, delta = ops.smooth_quant(self.xb, self.mod0, inv_t.view(1, -1))
        wq, wd = ops.quantize_weight(self.wt, s_t, bits=self.bits)
        xq = ops.dequantize_rows(q, delta)                   # [T][K]
        wq_t = ops.dequantize_rows(wq, wd)                   # Wq^T [N][K]
        g, _ = ops.mae_sign(ops.dgemm(xq, wq_t.T), self.ref, loss=loss_out)
        a = ops.dgemm(g, wq_t)                               # G Wq^T  [T][K]
        b = ops.dgemm(xq.T, g)                               # Xq^T G  [K][N]
        return ops.mas_gradient(self.x64, a, self.w64, b, s_t)

    def __call__(self, s32: np.ndarray):
        """(loss, dL/ds) at the host factors s32 [K] (float32), copied back:
        for tests and reports (the optimisation itself stays on the device)."""
        torch = self.torch
        dev = self.xb.device
        s_t = torch.from_numpy(np.ascontiguousarray(s32, np.float32)).to(dev)
        inv = torch.from_numpy((np.float32(1.0) / s32).astype(np.float32)).to(dev)
        loss = torch.empty((1,), dtype=torch.float64, device=dev)
        grad = self.device_step(s_t, inv, loss)
        return float(loss.item()), grad.cpu().numpy()


def optimise(x, modality, w, s_init, lam=None, epochs: int = 2, batch: int = 256,
             lr: float = 1e-2, bits: int = 8, device: str = "cuda:0"):
    """Optimised factors s32 [M][K] (float32) and each modality's per-step
    losses.  x [T][K] float32 calibration rows, modality [T] ids, w [K][N]
    float32 weight (paper layout), s_init [M][K] the MAS initial factors."""
    import torch

    from . import ops
    x = np.asarray(x, np.float32)
    modality = np.asarray(modality)
    s_init = np.asarray(s_init, np.float32)
    n_mod = s_init.shape[0]
    lam = np.ones(n_mod) if lam is None else np.asarray(lam, np.float64)
    dev = torch.device(device)
    wt = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(dev)
    w64 = wt.double()
    out = s_init.copy()
    losses = []
    for m in range(n_mod):
        rows = x[modality == m]
        hist = []
        if rows.shape[0] == 0 or lam[m] == 0:
            losses.append(hist)
            continue
        steps = [_Step(torch.from_numpy(np.ascontiguousarray(rows[b0:b0 + batch])).to(dev),
                       w64, wt, bits) for b0 in range(0, rows.shape[0], batch)]
        k_dim = s_init.shape[1]
        theta, m1, m2 = (torch.empty((k_dim,), dtype=torch.float64, device=dev)
                         for _ in range(3))
        s_t = torch.from_numpy(np.ascontiguousarray(s_init[m])).to(dev)
        inv_t = torch.empty_like(s_t)
        ops.adam_log_step(theta, m1, m2, None, s_t, inv_t, 0)     # theta = ln s, s = exp(theta)
        hist_t = torch.empty((epochs * len(steps),), dtype=torch.float64, device=dev)
        k = 0
        for _ in range(epochs):
            for st in steps:
                grad = st.device_step(s_t, inv_t, hist_t[k:k + 1])
                k += 1
                ops.adam_log_step(theta, m1, m2, grad, s_t, inv_t, k, lam=float(lam[m]), lr=lr)
        out[m] = s_t.cpu().numpy()
        losses.append(hist_t.cpu().numpy().tolist())
    return out, losses
