"""Synthetic analogues of the paper's two analyses of the compensation
(Sec. 4.3 and 5): the effective rank of the weight difference dW_m before
and after whitening, and the output SQNR (eq. sqnr) against the rank ratio
r / min(C_in, C_out), whitened (CMC) and not, beside the rank-0 shared
weight, the SmoothQuant comparator (one unified factor) and MAS-only (a
weight per modality).  Everything runs on the library's GPU calls: the
calibration (calibrate_layer_gpu with the compensation on the GPU), the
reference product X W (masq_dgemm) and the quantized layers.

Effective rank (the paper names the measure without defining it; this is
the usual entropy form of Roy and Vetterli, 2007): exp(-sum_i p_i ln p_i)
with p_i = sigma_i / sum_j sigma_j over the singular values of the matrix.
"""
from __future__ import annotations

import numpy as np


def effective_rank(sigma: np.ndarray) -> float:
    """exp of the Shannon entropy of the normalised singular values."""
    s = np.asarray(sigma, np.float64)
    s = s[s > 0]
    if s.size == 0:
        return 0.0
    p = s / s.sum()
    return float(np.exp(-np.sum(p * np.log(p))))


def sqnr_db(y_ref: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Per-token SQNR in dB: 10 log10(||y_ref||^2 / ||y_ref - y||^2)."""
    r = np.asarray(y_ref, np.float64)
    e = r - np.asarray(y, np.float64)
    num, den = np.einsum("ij,ij->i", r, r), np.einsum("ij,ij->i", e, e)
    with np.errstate(divide="ignore"):
        return np.where(den > 0, 10.0 * np.log10(num / np.where(den > 0, den, 1.0)), np.inf)


def _singular_values_gpu(a):
    """Singular values (decreasing) of a device fp64 matrix whose smaller
    dimension is at most 1024: the one-sided Jacobi SVD (masq_jacobi_svd) of
    the matrix whose columns are the rows (or the columns) of a."""
    from . import ops
    cols = a.clone() if a.shape[0] <= a.shape[1] else a.T.contiguous()
    sigma, _, _, _ = ops.jacobi_svd(cols)
    return sigma.cpu().numpy()


def cmc_study(workload: int, ranks=None, weight_bits: int = 4, device: str = "cuda:0"):
    """Rows of the two analyses for one projection of a benchmark workload.
    Returns a list of dicts (one per measurement)."""
    import torch

    import synth

    from . import calibrate, ops
    cfg = synth.CONFIGS[workload]
    p = cfg.projections[0]
    li = synth.make_layer_inputs(cfg, 0, projections=[p.name])
    x = np.asarray(li.x[p.input_key], np.float32)
    mod = np.asarray(li.modality, np.int32)
    w = np.asarray(li.w[p.name], np.float32)
    k, n = w.shape
    if ranks is None:
        ranks = [r for r in (0, 16, 32, 48, 64, 96, 128, 192, 256) if r <= min(k, n)]
    top = max(ranks)
    dev = torch.device(device)
    act = torch.bfloat16 if cfg.act_dtype == "bf16" else torch.float32
    xt = torch.from_numpy(x).to(dev, act)
    mt = torch.from_numpy(mod).to(dev)
    wt = torch.from_numpy(np.ascontiguousarray(w)).to(dev)
    y_ref = ops.dgemm(xt.double(), wt.double()).cpu().numpy()     # unquantised X W
    rows = []

    def sqnr_row(y, **tags):
        s = sqnr_db(y_ref, y.float().cpu().numpy())
        per = {str(m): round(float(np.mean(s[mod == m])), 3) for m in range(cfg.n_mod)
               if np.any(mod == m)}
        rows.append(dict(kind="sqnr", workload=cfg.name, weight_bits=weight_bits, **tags,
                         sqnr_db=per))

    # effective rank of dW_m before and after whitening
    r32 = ops.channel_range(xt, mt, cfg.n_mod)
    s_t, _ = ops.smoothing_factors(r32, wt)
    wq_t, ws_t = ops.quantize_weight(wt, s_t[0].contiguous(), bits=weight_bits)
    for m in range(1, cfg.n_mod):
        sel = torch.from_numpy(np.flatnonzero(mod == m).astype(np.int32)).to(dev)
        if sel.numel() == 0:
            continue
        sm = s_t[m].contiguous()
        z = ops.gather_smoothed(xt, sel, sm)
        dw = ops.weight_difference(wt, sm, wq_t, ws_t)
        wh = calibrate._CholeskyWhitening(z, 1e-6, torch.zeros((1,), dtype=torch.int32,
                                                                device=dev))
        rows.append(dict(kind="effective_rank", workload=cfg.name, modality=m,
                         weight_bits=weight_bits, c_in=k, c_out=n,
                         plain=round(effective_rank(_singular_values_gpu(dw)), 2),
                         whitened=round(effective_rank(_singular_values_gpu(wh.apply(dw))), 2)))
        del z, dw, wh
    # SQNR against the rank ratio: the factors at the largest rank, truncated
    for whiten in (True, False):
        art = calibrate.calibrate_layer_gpu(x, mod, w, cfg.n_mod, top, "f32",
                                            weight_bits=weight_bits, device=device,
                                            cmc_on_gpu=True, whiten=whiten)
        for r in ranks:
            if r == 0 and not whiten:
                continue
            a = dict(art, l_down=art["l_down"][:, :r], r_up=np.ascontiguousarray(art["r_up"][:, :, :r]),
                     lr_dtype=cfg.lr_dtype)
            y = ops.Linear.from_arrays(a, device)(xt, mt, out_dtype=torch.float32)
            sqnr_row(y, method="masquant" if r else "shared weight, rank 0",
                     whitened=whiten if r else None, rank=r,
                     rank_ratio=round(r / min(k, n), 4))
    # the comparators
    art = calibrate.calibrate_smoothquant(x, w, cfg.n_mod, cfg.lr_dtype, weight_bits=weight_bits)
    sqnr_row(ops.Linear.from_arrays(art, device)(xt, mt, out_dtype=torch.float32),
             method="smoothquant")
    if weight_bits == 8:
        art = calibrate.calibrate_mas_only(x, mod, w, cfg.n_mod, cfg.lr_dtype)
        sqnr_row(ops.MasOnlyLinear.from_arrays(art, device)(xt, mt, out_dtype=torch.float32),
                 method="mas-only")
    return rows
