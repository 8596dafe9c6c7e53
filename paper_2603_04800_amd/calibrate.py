"""Offline calibration: the per-layer artifacts the GPU linear consumes.

Host-side, fp64 NumPy, run once per layer before inference (the paper's
calibration stage, Sec. 4.2-4.3).  Produces, in the C library's layouts:

  inv_smooth [M][K] float32   fl(1 / s^m), s^m_i = sqrt(R^m_i / max_j |w_ji|)
                              (MAS initial factors, Sec. 4.2; R^m from Sec. 4.1)
  wq         [N][K] int8      Q(S_t W), symmetric per output channel (eq. PTQ)
  w_scale    [N]    float32   its scales
  l_down     [M-1][r][K]      (L1^m)^T, L1^m = T_m^-1 U_r        (eq. l1l2)
  r_up       [M-1][N][r]      (L2^m)^T, L2^m = Sigma_r V_r^T
                              from the truncated SVD of T_m dW_m, where
                              dW_m = S_m W - Q(S_t W) and T_m whitens
                              X_m S_m^-1 (Sec. 4.3)

Built for large layers: the whitening is never formed as a K x K matrix when
a modality has fewer calibration rows than channels (a thin SVD of the
smoothed activations gives it in closed form), and the rank-r truncation uses a
seeded randomized SVD (Halko, Martinsson and Tropp 2011, oversampling 10, two
power iterations) when min(K, N) is large.  For small layers the truncation
is an exact dense SVD.

The covariance gets a ridge eps * tr(C) / K * I (eps = 1e-6) so that T_m is
invertible when a modality has fewer rows than channels.
"""
from __future__ import annotations

import numpy as np

QMAX = 127
FLOOR = 1e-5
EXACT_SVD_MAX = 1024


def _to_bf16_values(a: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def smoothing_factors(x: np.ndarray, modality: np.ndarray, w: np.ndarray, n_mod: int):
    """(s32 [M][K], inv_s32 [M][K]) from per-modality activation ranges."""
    x = np.asarray(x, np.float32)
    wmax = np.abs(np.asarray(w, np.float32)).max(axis=1).astype(np.float64)
    s32 = np.empty((n_mod, x.shape[1]), np.float32)
    for m in range(n_mod):
        rows = x[modality == m]
        rng = np.abs(rows).max(axis=0).astype(np.float64) if rows.shape[0] else np.zeros(x.shape[1])
        s32[m] = np.sqrt(np.maximum(rng, FLOOR) / np.maximum(wmax, FLOOR)).astype(np.float32)
    inv = (np.float32(1.0) / s32).astype(np.float32)
    return s32, inv


def quantize_shared_weight(w: np.ndarray, s32_text: np.ndarray, bits: int = 8):
    """Q(diag(s_t) W) per output channel -> (wq [N][K] int8, w_scale [N] f32),
    b-bit codes in [-(2^(b-1) - 1), 2^(b-1) - 1] (8, or 4 for W4A8).

    fp64 throughout: s32 * w is exact, the step is one correctly rounded
    division, codes round half to even (torch.round)."""
    import torch
    qmax = (1 << (bits - 1)) - 1
    ws = torch.from_numpy(np.ascontiguousarray(w, np.float32)).double()
    ws.mul_(torch.from_numpy(np.asarray(s32_text, np.float32)).double()[:, None])
    step = ws.abs().amax(dim=0) / qmax
    safe = torch.where(step > 0, step, torch.ones_like(step))
    codes = torch.round(ws.div_(safe[None, :])).clamp_(-qmax, qmax)
    codes[:, step == 0] = 0
    return codes.t().contiguous().to(torch.int8).numpy(), step.float().numpy()


def _weight_difference(w: np.ndarray, s32_m: np.ndarray, wq: np.ndarray, w_scale: np.ndarray):
    """dW = S_m W - Q(S_t W) in fp64 [K][N] (Sec. 4.3)."""
    import torch
    dw = torch.from_numpy(np.ascontiguousarray(w, np.float32)).double()
    dw.mul_(torch.from_numpy(np.asarray(s32_m, np.float32)).double()[:, None])
    wdq = torch.from_numpy(wq).t().double()
    wdq.mul_(torch.from_numpy(np.asarray(w_scale, np.float32)).double()[None, :])
    dw.sub_(wdq)
    return dw.numpy()


class _Whitening:
    """T = C^1/2 and T^-1 for C = Z^T Z + eps' I, applied without forming K x K
    matrices when Z has fewer rows than columns."""

    def __init__(self, z: np.ndarray, ridge: float):
        k = z.shape[1]
        if z.shape[0] >= k:
            c = z.T @ z
            eps = ridge * np.trace(c) / k
            lam, p = np.linalg.eigh(c + eps * np.eye(k))
            lam = np.maximum(lam, 0.0)
            self.mode = "dense"
            self.p = p
            self.sq = np.sqrt(lam)
            self.isq = np.where(lam > 0, 1.0 / np.sqrt(np.where(lam > 0, lam, 1.0)), 0.0)
        else:
            # thin SVD of Z from the eigen-decomposition of its n x n Gram matrix
            mu, uz = np.linalg.eigh(z @ z.T)
            keep = mu > mu.max() * 1e-13 if mu.size and mu.max() > 0 else np.zeros(mu.shape, bool)
            mu, uz = mu[keep], uz[:, keep]
            sig = np.sqrt(mu)
            eps = ridge * np.sum(mu) / k
            self.mode = "thin"
            self.p = (z.T @ uz) / sig[None, :]               # [K][n] orthonormal columns
            self.root_eps = np.sqrt(eps)
            self.sq = np.sqrt(sig ** 2 + eps) - self.root_eps
            with np.errstate(divide="ignore"):
                base = 1.0 / self.root_eps if eps > 0 else 0.0
                self.isq = np.where(sig ** 2 + eps > 0, 1.0 / np.sqrt(sig ** 2 + eps), 0.0) - base
            self.inv_root_eps = base

    def apply(self, a: np.ndarray) -> np.ndarray:          # T @ a
        if self.mode == "dense":
            return self.p @ (self.sq[:, None] * (self.p.T @ a))
        return self.p @ (self.sq[:, None] * (self.p.T @ a)) + self.root_eps * a

    def apply_inv(self, a: np.ndarray) -> np.ndarray:      # T^-1 @ a
        if self.mode == "dense":
            return self.p @ (self.isq[:, None] * (self.p.T @ a))
        return self.p @ (self.isq[:, None] * (self.p.T @ a)) + self.inv_root_eps * a


def _truncated_svd(wh: "_Whitening", dw: np.ndarray, r: int, seed: int):
    """Top-r SVD of T dW.  Small problems: dense SVD of the explicit product.
    Large ones: randomized range finder on T dW applied implicitly (T is
    symmetric, so (T dW)^T q = dW^T (T q)); T dW is never formed."""
    k, n = dw.shape
    if min(k, n) <= EXACT_SVD_MAX or r >= min(k, n) // 2:
        u, s, vt = np.linalg.svd(wh.apply(dw), full_matrices=False)
        return u[:, :r], s[:r], vt[:r]
    rng = np.random.default_rng(seed)
    ell = min(r + 10, k, n)
    q, _ = np.linalg.qr(wh.apply(dw @ rng.standard_normal((n, ell))))
    for _ in range(2):
        q, _ = np.linalg.qr(dw.T @ wh.apply(q))
        q, _ = np.linalg.qr(wh.apply(dw @ q))
    b = (dw.T @ wh.apply(q)).T                           # q^T T dW, ell x n
    ub, s, vt = np.linalg.svd(b, full_matrices=False)
    return (q @ ub)[:, :r], s[:r], vt[:r]


def cmc_factors(z: np.ndarray, dw: np.ndarray, rank: int, ridge: float = 1e-6, seed: int = 0):
    """L1 [K][r], L2 [r][N] with dW ~ L1 L2 minimising ||Z (dW - L1 L2)||_F."""
    k, n = dw.shape
    l1 = np.zeros((k, rank))
    l2 = np.zeros((rank, n))
    if rank == 0 or z.shape[0] == 0 or not np.any(z):
        return l1, l2
    wh = _Whitening(z, ridge)
    u, s, vt = _truncated_svd(wh, dw, min(rank, k, n), seed)
    rr = s.shape[0]
    l1[:, :rr] = wh.apply_inv(u)
    l2[:rr] = s[:, None] * vt
    return l1, l2


class _CholeskyWhitening:
    """The whitening on the GPU: C = Z^T Z (masq_dgemm) + eps I with eps =
    ridge * tr(Z^T Z) / K, factored C = L L^T (masq_cholesky), T = L^T.  T is
    not the symmetric root that _Whitening applies, but T^T T = C is all the
    factors depend on: with T' = Q T (Q orthogonal) the SVD of T' dW has left
    vectors Q U and the same Sigma, V, so T'^-1 (Q U_r) = T^-1 U_r and L2 are
    unchanged (and the seeded range finder's subspaces rotate by Q alike)."""

    def __init__(self, z, ridge: float, info):
        from . import ops
        self.ops = ops
        self.l = ops.dgemm(z.T, z)                            # [K][K], then L in place
        _, self.trace = ops.cholesky(self.l, ridge, info=info)

    def apply(self, a):                                    # T a = L^T a
        return self.ops.dgemm(self.l.T, a)

    def apply_t(self, a):                                  # T^T a = L a
        return self.ops.dgemm(self.l, a)

    def solve_rows(self, ut):                              # rows of (T^-1 U)^T = U^T L^-1
        return self.ops.trsm_right(self.l, ut, trans=False)


class _NoWhitening:
    """T = I: the plain truncated SVD of dW, the non-whitened baseline that
    the paper's SQNR-against-rank comparison sets beside CMC (Sec. 5)."""

    l = None

    def apply(self, a):
        return a

    def apply_t(self, a):
        return a

    def solve_rows(self, ut):
        return ut


class _InfoSlots:
    """Device int32 slots for the info words of every Cholesky factorisation
    of one calibration, checked once at the end (no synchronisation
    between the steps)."""

    def __init__(self, device, n: int = 64):
        import torch
        self.buf = torch.zeros((n,), dtype=torch.int32, device=device)
        self.used = 0

    def next(self):
        if self.used == self.buf.shape[0]:
            raise RuntimeError("too many factorisations for the info slots")
        self.used += 1
        return self.buf[self.used - 1:self.used]

    def failed(self) -> bool:
        return bool(self.buf[:self.used].any().item())


def _cholqr(y, infos: _InfoSlots):
    """Q of Y [m][n] (m >= n) = Q R, in place of Y, by shifted CholeskyQR3
    (Fukaya, Kannan, Nakatsukasa, Yamamoto and Yanagisawa 2020): a first pass
    with G + s I, s = 11 (m n + n (n + 1)) u tr(G) (robust for condition
    numbers up to about 1/u), then two plain passes (CholeskyQR2); each pass
    is G = Y^T Y (masq_dgemm), G + s I = L L^T (masq_cholesky) and Y := Y
    L^-T (masq_trsm_right)."""
    from . import ops
    m, n = y.shape
    shift_ridge = 11.0 * (m * n + n * (n + 1)) * 2.0 ** -53 * n   # s = ridge * tr(G) / n
    for p in range(3):
        g = ops.dgemm(y.T, y)
        ops.cholesky(g, shift_ridge if p == 0 else 0.0, info=infos.next())
        ops.trsm_right(g, y, trans=True)
    return y


def _cmc_factors_device(wh, dw, r: int, seed: int, infos: _InfoSlots):
    """L1^T [r][K] and L2^T [N][r] on the GPU from the whitening wh and dW
    [K][N], as _truncated_svd and cmc_factors define them: the exact SVD of
    T dW for small layers, else the seeded randomized range finder (the same
    Gaussian test matrix as the host's, drawn by NumPy from the seed, with
    CholeskyQR orthogonalisations) and the SVD of q^T T dW.  Each SVD is the
    one-sided Jacobi SVD (masq_jacobi_svd) of the matrix whose columns are
    the rows of the factored matrix M: M^T = U S V^T, so M = V S U^T."""
    import torch

    from . import ops
    k, n = dw.shape
    dev = dw.device
    if min(k, n) <= EXACT_SVD_MAX or r >= min(k, n) // 2:
        if k <= n:
            # M = T dW [K][N]: left vectors V, L2^T = (U S)_r
            a = wh.apply(dw) if wh.l is not None else dw.clone()
            _, us_rows, v_rows, _ = ops.jacobi_svd(a, flags=1)
            return wh.solve_rows(v_rows[:r].contiguous()), us_rows[:r].T
        # M = (T dW)^T = dW^T L [N][K]: T dW = U S V^T with U, V the Jacobi
        # SVD's of the columns of T dW (the rows of M); L2 = S V^T
        at = ops.dgemm(dw.T, wh.l) if wh.l is not None else dw.T.contiguous()
        _, u_rows, vs_rows, _ = ops.jacobi_svd(at, flags=2)
        return wh.solve_rows(u_rows[:r].contiguous()), vs_rows[:r].T
    rng = np.random.default_rng(seed)
    ell = min(r + 10, k, n)
    omega = torch.from_numpy(rng.standard_normal((n, ell))).to(dev)
    q = _cholqr(wh.apply(ops.dgemm(dw, omega)), infos)                # [K][ell]
    for _ in range(2):
        q = _cholqr(ops.dgemm(dw.T, wh.apply_t(q)), infos)            # [N][ell]
        q = _cholqr(wh.apply(ops.dgemm(dw, q)), infos)                # [K][ell]
    # B = q^T T dW = (L q)^T dW [ell][N], its rows the columns of B^T = U S
    # V^T: B = V S U^T, the left vectors of T dW are q V, L2^T = (U S)_r
    b = ops.dgemm(wh.apply_t(q).T, dw)
    _, us_rows, v_rows, _ = ops.jacobi_svd(b, flags=1)
    return wh.solve_rows(ops.dgemm(v_rows[:r], q.T)), us_rows[:r].T


def cmc_factors_gpu(z, dw, rank: int, ridge: float = 1e-6, seed: int = 0,
                    whiten: bool = True):
    """cmc_factors from device inputs: z [n][K] and dw [K][N] fp64 tensors
    (masq_gather_smoothed, masq_weight_difference), every step on the GPU:
    the Gram matrix and its Cholesky factor (the whitening), the exact or
    seeded randomized truncated SVD (CholeskyQR orthogonalisations, Jacobi
    SVD of the small factor) and T^-1 U_r by triangular solves.  Returns host
    L1 [K][r], L2 [r][N] (copied back once, with the check of every
    factorisation's info word).  whiten=False drops the whitening (T = I):
    the best rank-r approximation of dW itself."""
    k, n = dw.shape
    l1 = np.zeros((k, rank))
    l2 = np.zeros((rank, n))
    if rank == 0 or z.shape[0] == 0:
        return l1, l2
    infos = _InfoSlots(dw.device)
    wh = _CholeskyWhitening(z, ridge, infos.next()) if whiten else _NoWhitening()
    rr = min(rank, k, n)
    l1t, l2t = _cmc_factors_device(wh, dw, rr, seed, infos)
    l1t_h, l2t_h = l1t.cpu().numpy(), l2t.cpu().numpy()
    if whiten and float(wh.trace.item()) == 0.0:          # Z = 0: no whitening, no compensation
        return l1, l2
    if infos.failed():
        raise RuntimeError("a Cholesky factorisation of the calibration failed "
                           "(matrix not positive definite)")
    l1[:, :rr] = l1t_h.T
    l2[:rr] = l2t_h.T
    return l1, l2


def calibrate_layer(x: np.ndarray, modality: np.ndarray, w: np.ndarray, n_mod: int,
                    rank: int, lr_dtype: str = "bf16", ridge: float = 1e-6,
                    seed: int = 0, weight_bits: int = 8) -> dict:
    """All inference artifacts of one linear from calibration activations.

    x: [T][K] float32 calibration rows, modality: [T] ids, w: [K][N] float
    weight in the paper's layout.  Returns a dict of NumPy arrays."""
    x = np.asarray(x, np.float32)
    modality = np.asarray(modality, np.int32)
    w = np.asarray(w, np.float32)
    s32, inv = smoothing_factors(x, modality, w, n_mod)
    wq, w_scale = quantize_shared_weight(w, s32[0], weight_bits)
    return _with_cmc_factors(x, modality, w, s32, inv, wq, w_scale, n_mod, rank, lr_dtype,
                             ridge, seed, weight_bits)


def calibrate_layer_gpu(x: np.ndarray, modality: np.ndarray, w: np.ndarray, n_mod: int,
                        rank: int, lr_dtype: str = "bf16", ridge: float = 1e-6,
                        seed: int = 0, weight_bits: int = 8, device: str = "cuda:0",
                        cmc_on_gpu: bool = False, whiten: bool = True) -> dict:
    """calibrate_layer with its exact steps on the GPU: the channel ranges,
    the MAS factors and Q(S_t W) (masq_channel_range, masq_smoothing_factors,
    masq_quantize_weight).  By default the compensation factors (whitening
    and the truncated SVD) are then formed on the host as in calibrate_layer,
    so the result is the same, array for array.  With cmc_on_gpu the
    smoothed rows, dW and every large product of the whitening and the
    truncated SVD run on the GPU too (masq_gather_smoothed,
    masq_weight_difference, masq_dgemm); the factors then equal the host's up
    to rounding.  whiten=False (with cmc_on_gpu) gives the non-whitened
    baseline's factors."""
    import torch

    from . import ops
    x = np.asarray(x, np.float32)
    modality = np.asarray(modality, np.int32)
    w = np.asarray(w, np.float32)
    xt = torch.from_numpy(x).to(device)
    mt = torch.from_numpy(modality).to(device)
    wt = torch.from_numpy(np.ascontiguousarray(w)).to(device)
    rng = ops.channel_range(xt, mt, n_mod)
    s_t, inv_t = ops.smoothing_factors(rng, wt)
    wq_t, ws_t = ops.quantize_weight(wt, s_t[0].contiguous(), bits=weight_bits)
    s32, inv = s_t.cpu().numpy(), inv_t.cpu().numpy()
    wq, w_scale = wq_t.cpu().numpy(), ws_t.cpu().numpy()
    if not cmc_on_gpu:
        return _with_cmc_factors(x, modality, w, s32, inv, wq, w_scale, n_mod, rank, lr_dtype,
                                 ridge, seed, weight_bits)
    k, n = w.shape
    l_down = np.zeros((max(n_mod - 1, 0), rank, k), np.float32)
    r_up = np.zeros((max(n_mod - 1, 0), n, rank), np.float32)
    if rank > 0 and n_mod > 1:
        for m in range(1, n_mod):
            rows = torch.from_numpy(np.flatnonzero(modality == m).astype(np.int32)).to(device)
            sm = s_t[m].contiguous()
            z = ops.gather_smoothed(xt, rows, sm)
            dw = ops.weight_difference(wt, sm, wq_t, ws_t)
            l1, l2 = cmc_factors_gpu(z, dw, rank, ridge, seed + m, whiten=whiten)
            l_down[m - 1] = l1.T
            r_up[m - 1] = l2.T
            del z, dw
    if lr_dtype == "bf16":
        l_down = _to_bf16_values(l_down)
        r_up = _to_bf16_values(r_up)
    return dict(inv_smooth=inv, s32=s32, wq=wq, w_scale=w_scale,
                l_down=np.ascontiguousarray(l_down), r_up=np.ascontiguousarray(r_up),
                rank=rank, n_mod=n_mod, lr_dtype=lr_dtype, weight_bits=weight_bits)


def _with_cmc_factors(x, modality, w, s32, inv, wq, w_scale, n_mod, rank, lr_dtype, ridge,
                      seed, weight_bits) -> dict:
    """The compensation factors of every non-text modality against the shared
    weight (wq, w_scale), and the artifact dict."""
    k, n = w.shape
    l_down = np.zeros((max(n_mod - 1, 0), rank, k), np.float32)
    r_up = np.zeros((max(n_mod - 1, 0), n, rank), np.float32)
    if rank > 0 and n_mod > 1:
        for m in range(1, n_mod):
            rows = x[modality == m].astype(np.float64)
            z = rows / s32[m].astype(np.float64)[None, :]
            dw = _weight_difference(w, s32[m], wq, w_scale)
            l1, l2 = cmc_factors(z, dw, rank, ridge, seed + m)
            l_down[m - 1] = l1.T
            r_up[m - 1] = l2.T
    if lr_dtype == "bf16":
        l_down = _to_bf16_values(l_down)
        r_up = _to_bf16_values(r_up)
    return dict(inv_smooth=inv, s32=s32, wq=wq, w_scale=w_scale,
                l_down=np.ascontiguousarray(l_down), r_up=np.ascontiguousarray(r_up),
                rank=rank, n_mod=n_mod, lr_dtype=lr_dtype, weight_bits=weight_bits)


def calibrate_smoothquant(x: np.ndarray, w: np.ndarray, n_mod: int, lr_dtype: str = "bf16",
                          weight_bits: int = 8) -> dict:
    """The SmoothQuant comparator on the same kernels: one unified factor for
    every token, s^uni_i = sqrt(max_t |x_ti| / max_j |w_ji|) over the rows of
    all modalities (Sec. 4.1), the shared weight Q(S^uni W), no compensation
    (rank 0).  inv_smooth repeats the unified factor for each modality id."""
    x = np.asarray(x, np.float32)
    w = np.asarray(w, np.float32)
    s32, _ = smoothing_factors(x, np.zeros(x.shape[0], np.int32), w, 1)
    wq, w_scale = quantize_shared_weight(w, s32[0], weight_bits)
    k, n = w.shape
    inv = (np.float32(1.0) / s32).astype(np.float32)
    return dict(inv_smooth=np.ascontiguousarray(np.repeat(inv, n_mod, axis=0)),
                s32=np.repeat(s32, n_mod, axis=0), wq=wq, w_scale=w_scale,
                l_down=np.zeros((max(n_mod - 1, 0), 0, k), np.float32),
                r_up=np.zeros((max(n_mod - 1, 0), n, 0), np.float32),
                rank=0, n_mod=n_mod, lr_dtype=lr_dtype, weight_bits=weight_bits)


def calibrate_mas_only(x: np.ndarray, modality: np.ndarray, w: np.ndarray, n_mod: int,
                       lr_dtype: str = "bf16") -> dict:
    """The MAS-only comparator (Sec. 4.2, without the shared weight): the
    per-modality MAS factors as for MASQuant, and one int8 weight per
    modality, Q(S_m W) per output channel; no compensation.  wq [M][N][K],
    w_scale [M][N]."""
    x = np.asarray(x, np.float32)
    w = np.asarray(w, np.float32)
    s32, inv = smoothing_factors(x, np.asarray(modality, np.int32), w, n_mod)
    qs = [quantize_shared_weight(w, s32[m], 8) for m in range(n_mod)]
    k, n = w.shape
    return dict(inv_smooth=inv, s32=s32, wq=np.stack([q for q, _ in qs]),
                w_scale=np.stack([sc for _, sc in qs]),
                l_down=np.zeros((max(n_mod - 1, 0), 0, k), np.float32),
                r_up=np.zeros((max(n_mod - 1, 0), n, 0), np.float32),
                rank=0, n_mod=n_mod, lr_dtype=lr_dtype, weight_bits=8)
