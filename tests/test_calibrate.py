"""The product's offline calibration against the oracle's dense, literal one,
and the seeded input generator.  CPU only."""
import numpy as np
import pytest

from oracle import calibration as ocal
from paper_2603_04800_amd import calibrate as pcal
import synth


def _layer(seed, counts=(80, 60, 40), K=48, N=40, scales=(1.0, 30.0, 2.0)):
    rng = np.random.default_rng(seed)
    mod = np.concatenate([np.full(c, m, np.int32) for m, c in enumerate(counts)])
    x = rng.standard_normal((mod.size, K)).astype(np.float32)
    for m in range(len(counts)):
        x[mod == m] *= np.float32(scales[m])
    x[:, 3:5] *= 20
    w = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    return x, mod, w


@pytest.mark.parametrize("counts", [(80, 60, 40), (50, 20, 8), (70, 0, 30)])
def test_product_calibration_matches_oracle(counts):
    x, mod, w = _layer(1, counts)
    p = pcal.calibrate_layer(x, mod, w, 3, rank=16, lr_dtype="f32")
    o = ocal.calibrate(x, mod, w, 3, rank=16, lr_dtype="f64")
    assert np.array_equal(p["s32"], o["s32"])
    assert np.array_equal(p["inv_smooth"], o["inv_smooth"])
    assert np.array_equal(p["wq"], o["wq"])
    assert np.array_equal(p["w_scale"], o["w_scale"])
    for m in (1, 2):
        lp = p["l_down"][m - 1].astype(np.float64).T @ p["r_up"][m - 1].astype(np.float64).T
        lo = o["l1"][m - 1] @ o["l2"][m - 1]
        scale = max(np.abs(lo).max(), 1e-30)
        assert np.abs(lp - lo).max() <= 1e-5 * scale, m


def test_randomized_truncation_is_near_optimal(monkeypatch):
    """Large layers use a randomized SVD; its whitened loss must sit within a
    few percent of the Eckart-Young optimum (Theorem 2)."""
    monkeypatch.setattr(pcal, "EXACT_SVD_MAX", 16)
    rng = np.random.default_rng(4)
    K, N, r = 96, 80, 8
    z = rng.standard_normal((50, K)) * rng.uniform(0.2, 4, K)[None, :]
    # a residual with a decaying spectrum, like a whitened modality difference
    u, _ = np.linalg.qr(rng.standard_normal((K, K)))
    v, _ = np.linalg.qr(rng.standard_normal((N, N)))
    dw = (u[:, :N] * (0.8 ** np.arange(N))) @ v.T
    l1, l2 = pcal.cmc_factors(z, dw, r, ridge=1e-6, seed=0)
    o1, o2 = ocal.cmc_factors(z, dw, r, ridge=1e-6)
    c = z.T @ z
    c += 1e-6 * np.trace(c) / K * np.eye(K)
    lam, p = np.linalg.eigh(c)
    t = (p * np.sqrt(lam)) @ p.T

    def loss(a, b):
        return np.linalg.norm(t @ (dw - a @ b)) ** 2

    assert loss(l1, l2) <= loss(o1, o2) * 1.02


def test_thin_whitening_equals_dense():
    rng = np.random.default_rng(5)
    z = rng.standard_normal((12, 40)) * rng.uniform(0.5, 3, 40)[None, :]
    a = rng.standard_normal((40, 7))
    thin = pcal._Whitening(z, 1e-3)
    assert thin.mode == "thin"
    t, t_inv = ocal.whitening(z, 1e-3)
    c = t.T @ t
    # T^T T equals the regularised covariance for both; the product's T is its symmetric root
    ta = thin.apply(np.eye(40))
    assert np.allclose(ta @ ta, c, rtol=1e-9, atol=1e-9 * np.abs(c).max())
    assert np.allclose(thin.apply_inv(thin.apply(a)), a, atol=1e-8)


def test_bf16_factor_rounding_matches_oracle():
    x, mod, w = _layer(2)
    p = pcal.calibrate_layer(x, mod, w, 3, rank=16, lr_dtype="bf16")
    from oracle.bf16 import bf16_round
    assert np.array_equal(p["l_down"], bf16_round(p["l_down"]))
    assert np.array_equal(p["r_up"], bf16_round(p["r_up"]))


def test_synth_is_deterministic_and_shaped():
    cfg = synth.CONFIGS[3]
    a = synth.make_modality_layout(cfg.counts, cfg.layout, cfg.index)
    b = synth.make_modality_layout(cfg.counts, cfg.layout, cfg.index)
    assert np.array_equal(a, b)
    assert [int((a == m).sum()) for m in range(3)] == list(cfg.counts)
    # runs of 64..512 tokens, adjacent runs of different modality
    edges = np.flatnonzero(np.diff(a)) + 1
    runs = np.diff(np.concatenate([[0], edges, [a.size]]))
    assert runs.min() >= 64 and runs.max() <= 1024


def test_synth_distributions():
    cfg = synth.CONFIGS[0]
    li = synth.make_layer_inputs(cfg)
    x = li.x["x"]
    mod = li.modality
    assert x.shape == (256, 512) and x.dtype == np.float32
    text, vis = x[mod == 0], x[mod == 1]
    big = np.abs(text).max(axis=0) > 15
    assert big.sum() == 8                                    # 8 outlier channels
    assert 20 < np.median(np.abs(vis)) / np.median(np.abs(text)) < 40
    w = li.w["linear"]
    assert w.shape == (512, 512) and abs(w.std() * np.sqrt(512) - 1) < 0.02
    again = synth.make_layer_inputs(cfg)
    assert np.array_equal(again.x["x"], x)


def test_synth_bf16_inputs_are_representable():
    cfg = synth.CONFIGS[2]
    li = synth.make_layer_inputs(cfg)
    x = li.x["x"]
    bits = x.view(np.uint32)
    assert not np.any(bits & 0xFFFF)


def _host_factorisation_calls(monkeypatch):
    """ops.dgemm, cholesky, trsm_right and jacobi_svd replaced by CPU
    computations that follow the C ABI's contracts (masq.h), so that the
    GPU calibration driver's host logic runs here."""
    import torch

    from paper_2603_04800_amd import ops

    def dgemm(a, b, c=None, beta=0.0, stream=None):
        out = a @ b
        if c is not None:
            c.copy_(out + beta * c)
            return c
        return out.contiguous()

    def cholesky(a, ridge=0.0, info=None, trace=None, stream=None):
        n = a.shape[0]
        info = torch.zeros((1,), dtype=torch.int32) if info is None else info
        trace = torch.zeros((1,), dtype=torch.float64) if trace is None else trace
        tr = torch.trace(a)
        trace.fill_(tr)
        a += ridge * tr / n * torch.eye(n, dtype=a.dtype)
        low, bad = torch.linalg.cholesky_ex(torch.tril(a) + torch.tril(a, -1).T)
        info.fill_(int(bad))
        a.copy_(low if int(bad) == 0 else torch.eye(n, dtype=a.dtype))
        return info, trace

    def trsm_right(l, y, trans, stream=None):
        # X L^T = Y  <=>  L X^T = Y^T;  X L = Y  <=>  L^T X^T = Y^T
        x = torch.linalg.solve_triangular(l if trans else l.T, y.T, upper=not trans).T
        y.copy_(x)
        return y

    def jacobi_svd(cols, flags=0, max_sweeps=60, stream=None):
        n, m = cols.shape
        u, s, vh = torch.linalg.svd(cols.T, full_matrices=True)     # [m][m], [k], [n][n]
        k = s.shape[0]
        sigma = torch.zeros(n, dtype=torch.float64)
        sigma[:k] = s
        ur = torch.zeros((n, m), dtype=torch.float64)
        ur[:k] = u[:, :k].T
        if flags & 1:
            ur *= sigma[:, None]
        vr = vh.clone()
        if flags & 2:
            vr *= sigma[:, None]
        return sigma, ur, vr, torch.ones(1, dtype=torch.int32)

    for name, fn in (("dgemm", dgemm), ("cholesky", cholesky), ("trsm_right", trsm_right),
                     ("jacobi_svd", jacobi_svd)):
        monkeypatch.setattr(ops, name, fn)


def test_gpu_cmc_driver_logic_with_host_products(monkeypatch):
    """The GPU compensation-factor driver (cmc_factors_gpu) with the GEMM and
    the factorisation calls replaced by CPU computations of their contracts:
    the same L1 L2 as the host calibration for more and fewer rows than
    channels, the exact SVD in both orientations (K <= N, K > N), the
    randomized truncation, and without whitening.  This checks the driver's
    host logic (which factor multiplies which, transposes, orientations);
    the kernels themselves are GPU tests."""
    import torch

    _host_factorisation_calls(monkeypatch)
    monkeypatch.setattr(pcal, "EXACT_SVD_MAX", 16)
    rng = np.random.default_rng(8)
    for n_rows, K, N, r in ((120, 64, 48, 8), (30, 64, 48, 8), (120, 40, 24, 20),
                            (120, 14, 40, 6), (90, 40, 12, 6)):
        z = rng.standard_normal((n_rows, K)) * rng.uniform(0.2, 4, K)[None, :]
        dw = rng.standard_normal((K, N))
        l1, l2 = pcal.cmc_factors_gpu(torch.from_numpy(z), torch.from_numpy(dw), r, seed=3)
        h1, h2 = pcal.cmc_factors(z, dw, r, seed=3)
        lp, lo = l1 @ l2, h1 @ h2
        assert np.abs(lp - lo).max() <= 1e-9 * np.abs(lo).max(), (n_rows, K, N, r)
    for K, N, r in ((14, 12, 4), (12, 14, 5)):                  # exact SVD, both orientations
        z = rng.standard_normal((50, K))
        dw = rng.standard_normal((K, N))
        l1, l2 = pcal.cmc_factors_gpu(torch.from_numpy(z), torch.from_numpy(dw), r, whiten=False)
        u, s, vt = np.linalg.svd(dw, full_matrices=False)
        best = (u[:, :r] * s[:r]) @ vt[:r]
        assert np.abs(l1 @ l2 - best).max() <= 1e-10 * np.abs(best).max()
    l1, l2 = pcal.cmc_factors_gpu(torch.zeros((0, 64), dtype=torch.float64),
                                  torch.from_numpy(rng.standard_normal((64, 48))), 8)
    assert not np.any(l1) and not np.any(l2)
    l1, l2 = pcal.cmc_factors_gpu(torch.zeros((10, 64), dtype=torch.float64),
                                  torch.from_numpy(rng.standard_normal((64, 48))), 8)
    assert not np.any(l1) and not np.any(l2)
