"""GPU parity of the MAS optimisation (Sec. 4.2, eq. mas_quant) against the
oracle (oracle/mas_opt.py), through the C ABI: the dequantisation exact,
the residual sign exact, the gradient within the fp64 rounding of its sums,
and whole optimisations step for step."""
import numpy as np
import pytest
import torch

from oracle import mas_opt as mo

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.fixture(scope="module")
def ops():
    assert torch.cuda.is_available(), "GPU tests need an MI355X visible to torch"
    from paper_2603_04800_amd import ops as o
    return o


@pytest.mark.parametrize("R,C", [(1, 16), (37, 80), (256, 3584)])
def test_dequantize_rows_is_exact(ops, R, C):
    rng = np.random.default_rng(R + C)
    codes = rng.integers(-127, 128, (R, C)).astype(np.int8)
    scale = rng.uniform(1e-4, 3.0, R).astype(np.float32)
    got = ops.dequantize_rows(torch.from_numpy(codes).to(DEV), torch.from_numpy(scale).to(DEV))
    want = codes.astype(np.float64) * scale.astype(np.float64)[:, None]
    assert np.array_equal(got.cpu().numpy().view(np.uint64), want.view(np.uint64))


@pytest.mark.parametrize("n", [1, 4095, 4097, 70000])
def test_mae_sign(ops, n):
    rng = np.random.default_rng(n)
    y = rng.standard_normal(n)
    ref = y + rng.standard_normal(n) * 0.1
    ref[::7] = y[::7]                                       # exact ties give 0
    g, loss_t = ops.mae_sign(torch.from_numpy(y).to(DEV), torch.from_numpy(ref).to(DEV))
    loss = float(loss_t.item())
    assert np.array_equal(g.cpu().numpy(), np.sign(y - ref) / n)
    assert loss == pytest.approx(np.mean(np.abs(y - ref)), rel=1e-13)


def test_mas_gradient_kernel(ops):
    rng = np.random.default_rng(9)
    T, K, N = 70, 96, 80
    x, a = rng.standard_normal((T, K)), rng.standard_normal((T, K))
    w, b = rng.standard_normal((K, N)), rng.standard_normal((K, N))
    s = rng.uniform(0.1, 5.0, K).astype(np.float32)
    got = ops.mas_gradient(*(torch.from_numpy(v).to(DEV) for v in (x, a, w, b, s))).cpu().numpy()
    s64 = s.astype(np.float64)
    want = -np.sum(x * a, 0) / (s64 * s64) + np.sum(w * b, 1)
    scale = np.sum(np.abs(x * a), 0) / (s64 * s64) + np.sum(np.abs(w * b), 1)
    assert np.all(np.abs(got - want) <= 4 * (T + N) * 2.0 ** -53 * scale)


def _case(seed, T, K, N):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((T, K)) * rng.uniform(0.2, 8.0, K)).astype(np.float32)
    x[:, :3] *= 20                                          # outlier channels
    w = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    s = rng.uniform(0.3, 3.0, K).astype(np.float32)
    return x, w, s


def _grad_scale(x, s, w, bits):
    """sum_{t,o} |G_to| (|x_ti| |Wq_io| / s_i^2 + |Xq_ti| |w_io|): the size of
    the terms whose fp64 sums the two sides order differently."""
    xq, wq, r = mo.forward(x, s, w, bits)
    g = np.ones_like(r) / r.size
    s64 = s.astype(np.float64)
    return (np.abs(x).astype(np.float64) * (g @ np.abs(wq).T)).sum(0) / (s64 * s64) + \
        (np.abs(w).astype(np.float64) * (np.abs(xq).T @ g)).sum(1)


@pytest.mark.parametrize("T,K,N,bits", [(70, 96, 80, 8), (70, 96, 80, 4), (256, 512, 512, 8),
                                        (1, 16, 16, 8)])
def test_one_step_matches_the_oracle(ops, T, K, N, bits):
    from paper_2603_04800_amd import mas_opt
    x, w, s = _case(T + K, T, K, N)
    wt = torch.from_numpy(w).to(DEV)
    step = mas_opt._Step(torch.from_numpy(x).to(DEV), wt.double(), wt, bits)
    loss, g = step(s)
    loss_ref, g_ref = mo.ste_gradient(x, s, w, bits)
    assert loss == pytest.approx(loss_ref, rel=1e-12)
    tol = 4 * (K + N + T) * 2.0 ** -53 * _grad_scale(x, s, w, bits)
    assert np.all(np.abs(g - g_ref) <= tol)


@pytest.mark.parametrize("bits", [8, 4])
def test_optimisation_matches_the_oracle(ops, bits):
    """Two epochs over two modalities in ragged batches: the same losses at
    every step and the same final factors (up to the rounding of the
    gradient's fp64 sums carried through Adam)."""
    from paper_2603_04800_amd import mas_opt
    rng = np.random.default_rng(bits)
    x, w, _ = _case(7, 150, 64, 48)
    mod = rng.integers(0, 2, 150).astype(np.int32)
    s0 = rng.uniform(0.3, 3.0, (2, 64)).astype(np.float32)
    got, hist = mas_opt.optimise(x, mod, w, s0, epochs=2, batch=32, lr=1e-2, bits=bits)
    want, hist_ref = mo.optimise(x, mod, w, s0, epochs=2, batch=32, lr=1e-2, bits=bits)
    for h, hr in zip(hist, hist_ref):
        assert len(h) == len(hr) and np.allclose(h, hr, rtol=1e-9)
    assert np.allclose(got, want, rtol=1e-6)


def test_adam_log_step_matches_its_formula(ops):
    """masq_adam_log_step: the moments exactly as their formula in fp64 (one
    rounding an operation), theta within one ulp of it (the square root is
    the device's), the next factors fl32(exp(theta)) within one ulp of the
    host's exp, and their reciprocals correctly rounded from them.  Step 0
    initialises theta = ln s."""
    rng = np.random.default_rng(3)
    K = 1000
    s0 = rng.uniform(0.2, 5.0, K).astype(np.float32)
    theta, m1, m2 = (torch.empty(K, dtype=torch.float64, device=DEV) for _ in range(3))
    s_t = torch.from_numpy(s0.copy()).to(DEV)
    inv_t = torch.empty_like(s_t)
    ops.adam_log_step(theta, m1, m2, None, s_t, inv_t, 0)
    th = np.log(s0.astype(np.float64))
    assert np.all(np.abs(theta.cpu().numpy() - th) <= np.spacing(np.abs(th)))
    assert not m1.cpu().numpy().any() and not m2.cpu().numpy().any()
    s_host = np.exp(theta.cpu().numpy()).astype(np.float32)
    assert np.all(np.abs(s_t.cpu().numpy().view(np.int32) - s_host.view(np.int32)) <= 1)
    lam, lr, b1, b2, eps = 0.7, 1e-2, 0.9, 0.999, 1e-8
    for step in (1, 2, 3):
        g = rng.standard_normal(K)
        s_in = s_t.cpu().numpy().astype(np.float64)
        th, a, v = theta.cpu().numpy(), m1.cpu().numpy(), m2.cpu().numpy()
        ops.adam_log_step(theta, m1, m2, torch.from_numpy(g).to(DEV), s_t, inv_t, step,
                          lam=lam, lr=lr, b1=b1, b2=b2, eps=eps)
        gg = (lam * s_in) * g
        a = b1 * a + (1 - b1) * gg
        v = b2 * v + ((1 - b2) * gg) * gg
        th = th - (lr * (a / (1 - b1 ** step))) / (np.sqrt(v / (1 - b2 ** step)) + eps)
        assert np.array_equal(m1.cpu().numpy(), a) and np.array_equal(m2.cpu().numpy(), v)
        # (sqrt and exp are the device's: theta within one ulp of the host's)
        assert np.all(np.abs(theta.cpu().numpy() - th) <= np.spacing(np.abs(th)))
        th = theta.cpu().numpy()
        s_new = s_t.cpu().numpy()
        assert np.all(np.abs(s_new.view(np.int32) - np.exp(th).astype(np.float32).view(np.int32))
                      <= 1)
        assert np.array_equal(inv_t.cpu().numpy(), np.float32(1.0) / s_new)


def test_mae_loss_sums_the_blocks_in_order(ops):
    """The loss of masq_mae_loss is the blocks' sum in index order over the
    count, exactly (and 0 for an empty problem)."""
    rng = np.random.default_rng(4)
    n = 3 * 4096 + 17
    y, ref = rng.standard_normal(n), rng.standard_normal(n)
    g, loss = ops.mae_sign(torch.from_numpy(y).to(DEV), torch.from_numpy(ref).to(DEV))
    blocks = [np.abs(y[b:b + 4096] - ref[b:b + 4096]) for b in range(0, n, 4096)]
    assert abs(float(loss.item()) - np.mean(np.abs(y - ref))) <= 1e-14
    assert len(blocks) == int(ops._lib.masq_mae_partials(n))
