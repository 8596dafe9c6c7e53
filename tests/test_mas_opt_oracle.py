"""Pins of the MAS optimisation oracle (Sec. 4.2, eq. mas_quant; CPU)."""
import numpy as np
import pytest

from oracle import comparators as cmp
from oracle import mas_opt as mo
from oracle.calibration import quantize_weight


def _case(seed, T=24, K=32, N=16):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((T, K)) * rng.uniform(0.2, 8.0, K)).astype(np.float32)
    w = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    s = rng.uniform(0.3, 3.0, K).astype(np.float32)
    return x, w, s


@pytest.mark.parametrize("bits", [8, 4])
def test_ste_gradient_brute_force(bits):
    """The vectorised straight-through gradient against its sum written out
    term by term: dL/ds_i = sum_{t,o} G_to (-(x_ti / s_i^2) Wq_io + Xq_ti w_io)."""
    x, w, s = _case(1, T=3, K=16, N=4)
    xq, wq, r = mo.forward(x, s, w, bits)
    T, K = x.shape
    N = w.shape[1]
    want = np.zeros(K)
    for i in range(K):
        acc = 0.0
        for t in range(T):
            for o in range(N):
                gto = (1.0 if r[t, o] > 0 else -1.0 if r[t, o] < 0 else 0.0) / (T * N)
                acc += gto * (-(float(x[t, i]) / float(s[i]) ** 2) * wq[i, o]
                              + xq[t, i] * float(w[i, o]))
        want[i] = acc
    loss, got = mo.ste_gradient(x, s, w, bits)
    assert np.allclose(got, want, rtol=1e-10, atol=1e-14 * np.abs(want).max())
    assert loss == pytest.approx(np.abs(r).mean(), rel=1e-15)


def test_ste_gradient_is_the_derivative_with_frozen_quantisation_error():
    """With each quantizer's error held at its value at s, the objective is
    smooth in s and its derivative there is the straight-through gradient
    (central differences)."""
    x, w, s = _case(2)
    xq, wq, _ = mo.forward(x, s, w, 8)
    s64 = s.astype(np.float64)
    ex = xq - x.astype(np.float64) / s64[None, :]
    ew = wq - s64[:, None] * w.astype(np.float64)
    xw = x.astype(np.float64) @ w.astype(np.float64)

    def surrogate(sv):
        y = (x.astype(np.float64) / sv[None, :] + ex) @ (sv[:, None] * w.astype(np.float64) + ew)
        return np.mean(np.abs(y - xw))

    _, g = mo.ste_gradient(x, s, w, 8)
    h = 1e-7
    fd = np.array([(surrogate(s64 + h * e) - surrogate(s64 - h * e)) / (2 * h)
                   for e in np.eye(s.size)])
    assert np.allclose(g, fd, rtol=1e-5, atol=1e-7 * np.abs(g).max())


def test_loss_at_the_factors_equals_the_mas_only_layer():
    """eq. mas_quant evaluated through the MAS-only comparator's layer (a
    weight Q(S_m W) per modality, fp32 dequantisation) at the same factors."""
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((40, 48)) * 5).astype(np.float32)
    mod = np.repeat([0, 1], 20).astype(np.int32)
    w = (rng.standard_normal((48, 32)) / 7).astype(np.float32)
    s = rng.uniform(0.5, 2.0, (2, 48)).astype(np.float32)
    y = cmp.mas_only_linear(x, mod, w, 2, smoothing=s)
    xw = x.astype(np.float64) @ w.astype(np.float64)
    for m in (0, 1):
        direct = np.mean(np.abs(y[mod == m].astype(np.float64) - xw[mod == m]))
        assert mo.mae_loss(x[mod == m], s[m], w) == pytest.approx(direct, rel=1e-5)


def test_first_adam_step_moves_every_coordinate_by_lr_against_the_sign():
    g = np.array([3.0, -1e-3, 0.5, -7.0])
    th, _, _ = mo.adam_step(np.zeros(4), np.zeros(4), np.zeros(4), g, 1, 0.1)
    assert np.allclose(th, -0.1 * np.sign(g), rtol=1e-4)


def test_optimisation_lowers_the_loss_from_a_poor_start():
    x, w, s = _case(4, T=64, K=32, N=24)
    s_bad = (s * np.where(np.arange(32) % 2 == 0, 4.0, 0.25)).astype(np.float32)
    mod = np.zeros(64, np.int32)
    s_opt, losses = mo.optimise(x, mod, w, s_bad[None, :], epochs=30, batch=64, lr=0.05)
    assert len(losses[0]) == 30
    assert mo.mae_loss(x, s_opt[0], w) < 0.9 * losses[0][0]


def test_zero_weight_or_absent_modality_keeps_the_initial_factors():
    x, w, s = _case(5)
    mod = np.zeros(x.shape[0], np.int32)                  # modality 1 has no rows
    s2 = np.stack([s, s * 2]).astype(np.float32)
    out, losses = mo.optimise(x, mod, w, s2, lam=[0.0, 1.0], epochs=1, batch=8)
    assert np.array_equal(out, s2) and losses == [[], []]
    out, losses = mo.optimise(x, mod, w, s2, epochs=2, batch=8)
    assert len(losses[0]) == 2 * 3 and not np.array_equal(out[0], s2[0])


def test_weight_quantizer_is_the_inference_one():
    """The forward pass's Wq is Q(S W) of the calibration (eq. PTQ per output
    channel), dequantized."""
    x, w, s = _case(6)
    _, wq, _ = mo.forward(x, s, w, 4)
    codes, scale, wdq = quantize_weight(w, s, 4)
    assert np.array_equal(wq, wdq)
    assert np.abs(codes).max() <= 7
