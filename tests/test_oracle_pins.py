"""Pins of the CPU oracle to facts fixed by the paper and by mathematics.

None of these re-types an oracle formula: each checks a property, a special
case, a brute-force enumeration with scalar arithmetic, or an independent
library routine.  Runs on the CPU only.
"""
import numpy as np
import pytest
import torch

from oracle import bf16 as obf
from oracle import calibration as cal
from oracle import inference as inf


# --------------------------------------------------------------------------- bf16
def test_bf16_widening_exhaustive():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = obf.bf16_bits_to_f32(bits)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    same = (ours.view(np.uint32) == ref.view(np.uint32)) | (np.isnan(ours) & np.isnan(ref))
    assert same.all()


def test_bf16_narrowing_matches_torch():
    rng = np.random.default_rng(7)
    mags = rng.standard_normal(200000) * 10.0 ** rng.integers(-30, 30, 200000)
    vals = [mags.astype(np.float32)]
    # exact ties (low 16 bits = 0x8000) with both parities, and neighbours
    hi = rng.integers(0, 1 << 15, 50000).astype(np.uint32) << np.uint32(16)
    for low in (0x7FFF, 0x8000, 0x8001):
        vals.append((hi | np.uint32(low)).view(np.float32))
    vals.append(np.array([0.0, -0.0, 3.4e38, -3.4e38, 1e-40, -1e-40, np.inf, -np.inf], np.float32))
    x = np.concatenate(vals).astype(np.float32)
    ours = obf.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(x)
    assert nan.sum() > 0 and np.array_equal(ours[~nan], ref[~nan])
    # NaN payloads are not canonicalised alike; both must stay NaN
    assert np.isnan(obf.bf16_bits_to_f32(ours[nan])).all()


# ----------------------------------------------------------- quantization (O2-O4)
def _brute_quant(x, mod, inv):
    """Scalar loops with numpy.float32 scalars and Python's round (half to even)."""
    T, K = x.shape
    q = np.zeros((T, K), np.int64)
    d = np.zeros(T, np.float32)
    for t in range(T):
        xs = [np.float32(x[t, i]) * np.float32(inv[mod[t], i]) for i in range(K)]
        a = np.float32(0)
        for v in xs:
            a = max(a, abs(v))
        if a == 0:
            continue
        d[t] = np.float32(a) / np.float32(127)
        rq = np.float32(127) / np.float32(a)
        for i in range(K):
            v = round(float(np.float32(xs[i] * rq)))
            q[t, i] = min(127, max(-127, v))
    return q, d


@pytest.mark.parametrize("seed", range(6))
def test_quant_brute_force(seed):
    rng = np.random.default_rng(seed)
    T, K, M = 8, 32, 3
    x = (rng.standard_normal((T, K)) * rng.choice([0.01, 1, 30, 1e4], (T, 1))).astype(np.float32)
    x[3] = 0.0                                       # all-zero row
    x[5, :4] = np.float32(2.5)                       # repeated magnitudes
    mod = rng.integers(0, M, T).astype(np.int32)
    inv = rng.uniform(0.05, 4, (M, K)).astype(np.float32)
    q_ref, d_ref = _brute_quant(x, mod, inv)
    q, d = inf.smooth_quant(x, mod, inv)
    assert np.array_equal(q.astype(np.int64), q_ref)
    assert np.array_equal(d.view(np.uint32), d_ref.view(np.uint32))


def test_quant_ties_round_to_even():
    # rq = 127 / 127 = 1 exactly, so the codes are rint of the values themselves
    xs = np.array([[127.0, 0.5, 1.5, 2.5, -0.5, -1.5, 3.5, -126.5]], np.float32)
    q, d = inf.quantize_per_token(xs)
    assert d[0] == np.float32(1.0)
    assert q[0].tolist() == [127, 0, 2, 2, 0, -2, 4, -126]


def test_quant_properties():
    rng = np.random.default_rng(11)
    xs = (rng.standard_normal((4000, 96)) * rng.lognormal(0, 3, (4000, 1))).astype(np.float32)
    xs[17] = 0
    q, d = inf.quantize_per_token(xs)
    nz = d > 0
    # the largest magnitude maps to +-127 and nothing exceeds it
    assert np.all(np.abs(q).max(axis=1)[nz] == 127)
    assert np.abs(q.astype(int)).max() <= 127 and (q != -128).all()
    # zero rows give a zero scale and zero codes
    assert d[17] == 0 and not q[17].any()
    # eq. PTQ rounds to the nearest level: |x - q * delta| <= delta / 2
    err = np.abs(xs.astype(np.float64) - q.astype(np.float64) * d[:, None].astype(np.float64))
    assert np.all(err <= d[:, None] * (0.5 + 1e-5))
    # re-quantizing the dequantized row returns the same codes
    q2, _ = inf.quantize_per_token((q.astype(np.float32) * d[:, None]).astype(np.float32))
    assert np.array_equal(q, q2)
    # sign symmetry of the symmetric quantizer
    qn, dn = inf.quantize_per_token(-xs)
    assert np.array_equal(qn, -q) and np.array_equal(dn, d)


def test_smoothing_reduces_to_plain_per_token_quant_when_s_is_one():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((16, 64)).astype(np.float32)
    mod = np.zeros(16, np.int32)
    q, d = inf.smooth_quant(x, mod, np.ones((1, 64), np.float32))
    scale = np.abs(x).max(axis=1) / 127
    ref = np.clip(np.rint(x / scale[:, None]), -127, 127)
    # multiply-by-reciprocal and divide may differ by one code at a tie boundary
    assert np.abs(q - ref).max() <= 1 and np.mean(q == ref) > 0.999


# -------------------------------------------------------------- int GEMM (O5-O6)
def test_int_gemm_two_exact_methods():
    rng = np.random.default_rng(5)
    q = rng.integers(-127, 128, (37, 300)).astype(np.int8)
    w = rng.integers(-127, 128, (53, 300)).astype(np.int8)
    ref = np.einsum("ti,oi->to", q.astype(np.int64), w.astype(np.int64))
    assert np.array_equal(inf.int_gemm(q, w).astype(np.int64), ref)


def test_int_gemm_extreme_magnitude_is_exact():
    k = 18944
    q = np.full((2, k), 127, np.int8)
    q[1] = -127
    w = np.full((3, k), 127, np.int8)
    w[2, ::2] = -127
    acc = inf.int_gemm(q, w)
    assert acc[0, 0] == 127 * 127 * k and acc[1, 1] == -127 * 127 * k and acc[0, 2] == 0


def test_int_gemm_known_answers():
    rng = np.random.default_rng(6)
    w = rng.integers(-127, 128, (24, 64)).astype(np.int8)
    ones = np.ones((3, 64), np.int8)
    assert np.array_equal(inf.int_gemm(ones, w), np.tile(w.astype(np.int64).sum(1), (3, 1)))
    q = rng.integers(-127, 128, (5, 64)).astype(np.int8)
    eye = (127 * np.eye(64)).astype(np.int8)
    assert np.array_equal(inf.int_gemm(q, eye), 127 * q.astype(np.int32))


def test_dequant_brute_force():
    rng = np.random.default_rng(8)
    acc = rng.integers(-(2 ** 30), 2 ** 30, (6, 9)).astype(np.int32)
    acc[0, 0] = 2 ** 24 + 1                           # not representable in fp32
    dx = rng.uniform(1e-3, 5, 6).astype(np.float32)
    ws = rng.uniform(1e-4, 1, 9).astype(np.float32)
    y = inf.dequant(acc, dx, ws)
    for t in range(6):
        for o in range(9):
            ref = np.float32(np.float32(float(acc[t, o])) * dx[t]) * ws[o]
            assert y[t, o].view(np.uint32) == np.float32(ref).view(np.uint32)


# -------------------------------------------------------- compensation (O7)
def test_compensation_brute_force_and_routing():
    rng = np.random.default_rng(9)
    T, K, N, r, M = 7, 12, 10, 3, 3
    xs = rng.standard_normal((T, K)).astype(np.float32)
    mod = np.array([0, 1, 2, 2, 0, 1, 2], np.int32)
    ld = rng.standard_normal((M - 1, r, K))
    ru = rng.standard_normal((M - 1, N, r))
    c = inf.compensation(xs, mod, ld, ru)
    for t in range(T):
        for o in range(N):
            if mod[t] == 0:
                assert c[t, o] == 0.0
                continue
            s = 0.0
            for k in range(r):
                u = sum(float(xs[t, i]) * ld[mod[t] - 1, k, i] for i in range(K))
                s += u * ru[mod[t] - 1, o, k]
            assert abs(c[t, o] - s) <= 1e-12 * (1 + abs(s))


def _round_f32_once(v):
    """The binary32 value nearest to the rational v, ties to even: one rounding
    of the exact value (the nearest double's binary32 neighbours are the only
    candidates, chosen by exact rational distance)."""
    from fractions import Fraction
    f = np.float32(float(v))
    cands = [f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(-np.inf))]
    dist = [abs(Fraction(float(c)) - v) for c in cands]
    best = min(dist)
    tied = [c for c, d in zip(cands, dist) if d == best]
    if len(tied) > 1:
        tied = [c for c in tied if int(c.view(np.uint32)) % 2 == 0]
    return np.float32(tied[0])


def test_lowrank_comp_brute_force_one_rounding():
    """The reference of the standalone compensation call (Sec. 4.3, final case
    equation): text rows of y_in come back bit for bit; a row of modality m is
    y_in + (xs L1^m) L2^m computed exactly in rationals, with xs = fl(x inv_s)
    in float32 scalars, and rounded once to binary32."""
    from fractions import Fraction
    rng = np.random.default_rng(11)
    T, K, N, r, M = 9, 8, 6, 2, 3
    x = (rng.standard_normal((T, K)) * 3).astype(np.float32)
    mod = np.array([0, 1, 2, 0, 2, 1, 1, 0, 2], np.int32)
    inv = rng.uniform(0.2, 3, (M, K)).astype(np.float32)
    ld = rng.standard_normal((M - 1, r, K)).astype(np.float32)
    ru = rng.standard_normal((M - 1, N, r)).astype(np.float32)
    y_in = rng.standard_normal((T, N)).astype(np.float32)
    out = inf.lowrank_comp(x, mod, inv, ld, ru, y_in)
    assert out.dtype == np.float32 and out.shape == (T, N)
    twice = 0                         # elements where rounding the term first would differ
    for t in range(T):
        m = int(mod[t])
        if m == 0:
            assert np.array_equal(out[t].view(np.uint32), y_in[t].view(np.uint32))
            continue
        xs = [Fraction(float(np.float32(x[t, i]) * np.float32(inv[m, i]))) for i in range(K)]
        u = [sum(xs[i] * Fraction(float(ld[m - 1, k, i])) for i in range(K)) for k in range(r)]
        for o in range(N):
            c = sum(u[k] * Fraction(float(ru[m - 1, o, k])) for k in range(r))
            ref = _round_f32_once(Fraction(float(y_in[t, o])) + c)
            assert out[t, o].view(np.uint32) == ref.view(np.uint32), (t, o)
            alt = _round_f32_once(Fraction(float(y_in[t, o])) + Fraction(float(np.float32(float(c)))))
            twice += int(alt.view(np.uint32) != ref.view(np.uint32))
    assert twice > 0, "the case does not tell one rounding from two"


def test_whole_layer_brute_force():
    """The whole layer (Sec. 4.3, final case equation; eq. PTQ) element by
    element in Python scalars and exact rationals, on tiny inputs of three
    modalities: xs = fl32(x inv_s[m]); Delta = fl32(a / 127) and
    rq = fl32(127 / a) from the row's absmax a, each one correctly rounded
    division; codes = clip(rne(fl32(xs rq)), +-127); the integer sum of the
    code products; y0 = fl32(fl32(acc Delta) w_scale); text rows y0, other
    rows y0 + (xs L1^m) L2^m taken exactly and rounded once to binary32."""
    from fractions import Fraction
    rng = np.random.default_rng(21)
    T, K, N, r, M = 7, 10, 6, 3, 3
    x = (rng.standard_normal((T, K)) * 4).astype(np.float32)
    x[3] = 0                                           # a zero row: zero scale and codes
    mod = np.array([0, 1, 2, 0, 2, 1, 2], np.int32)
    inv = rng.uniform(0.2, 3, (M, K)).astype(np.float32)
    wq = rng.integers(-127, 128, (N, K)).astype(np.int8)
    ws = rng.uniform(1e-3, 1e-2, N).astype(np.float32)
    ld = rng.standard_normal((M - 1, r, K)).astype(np.float32)
    ru = (rng.standard_normal((M - 1, N, r)) * 0.1).astype(np.float32)
    y = inf.linear(x, mod, inv, wq, ws, ld, ru)
    assert y.dtype == np.float32 and y.shape == (T, N)
    for t in range(T):
        m = int(mod[t])
        xs = [np.float32(x[t, i]) * np.float32(inv[m, i]) for i in range(K)]
        a = max(abs(float(v)) for v in xs)
        if a == 0:
            delta, rq = np.float32(0), np.float32(0)
        else:
            delta = _round_f32_once(Fraction(a) / 127)
            rq = _round_f32_once(Fraction(127) / Fraction(a))
        codes = []
        for v in xs:
            p = np.float32(v) * rq                     # one binary32 product
            c = round(Fraction(float(p)))              # Python's round: ties to even
            codes.append(max(-127, min(127, c)))
        for o in range(N):
            acc = sum(codes[i] * int(wq[o, i]) for i in range(K))
            y0 = np.float32(np.float32(float(acc)) * delta) * np.float32(ws[o])
            if m == 0:
                assert y[t, o].view(np.uint32) == np.float32(y0).view(np.uint32), (t, o)
                continue
            u = [sum(Fraction(float(xs[i])) * Fraction(float(ld[m - 1, k, i])) for i in range(K))
                 for k in range(r)]
            cterm = sum(u[k] * Fraction(float(ru[m - 1, o, k])) for k in range(r))
            ref = _round_f32_once(Fraction(float(y0)) + cterm)
            assert y[t, o].view(np.uint32) == ref.view(np.uint32), (t, o)
    assert np.all(y[3] == 0)


def test_text_rows_equal_the_plain_w8a8_product():
    rng = np.random.default_rng(10)
    T, K, N = 12, 64, 40
    x = rng.standard_normal((T, K)).astype(np.float32)
    mod = np.array([0, 1] * 6, np.int32)
    inv = rng.uniform(0.5, 2, (2, K)).astype(np.float32)
    wq = rng.integers(-127, 128, (N, K)).astype(np.int8)
    ws = rng.uniform(1e-3, 1e-2, N).astype(np.float32)
    ld = rng.standard_normal((1, 8, K)).astype(np.float32)
    ru = rng.standard_normal((1, N, 8)).astype(np.float32)
    y = inf.linear(x, mod, inv, wq, ws, ld, ru)
    q, d = inf.smooth_quant(x, mod, inv)
    _, y0 = inf.w8a8_gemm(q, d, wq, ws)
    assert np.array_equal(y[mod == 0], y0[mod == 0])
    assert not np.allclose(y[mod == 1], y0[mod == 1])
    # rank 0 and zero factors leave every row at the plain product
    assert np.array_equal(inf.linear(x, mod, inv, wq, ws, ld * 0, ru * 0), y0)
    assert np.array_equal(inf.linear(x, mod, inv, wq, ws, ld[:, :0], ru[:, :, :0]), y0)


# ------------------------------------------------------------- calibration pins
def _small_layer(seed, T=(96, 80, 72), K=24, N=20, scales=(1.0, 30.0, 2.0)):
    rng = np.random.default_rng(seed)
    mod = np.concatenate([np.full(c, m, np.int32) for m, c in enumerate(T)])
    x = rng.standard_normal((mod.size, K)).astype(np.float32)
    for m, s in enumerate(scales[:len(T)]):
        x[mod == m] *= np.float32(s)
    x[:, :2] *= 20
    if len(T) > 2:
        x[mod == 2, 5:7] *= 10
    w = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    return x, mod, w


@pytest.mark.parametrize("base,bits", [("quantized", 8), ("fp", 8), ("quantized", 4)])
def test_full_rank_reconstructs_modality_smoothed_weight(base, bits):
    """At full rank the compensation restores S_m W exactly on top of the
    shared weight, whatever its bit width (8, or 4 in the W4A8 setting)."""
    x, mod, w = _small_layer(1)
    art = cal.calibrate(x, mod, w, 3, rank=min(w.shape), lr_dtype="f64", base=base,
                        weight_bits=bits)
    base_w = art["wdq"] if base == "quantized" else art["s32"][0][:, None].astype(np.float64) * w
    for m in (1, 2):
        target = art["s32"][m][:, None].astype(np.float64) * w
        recon = base_w + art["l1"][m - 1] @ art["l2"][m - 1]
        assert np.abs(recon - target).max() <= 1e-9 * np.abs(target).max()


def test_computational_invariance_quantization_off():
    """(X S_m^-1)(S_m W) = X W (Sec. 3.1).  With the activation quantizer off and
    full-rank compensation, non-text rows reproduce X W exactly: the residual
    dW = S_m W - Q(S_t W) absorbs the weight rounding too.  Text rows take no
    compensation (Sec. 4.3), so they differ from X W only by the weight
    rounding, which eq. PTQ bounds by half a step per channel."""
    x, mod, w = _small_layer(2)
    art = cal.calibrate(x, mod, w, 3, rank=min(w.shape), lr_dtype="f64")
    y = inf.linear(x, mod, art["inv_smooth"], art["wq"], art["w_scale"],
                   art["l_down"], art["r_up"], quantize_activations=False)
    ref = x.astype(np.float64) @ w.astype(np.float64)
    for m in (1, 2):
        rows = mod == m
        err = np.linalg.norm(y[rows] - ref[rows]) / np.linalg.norm(ref[rows])
        # only the fp32 rounding of S_m^-1 and of the smoothed row remains
        assert err < 2e-6, (m, err)
    rows = mod == 0
    xs = np.abs(x[rows].astype(np.float64) * art["inv_smooth"][0].astype(np.float64))
    bound = xs.sum(axis=1, keepdims=True) * art["w_scale"][None, :].astype(np.float64) * 0.5
    assert np.all(np.abs(y[rows] - ref[rows]) <= bound * (1 + 1e-5) + 1e-6 * np.abs(ref[rows]))
    assert np.abs(y[rows] - ref[rows]).max() > 0
    # without the compensation the non-text rows are visibly off
    y_nc = inf.linear(x, mod, art["inv_smooth"], art["wq"], art["w_scale"],
                      quantize_activations=False)
    rows = mod == 1
    assert np.linalg.norm(y_nc[rows] - ref[rows]) / np.linalg.norm(ref[rows]) > 1e-2


def test_equal_smoothing_with_fp_base_is_smoothquant():
    """s_m = s_t: the float difference vanishes, so L2 = Sigma_r V_r^T = 0 and
    the layer is SmoothQuant W8A8 bit-for-bit on every row."""
    x, mod, w = _small_layer(3)
    s_t = cal.smoothing_factor(cal.channel_range(x, mod, 0), cal.weight_range(w))[0]
    smoothing = np.stack([s_t] * 3)
    art = cal.calibrate(x, mod, w, 3, rank=4, lr_dtype="f32", base="fp", smoothing=smoothing)
    assert not np.any(art["r_up"])
    y = inf.linear(x, mod, art["inv_smooth"], art["wq"], art["w_scale"], art["l_down"], art["r_up"])
    q, d = inf.smooth_quant(x, mod, art["inv_smooth"])
    _, y0 = inf.w8a8_gemm(q, d, art["wq"], art["w_scale"])
    assert np.array_equal(y, y0)


def test_weight_quantizer_properties():
    x, mod, w = _small_layer(4, K=40, N=33)
    s32 = cal.smoothing_factor(cal.channel_range(x, mod, 0), cal.weight_range(w))[0]
    wq, scale, wdq = cal.quantize_weight(w, s32)
    ws = s32[:, None].astype(np.float64) * w
    assert np.all(np.abs(wq).max(axis=1) == 127)
    err = np.abs(wdq - ws)
    assert np.all(err <= scale[None, :].astype(np.float64) * 0.5 * (1 + 1e-6))


def test_weight_quantizer_4bit_brute_force():
    """The 4-bit shared weight of the W4A8 setting (Tables 1-2) under eq. PTQ:
    per output channel the step is max |S_t W| / 7 and each code is the
    ratio rounded half to even, clamped to [-7, 7]; checked element by
    element with Python floats and round()."""
    rng = np.random.default_rng(5)
    K, N = 24, 7
    w = rng.standard_normal((K, N))
    w[3, 2] = 0.0
    s32 = rng.uniform(0.3, 3.0, K).astype(np.float32)
    wq, scale, wdq = cal.quantize_weight(w, s32, bits=4)
    assert wq.dtype == np.int8 and wq.shape == (N, K)
    for o in range(N):
        col = [float(s32[i]) * float(w[i, o]) for i in range(K)]
        step = max(abs(v) for v in col) / 7
        assert scale[o] == np.float32(step)
        for i in range(K):
            assert int(wq[o, i]) == max(-7, min(7, round(col[i] / step)))
    assert np.all(np.abs(wq).max(axis=1) == 7)
    err = np.abs(wdq - s32[:, None].astype(np.float64) * w)
    assert np.all(err <= scale[None, :].astype(np.float64) * 0.5 * (1 + 1e-6))
    # a weight already on the 4-bit grid quantizes to itself
    wq2, scale2, _ = cal.quantize_weight(wdq / s32[:, None].astype(np.float64), s32, bits=4)
    assert np.array_equal(wq2, wq)


def test_theorem2_eckart_young():
    """Theorem 2: the whitened truncation minimises ||Z (dW - L)||_F over rank-r L,
    with minimum sum_{j>r} sigma_j(Z dW)^2 (an independent SVD of Z dW)."""
    rng = np.random.default_rng(12)
    K, N, r, Tm = 16, 12, 3, 80
    z = rng.standard_normal((Tm, K)) * rng.uniform(0.1, 10, K)[None, :]
    dw = rng.standard_normal((K, N))
    l1, l2 = cal.cmc_factors(z, dw, r, ridge=0.0)
    loss = np.linalg.norm(z @ (dw - l1 @ l2)) ** 2
    sig = np.linalg.svd(z @ dw, compute_uv=False)
    assert abs(loss / np.sum(sig[r:] ** 2) - 1) < 1e-9
    # any other rank-r choice is no better: unwhitened truncation, random
    u, s, vt = np.linalg.svd(dw, full_matrices=False)
    plain = u[:, :r] * s[:r] @ vt[:r]
    assert np.linalg.norm(z @ (dw - plain)) ** 2 >= loss * (1 - 1e-12)
    for _ in range(20):
        lr = rng.standard_normal((K, r)) @ rng.standard_normal((r, N))
        assert np.linalg.norm(z @ (dw - lr)) ** 2 >= loss


def test_whitening_orthonormalises():
    """Sec. 4.3: (X_v S_v^-1) T^-1 has orthonormal columns."""
    rng = np.random.default_rng(13)
    z = rng.standard_normal((64, 10)) * rng.uniform(0.1, 5, 10)[None, :]
    t, t_inv = cal.whitening(z, ridge=0.0)
    g = (z @ t_inv).T @ (z @ t_inv)
    assert np.abs(g - np.eye(10)).max() < 1e-10
    assert np.abs(t @ t_inv - np.eye(10)).max() < 1e-10


def test_smoothing_factor_closed_form():
    """Sec. 4.2: s_i = sqrt(max_t |x_ti| / max_j |w_ji|); the smoothed weight and
    smoothed activations then share one per-channel range (alpha = 1/2)."""
    x, mod, w = _small_layer(14)
    wmax = cal.weight_range(w)
    for m in range(3):
        s32, inv = cal.smoothing_factor(cal.channel_range(x, mod, m), wmax)
        xr = np.abs(x[mod == m]).max(axis=0) / s32.astype(np.float64)
        wr = np.abs(w).max(axis=1) * s32.astype(np.float64)
        assert np.allclose(xr, wr, rtol=1e-6)
        assert np.array_equal(inv, (np.float32(1) / s32).astype(np.float32))


def test_mas_recovers_audio_sqnr_lost_to_unified_smoothing():
    """Sec. 4.1 / Theorem 1: a unified factor set by the dominant modality lowers
    the activation SQNR of a modality whose range ratio is non-uniform."""
    x, mod, w = _small_layer(15, T=(64, 64, 64), K=48, N=8)
    wmax = cal.weight_range(w)
    uni = cal.smoothing_factor(np.abs(x).max(axis=0), wmax)[1]
    aud = cal.smoothing_factor(cal.channel_range(x, mod, 2), wmax)[1]
    xa = x[mod == 2]

    def sqnr(inv):
        xs = inf.smooth(xa, np.zeros(len(xa), np.int32), inv[None, :])
        q, d = inf.quantize_per_token(xs)
        e = xs - q * d[:, None]
        return 10 * np.log10((xs.astype(np.float64) ** 2).sum() / (e.astype(np.float64) ** 2).sum())

    assert sqnr(aud) > sqnr(uni) + 1.0


def test_relerr_metric():
    ref = np.array([[1.0, -2.0, 0.0, 4.0]])
    assert inf.relerr(ref, ref) == 0.0
    y = ref.copy()
    y[0, 2] = 0.01                       # near-zero reference element: scaled by the row rms
    assert abs(inf.relerr(y, ref) - 0.01 / np.sqrt(21 / 4)) < 1e-12
