"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Bar: int8 codes, per-token scales and int32 accumulators bit-exact; the
dequantised shared-weight product bit-exact; the layer output within
max relative error 1e-3 (fp32 workloads) or 1e-2 (bf16 workloads) under the
row-rms-guarded metric ``oracle.inference.relerr``; text rows, which take no
compensation, bit-exact.  Every case, the full-size workloads included,
compares every row: the codes and scales of the standalone call and of the
fused layer's own stage 1 (read from its workspace), every int32 accumulator,
and, with the up-projection factors set to zero, every row of the fused
layer against the oracle's dequantised product bit for bit (which pins the
non-text codes and the accumulators of whichever fused GEMM variant runs).
The 4-bit shared weight (W4A8) is held to the same bar: the device gets the
oracle's 4-bit codes packed two per byte, the oracle uses the codes as they
are.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import inference as oinf

pytestmark = pytest.mark.gpu


def _require_gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X visible to torch"


@pytest.fixture(scope="module")
def ops():
    _require_gpu()
    from paper_2603_04800_amd import ops as o
    return o


def _np(t):
    return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()


def _tol(act_dtype, lr_dtype="f32"):
    return 1e-3 if act_dtype == "f32" and lr_dtype == "f32" else 1e-2


def _ws_codes(ws, T, K):
    """The codes q [T][K] and scales [T] stage 1 leaves in the fused layer's
    workspace: q at offset 0, the scales at the next 256-byte boundary.  Past
    the small-batch path (T > 16) with K % 64 == 0 the codes are row-paired:
    rows 2i and 2i + 1 alternate in 64-byte pieces ([T/2][K/64][2][64]), the
    batch rounded up to whole pairs."""
    paired = T > 16 and K % 64 == 0
    rows = (T + 1) // 2 * 2 if paired else T
    off = (rows * K + 255) // 256 * 256
    q = ws[: rows * K].view(torch.int8)
    if paired:
        q = q.view(rows // 2, K // 64, 2, 64).permute(0, 2, 1, 3).reshape(rows, K)[:T]
    else:
        q = q.view(T, K)
    dx = ws[off: off + 4 * T].view(torch.float32)
    return q, dx


def _check_layer(ops, L, name=""):
    """Run every entry point on one layer and compare every row with the oracle."""
    from paper_2603_04800_amd import workload
    x, mod, lin = workload.to_device(L)
    xs_np, mod_np = L["x"], L["modality"]
    act = L["act_dtype"]
    out_dtype = torch.bfloat16 if act == "bf16" else torch.float32
    T, K = xs_np.shape
    w4 = int(L.get("weight_bits", 8)) == 4
    assert w4 == lin.w4
    cmc = lin.rank > 0 and lin.n_mod > 1
    print(f"[parity] {name} T={T} K={K} N={L['wq'].shape[0]} r={L['rank']} "
          f"M={L['n_mod']} wbits={8 - 4 * w4}", flush=True)

    # smoothing + quantisation: every code and scale
    q, dx = ops.smooth_quant(x, mod, lin.inv_smooth)
    q_ref, dx_ref = oinf.smooth_quant(xs_np, mod_np, L["inv_smooth"])
    torch.cuda.synchronize()
    assert np.array_equal(q.cpu().numpy(), q_ref), "int8 codes differ"
    assert np.array_equal(dx.cpu().numpy().view(np.uint32), dx_ref.view(np.uint32)), "scales differ"

    # shared-weight GEMM: every int32 accumulator and dequantised value
    gemm = ops.w4a8_gemm if w4 else ops.w8a8_gemm
    acc, y0 = gemm(q, dx, lin.wq, lin.w_scale, want_acc=True, out_dtype=torch.float32)
    acc_ref, y0_ref = oinf.w8a8_gemm(q_ref, dx_ref, L["wq"], L["w_scale"])
    acc_np = acc.cpu().numpy()
    assert np.array_equal(acc_np, acc_ref), f"int32 accumulators differ ({np.sum(acc_np != acc_ref)})"
    del acc, acc_np
    y0_np = y0.cpu().numpy()
    assert np.array_equal(y0_np.view(np.uint32), y0_ref.view(np.uint32)), "dequantised product differs"
    y0_out = oinf.to_output(y0_ref, act)

    # the fused layer
    y = lin(x, mod, out_dtype=out_dtype)
    y_ref = oinf.to_output(oinf.linear(xs_np, mod_np, L["inv_smooth"], L["wq"],
                                       L["w_scale"], L["l_down"], L["r_up"]), act)
    y_np = _np(y)
    err = oinf.relerr(y_np, y_ref)
    print(f"[parity] {name} fused relerr {err:.3e} (bar {_tol(act, L['lr_dtype']):.0e})", flush=True)
    assert err <= _tol(act, L["lr_dtype"]), f"fused relerr {err}"
    text = mod_np == 0
    assert np.array_equal(y_np[text], y0_out[text]), "text rows not exact"
    if not cmc:
        assert np.array_equal(y_np, y0_out), "rows without compensation not exact"
    del y_ref

    # stage 1 of the fused layer (whichever kernel this shape dispatches to)
    # leaves the codes and scales of every row in its workspace; stage1 +
    # stage2 equals the fused call, and reruns are bitwise identical
    y2 = torch.empty_like(y)
    ws = lin.workspace(T, x.device)
    lin.stage1(x, mod, y2, ws)
    qw, dxw = _ws_codes(ws, T, K)
    assert np.array_equal(qw.cpu().numpy(), q_ref), "fused stage 1: int8 codes differ"
    assert np.array_equal(dxw.cpu().numpy().view(np.uint32), dx_ref.view(np.uint32)), \
        "fused stage 1: scales differ"
    lin.stage2(x, mod, y2, ws)
    y3 = lin(x, mod, out_dtype=out_dtype)
    torch.cuda.synchronize()
    assert torch.equal(y2.view(torch.int16) if y2.dtype == torch.bfloat16 else y2.view(torch.int32),
                       y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))
    assert torch.equal(y3, y)
    del y2, y3

    if cmc:
        # the same layer, dispatch and rank with L2 = 0: the compensation adds
        # exact zeros, so every row (non-text codes, accumulators of the fused
        # GEMM variant, dequantisation) must equal the oracle's y0 bit for bit
        from paper_2603_04800_amd import ops as _o
        lin0 = _o.Linear(lin.inv_smooth, lin.wq, lin.w_scale, lin.l_down, torch.zeros_like(lin.r_up))
        yz = _np(lin0(x, mod, out_dtype=out_dtype))
        bad = np.flatnonzero(np.any(yz.view(np.uint32 if yz.dtype == np.float32 else np.uint16)
                                    != y0_out.view(np.uint32 if y0_out.dtype == np.float32
                                                   else np.uint16), axis=1))
        assert bad.size == 0, f"L2 = 0: {bad.size} rows differ from y0 (first {bad[:8]})"

    # standalone compensation on top of the fp32 dequantised product
    if cmc:
        yl = ops.lowrank_comp(x, mod, lin.inv_smooth, lin.l_down, lin.r_up, y0.clone())
        yl_ref = oinf.lowrank_comp(xs_np, mod_np, L["inv_smooth"], L["l_down"], L["r_up"], y0_ref)
        yl_np = yl.cpu().numpy()
        err = oinf.relerr(yl_np, yl_ref)
        assert err <= _tol(act, L["lr_dtype"]), f"lowrank_comp relerr {err}"
        assert np.array_equal(yl_np[text].view(np.uint32), y0_ref[text].view(np.uint32))
    return err


# ------------------------------------------------------------------ workloads
_FULL = [(c.index, p.name) for c in synth.CONFIGS for p in c.projections]


@pytest.mark.parametrize("cfg_index,proj", _FULL, ids=[f"cfg{c}-{p}" for c, p in _FULL])
def test_workload_parity(ops, cfg_index, proj):
    from paper_2603_04800_amd import workload
    L = workload.layer(cfg_index, proj)
    _check_layer(ops, L, name=f"cfg{cfg_index}/{proj}")


# ------------------------------------------------------------------ random sweep
def _sweep_cases(n=24, seed=2024):
    """Seeded random valid shapes across the dispatch boundaries: batches of
    1-16 tokens (small-batch and decode GEMMs), 17-300 and 300-1300 tokens
    (tiled GEMM, split K on small grids); K a multiple of 64 (direct-to-LDS,
    decode, W4A8) or, every fifth case, a ragged multiple of 16 (general-K
    GEMM); N a multiple of 16; rank 0-64; one to four modalities; fp32 or
    bf16 activations and factors; contiguous, alternating or run layouts."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        lo, hi = [(1, 17), (17, 301), (301, 1301), (1, 1301)][i % 4]
        T = int(rng.integers(lo, hi))
        ragged = i % 5 == 0
        K = 16 * (4 * int(rng.integers(1, 40)) + int(rng.integers(1, 4))) if ragged \
            else 64 * int(rng.integers(1, 40))
        w4 = not ragged and i % 3 == 1
        N = 16 * int(rng.integers(1, 48))
        M = int(rng.integers(1, 5))
        r = 0 if M == 1 else 16 * int(rng.integers(0, 5))
        act = str(rng.choice(["f32", "bf16"]))
        lr = str(rng.choice(["f32", "bf16"]))
        layout = str(rng.choice(["contiguous", "alternating", "runs"]))
        cases.append(dict(T=T, K=K, N=N, r=r, M=M, act=act, lr=lr, layout=layout,
                          weight_bits=4 if w4 else 8, seed=int(seed + i)))
    return cases


_SWEEP = _sweep_cases()


@pytest.mark.parametrize("case", _SWEEP, ids=[
    f"T{c['T']}_K{c['K']}_N{c['N']}_r{c['r']}_M{c['M']}_{c['act']}_{c['lr']}_{c['layout']}_w{c['weight_bits']}"
    for c in _SWEEP])
def test_random_shape_parity(ops, case):
    kw = dict(case)
    L = _random_layer(kw.pop("T"), kw.pop("K"), kw.pop("N"), kw.pop("r"), kw.pop("M"),
                      kw.pop("act"), kw.pop("lr"), **kw)
    if L["rank"] == 0:
        L["l_down"] = L["l_down"][:, :0]
        L["r_up"] = L["r_up"][:, :, :0]
    _check_layer(ops, L, name="sweep")


def _split_cases(n=16, seed=79):
    """Seeded random shapes for the split stage 1 (bf16 activations and
    factors, rank 16-64, two to four modalities, 17-4095 tokens, K a
    multiple of 64 up to 8960): the quarter-streamed down-projection with
    slices of one or more chunks, last chunks of one to four quarters,
    ragged row tiles, tiles holding one, two or three non-text modalities,
    and both row quantisers (a wave per row up to 4096 columns, a workgroup
    per row beyond)."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        T = int(rng.integers(17, 4096))
        K = 64 * int(rng.integers(2, 141))
        N = 16 * int(rng.integers(1, 7))
        M = int(rng.integers(2, 5))
        r = 16 * int(rng.integers(1, 5))
        layout = str(rng.choice(["contiguous", "alternating", "runs"]))
        cases.append(dict(T=T, K=K, N=N, r=r, M=M, act="bf16", lr="bf16", layout=layout,
                          seed=int(seed + i)))
    return cases


_SPLIT = _split_cases()


@pytest.mark.parametrize("case", _SPLIT, ids=[
    f"T{c['T']}_K{c['K']}_N{c['N']}_r{c['r']}_M{c['M']}_{c['layout']}" for c in _SPLIT])
def test_split_stage1_sweep(ops, case):
    kw = dict(case)
    L = _random_layer(kw.pop("T"), kw.pop("K"), kw.pop("N"), kw.pop("r"), kw.pop("M"),
                      kw.pop("act"), kw.pop("lr"), **kw)
    _check_layer(ops, L, name="split-sweep")


# ------------------------------------------------------------------ comparator
@pytest.mark.parametrize("cfg_index", [0, 2, 3])
def test_smoothquant_comparator_parity(ops, cfg_index):
    """The SmoothQuant comparator (one unified smoothing factor, no
    compensation; Sec. 4.1) runs through the same kernels and C ABI at the
    workload's full size, held to the same bar."""
    from paper_2603_04800_amd import workload
    L = workload.layer(cfg_index, method="smoothquant")
    assert L["rank"] == 0
    _check_layer(ops, L, name=f"smoothquant/cfg{cfg_index}")


def _check_mas_only(L, mod_gpu=None, name=""):
    """MAS-only layer through masq_mas_only_linear against the oracle's
    layer run with each modality's own artifacts, every row bit for bit."""
    from paper_2603_04800_amd import workload
    x, mod, lin = workload.to_device(L)
    if mod_gpu is not None:
        mod = torch.from_numpy(mod_gpu).to(x.device)
    act = L["act_dtype"]
    print(f"[mas-only] {name} T={x.shape[0]} K={lin.c_in} N={lin.c_out} M={lin.n_mod}", flush=True)
    y = lin(x, mod, out_dtype=torch.bfloat16 if act == "bf16" else torch.float32)
    y2 = lin(x, mod, out_dtype=torch.bfloat16 if act == "bf16" else torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(y, y2), "reruns differ"
    mod_np = L["modality"]
    y_np = _np(y)
    for m in range(L["n_mod"]):
        rm = np.flatnonzero(mod_np == m)
        if rm.size == 0:
            continue
        ref = oinf.linear(L["x"][rm], np.zeros(rm.size, np.int32), L["inv_smooth"][m][None],
                          L["wq"][m], L["w_scale"][m])
        ref = oinf.to_output(ref, act)
        bad = np.flatnonzero(np.any(y_np[rm] != ref, axis=1))
        assert bad.size == 0, f"modality {m}: {bad.size} rows differ (first token {rm[bad[:4]]})"


_MAS = [(c.index, p.name) for c in synth.CONFIGS for p in c.projections]


@pytest.mark.parametrize("cfg_index,proj", _MAS, ids=[f"cfg{c}-{p}" for c, p in _MAS])
def test_mas_only_comparator_parity(ops, cfg_index, proj):
    """The MAS-only comparator (a weight per modality, no compensation;
    Sec. 4.2) through masq_mas_only_linear: rows grouped by modality on the
    device, every row bit-exact against the oracle's layer, on every
    workload (interleaved runs included)."""
    from paper_2603_04800_amd import workload
    L = workload.layer(cfg_index, proj, method="mas")
    _check_mas_only(L, name=f"cfg{cfg_index}/{proj}")


def _random_mas_layer(T, K, N, M, act, layout="alternating", seed=0, counts=None):
    rng = np.random.default_rng(seed)
    if counts is None:
        counts = [T // M + (1 if m < T % M else 0) for m in range(M)]
    mod = synth.make_modality_layout(counts, layout, 0, seed)
    x = rng.standard_normal((T, K)).astype(np.float32)
    for m, sc in enumerate([1.0, 30.0, 2.0, 5.0][:M]):
        x[mod == m] *= np.float32(sc)
    from oracle.bf16 import bf16_round
    if act == "bf16":
        x = bf16_round(x)
    return dict(x=x, modality=mod, inv_smooth=rng.uniform(0.05, 3.0, (M, K)).astype(np.float32),
                wq=rng.integers(-127, 128, (M, N, K)).astype(np.int8),
                w_scale=rng.uniform(1e-4, 1e-2, (M, N)).astype(np.float32),
                l_down=np.zeros((max(M - 1, 0), 0, K), np.float32),
                r_up=np.zeros((max(M - 1, 0), N, 0), np.float32), n_mod=M, rank=0,
                act_dtype=act, lr_dtype="bf16", weight_bits=8, method="mas")


_MAS_EDGE = {
    "T1": dict(T=1, K=64, N=32, M=2, act="bf16"),
    "alternating_3mod_ragged": dict(T=517, K=192, N=272, M=3, act="bf16"),
    "runs_4mod_fp32": dict(T=1300, K=256, N=96, M=4, act="f32", layout="runs"),
    "empty_modality": dict(T=300, K=128, N=64, M=3, act="bf16", counts=[150, 0, 150]),
    "single_modality": dict(T=257, K=64, N=48, M=1, act="bf16"),
    "all_vision": dict(T=600, K=128, N=80, M=2, act="bf16", counts=[0, 600]),
    "decode_t16_split_k": dict(T=16, K=4096, N=512, M=2, act="bf16"),
    "few_tiles_split_k": dict(T=700, K=2048, N=528, M=3, act="bf16", layout="runs"),
}


@pytest.mark.parametrize("name", list(_MAS_EDGE))
def test_mas_only_edge_cases(ops, name):
    kw = dict(_MAS_EDGE[name])
    L = _random_mas_layer(kw.pop("T"), kw.pop("K"), kw.pop("N"), kw.pop("M"), kw.pop("act"),
                          seed=11, **kw)
    _check_mas_only(L, name=name)


def test_mas_only_invalid_ids_read_as_text(ops):
    L = _random_mas_layer(300, 128, 64, 3, "bf16", seed=5)
    bad = np.array([0, 7, 150, 299])
    mod_gpu = L["modality"].copy()
    mod_gpu[bad] = np.array([3, -1, 1 << 20, 9], np.int32)
    L["modality"][bad] = 0
    _check_mas_only(L, mod_gpu=mod_gpu, name="invalid ids")


# ------------------------------------------------------------------ edge cases
def _random_layer(T, K, N, r, M, act, lr, layout="alternating", zero_rows=(), seed=0,
                  counts=None, weight_bits=8):
    rng = np.random.default_rng(seed)
    if counts is None:
        counts = [T // M + (1 if m < T % M else 0) for m in range(M)]
    mod = synth.make_modality_layout(counts, layout, 0, seed)
    x = rng.standard_normal((T, K)).astype(np.float32)
    for m, s in enumerate([1.0, 30.0, 2.0, 5.0][:M]):
        x[mod == m] *= np.float32(s)
    x[:, : max(1, K // 64)] *= 20
    for t in zero_rows:
        x[t] = 0
    from oracle.bf16 import bf16_round
    if act == "bf16":
        x = bf16_round(x)
    inv = rng.uniform(0.05, 3.0, (M, K)).astype(np.float32)
    qmax = (1 << (weight_bits - 1)) - 1
    wq = rng.integers(-qmax, qmax + 1, (N, K)).astype(np.int8)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    ld = (rng.standard_normal((max(M - 1, 0), r, K)) / np.sqrt(K)).astype(np.float32)
    ru = (rng.standard_normal((max(M - 1, 0), N, r)) * 0.05).astype(np.float32)
    if lr == "bf16":
        ld, ru = bf16_round(ld), bf16_round(ru)
    return dict(x=x, modality=mod, inv_smooth=inv, wq=wq, w_scale=ws, l_down=ld, r_up=ru,
                n_mod=M, rank=r, act_dtype=act, lr_dtype=lr, weight_bits=weight_bits)


_EDGE = {
    "T1_single_token": dict(T=1, K=64, N=32, r=16, M=2, act="bf16", lr="bf16"),
    "ragged_T_N_K48_fp32": dict(T=300, K=48, N=80, r=16, M=2, act="f32", lr="f32",
                                layout="contiguous"),
    "tri_modal_alternating": dict(T=257, K=128, N=272, r=32, M=3, act="bf16", lr="bf16"),
    "runs_bf16_multi_tile": dict(T=700, K=1024, N=528, r=64, M=3, act="bf16", lr="bf16",
                                 layout="runs"),
    "rank128_two_slots_global_path": dict(T=96, K=256, N=256, r=128, M=3, act="bf16", lr="bf16"),
    "fp32_rank64_two_slots_global_path": dict(T=96, K=256, N=256, r=64, M=3, act="f32", lr="f32"),
    "bf16_act_fp32_factors": dict(T=130, K=192, N=64, r=16, M=2, act="bf16", lr="f32"),
    "fp32_act_bf16_factors": dict(T=130, K=192, N=64, r=16, M=2, act="f32", lr="bf16"),
    "zero_rows": dict(T=40, K=64, N=48, r=16, M=2, act="bf16", lr="bf16", zero_rows=(0, 7, 39)),
    "all_text": dict(T=100, K=128, N=64, r=16, M=2, act="bf16", lr="bf16", counts=[100, 0]),
    "all_vision": dict(T=100, K=128, N=64, r=16, M=2, act="bf16", lr="bf16", counts=[0, 100]),
    "rank0": dict(T=70, K=64, N=64, r=0, M=2, act="f32", lr="f32"),
    "single_modality": dict(T=70, K=64, N=64, r=16, M=1, act="bf16", lr="bf16"),
    "four_modalities": dict(T=260, K=128, N=96, r=16, M=4, act="bf16", lr="bf16"),
    # small batches split the down-projection along k (ragged last slice)
    "sliced_down_ragged_k": dict(T=40, K=1552, N=160, r=32, M=3, act="bf16", lr="bf16"),
    "sliced_down_rank128": dict(T=20, K=1024, N=96, r=128, M=2, act="bf16", lr="bf16"),
    "sliced_down_fp32": dict(T=9, K=2064, N=48, r=16, M=3, act="f32", lr="f32"),
    "decode_t16_k4096": dict(T=16, K=4096, N=512, r=64, M=2, act="bf16", lr="bf16"),
    "decode_t5_alternating": dict(T=5, K=1024, N=272, r=64, M=3, act="bf16", lr="bf16"),
    # k-sliced decode GEMM: ragged last slice, a partial last channel group
    "decode_t7_k2624_n208_two_slices": dict(T=7, K=2624, N=208, r=32, M=3, act="bf16",
                                            lr="bf16"),
    "decode_t16_k5184_fp32_three_slices": dict(T=16, K=5184, N=96, r=16, M=2, act="f32",
                                               lr="f32"),
    # grids with few tiles split K across workgroups (raw int32 slices added exactly)
    "splitk_bf16": dict(T=300, K=2048, N=512, r=64, M=3, act="bf16", lr="bf16"),
    "splitk_fp32_ragged": dict(T=260, K=1600, N=272, r=16, M=2, act="f32", lr="f32"),
    # the compensation operands loaded as extra stages of the K ring: the
    # shortest ring (four 64-byte stages), ranks below 64, mixed tiles
    # wide down-projection (rows of 2048 columns and more below 4096 tokens,
    # of 8192 and more at any batch): ragged last k slice, ranks below 64,
    # fp32 activations, the smallest batch above the decode path, and the
    # batches either side of the 4096-token switch to the fused stage 1
    "down_wide_t17_k2048": dict(T=17, K=2048, N=32, r=64, M=3, act="bf16", lr="bf16",
                                layout="alternating"),
    "down_wide_t600_k2112_f32": dict(T=600, K=2112, N=48, r=16, M=2, act="f32", lr="bf16"),
    "down_wide_t4095_k2048": dict(T=4095, K=2048, N=16, r=64, M=3, act="bf16", lr="bf16",
                                  layout="runs"),
    "stage1_fused_t4096_k2048": dict(T=4096, K=2048, N=16, r=64, M=3, act="bf16", lr="bf16",
                                     layout="runs"),
    "stage1_fused_t300_k1984": dict(T=300, K=1984, N=48, r=32, M=2, act="bf16", lr="bf16"),
    "down_wide_t1100_k8208_r32": dict(T=1100, K=8208, N=32, r=32, M=3, act="bf16", lr="bf16",
                                      layout="runs"),
    "down_wide_f32_t1030_k8192_r48": dict(T=1030, K=8192, N=16, r=48, M=2, act="f32",
                                          lr="bf16"),
    # down-projection with the L1 fragments in LDS (rows too long for the
    # register-resident stage 1, or four modalities' factors too large for
    # its LDS), then the quantisation adding the slice partials: ragged
    # batch, rank 48, and a third non-text modality in one 128-row tile
    # (its fragments read from global memory)
    "down_lds_t600_k5120_r48": dict(T=600, K=5120, N=48, r=48, M=3, act="bf16", lr="bf16",
                                    layout="runs"),
    "down_lds_four_mod_alternating_k3584": dict(T=300, K=3584, N=32, r=64, M=4, act="bf16",
                                                lr="bf16"),
    "down_lds_t40_k4160_r16": dict(T=40, K=4160, N=64, r=16, M=2, act="bf16", lr="bf16"),
    # k slices of two and five 256-column chunks streamed in 64-column
    # quarters (long rows, large grids), the last slice short of chunks and
    # its last chunk one quarter long; a ragged last row tile of two rows
    # whose slice ends in an odd number of quarters
    "down_lds_two_chunk_slices_t4096_k8192": dict(T=4096, K=8192, N=32, r=64, M=3,
                                                  act="bf16", lr="bf16", layout="runs"),
    "down_lds_five_chunk_slices_ragged_t8192_k8256": dict(T=8192, K=8256, N=16, r=32, M=2,
                                                          act="bf16", lr="bf16",
                                                          layout="contiguous"),
    "down_lds_ragged_tile_t130_k1216_r32": dict(T=130, K=1216, N=32, r=32, M=3, act="bf16",
                                                lr="bf16"),
    # 32-row stage-1 workgroups (batches of 8192 tokens and more), ragged tail
    "stage1_wide_ragged_t8200": dict(T=8200, K=128, N=32, r=64, M=3, act="bf16", lr="bf16",
                                     layout="runs"),
    "ring_tail_k256_rank16": dict(T=520, K=256, N=272, r=16, M=2, act="bf16", lr="bf16",
                                  layout="runs"),
    "ring_tail_k320_rank32": dict(T=300, K=320, N=256, r=32, M=3, act="bf16", lr="bf16"),
    "ring_tail_k512_rank48_f32_out": dict(T=400, K=512, N=336, r=48, M=3, act="f32", lr="bf16",
                                          layout="runs"),
    # the stage-1 choice: the register-resident kernel for 4096 tokens and
    # more with one non-text modality, the split form just below (odd batch:
    # row-paired codes with an unused last row)
    "fr_first_t4096_two_mod": dict(T=4096, K=1024, N=32, r=64, M=2, act="bf16", lr="bf16",
                                   layout="contiguous"),
    "split_t4095_two_mod": dict(T=4095, K=1024, N=32, r=64, M=2, act="bf16", lr="bf16",
                                layout="runs"),
    # more tiles than compute units: persistent GEMM workgroups take a second
    # tile, with the next tile's first stages queued during the epilogue
    # (three stages after text-only tiles, one after one-modality tiles,
    # none after two-modality ones), and rings of 4, 2 and 1 stages
    "persistent_two_tiles_k256": dict(T=2304, K=256, N=8192, r=64, M=3, act="bf16", lr="bf16",
                                      layout="runs"),
    "persistent_two_tiles_k128": dict(T=2304, K=128, N=8192, r=32, M=2, act="bf16", lr="bf16",
                                      layout="runs"),
    "persistent_two_tiles_k64_f32_out": dict(T=2304, K=64, N=8192, r=16, M=3, act="f32",
                                             lr="bf16", layout="runs"),
}


@pytest.mark.parametrize("name", list(_EDGE))
def test_edge_case_parity(ops, name):
    kw = dict(_EDGE[name])
    L = _random_layer(kw.pop("T"), kw.pop("K"), kw.pop("N"), kw.pop("r"), kw.pop("M"),
                      kw.pop("act"), kw.pop("lr"), **kw)
    if L["rank"] == 0:
        L["l_down"] = L["l_down"][:, :0]
        L["r_up"] = L["r_up"][:, :, :0]
    _check_layer(ops, L, name=name)


def test_zero_row_gives_zero_scale_and_codes(ops):
    L = _random_layer(8, 64, 32, 16, 2, "f32", "f32", zero_rows=(3,))
    from paper_2603_04800_amd import workload
    x, mod, lin = workload.to_device(L)
    q, dx = ops.smooth_quant(x, mod, lin.inv_smooth)
    assert float(dx[3]) == 0.0 and int(q[3].abs().sum()) == 0


def test_empty_batch_is_a_noop(ops):
    L = _random_layer(4, 64, 32, 16, 2, "bf16", "bf16")
    from paper_2603_04800_amd import workload
    x, mod, lin = workload.to_device(L)
    y = lin(x[:0], mod[:0])
    assert y.shape == (0, 32)


@pytest.mark.parametrize("T,K", [(16, 2048), (300, 512)])
def test_bound_calls_equal_the_layer(ops, T, K):
    """Linear.bind: the pre-marshalled fused call and its two stages give the
    layer's output bit for bit (small-batch and tiled paths)."""
    from paper_2603_04800_amd import workload
    L = _random_layer(T, K, 128, 32, 3, "bf16", "bf16")
    x, mod, lin = workload.to_device(L)
    y_ref = lin(x, mod)
    y1, y2 = torch.empty_like(y_ref), torch.empty_like(y_ref)
    b1, b2 = lin.bind(x, mod, y1), lin.bind(x, mod, y2)
    b1()
    b2.stage1()
    b2.stage2()
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y_ref.view(torch.int16))
    assert torch.equal(y2.view(torch.int16), y_ref.view(torch.int16))


@pytest.mark.parametrize("K,r", [(128, 16), (512, 64)])
def test_invalid_modality_ids_read_as_text(ops, K, r):
    """Ids outside [0, n_mod) are documented to be read as text: the layer then
    equals the oracle run with those ids replaced by 0 (text rows exact)."""
    from paper_2603_04800_amd import workload
    L = _random_layer(300, K, 96, r, 3, "bf16", "bf16")
    bad = np.array([0, 5, 17, 100, 257, 299])
    mod_gpu = L["modality"].copy()
    mod_gpu[bad] = np.array([3, -1, 4, 1 << 20, -(1 << 30), 7], np.int32)
    L["modality"][bad] = 0
    x, _, lin = workload.to_device(L)
    y = lin(x, torch.from_numpy(mod_gpu).to(x.device), out_dtype=torch.bfloat16)
    y_ref = oinf.to_output(oinf.linear(L["x"], L["modality"], L["inv_smooth"], L["wq"],
                                       L["w_scale"], L["l_down"], L["r_up"]), "bf16")
    y_np = _np(y)
    assert oinf.relerr(y_np, y_ref) <= 1e-2
    assert np.array_equal(y_np[bad], y_ref[bad])


# ------------------------------------------------------------------ 4-bit shared weight
# Full-size prefill (every tile of the direct-to-LDS GEMM) and decode (the
# k-sliced Wq-streaming GEMM) with the weight calibrated to 4 bits.
_FULL_W4 = [(1, None), (2, None)]


@pytest.mark.parametrize("cfg_index,proj", _FULL_W4, ids=[f"cfg{c}" for c, _ in _FULL_W4])
def test_w4a8_workload_parity(ops, cfg_index, proj):
    from paper_2603_04800_amd import workload
    L = workload.layer(cfg_index, proj, weight_bits=4)
    assert np.abs(L["wq"]).max() <= 7
    _check_layer(ops, L, name=f"w4/cfg{cfg_index}")


_EDGE_W4 = {
    # decode GEMM (fused) and small-batch GEMM (int32 accumulators requested)
    "w4_T1_k64": dict(T=1, K=64, N=32, r=16, M=2, act="bf16", lr="bf16"),
    "w4_decode_t16_k4096": dict(T=16, K=4096, N=512, r=64, M=2, act="bf16", lr="bf16"),
    "w4_decode_t7_k2624_n208": dict(T=7, K=2624, N=208, r=32, M=3, act="bf16", lr="bf16"),
    "w4_decode_fp32_t9_k5184": dict(T=9, K=5184, N=96, r=16, M=2, act="f32", lr="f32"),
    # rows too long for the k-sliced decode GEMM: the single-pass small-batch GEMM
    "w4_small_t3_k20544": dict(T=3, K=20544, N=48, r=16, M=2, act="bf16", lr="bf16"),
    # direct-to-LDS GEMM: split K over few tiles, one K stage ring tail,
    # ragged T and N, fp32 activations and factors, four modalities, no split
    "w4_splitk_runs_t700_k1024": dict(T=700, K=1024, N=528, r=64, M=3, act="bf16", lr="bf16",
                                      layout="runs"),
    "w4_ring_tail_k256": dict(T=520, K=256, N=272, r=16, M=2, act="bf16", lr="bf16",
                              layout="runs"),
    "w4_fp32_ragged_t300_k192": dict(T=300, K=192, N=80, r=16, M=2, act="f32", lr="f32",
                                     layout="contiguous"),
    "w4_bf16_act_fp32_factors": dict(T=130, K=192, N=64, r=16, M=2, act="bf16", lr="f32"),
    "w4_four_modalities": dict(T=260, K=128, N=96, r=16, M=4, act="bf16", lr="bf16"),
    "w4_rank0": dict(T=70, K=64, N=64, r=0, M=2, act="f32", lr="f32"),
    "w4_no_split_t4096_n2048": dict(T=4096, K=128, N=2048, r=32, M=2, act="bf16", lr="bf16",
                                    layout="runs"),
}


@pytest.mark.parametrize("name", list(_EDGE_W4))
def test_w4a8_edge_case_parity(ops, name):
    kw = dict(_EDGE_W4[name])
    L = _random_layer(kw.pop("T"), kw.pop("K"), kw.pop("N"), kw.pop("r"), kw.pop("M"),
                      kw.pop("act"), kw.pop("lr"), weight_bits=4, **kw)
    if L["rank"] == 0:
        L["l_down"] = L["l_down"][:, :0]
        L["r_up"] = L["r_up"][:, :, :0]
    _check_layer(ops, L, name=name)


def test_w4a8_equals_w8a8_on_the_same_codes(ops):
    """The packed path and the int8 path given the same (4-bit) codes agree
    bit for bit, on the decode and on the prefill GEMM."""
    from paper_2603_04800_amd import int4, workload
    for T in (12, 600):
        L = _random_layer(T, 1024, 256, 32, 3, "bf16", "bf16", weight_bits=4, seed=3)
        x, mod, lin4 = workload.to_device(L)
        L8 = dict(L, weight_bits=8)
        _, _, lin8 = workload.to_device(L8)
        assert lin4.w4 and not lin8.w4
        assert torch.equal(lin4.wq.cpu(), torch.from_numpy(int4.pack(L["wq"])))
        y4 = lin4(x, mod)
        y8 = lin8(x, mod)
        torch.cuda.synchronize()
        assert torch.equal(y4.view(torch.int16), y8.view(torch.int16)), f"T={T}"
