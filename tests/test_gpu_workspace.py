"""The workspace contract of masq_linear_fused, masq_linear_fused_w4a8 and
masq_mas_only_linear: its contents need not be initialised.  Every dispatch
path that keeps arrival counters, slice partials or row tables in the
workspace runs once on a zeroed workspace and then on workspaces filled with
byte patterns (every counter starting far from zero, every partial slot and
table entry holding garbage, negative or huge values); the outputs must be
bit-identical, also on a second call over the same dirty workspace.  (No
kernel here waits on a counter: a counter left uncleared would show up as
missing or wrong outputs, never as a hang.)"""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _layer(T, K, N, r, M, act="bf16", lr="bf16", layout="runs", weight_bits=8, mas=False,
           seed=0):
    from oracle.bf16 import bf16_round
    rng = np.random.default_rng(seed)
    counts = [T // M + (1 if m < T % M else 0) for m in range(M)]
    mod = synth.make_modality_layout(counts, layout if T >= 256 else "alternating", 0, seed)
    x = rng.standard_normal((T, K)).astype(np.float32)
    for m, s in enumerate([1.0, 30.0, 2.0][:M]):
        x[mod == m] *= np.float32(s)
    if act == "bf16":
        x = bf16_round(x)
    inv = rng.uniform(0.05, 3.0, (M, K)).astype(np.float32)
    qmax = (1 << (weight_bits - 1)) - 1
    shape = (M, N, K) if mas else (N, K)
    wq = rng.integers(-qmax, qmax + 1, shape).astype(np.int8)
    ws = rng.uniform(1e-4, 1e-2, (M, N) if mas else N).astype(np.float32)
    rr = 0 if mas else r
    ld = (rng.standard_normal((M - 1, rr, K)) / np.sqrt(K)).astype(np.float32)
    ru = (rng.standard_normal((M - 1, N, rr)) * 0.05).astype(np.float32)
    if lr == "bf16":
        ld, ru = bf16_round(ld), bf16_round(ru)
    L = dict(x=x, modality=mod, inv_smooth=inv, wq=wq, w_scale=ws, l_down=ld, r_up=ru,
             n_mod=M, rank=rr, act_dtype=act, lr_dtype=lr, weight_bits=weight_bits)
    if mas:
        L["method"] = "mas"
    return L


_CASES = {
    # register-resident stage 1, persistent tiled GEMM (128 tiles)
    "fr_persistent_t4096_k3584_n2048_m2": dict(T=4096, K=3584, N=2048, r=64, M=2),
    # k_down_lds + the row quantiser adding its partials, split-K GEMM (16 tiles)
    "down_lds_split_k_t2048_k3584_n512_m3": dict(T=2048, K=3584, N=512, r=64, M=3),
    # rows longer than the registers hold: k_down_lds over many slices
    "down_lds_long_rows_t512_k18944_n256_m3": dict(T=512, K=18944, N=256, r=64, M=3),
    # fp32 activations, bf16 factors: the wide down-projection's partials
    "down_wide_f32_t2048_k2048_n512_m3": dict(T=2048, K=2048, N=512, r=64, M=3, act="f32"),
    # fp32 factors: quantiser, then the k-sliced down-projection's tickets
    "lowrank_down_f32_t1024_k2048_n512_m3": dict(T=1024, K=2048, N=512, r=64, M=3, act="f32",
                                                 lr="f32"),
    # small batch: the decode GEMM's slice partials and counters
    "decode_t16_k4096_n512_m2": dict(T=16, K=4096, N=512, r=64, M=2),
    # the 4-bit shared weight over few tiles (split K)
    "w4a8_split_k_t700_k1024_n528_m3": dict(T=700, K=1024, N=528, r=32, M=3, weight_bits=4),
    # MAS-only: the rows grouped by modality, its tile table and counters
    "mas_only_few_tiles_t700_k2048_n528_m3": dict(T=700, K=2048, N=528, r=0, M=3, mas=True),
    "mas_only_decode_t16_k4096_n512_m2": dict(T=16, K=4096, N=512, r=0, M=2, mas=True),
}


def _bits(y):
    return y.view(torch.int16 if y.dtype == torch.bfloat16 else torch.int32).clone()


@pytest.mark.parametrize("name", list(_CASES))
def test_dirty_workspace_gives_identical_outputs(name):
    assert torch.cuda.is_available()
    from paper_2603_04800_amd import ops, workload
    kw = _CASES[name]
    L = _layer(seed=31, **kw)
    x, mod, lin = workload.to_device(L)
    T = x.shape[0]
    if kw.get("mas"):
        need = int(ops._lib.masq_mas_only_workspace_bytes(T, lin.c_in, lin.c_out, lin.n_mod))
    else:
        need = ops.workspace_bytes(T, lin.c_in, lin.c_out, lin.rank, lin.n_mod)
    print(f"[workspace] {name}: T={T} K={lin.c_in} N={lin.c_out} {need} bytes", flush=True)
    out_dt = torch.bfloat16 if kw.get("act", "bf16") == "bf16" else torch.float32
    dev = x.device

    def run(ws):
        y = torch.full((T, lin.c_out), float("nan"), dtype=out_dt, device=dev)
        lin(x, mod, out=y, workspace=ws)
        torch.cuda.synchronize()
        return _bits(y)

    ref = run(torch.zeros(max(need, 256), dtype=torch.uint8, device=dev))
    assert not torch.isnan(ref.view(out_dt).float()).any()
    for fill in (0xA5, 0x7F, 0xFF):
        ws = torch.full((max(need, 256),), fill, dtype=torch.uint8, device=dev)
        for rep in range(2):
            got = run(ws)
            assert torch.equal(got, ref), f"{name}: fill {fill:#x}, call {rep}"
