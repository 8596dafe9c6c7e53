"""The allocation-free entry point masq_linear_fused_noalloc against
masq_linear_fused: same kernels, so every output must agree bit for bit, on
consecutive calls that share the static scratch (each later call smaller than
the one before it, so leftovers of the larger call lie in the scratch), across
the dispatch paths (tiled GEMM with the fused stage 1, split K over few tiles,
the small-batch decode path).  The larger calls are also held to the oracle's
bar."""
import numpy as np
import pytest
import torch

from oracle import inference as oinf

pytestmark = pytest.mark.gpu


def _layer(T, K, N, r, M, seed):
    import synth
    from oracle.bf16 import bf16_round
    rng = np.random.default_rng(seed)
    counts = [T // M + (1 if m < T % M else 0) for m in range(M)]
    mod = synth.make_modality_layout(counts, "runs" if T >= 256 else "alternating", 0, seed)
    x = rng.standard_normal((T, K)).astype(np.float32)
    for m, s in enumerate([1.0, 30.0, 2.0][:M]):
        x[mod == m] *= np.float32(s)
    x = bf16_round(x)
    inv = rng.uniform(0.05, 3.0, (M, K)).astype(np.float32)
    wq = rng.integers(-127, 128, (N, K)).astype(np.int8)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    ld = bf16_round((rng.standard_normal((M - 1, r, K)) / np.sqrt(K)).astype(np.float32))
    ru = bf16_round((rng.standard_normal((M - 1, N, r)) * 0.05).astype(np.float32))
    return dict(x=x, modality=mod, inv_smooth=inv, wq=wq, w_scale=ws, l_down=ld, r_up=ru,
                n_mod=M, rank=r, act_dtype="bf16", lr_dtype="bf16", weight_bits=8)


def _run_pair(L, oracle=True):
    from paper_2603_04800_amd import workload
    x, mod, lin = workload.to_device(L)
    T = x.shape[0]
    print(f"[noalloc] T={T} K={lin.c_in} N={lin.c_out} r={lin.rank} M={lin.n_mod}", flush=True)
    y_ref = lin(x, mod, out_dtype=torch.bfloat16)
    y = torch.full_like(y_ref, float("nan"))
    lin.noalloc(x, mod, y)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16)), \
        "noalloc differs from masq_linear_fused"
    if oracle:
        ref = oinf.to_output(oinf.linear(L["x"], L["modality"], L["inv_smooth"], L["wq"],
                                         L["w_scale"], L["l_down"], L["r_up"]), "bf16")
        got = y.float().cpu().numpy()
        assert oinf.relerr(got, ref) <= 1e-2
        text = L["modality"] == 0
        assert np.array_equal(got[text], ref[text])


def test_noalloc_equals_fused_on_consecutive_shrinking_calls():
    assert torch.cuda.is_available()
    from paper_2603_04800_amd import ops
    sizes = [
        (4096, 3584, 4096, 64, 3, True),    # fused stage 1, tiled GEMM: 14.7 MB of codes
        (700, 1024, 528, 64, 3, True),      # few tiles: split K (arrival counters)
        (300, 512, 256, 32, 2, True),
        (16, 4096, 512, 64, 2, True),       # small batch: decode GEMM (its own counters)
        (5, 1024, 272, 32, 3, False),
    ]
    for i, (T, K, N, r, M, check) in enumerate(sizes):
        need = ops.workspace_bytes(T, K, N, r, M)
        assert need <= 64 << 20, f"case {i} needs {need} bytes"
        _run_pair(_layer(T, K, N, r, M, seed=100 + i), oracle=check)


def test_noalloc_rejects_a_problem_beyond_the_scratch_and_leaves_y_alone():
    from paper_2603_04800_amd import ops, workload
    T, K, N = 20000, 3584, 64
    assert ops.workspace_bytes(T, K, N, 16, 2) > 64 << 20
    L = _layer(64, 64, 64, 16, 2, seed=7)
    _, _, lin = workload.to_device(L)
    dev = torch.device("cuda")
    x = torch.zeros((T, K), dtype=torch.bfloat16, device=dev)
    mod = torch.zeros(T, dtype=torch.int32, device=dev)
    lin_big = ops.Linear(torch.ones((2, K), device=dev), torch.zeros((N, K), dtype=torch.int8,
                                                                     device=dev),
                         torch.ones(N, device=dev),
                         torch.zeros((1, 16, K), dtype=torch.bfloat16, device=dev),
                         torch.zeros((1, N, 16), dtype=torch.bfloat16, device=dev))
    y = torch.full((T, N), 3.0, dtype=torch.bfloat16, device=dev)
    with pytest.raises(ops.MasqError) as e:
        lin_big.noalloc(x, mod, y)
    assert e.value.code == 8
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())
    # an empty batch is a no-op
    y0 = torch.empty((0, lin.c_out), dtype=torch.bfloat16, device=dev)
    lin.noalloc(torch.empty((0, lin.c_in), dtype=torch.bfloat16, device=dev),
                torch.empty(0, dtype=torch.int32, device=dev), y0)
