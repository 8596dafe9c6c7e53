"""The whole layer on a batch whose codes pass 2^31 bytes and whose
activations pass 2^32 bytes (640000 tokens x 3584 columns, and 120000
tokens x 18944 columns with three modalities, the paper's decoder widths,
so that both stage-1 forms run: rows held in registers, and the streamed
down-projection with the row quantiser): every per-token offset must be
64-bit.  The layer
works row by row (per-token smoothing and quantisation, a GEMM row, the
row's compensation), so the oracle checks sampled rows one by one, among
them the rows on both sides of the 2^31-byte boundary of the codes and the
last rows of the batch: text rows bit for bit, all rows within 1e-2."""
import numpy as np
import pytest
import torch

from oracle import inference as oinf

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T,K,r,M", [(640000, 3584, 16, 2), (120000, 18944, 64, 3)],
                         ids=["register_resident_stage1_t640000_k3584",
                              "down_lds_row_quantiser_t120000_k18944"])
def test_layer_past_2_31_bytes_of_codes(T, K, r, M):
    assert torch.cuda.is_available()
    from oracle.bf16 import bf16_round
    from paper_2603_04800_amd import ops
    N = 64
    assert T * K > 2 ** 31
    dev = torch.device("cuda")
    print(f"[large] T={T} K={K} N={N}", flush=True)
    g = torch.Generator(device=dev).manual_seed(12)
    x = torch.randn((T, K), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    mod = torch.randint(0, M, (T,), generator=g, device=dev, dtype=torch.int32)
    x[mod == 1] *= 30
    x[mod == 2] *= 2
    rng = np.random.default_rng(12)
    inv = rng.uniform(0.05, 3.0, (M, K)).astype(np.float32)
    wq = rng.integers(-127, 128, (N, K)).astype(np.int8)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    ld = bf16_round((rng.standard_normal((M - 1, r, K)) / np.sqrt(K)).astype(np.float32))
    ru = bf16_round((rng.standard_normal((M - 1, N, r)) * 0.05).astype(np.float32))
    lin = ops.Linear(torch.from_numpy(inv).to(dev), torch.from_numpy(wq).to(dev),
                     torch.from_numpy(ws).to(dev),
                     torch.from_numpy(ld).to(dev, torch.bfloat16),
                     torch.from_numpy(ru).to(dev, torch.bfloat16))
    y = lin(x, mod, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    edge = (2 ** 31) // K
    rows = sorted(set([0, 1, 2, edge - 2, edge - 1, edge, edge + 1, edge + 2, T - 3, T - 2, T - 1] +
                      rng.integers(0, T, 40).tolist()))
    idx = torch.tensor(rows, device=dev)
    xr = x[idx].float().cpu().numpy()
    mr = mod[idx].cpu().numpy()
    got = y[idx].float().cpu().numpy()
    ref = oinf.to_output(oinf.linear(xr, mr, inv, wq, ws, ld, ru), "bf16")
    assert oinf.relerr(got, ref) <= 1e-2
    text = mr == 0
    assert text.any() and np.array_equal(got[text], ref[text])
