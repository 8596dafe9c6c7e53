"""The int8 GEMM at the longest rows the ABI accepts, with codes at the ends
of their range, so that the int32 accumulators come within a hair of 2^31
(eq. PTQ codes in [-127, 127]; 4-bit weight codes in [-7, 7], which the
kernels scale by 16 on the way into the int8 MFMA and back).  Every
accumulator must equal the oracle's exact product bit for bit, and the
dequantised outputs too (the same two fp32 multiplies), on each GEMM the
dispatch picks for such rows: the generic kernel (c_in % 64 != 0), the
direct-to-LDS GEMM, and the small-batch GEMM (16 tokens, rows longer than
the decode GEMM takes)."""
import numpy as np
import pytest
import torch

from oracle import inference as oinf

pytestmark = pytest.mark.gpu

W8_MAX_K = 133136     # 127 * 127 * K < 2^31, K % 16 == 0
W4_MAX_K = 150976     # 127 * 7 * 16 * K < 2^31, K % 64 == 0


def _codes(T, K, N, qmax_w, seed):
    """q [T][K] and w [N][K]: rows 0 and 1 of each all +max and all -max (so
    that acc[0][0], acc[1][1] reach +max*max*K and acc[0][1], acc[1][0]
    -max*max*K), the rest random over the whole range."""
    rng = np.random.default_rng(seed)
    q = rng.integers(-127, 128, (T, K)).astype(np.int8)
    w = rng.integers(-qmax_w, qmax_w + 1, (N, K)).astype(np.int8)
    q[0], q[1] = 127, -127
    w[0], w[1] = qmax_w, -qmax_w
    return q, w


@pytest.mark.parametrize("T,K", [(64, W8_MAX_K), (64, W8_MAX_K - 16), (16, W8_MAX_K - 16)],
                         ids=["generic_k133136", "dma_k133120", "small_batch_t16_k133120"])
def test_w8a8_accumulators_at_the_longest_rows(T, K):
    assert torch.cuda.is_available()
    from paper_2603_04800_amd import ops
    N = 48
    q, w = _codes(T, K, N, 127, seed=K + T)
    rng = np.random.default_rng(3)
    xs = rng.uniform(1e-3, 1.0, T).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    print(f"[limits] w8 T={T} K={K}", flush=True)
    acc_ref, y_ref = oinf.w8a8_gemm(q, xs, w, ws)
    assert acc_ref[0, 0] == 127 * 127 * K and acc_ref[0, 1] == -127 * 127 * K
    dev = torch.device("cuda")
    acc, y = ops.w8a8_gemm(torch.from_numpy(q).to(dev), torch.from_numpy(xs).to(dev),
                           torch.from_numpy(w).to(dev), torch.from_numpy(ws).to(dev))
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert np.array_equal(y.cpu().numpy().view(np.int32), y_ref.view(np.int32))


@pytest.mark.parametrize("T", [64, 16], ids=["dma_t64", "small_batch_t16"])
def test_w4a8_accumulators_at_the_longest_rows(T):
    assert torch.cuda.is_available()
    from paper_2603_04800_amd import int4, ops
    K, N = W4_MAX_K, 48
    q, w = _codes(T, K, N, 7, seed=K + T)
    rng = np.random.default_rng(4)
    xs = rng.uniform(1e-3, 1.0, T).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    print(f"[limits] w4 T={T} K={K}", flush=True)
    acc_ref, y_ref = oinf.w8a8_gemm(q, xs, w, ws)
    assert acc_ref[0, 0] == 127 * 7 * K
    dev = torch.device("cuda")
    acc, y = ops.w4a8_gemm(torch.from_numpy(q).to(dev), torch.from_numpy(xs).to(dev),
                           torch.from_numpy(int4.pack(w)).to(dev), torch.from_numpy(ws).to(dev))
    torch.cuda.synchronize()
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert np.array_equal(y.cpu().numpy().view(np.int32), y_ref.view(np.int32))
