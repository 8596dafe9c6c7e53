// Peak probes: the measured denominators the benchmark reports beside the
// MI355X spec-sheet peaks.  Not part of the layer; built as its own library
// (libmasq_probe.so) and declared in masq_probe.h.
//
//  k_probe_mfma_i8  int8 MFMA issue with no memory traffic: the rate the
//                   matrix cores sustain (at whatever clock the chip holds
//                   under that load) when nothing else limits them.
//  k_probe_read     a linear, coalesced 16-byte read of a large buffer: the
//                   HBM read rate a streaming kernel can reach.
//  k_probe_lds_dma  L2 -> LDS transfer by LDS DMA in the GEMM's stage-row
//                   pattern: what the GEMM's K-stage feed can sustain per CU.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "masq_probe.h"

namespace {

typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef int32_t v16i __attribute__((ext_vector_type(16)));

constexpr int kChains = 8;     // independent accumulator chains per wave

__global__ __launch_bounds__(256) void k_probe_mfma_i8(int iters, int32_t* __restrict__ out) {
    const int tid = static_cast<int>(threadIdx.x);
    const v4i a = {tid, 3 * tid + 1, 5, 7};
    const v4i b = {11, tid ^ 5, 13, 17};
    v16i acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = v16i{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < kChains; ++c)
            acc[c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[c], 0, 0, 0);
    }
    int32_t s = 0;
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) s += acc[c][e];
    out[static_cast<int64_t>(blockIdx.x) * blockDim.x + tid] = s;
}

constexpr int kReadUnroll = 4;

__global__ __launch_bounds__(256) void k_probe_read(const v4i* __restrict__ p, int64_t n16,
                                                     int32_t* __restrict__ out) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    v4i s = {0, 0, 0, 0};
    for (; i + (kReadUnroll - 1) * stride < n16; i += kReadUnroll * stride) {
        v4i v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) v[u] = p[i + u * stride];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) s ^= v[u];
    }
    for (; i < n16; i += stride) s ^= p[i];
    out[static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x] = s.x ^ s.y ^ s.z ^ s.w;
}

// L2 -> LDS transfer by LDS DMA (global_load_lds_dwordx4), the path that
// feeds the GEMM's K stages: every wave of a 512-thread workgroup moves
// 4 KB per round (four 1 KB instructions, 16 rows x 64 bytes each, the
// GEMM's stage-row pattern) into its own LDS area, at most three rounds in
// flight, over `iters` rounds; the rows lie in a region of `region` bytes
// with a 4 KB pitch (an L2-resident region measures the L2 path).
__device__ __forceinline__ void probe_lds_dma16(const void* src, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(src), "s"(lds_addr) : "memory", "m0");
}

__global__ __launch_bounds__(512) void k_probe_lds_dma(const uint8_t* __restrict__ src,
                                                       int64_t region, int iters,
                                                       int32_t* __restrict__ out) {
    __shared__ __attribute__((aligned(16))) uint8_t lds[8][4][1024];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int64_t kPitch = 4096;
    const int64_t nrows = region / kPitch;
    int64_t row = (static_cast<int64_t>(blockIdx.x) * 8 + wave) * 64 % nrows;
    const uint32_t base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&lds[wave][0][0]));
    for (int it = 0; it < iters; ++it) {
        for (int j = 0; j < 4; ++j) {
            const int64_t r = (row + 16 * j + lane / 4) % nrows;
            const int col = (it % 64) * 64 + 16 * (lane % 4);
            probe_lds_dma16(src + r * kPitch + col,
                            static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(
                                static_cast<int>(base) + j * 1024)));
        }
        row = (row + 64) % nrows;
        if ((it & 3) == 3) __builtin_amdgcn_s_waitcnt((8 & 15) | (7 << 4));    // vmcnt(8)
    }
    __builtin_amdgcn_s_waitcnt(7 << 4);                                        // vmcnt(0)
    __syncthreads();
    if (threadIdx.x == 0) out[blockIdx.x] = lds[0][0][0];
}

}  // namespace

extern "C" {

int masq_probe_lds_dma(const void* buf, int64_t region, int32_t blocks, int32_t iters,
                       int32_t* out, void* stream) {
    if (buf == nullptr || out == nullptr || blocks <= 0 || iters <= 0 || region < 4096 * 64 ||
        (reinterpret_cast<uintptr_t>(buf) & 15u) != 0)
        return -1;
    (void)hipGetLastError();
    k_probe_lds_dma<<<blocks, 512, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<const uint8_t*>(buf), region, iters, out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

int64_t masq_probe_lds_dma_bytes(int32_t blocks, int32_t iters) {
    return static_cast<int64_t>(blocks) * 8 * iters * 4 * 1024;
}

int masq_probe_mfma_i8(int32_t blocks, int32_t iters, int32_t* out, void* stream) {
    if (blocks <= 0 || iters <= 0 || out == nullptr) return -1;
    (void)hipGetLastError();
    k_probe_mfma_i8<<<blocks, 256, 0, static_cast<hipStream_t>(stream)>>>(iters, out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

int64_t masq_probe_mfma_i8_ops(int32_t blocks, int32_t iters) {
    return static_cast<int64_t>(blocks) * 4 * iters * kChains * (2LL * 32 * 32 * 32);
}

int masq_probe_read(const void* buf, int64_t bytes, int32_t blocks, int32_t* out, void* stream) {
    if (buf == nullptr || out == nullptr || blocks <= 0 || bytes < 0 || bytes % 16 != 0 ||
        (reinterpret_cast<uintptr_t>(buf) & 15u) != 0)
        return -1;
    (void)hipGetLastError();
    k_probe_read<<<blocks, 256, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<const v4i*>(buf), bytes / 16, out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

}  // extern "C"
