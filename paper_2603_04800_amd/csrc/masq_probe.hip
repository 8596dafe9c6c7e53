// Peak probes: the measured denominators the benchmark reports beside the
// MI355X spec-sheet peaks.  Not part of the layer; built as its own library
// (libmasq_probe.so) and declared in masq_probe.h.
//
//  k_probe_mfma_i8  int8 MFMA issue with no memory traffic: the rate the
//                   matrix cores sustain (at whatever clock the chip holds
//                   under that load) when nothing else limits them.
//  k_probe_read     a linear, coalesced 16-byte read of a large buffer: the
//                   HBM read rate a streaming kernel can reach.

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

}  // namespace

extern "C" {

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
