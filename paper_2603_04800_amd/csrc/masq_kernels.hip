// HIP kernels of the modality-aware W8A8 + low-rank linear for gfx950 (CDNA4).
//
// Layer (MASQuant, Sec. 4.3 final case equation):
//   y_t = Q(x_t S_m^-1) . Q(S_t W)                       for every row
//       + (x_t S_m^-1) L1^m L2^m                          for rows of modality m != text
//
// Kernels
//   k_smooth_quant   one workgroup per token row: x * inv_s[m], wave64 + LDS
//                    absmax, delta = amax/127, int8 codes (eq. PTQ, z = 0).
//   k_lowrank_down   u = (x S_m^-1) L1^m on 16-row tiles with bf16 (or fp32)
//                    MFMA; rows of other modalities are masked to zero, tiles
//                    without non-text rows exit at once.
//   k_gemm           q . Wq^T on int8 MFMA (v_mfma_i32_32x32x32_i8), 256x256
//                    tiles, 128-byte K stages double-buffered in LDS with an
//                    XOR swizzle; epilogue: dequantisation, then on tiles that
//                    hold non-text rows the rank-r up-projection u L2^m on
//                    bf16 (fp32) MFMA accumulating into the dequantised fp32
//                    tile, then the cast and store.
//   k_lowrank_comp   standalone y += (x S_m^-1 L1^m) L2^m.
//
// Bit-exact contract: the smoothing is a single fp32 multiply, the scale and
// its reciprocal are correctly rounded divisions (the default for HIP), codes
// round half to even (v_rndne_f32), int32 accumulation is exact, the
// dequantisation is two fp32 multiplies in a fixed order.  The library is
// compiled without FP contraction.

#include <type_traits>

#include "masq_common.h"

namespace masq {
namespace {

typedef int32_t v2i __attribute__((ext_vector_type(2)));
typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef int32_t v16i __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

typedef uint16_t bf16_t;   // bfloat16 stored as its bit pattern

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// Two fp32 values narrowed to bf16 bits (a in the low half), round to nearest
// even: one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v2f{a, b}, v2bf));
}
__device__ __forceinline__ uint32_t f32_to_bf16(float f) { return pack_bf16x2(f, 0.f) & 0xFFFFu; }

// ---------------------------------------------------------------- element IO
template <typename T> struct Elem;
template <> struct Elem<float> {
    static __device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
        const v4f a = *reinterpret_cast<const v4f*>(p);
        const v4f b = *reinterpret_cast<const v4f*>(p + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
    static __device__ __forceinline__ float load1(const float* p) { return *p; }
    static __device__ __forceinline__ void store1(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16_t> {
    static __device__ __forceinline__ void load8(const bf16_t* p, float (&v)[8]) {
        const v4i a = *reinterpret_cast<const v4i*>(p);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = __uint_as_float(static_cast<uint32_t>(a[j]) << 16);
            v[2 * j + 1] = __uint_as_float(static_cast<uint32_t>(a[j]) & 0xFFFF0000u);
        }
    }
    static __device__ __forceinline__ float load1(const bf16_t* p) { return bf16_to_f32(*p); }
    static __device__ __forceinline__ void store1(bf16_t* p, float v) {
        *p = static_cast<bf16_t>(f32_to_bf16(v));
    }
};

__device__ __forceinline__ void load8_f32(const float* p, float (&v)[8]) { Elem<float>::load8(p, v); }

// Eight elements as loaded (16 or 32 bytes), converted to fp32 only when
// used, so that a software pipeline can keep the load in flight meanwhile.
template <typename T> struct Raw8;
template <> struct Raw8<bf16_t> {
    v4i a;
    __device__ __forceinline__ void load(const bf16_t* p) { a = *reinterpret_cast<const v4i*>(p); }
    __device__ __forceinline__ void to_f32(float (&v)[8]) const {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = __uint_as_float(static_cast<uint32_t>(a[j]) << 16);
            v[2 * j + 1] = __uint_as_float(static_cast<uint32_t>(a[j]) & 0xFFFF0000u);
        }
    }
};
template <> struct Raw8<float> {
    v4f a, b;
    __device__ __forceinline__ void load(const float* p) {
        a = *reinterpret_cast<const v4f*>(p);
        b = *reinterpret_cast<const v4f*>(p + 4);
    }
    __device__ __forceinline__ void to_f32(float (&v)[8]) const {
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
};

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

// Modality ids outside [0, n_mod) are treated as text, so that a bad id can
// never index past the smoothing or factor arrays.
__device__ __forceinline__ int sane_mod(int m, int n_mod) {
    return (m >= 0 && m < n_mod) ? m : 0;
}

// XOR swizzle of the 16-byte chunk index inside a 128-byte LDS row: any 8
// (or 16) consecutive rows read at one logical chunk land on distinct banks.
__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }

// 4-bit shared weight.  A row of K codes is packed two per byte, in 4-byte
// words of 8 codes: byte b of the word holding codes 8g .. 8g + 7 carries
// code 8g + b in its low nibble and code 8g + b + 4 in its high nibble
// (two's complement).  Two packed words (16 codes) become one 16-byte int8
// MFMA operand in k order, each code multiplied by 16: masking leaves every
// nibble in the high half of its byte, so the int8 byte reads 16 c.  An int32
// sum of such products is 16 times the true one and a multiple of 16, so an
// arithmetic shift right by 4 recovers it exactly.  (|16 c q| <= 112 * 127:
// any K below 2^31 / 14224 stays in range.)
__device__ __forceinline__ v4i w4_operand(v2i p) {
    constexpr int kHi = static_cast<int>(0xF0F0F0F0u);
    return v4i{(p.x << 4) & kHi, p.x & kHi, (p.y << 4) & kHi, p.y & kHi};
}

// ================================================================ LDS DMA
// One 16-byte lane of an LDS-DMA load: the wave writes 64 x 16 contiguous
// bytes at LDS address m0 (wave-uniform), lane i at m0 + 16 i.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(src), "s"(lds_addr) : "memory", "m0");
}

// Scheduling fence: the compiler may move no instruction across it, so the
// software pipeline below keeps the order it is written in.
#define MASQ_SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)

// s_waitcnt vmcnt(n) lgkmcnt(0) (expcnt unconstrained).
#define MASQ_WAIT_VMCNT_LGKM0(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (0 << 8))

// One 4-byte lane of an LDS-DMA load: lane i writes LDS address m0 + 4 i.
__device__ __forceinline__ void lds_dma4(const void* src, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
                 :: "v"(src), "s"(lds_addr) : "memory", "m0");
}

// ================================================================ smoothing + quant
// One workgroup per token row (small batches, where a row's latency
// matters): the first 256 x 8 x kSqChunks elements of the row are loaded
// with all requests in flight at once and kept in registers between the
// absmax and the quantisation; a longer row streams its remainder twice.
constexpr int kSqChunks = 10;

// Row t quantised by a workgroup of NT threads keeping NT x 8 x NCH elements
// of the row in registers.
template <typename XT, int NT, int NCH>
__device__ __forceinline__ void sq_row(const XT* __restrict__ x, const int32_t* __restrict__ mod,
                                       const float* __restrict__ inv_s, int K, int n_mod,
                                       int8_t* __restrict__ q, float* __restrict__ x_scale,
                                       int64_t t, bool pair) {
    __shared__ float red[NT / 64];
    const int m = sane_mod(mod[t], n_mod);
    const XT* xr = x + t * static_cast<int64_t>(K);
    const float* sr = inv_s + static_cast<int64_t>(m) * K;
    int8_t* qr = q + code_row(t, K, pair);
    const int nv = K >> 3;

    float xs[NCH][8];
    float amax = 0.f;
    {
        float xv[NCH][8], sv[NCH][8];
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int v = min(static_cast<int>(threadIdx.x) + NT * c, nv - 1);   // clamped
            Elem<XT>::load8(xr + 8 * v, xv[c]);
            load8_f32(sr + 8 * v, sv[c]);
        }
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const bool in = static_cast<int>(threadIdx.x) + NT * c < nv;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                xs[c][j] = xv[c][j] * sv[c][j];
                if (in) amax = fmaxf(amax, fabsf(xs[c][j]));
            }
        }
    }
    for (int v = threadIdx.x + NT * NCH; v < nv; v += NT) {
        float xv[8], sv[8];
        Elem<XT>::load8(xr + 8 * v, xv);
        load8_f32(sr + 8 * v, sv);
#pragma unroll
        for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(xv[j] * sv[j]));
    }
    amax = wave_max(amax);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
    __syncthreads();
    amax = red[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) amax = fmaxf(amax, red[w]);

    const bool nz = amax > 0.f;
    const float dx = nz ? amax / 127.0f : 0.f;     // correctly rounded
    const float rq = nz ? 127.0f / amax : 0.f;
    if (threadIdx.x == 0) x_scale[t] = dx;

    auto put8 = [&](int v, const float (&val)[8]) {
        uint32_t w[2] = {0u, 0u};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float c = rintf(val[j] * rq);
            c = fminf(fmaxf(c, -127.0f), 127.0f);
            w[j >> 2] |= (static_cast<uint32_t>(static_cast<int32_t>(c)) & 0xFFu) << (8 * (j & 3));
        }
        v2i out;
        out.x = static_cast<int32_t>(w[0]);
        out.y = static_cast<int32_t>(w[1]);
        *reinterpret_cast<v2i*>(qr + code_col(8 * v, pair)) = out;
    };
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int v = static_cast<int>(threadIdx.x) + NT * c;
        if (v < nv) put8(v, xs[c]);
    }
    for (int v = threadIdx.x + NT * NCH; v < nv; v += NT) {
        float xv[8], sv[8], val[8];
        Elem<XT>::load8(xr + 8 * v, xv);
        load8_f32(sr + 8 * v, sv);
#pragma unroll
        for (int j = 0; j < 8; ++j) val[j] = xv[j] * sv[j];
        put8(v, val);
    }
}

// u of row t from the wide down-projection's slice partials (one wave, lane
// k = rank column k < r <= 64): the slices added in slice order; also its
// bf16 hi/lo row [hi 64 | lo 64] (zero for text rows and columns past r).
__device__ __forceinline__ void finish_u_row(int64_t t, int64_t T, bool text, const float* part,
                                             int slices, int r, float* u, uint8_t* u_hl,
                                             int lane) {
    const int k = lane;
    float v = 0.f;                      // text rows: u = 0 (their partials are not written)
    if (k < r && !text) {
        // the slices' partials in flight together (16 a batch; past the last
        // slice the last is re-read and not added), added in slice order
        const float* p = part + t * r + k;
        const int64_t step = T * r;
        for (int s0 = 0; s0 < slices; s0 += 16) {
            float pv[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) pv[q] = p[min(s0 + q, slices - 1) * step];
            v = s0 == 0 ? pv[0] : v + pv[0];
#pragma unroll
            for (int q = 1; q < 16; ++q)
                if (s0 + q < slices) v += pv[q];
        }
    }
    if (k < r) u[t * r + k] = v;
    if (u_hl != nullptr) {
        const bool live = !text && k < r;
        const uint32_t hb = f32_to_bf16(v);
        const uint32_t lb = f32_to_bf16(v - __uint_as_float(hb << 16));
        reinterpret_cast<uint16_t*>(u_hl + t * 256)[k] = static_cast<uint16_t>(live ? hb : 0u);
        reinterpret_cast<uint16_t*>(u_hl + t * 256 + 128)[k] = static_cast<uint16_t>(live ? lb : 0u);
    }
}

template <typename XT>
__global__ __launch_bounds__(256) void k_smooth_quant(const XT* __restrict__ x,
                                                      const int32_t* __restrict__ mod,
                                                      const float* __restrict__ inv_s, int K,
                                                      int n_mod, int8_t* __restrict__ q,
                                                      float* __restrict__ x_scale,
                                                      int* __restrict__ zero_ints, int n_zero,
                                                      int64_t T, UFinish fin, bool pair) {
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < n_zero; i += 256) zero_ints[i] = 0;
    if (fin.part != nullptr && threadIdx.x < 64)
        finish_u_row(blockIdx.x, T, sane_mod(mod[blockIdx.x], n_mod) == 0, fin.part, fin.slices,
                     fin.r, fin.u, fin.u_hl, threadIdx.x);
    sq_row<XT, 256, kSqChunks>(x, mod, inv_s, K, n_mod, q, x_scale, blockIdx.x, pair);
}

__device__ __forceinline__ void split_bf16x8(const float (&v)[8], v4i& hi, v4i& lo) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t h = pack_bf16x2(v[2 * j], v[2 * j + 1]);
        const float h0 = __uint_as_float(h << 16), h1 = __uint_as_float(h & 0xFFFF0000u);
        hi[j] = static_cast<int32_t>(h);
        lo[j] = static_cast<int32_t>(pack_bf16x2(v[2 * j] - h0, v[2 * j + 1] - h1));
    }
}

// One row t quantised by one wave (lane = this lane), its smoothed values
// kept in registers between the absmax and the codes for rows of up to
// 64 * 8 * NC elements; longer rows stream their remainder twice.
template <typename XT, int NC>
__device__ __forceinline__ void quant_row_wave(const XT* __restrict__ x, const int32_t* __restrict__ mod,
                                               const float* __restrict__ inv_s, int K, int n_mod,
                                               int8_t* __restrict__ q, float* __restrict__ x_scale,
                                               int64_t t, bool pair, int lane) {
    const int m = sane_mod(mod[t], n_mod);
    const XT* xr = x + t * static_cast<int64_t>(K);
    const float* sr = inv_s + static_cast<int64_t>(m) * K;
    int8_t* qr = q + code_row(t, K, pair);
    const int nv = K >> 3;

    float xs[NC][8];
    float amax = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int v = lane + 64 * c;
        if (v < nv) {
            float xv[8], sv[8];
            Elem<XT>::load8(xr + 8 * v, xv);
            load8_f32(sr + 8 * v, sv);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                xs[c][j] = xv[j] * sv[j];
                amax = fmaxf(amax, fabsf(xs[c][j]));
            }
        }
    }
    for (int v = lane + 64 * NC; v < nv; v += 64) {
        float xv[8], sv[8];
        Elem<XT>::load8(xr + 8 * v, xv);
        load8_f32(sr + 8 * v, sv);
#pragma unroll
        for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(xv[j] * sv[j]));
    }
    amax = wave_max(amax);
    const bool nz = amax > 0.f;
    const float dx = nz ? amax / 127.0f : 0.f;     // correctly rounded
    const float rq = nz ? 127.0f / amax : 0.f;
    if (lane == 0) x_scale[t] = dx;

    auto store8 = [&](int v, const float (&vals)[8]) {
        uint32_t w[2] = {0u, 0u};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float c = rintf(vals[j] * rq);
            c = fminf(fmaxf(c, -127.0f), 127.0f);
            w[j >> 2] |= (static_cast<uint32_t>(static_cast<int32_t>(c)) & 0xFFu) << (8 * (j & 3));
        }
        v2i out;
        out.x = static_cast<int32_t>(w[0]);
        out.y = static_cast<int32_t>(w[1]);
        *reinterpret_cast<v2i*>(qr + code_col(8 * v, pair)) = out;
    };
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int v = lane + 64 * c;
        if (v < nv) store8(v, xs[c]);
    }
    for (int v = lane + 64 * NC; v < nv; v += 64) {
        float xv[8], sv[8], vals[8];
        Elem<XT>::load8(xr + 8 * v, xv);
        load8_f32(sr + 8 * v, sv);
#pragma unroll
        for (int j = 0; j < 8; ++j) vals[j] = xv[j] * sv[j];
        store8(v, vals);
    }
}

// One wave per token row (four rows per workgroup).  Used for large
// batches; k_smooth_quant (a whole workgroup per row) serves small ones,
// where a row's latency matters more than the number of rows in flight.
template <typename XT, int NC>
__global__ __launch_bounds__(256) void k_smooth_quant_rows(const XT* __restrict__ x,
                                                           const int32_t* __restrict__ mod,
                                                           const float* __restrict__ inv_s,
                                                           int64_t T, int K, int n_mod,
                                                           int8_t* __restrict__ q,
                                                           float* __restrict__ x_scale,
                                                           int* __restrict__ zero_ints,
                                                           int n_zero, UFinish fin, bool pair) {
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < n_zero; i += 256) zero_ints[i] = 0;
    const int lane = threadIdx.x & 63;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (t >= T) return;
    if (fin.part != nullptr)
        finish_u_row(t, T, sane_mod(mod[t], n_mod) == 0, fin.part, fin.slices, fin.r, fin.u, fin.u_hl, lane);
    quant_row_wave<XT, NC>(x, mod, inv_s, K, n_mod, q, x_scale, t, pair, lane);
}

// ================================================================ down-projection
// u = (x S_m^-1) L1^m for a tile of 16 token rows and a group of up to 64 rank
// columns.  Each of the four waves takes a quarter of the k range for all the
// group's columns (4 MFMA column blocks share one A fragment); the partial
// sums are added across waves in LDS in a fixed order.  Rows whose modality
// is not m contribute zeros.  MFMA operand layout: lane l holds row/column
// (l % 16) and the k group (l / 16); A and B use the same k assignment.
template <typename XT, typename LT> struct DownK;

// bf16 factors: the smoothed row enters as two bf16 terms, hi = bf16(xs) and
// lo = bf16(xs - hi), both multiplied with the exactly-bf16 factor, so the
// product keeps about 16 significant bits of the fp32 row.
template <typename XT> struct DownK<XT, bf16_t> {
    static constexpr int kStep = 32;
    static constexpr int kUnroll = 4;
    static __device__ __forceinline__ void run(const XT* x, const float* inv_s_m,
                                               const bf16_t* ld_m, int64_t row0, int64_t T,
                                               int K, int kb, int ke, int c0, int ncb,
                                               const int* smod, int m, v4f (&acc)[4], int lane) {
        const int ar = lane & 15, kg = lane >> 4;
        const int64_t t = row0 + ar;
        const bool live = (t < T) && (smod[ar] == m);
        const XT* xrow = x + (live ? t : row0) * static_cast<int64_t>(K);
        const bf16_t* lrow[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            lrow[j] = ld_m + static_cast<int64_t>(c0 + 16 * min(j, ncb - 1) + ar) * K;
        const v4i zero = {0, 0, 0, 0};
        for (int k0 = kb; k0 < ke; k0 += kStep * kUnroll) {
            float xv[kUnroll][8], sv[kUnroll][8];
            v4i bv[kUnroll][4];
            bool ok[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {       // all loads of the unrolled steps first
                const int k = k0 + kStep * u + 8 * kg;
                ok[u] = k < ke;
                const int kc = ok[u] ? k : ke - 8;
                Elem<XT>::load8(xrow + kc, xv[u]);
                load8_f32(inv_s_m + kc, sv[u]);
#pragma unroll
                for (int j = 0; j < 4; ++j) bv[u][j] = *reinterpret_cast<const v4i*>(lrow[j] + kc);
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                if (k0 + kStep * u >= ke) break;
                float xs[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) xs[e] = xv[u][e] * sv[u][e];
                v4i hi, lo;
                split_bf16x8(xs, hi, lo);
                const bool use = live && ok[u];
                hi = use ? hi : zero;
                lo = use ? lo : zero;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (j >= ncb) break;
                    const v4i b = ok[u] ? bv[u][j] : zero;
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(v8bf, hi), __builtin_bit_cast(v8bf, b), acc[j], 0, 0, 0);
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(v8bf, lo), __builtin_bit_cast(v8bf, b), acc[j], 0, 0, 0);
                }
            }
        }
    }
};

template <typename XT> struct DownK<XT, float> {   // fp32 factors: fp32 MFMA
    static constexpr int kStep = 4;
    static __device__ __forceinline__ void run(const XT* x, const float* inv_s_m,
                                               const float* ld_m, int64_t row0, int64_t T, int K,
                                               int kb, int ke, int c0, int ncb, const int* smod,
                                               int m, v4f (&acc)[4], int lane) {
        const int ar = lane & 15, kg = lane >> 4;
        const int64_t t = row0 + ar;
        const bool live = (t < T) && (smod[ar] == m);
        const XT* xrow = x + (live ? t : row0) * static_cast<int64_t>(K);
        for (int k0 = kb; k0 < ke; k0 += kStep) {
            const int k = k0 + kg;
            const bool ok = k < ke;
            const int kc = ok ? k : ke - 1;
            const float xs = Elem<XT>::load1(xrow + kc) * inv_s_m[kc];
            const float a = (live && ok) ? xs : 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (j >= ncb) break;
                const float b = ok ? ld_m[static_cast<int64_t>(c0 + 16 * j + ar) * K + kc] : 0.f;
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[j], 0, 0, 0);
            }
        }
    }
};

// The 16 x rc block of u (rank columns c0..c0+rc) over k in [kb, ke), summed
// over the modalities present, written as red-reduced fp32 to out(row, col).
template <int NW, typename XT, typename LT, typename Out>
__device__ __forceinline__ void down_group(const XT* x, const float* inv_s, const LT* l_down,
                                           int64_t row0, int64_t T, int K, int r, int n_mod,
                                           int kb, int ke, int c0, const int* smod,
                                           unsigned present, float (*red)[kRowsDown][64],
                                           Out out) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rc = min(64, r - c0);
    const int ncb = rc >> 4;
    constexpr int step = DownK<XT, LT>::kStep;
    const int span = ke - kb;
    const int q = ((span + NW * step - 1) / (NW * step)) * step;  // k per wave, step-aligned
    const int wkb = min(ke, kb + wave * q);
    const int wke = min(ke, wkb + q);
    v4f acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};
    for (int m = 1; m < n_mod; ++m) {
        if (!(present & (1u << m))) continue;
        DownK<XT, LT>::run(x, inv_s + static_cast<int64_t>(m) * K,
                           l_down + static_cast<int64_t>(m - 1) * r * K, row0, T, K, wkb, wke,
                           c0, ncb, smod, m, acc, lane);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (j >= ncb) break;
#pragma unroll
        for (int i = 0; i < 4; ++i) red[wave][4 * (lane >> 4) + i][16 * j + (lane & 15)] = acc[j][i];
    }
    __syncthreads();
    for (int idx = tid; idx < kRowsDown * rc; idx += 64 * NW) {
        const int row = idx / rc, col = idx - row * rc;
        float v = red[0][row][col];
#pragma unroll
        for (int w = 1; w < NW; ++w) v += red[w][row][col];       // fixed order
        out(row, c0 + col, v);
    }
    __syncthreads();
}

__device__ __forceinline__ unsigned tile_presence(const int* smod) {
    unsigned present = 0;
#pragma unroll
    for (int i = 0; i < kRowsDown; ++i)
        if (smod[i] > 0) present |= 1u << smod[i];
    return present;
}

// Down-projection u = (x S_m^-1) L1^m of the non-text rows (Sec. 4.3,
// eq. l1l2).  grid: (ceil(T / 16), n_kslices).  A workgroup takes 16 rows
// over the k slice [s kslice, (s + 1) kslice), split among its four waves
// and summed across them in LDS (down_group).  With one slice the result
// goes straight to u; otherwise each slice writes its partial sums to
// u_part[s], and the last slice workgroup of a row tile to arrive (counted
// on tickets[tile], cleared beforehand by the quantisation kernel) adds the
// partials in slice order, so the result does not depend on timing.  Tiles
// without non-text rows are skipped (their u rows are never read).
constexpr int kDownWaves = 8;

template <int NW, typename XT, typename LT>
__device__ __forceinline__ void down_tile_in(const XT* __restrict__ x, const int32_t* __restrict__ mod,
                                             const float* __restrict__ inv_s,
                                             const LT* __restrict__ l_down, int64_t T, int K, int r,
                                             int n_mod, int kslice, int n_kslices,
                                             float* __restrict__ u, float* __restrict__ u_part,
                                             int* __restrict__ tickets, int tile, int s, int* smod,
                                             float (*red)[kRowsDown][64], int* last_flag) {
    const int tid = threadIdx.x;
    const int64_t row0 = static_cast<int64_t>(tile) * kRowsDown;
    const int kb = s * kslice;
    const int ke = min(K, kb + kslice);
    if (tid < kRowsDown) {
        const int64_t t = row0 + tid;
        smod[tid] = t < T ? sane_mod(mod[t], n_mod) : 0;
    }
    __syncthreads();
    const unsigned present = tile_presence(smod);
    if (!present) return;                                            // uniform per tile
    float* out = n_kslices > 1 ? u_part + static_cast<int64_t>(s) * T * r : u;
    for (int c0 = 0; c0 < r; c0 += 64)
        down_group<NW, XT, LT>(x, inv_s, l_down, row0, T, K, r, n_mod, kb, ke, c0, smod, present,
                               red, [&](int row, int col, float v) {
                                   const int64_t t = row0 + row;
                                   if (t < T) out[t * r + col] = v;
                               });
    if (n_kslices == 1 || tickets == nullptr) return;   // the consumer adds the partials

    __threadfence();                 // this slice's partials are visible device-wide ...
    __syncthreads();
    if (tid == 0) *last_flag = atomicAdd(&tickets[tile], 1) == n_kslices - 1;
    __syncthreads();
    if (!*last_flag) return;
    __threadfence();                 // ... before the last arrival reads them all
    // 4 consecutive values per thread (r % 16 == 0); the partials of 8 slices
    // are loaded together and added in slice order
    const int rows = static_cast<int>(min<int64_t>(kDownRows, T - row0));
    const int64_t slice = T * r;
    for (int idx = 4 * tid; idx < rows * r; idx += 4 * 64 * NW) {
        const int64_t e = row0 * r + idx;
        v4f v = *reinterpret_cast<const v4f*>(u_part + e);
        for (int q0 = 1; q0 < n_kslices; q0 += 8) {
            v4f part[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int q = min(q0 + k, n_kslices - 1);
                part[k] = *reinterpret_cast<const v4f*>(u_part + q * slice + e);
            }
#pragma unroll
            for (int k = 0; k < 8; ++k)
                if (q0 + k < n_kslices) v += part[k];
        }
        *reinterpret_cast<v4f*>(u + e) = v;
    }
}

template <typename XT, typename LT>
__device__ __forceinline__ void down_tile(const XT* __restrict__ x, const int32_t* __restrict__ mod,
                                          const float* __restrict__ inv_s,
                                          const LT* __restrict__ l_down, int64_t T, int K, int r,
                                          int n_mod, int kslice, int n_kslices,
                                          float* __restrict__ u, float* __restrict__ u_part,
                                          int* __restrict__ tickets, int tile, int s) {
    __shared__ int smod[kRowsDown];
    __shared__ float red[kDownWaves][kRowsDown][64];
    __shared__ int last;
    down_tile_in<kDownWaves, XT, LT>(x, mod, inv_s, l_down, T, K, r, n_mod, kslice, n_kslices, u,
                                     u_part, tickets, tile, s, smod, red, &last);
}

template <typename XT, typename LT>
__global__ __launch_bounds__(64 * kDownWaves) void k_lowrank_down(const XT* __restrict__ x,
                                                      const int32_t* __restrict__ mod,
                                                      const float* __restrict__ inv_s,
                                                      const LT* __restrict__ l_down, int64_t T,
                                                      int K, int r, int n_mod, int kslice,
                                                      int n_kslices, float* __restrict__ u,
                                                      float* __restrict__ u_part,
                                                      int* __restrict__ tickets) {
    down_tile<XT, LT>(x, mod, inv_s, l_down, T, K, r, n_mod, kslice, n_kslices, u, u_part, tickets,
                      blockIdx.x, blockIdx.y);
}

// Down-projection of large batches (bf16 factors, rank <= 64): u = (x S_m^-1)
// L1^m of the non-text rows over 128-row tiles (each L1 fragment serves 128
// rows) and k slices [s kslice, (s + 1) kslice); grid (ceil(T / 128), S).
// Wave w takes rows 32 w .. 32 w + 31 of the tile (skipping out when none of
// them is non-text) and accumulates on v_mfma_f32_32x32x16_bf16 with the L1
// rows as operand A, the hi/lo split of the smoothed rows as operand B, so
// that each lane ends up with one token and 16 rank columns.  The slice's
// fp32 partials go to part[s]; the quantisation kernel adds the slices in
// slice order.
template <typename XT>
__global__ __launch_bounds__(256, 2) void k_down_wide(const XT* __restrict__ x,
                                                   const int32_t* __restrict__ mod,
                                                   const float* __restrict__ inv_s,
                                                   const bf16_t* __restrict__ l_down, int64_t T,
                                                   int K, int r, int n_mod, int kslice,
                                                   float* __restrict__ part) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int rl = lane & 31, kg = lane >> 5;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * kDownWideRows + 32 * wave + rl;
    const bool valid = t < T;
    const int mrow = valid ? sane_mod(mod[t], n_mod) : 0;
    unsigned pres = 0;
    for (int m = 1; m < n_mod; ++m)
        if (__ballot(valid && mrow == m) != 0ull) pres |= 1u << m;
    const unsigned present = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<int>(pres)));
    if (present == 0) return;                                 // uniform: no non-text row here
    int mods[3] = {0, 0, 0};
    int np = 0;
    for (int m = 1; m < n_mod; ++m)
        if (present & (1u << m)) mods[np++] = m;
    const int kb = blockIdx.y * kslice, ke = min(K, kb + kslice);
    const XT* xrow = x + (valid ? t : 0) * static_cast<int64_t>(K);
    const float* srow = inv_s + static_cast<int64_t>(mrow) * K;
    const int nrb = (r + 31) >> 5;                            // 32-rank blocks (1 or 2)
    v16f acc[2];
    acc[0] = v16f{0.f};
    acc[1] = v16f{0.f};
    const v4i zero = {0, 0, 0, 0};
    // two-deep software pipeline over rounds of kSteps 16-column MFMA steps:
    // the next round's loads (rows, smoothing factors, L1 rows of the first
    // modality present) are in flight while the current round is used
    constexpr int kSteps = 2;
    struct Stage {
        Raw8<XT> xr[kSteps];
        Raw8<float> sr[kSteps];
        v4i bv[kSteps][2];
    };
    const bf16_t* lm0 = l_down + static_cast<int64_t>(mods[0] - 1) * r * K;
    auto issue = [&](int k0, Stage& S) __attribute__((always_inline)) {
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            const int k = k0 + 16 * st + 8 * kg;
            const int kc = k < ke ? k : ke - 8;
            S.xr[st].load(xrow + kc);
            S.sr[st].load(srow + kc);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
                S.bv[st][rb] = *reinterpret_cast<const v4i*>(
                    lm0 + static_cast<int64_t>(min(32 * rb + rl, r - 1)) * K + kc);
        }
    };
    auto compute = [&](int k0, const Stage& S) __attribute__((always_inline)) {
        bool ok[kSteps];
        v4i hi[kSteps], lo[kSteps];
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            ok[st] = k0 + 16 * st + 8 * kg < ke;
            float xv[8], sv[8], xs[8];
            S.xr[st].to_f32(xv);
            S.sr[st].to_f32(sv);
#pragma unroll
            for (int e = 0; e < 8; ++e) xs[e] = xv[e] * sv[e];
            split_bf16x8(xs, hi[st], lo[st]);
        }
        for (int p = 0; p < np; ++p) {                        // usually one modality
            v4i bv[kSteps][2];
            if (p == 0) {
#pragma unroll
                for (int st = 0; st < kSteps; ++st) {
                    bv[st][0] = S.bv[st][0];
                    bv[st][1] = S.bv[st][1];
                }
            } else {
                const bf16_t* lm = l_down + static_cast<int64_t>(mods[p] - 1) * r * K;
#pragma unroll
                for (int st = 0; st < kSteps; ++st) {
                    const int k = k0 + 16 * st + 8 * kg;
                    const int kc = ok[st] ? k : ke - 8;
#pragma unroll
                    for (int rb = 0; rb < 2; ++rb)
                        bv[st][rb] = *reinterpret_cast<const v4i*>(
                            lm + static_cast<int64_t>(min(32 * rb + rl, r - 1)) * K + kc);
                }
            }
            const bool mine = valid && mrow == mods[p];
#pragma unroll
            for (int st = 0; st < kSteps; ++st) {
                const bool use = mine && ok[st];
                const v4i h = use ? hi[st] : zero, l = use ? lo[st] : zero;
#pragma unroll
                for (int rb = 0; rb < 2; ++rb) {
                    if (rb >= nrb) break;
                    // rank rows past r multiply zeros
                    const v4i bb = (32 * rb + rl < r) ? bv[st][rb] : zero;
                    acc[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(v8bf, bb), __builtin_bit_cast(v8bf, h), acc[rb], 0, 0, 0);
                    acc[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(v8bf, bb), __builtin_bit_cast(v8bf, l), acc[rb], 0, 0, 0);
                }
            }
        }
    };
    constexpr int kSpan = 16 * kSteps;
    {
        Stage A, B;
        issue(kb, A);
        for (int k0 = kb; k0 < ke; k0 += 2 * kSpan) {
            if (k0 + kSpan < ke) issue(k0 + kSpan, B);
            compute(k0, A);
            if (k0 + kSpan >= ke) break;
            if (k0 + 2 * kSpan < ke) issue(k0 + 2 * kSpan, A);
            compute(k0 + kSpan, B);
        }
    }
    // acc[rb][e]: token t, rank 32 rb + 8 (e / 4) + 4 kg + e % 4
    if (!valid) return;
    float* out = part + (static_cast<int64_t>(blockIdx.y) * T + t) * r;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
        if (rb >= nrb) break;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int rk = 32 * rb + 8 * g + 4 * kg;
            if (rk < r)
                *reinterpret_cast<v4f*>(out + rk) =
                    v4f{acc[rb][4 * g], acc[rb][4 * g + 1], acc[rb][4 * g + 2], acc[rb][4 * g + 3]};
        }
    }
}

// Stage 1 of the small-batch path in one launch: workgroups [0, T) quantise
// one row each, workgroups [T, T + n_kslices) compute one k slice of the
// down-projection (partials left for the GEMM to add).  256 threads: four
// waves per slice of 512 columns, so the many small slices start at once.
// Workgroup 0 also clears zero_ints (the decode GEMM's arrival counters).
template <typename XT, typename LT>
__global__ __launch_bounds__(256) void k_stage1_small(
    const XT* __restrict__ x, const int32_t* __restrict__ mod, const float* __restrict__ inv_s,
    const LT* __restrict__ l_down, int T, int K, int r, int n_mod, int kslice, int n_kslices,
    int8_t* __restrict__ q, float* __restrict__ x_scale, float* __restrict__ u,
    float* __restrict__ u_part, int* __restrict__ zero_ints, int n_zero) {
    __shared__ int smod[kRowsDown];
    __shared__ float red[4][kRowsDown][64];
    __shared__ int last;
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < n_zero; i += blockDim.x) zero_ints[i] = 0;
    if (static_cast<int>(blockIdx.x) < T) {
        sq_row<XT, 256, kSqChunks>(x, mod, inv_s, K, n_mod, q, x_scale, blockIdx.x, false);
    } else if (l_down != nullptr) {
        down_tile_in<4, XT, LT>(x, mod, inv_s, l_down, T, K, r, n_mod, kslice, n_kslices, u,
                                u_part, nullptr, 0, blockIdx.x - T, smod, red, &last);
    }
}

// ================================================================ fused stage 1
// Smoothing, per-token quantisation and the down-projection in one kernel
// (bf16 factors, rank <= 64, batches above the small path).  A workgroup
// takes 16 rows; its 8 waves split K.  Pass 1 streams the rows once: each
// wave keeps the absmax of its part of every row and accumulates u on
// bf16 MFMA (hi/lo split of the smoothed values, rows masked to each
// non-text modality present).  Absmax and u are combined across waves in
// LDS in a fixed order.  Pass 2 re-reads the wave's part (from cache) and
// writes the int8 codes with the row's reciprocal scale.
// SL (32 rows): the smoothing factors of every modality ([n_mod][K] fp32,
// at most kFuseInvBytes) are copied to LDS by DMA at the start and read from
// there instead of being loaded with every step of every row group.
constexpr int kFuseWaves = 8;
constexpr int kFuseWideMinT = 8192;    // batches from this size take 32 rows per workgroup
constexpr int kFuseInvBytes = 65536;

template <typename XT, int RG, bool SL = false>
__global__ __launch_bounds__(64 * kFuseWaves) void k_stage1_fused(
    const XT* __restrict__ x, const int32_t* __restrict__ mod, const float* __restrict__ inv_s,
    const bf16_t* __restrict__ l_down, int64_t T, int K, int r, int n_mod,
    int8_t* __restrict__ q, float* __restrict__ x_scale, float* __restrict__ u,
    uint8_t* __restrict__ u_hl, int* __restrict__ zero_ints, int n_zero, bool pair) {
    constexpr int kRows = 16 * RG;                 // RG groups of 16 rows share each L1 fragment
    if (blockIdx.x == 0)                           // arrival counters of stage 2
        for (int i = threadIdx.x; i < n_zero; i += blockDim.x) zero_ints[i] = 0;
    __shared__ int smod[kRows];
    __shared__ float samax[kFuseWaves][kRows];
    __shared__ float red[kFuseWaves][kRows][64];
    __shared__ float srq[kRows];
    __shared__ __attribute__((aligned(16))) float s_inv[SL ? kFuseInvBytes / 4 : 4];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kRows;
    if constexpr (SL) {
        // n_mod K / 4 pieces of 16 bytes in 1 KB blocks (the last block's
        // pieces past the end repeat the last piece; the host checks the fit)
        const int pieces = n_mod * K / 4;
        const uint32_t b0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(s_inv));
        for (int i = wave; i * 64 < pieces; i += kFuseWaves)
            lds_dma16(inv_s + 4 * min(i * 64 + lane, pieces - 1), b0 + i * 1024);
    }
    if (tid < kRows) {
        const int64_t t = row0 + tid;
        smod[tid] = t < T ? sane_mod(mod[t], n_mod) : 0;
    }
    if constexpr (SL) MASQ_WAIT_VMCNT_LGKM0(0);      // this wave's share of the factors
    __syncthreads();
    // non-text modalities present in the tile, as a list (scalar registers:
    // the MFMA loop below must branch on it, MFMA ignores EXEC)
    unsigned pres = 0;
#pragma unroll
    for (int i = 0; i < kRows; ++i)
        if (smod[i] > 0) pres |= 1u << smod[i];
    const unsigned present = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<int>(pres)));
    int mods[3] = {0, 0, 0};
    int np = 0;
    for (int m = 1; m < n_mod; ++m)
        if (present & (1u << m)) mods[np++] = m;
    const int ncb = r >> 4;                                   // 16-column MFMA blocks (<= 4)

    constexpr int kStep = 32, kU = 2;
    const int per = ((K + kFuseWaves * kStep - 1) / (kFuseWaves * kStep)) * kStep;
    const int kb = min(K, wave * per), ke = min(K, kb + per);
    const int ar = lane & 15, kg = lane >> 4;
    bool valid[RG];
    int mrow[RG];
    const XT* xrow[RG];
    const float* srow[RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        const int64_t t = row0 + 16 * g + ar;
        valid[g] = t < T;
        mrow[g] = smod[16 * g + ar];
        xrow[g] = x + (valid[g] ? t : row0) * static_cast<int64_t>(K);
        srow[g] = inv_s + static_cast<int64_t>(mrow[g]) * K;
    }

    v4f acc[RG][4];
    float amax[RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        amax[g] = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[g][j] = v4f{0.f, 0.f, 0.f, 0.f};
    }
    const v4i zero = {0, 0, 0, 0};
    // Pass 1 as a two-deep software pipeline (one row group): the loads of
    // the next 64 columns (rows, smoothing factors, L1 rows of the first
    // modality present) are issued before the current ones are used; the L1
    // rows of further modalities are loaded in place.
    struct Stage {
        Raw8<XT> xr[RG][kU];
        Raw8<float> sr[RG][kU];
        v4i bv[kU][4];
    };
    const bf16_t* lm0 = l_down + static_cast<int64_t>(max(mods[0] - 1, 0)) * r * K;
    auto issue = [&](int k0, Stage& S) __attribute__((always_inline)) {
#pragma unroll
        for (int uu = 0; uu < kU; ++uu) {
            const int k = k0 + kStep * uu + 8 * kg;
            const int kc = k < ke ? k : ke - 8;
#pragma unroll
            for (int g = 0; g < RG; ++g) {
                S.xr[g][uu].load(xrow[g] + kc);
                if constexpr (!SL) S.sr[g][uu].load(srow[g] + kc);
            }
            if (np > 0) {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    S.bv[uu][j] = *reinterpret_cast<const v4i*>(
                        lm0 + static_cast<int64_t>(16 * min(j, ncb - 1) + ar) * K + kc);
            }
        }
    };
    auto compute = [&](int k0, const Stage& S) __attribute__((always_inline)) {
        bool ok[kU];
#pragma unroll
        for (int uu = 0; uu < kU; ++uu) ok[uu] = k0 + kStep * uu + 8 * kg < ke;
        v4i hi[RG][kU], lo[RG][kU];
#pragma unroll
        for (int g = 0; g < RG; ++g)
#pragma unroll
            for (int uu = 0; uu < kU; ++uu) {
                float xv[8], sv[8], xs[8];
                S.xr[g][uu].to_f32(xv);
                if constexpr (SL) {
                    const int k = k0 + kStep * uu + 8 * kg;
                    const float* sp = s_inv + mrow[g] * K + (k < ke ? k : ke - 8);
                    *reinterpret_cast<v4f*>(sv) = *reinterpret_cast<const v4f*>(sp);
                    *reinterpret_cast<v4f*>(sv + 4) = *reinterpret_cast<const v4f*>(sp + 4);
                } else {
                    S.sr[g][uu].to_f32(sv);
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    xs[e] = xv[e] * sv[e];
                    if (valid[g] && ok[uu]) amax[g] = fmaxf(amax[g], fabsf(xs[e]));
                }
                split_bf16x8(xs, hi[g][uu], lo[g][uu]);
            }
        for (int p = 0; p < np; ++p) {                        // usually one modality
            v4i bv[kU][4];
            if (p == 0) {
#pragma unroll
                for (int uu = 0; uu < kU; ++uu)
#pragma unroll
                    for (int j = 0; j < 4; ++j) bv[uu][j] = S.bv[uu][j];
            } else {
                const bf16_t* lm = l_down + static_cast<int64_t>(mods[p] - 1) * r * K;
#pragma unroll
                for (int uu = 0; uu < kU; ++uu) {
                    const int k = k0 + kStep * uu + 8 * kg;
                    const int kc = ok[uu] ? k : ke - 8;
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        bv[uu][j] = *reinterpret_cast<const v4i*>(
                            lm + static_cast<int64_t>(16 * min(j, ncb - 1) + ar) * K + kc);
                }
            }
#pragma unroll
            for (int g = 0; g < RG; ++g) {
                const bool mine = valid[g] && mrow[g] == mods[p];
#pragma unroll
                for (int uu = 0; uu < kU; ++uu) {
                    const bool use = mine && ok[uu];
                    const v4i h = use ? hi[g][uu] : zero, l = use ? lo[g][uu] : zero;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (j >= ncb) break;
                        acc[g][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(v8bf, h), __builtin_bit_cast(v8bf, bv[uu][j]), acc[g][j], 0, 0, 0);
                        acc[g][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(v8bf, l), __builtin_bit_cast(v8bf, bv[uu][j]), acc[g][j], 0, 0, 0);
                    }
                }
            }
        }
    };
    constexpr int kSpan = kStep * kU;
    if constexpr (RG == 1) {
        if (kb < ke) {
            Stage A, B;
            issue(kb, A);
            for (int k0 = kb; k0 < ke; k0 += 2 * kSpan) {
                if (k0 + kSpan < ke) issue(k0 + kSpan, B);
                compute(k0, A);
                if (k0 + kSpan >= ke) break;
                if (k0 + 2 * kSpan < ke) issue(k0 + 2 * kSpan, A);
                compute(k0 + kSpan, B);
            }
        }
    } else {                          // two row groups: no registers for a second stage
        for (int k0 = kb; k0 < ke; k0 += kSpan) {
            Stage A;
            issue(k0, A);
            compute(k0, A);
        }
    }
    // the four lanes of a row (lane % 16) hold its four k groups
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        float a = amax[g];
        a = fmaxf(a, __shfl_xor(a, 16));
        a = fmaxf(a, __shfl_xor(a, 32));
        if (lane < 16) samax[wave][16 * g + lane] = a;
    }
    if (np > 0) {
#pragma unroll
        for (int g = 0; g < RG; ++g)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (j >= ncb) break;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    red[wave][16 * g + 4 * (lane >> 4) + i][16 * j + (lane & 15)] = acc[g][j][i];
            }
    }
    __syncthreads();
    if (tid < kRows) {
        float a = samax[0][tid];
#pragma unroll
        for (int w = 1; w < kFuseWaves; ++w) a = fmaxf(a, samax[w][tid]);
        const bool nz = a > 0.f;
        srq[tid] = nz ? 127.0f / a : 0.f;                     // correctly rounded
        if (row0 + tid < T) x_scale[row0 + tid] = nz ? a / 127.0f : 0.f;
    }
    // u (fp32; written when the tile has non-text rows) and its bf16 hi/lo
    // rows [hi 64 | lo 64] for the GEMM epilogue (text rows and columns past
    // r zero there): thread (row, g) sums columns 8 g .. 8 g + 7 over the
    // waves in a fixed order
    static_assert(kRows * 8 <= 64 * kFuseWaves, "one thread per (row, 8 columns)");
    if (tid < kRows * 8 && (np > 0 || u_hl != nullptr)) {
        const int row = tid >> 3, g = tid & 7;
        const int64_t t = row0 + row;
        if (t < T) {
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = 0.f;
            if (np > 0 && 8 * g < r) {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    v4f a = *reinterpret_cast<const v4f*>(&red[0][row][8 * g + 4 * h]);
#pragma unroll
                    for (int w = 1; w < kFuseWaves; ++w)
                        a += *reinterpret_cast<const v4f*>(&red[w][row][8 * g + 4 * h]);
                    v[4 * h] = a.x; v[4 * h + 1] = a.y; v[4 * h + 2] = a.z; v[4 * h + 3] = a.w;
                    *reinterpret_cast<v4f*>(u + t * r + 8 * g + 4 * h) = a;
                }
            }
            if (u_hl != nullptr) {
                v4i hi, lo;
                split_bf16x8(v, hi, lo);
                const bool live = smod[row] > 0;
                *reinterpret_cast<v4i*>(u_hl + t * 256 + 16 * g) = live ? hi : zero;
                *reinterpret_cast<v4i*>(u_hl + t * 256 + 128 + 16 * g) = live ? lo : zero;
            }
        }
    }
    __syncthreads();

    // pass 2: lane -> row 16 g + lane / 4 of each row group, 16 consecutive
    // elements at 16 (lane % 4); the row groups' loads go out together
    const int qc = 16 * (lane & 3);
    for (int k0 = kb; k0 < ke; k0 += 64) {
        const int k = k0 + qc;
        float xv[RG][16], sv[RG][16];
        bool live[RG];
#pragma unroll
        for (int g = 0; g < RG; ++g) {
            const int qr = 16 * g + (lane >> 2);
            const int64_t tq = row0 + qr;
            live[g] = tq < T && k < ke;
            const int64_t tl = live[g] ? tq : row0;
            const int kl = live[g] ? k : kb;
            const XT* xr2 = x + tl * static_cast<int64_t>(K);
            const float* sr2 = (SL ? s_inv : inv_s) + static_cast<int64_t>(smod[qr]) * K;
            Elem<XT>::load8(xr2 + kl, *reinterpret_cast<float(*)[8]>(xv[g]));
            Elem<XT>::load8(xr2 + kl + 8, *reinterpret_cast<float(*)[8]>(xv[g] + 8));
            load8_f32(sr2 + kl, *reinterpret_cast<float(*)[8]>(sv[g]));
            load8_f32(sr2 + kl + 8, *reinterpret_cast<float(*)[8]>(sv[g] + 8));
        }
#pragma unroll
        for (int g = 0; g < RG; ++g) {
            if (!live[g]) continue;
            const int qr = 16 * g + (lane >> 2);
            const float rq = srq[qr];
            uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                float c = rintf((xv[g][e] * sv[g][e]) * rq);
                c = fminf(fmaxf(c, -127.0f), 127.0f);
                w[e >> 2] |= (static_cast<uint32_t>(static_cast<int32_t>(c)) & 0xFFu) << (8 * (e & 3));
            }
            *reinterpret_cast<v4i*>(q + code_row(row0 + qr, K, pair) + code_col(k, pair)) =
                v4i{static_cast<int32_t>(w[0]), static_cast<int32_t>(w[1]), static_cast<int32_t>(w[2]),
                    static_cast<int32_t>(w[3])};
        }
    }
}

// ---------------------------------------------------------------- down-projection, operands in LDS
// u = xs L1^m for bf16 activations and factors (rank <= 64), as slice
// partials part[s][t][0 .. r) over k slices of nchunk chunks of kDlCols
// columns; grid (ceil(T / 128), S).  A workgroup of 8 waves owns 128 rows
// and one slice, which it streams in 64-column quarters through a ring of
// kDlBufs LDS buffers filled by DMA, kDlAhead quarters ahead of the one
// being multiplied (one barrier a quarter).  A quarter's buffer holds the
// 128 rows of X, the 64 (L1^m)^T rows of up to two non-text modalities
// present in the rows, and the smoothing factors of every modality.  Each
// DMA instruction reads whole 128-byte lines (eight lanes a row, 16 bytes
// each); the rows are stored 128 bytes apart with the 16-byte pieces of
// row i at piece ^ (i % 8), so that the operand reads (8 consecutive rows,
// one piece each, per 128-byte bank cycle) fall on distinct banks.  Wave w
// multiplies its rows 16 w .. + 15 (lane l: row l % 16, columns
// 32 st + 8 (l / 16) .. + 7 of k step st), each step's smoothed values
// entering v_mfma_f32_16x16x32_bf16 as bf16 hi + lo.  L1^m is read from L2
// once per 128 rows, not once per 16.  Rows of a third non-text modality in
// the same 128 rows read their operands from global memory afterwards.
// Tiles without non-text rows return at once: text rows' partials are never
// read (finish_u_row).
constexpr int kDlCols = 256;                        // chunk width of the slice plan
static_assert(kDlCols == kDownLdsCols, "chunk width of the workspace plan");
constexpr int kDlRows = 128;
static_assert(kDlRows == kDownLdsRows, "row tile of the workspace plan");
constexpr int kDlWaves = kDlRows / 16;
constexpr int kDlBufs = 2;                          // LDS ring of 64-column quarters
constexpr int kDlAhead = kDlBufs - 1;               // quarters in flight ahead
constexpr int kDlFragOps = 64 / (8 * kDlWaves);    // DMA instructions per wave for 64 rank rows
static_assert(kDlFragOps * 8 * kDlWaves == 64 && 2 * 8 * kDlWaves == kDlRows,
              "whole DMA instructions of 8 rows per wave");
struct DlQuarter {
    v4i x[kDlRows * 8];                             // the tile's rows x 8 pieces
    v4i f[2][64 * 8];                               // two modalities x 64 rank rows
    v4i s[64];                                      // 4 modalities x 64 factors
};
__device__ __forceinline__ int dl_swz(int row) { return row & 7; }
// s_waitcnt vmcnt(n) for the few counts the ring needs (n wave-uniform)
__device__ __forceinline__ void dl_wait(int n) {
    switch (n) {
        case 0: MASQ_WAIT_VMCNT_LGKM0(0); break;
        case 3: MASQ_WAIT_VMCNT_LGKM0(3); break;
        case 4: MASQ_WAIT_VMCNT_LGKM0(4); break;
        case 5: MASQ_WAIT_VMCNT_LGKM0(5); break;
        case 6: MASQ_WAIT_VMCNT_LGKM0(6); break;
        case 8: MASQ_WAIT_VMCNT_LGKM0(8); break;
        case 9: MASQ_WAIT_VMCNT_LGKM0(9); break;
        case 10: MASQ_WAIT_VMCNT_LGKM0(10); break;
        case 12: MASQ_WAIT_VMCNT_LGKM0(12); break;
        case 15: MASQ_WAIT_VMCNT_LGKM0(15); break;
        default: MASQ_WAIT_VMCNT_LGKM0(0); break;  // (over-waits)
    }
}

__device__ __forceinline__ void down_lds_tile(
    const bf16_t* __restrict__ x, const int32_t* __restrict__ mod, const float* __restrict__ inv_s,
    const bf16_t* __restrict__ l_down, int64_t T, int K, int r, int n_mod, int nchunk,
    float* __restrict__ part, int tile, int s) {
    __shared__ __attribute__((aligned(16))) DlQuarter sb[kDlBufs];          // 132 KB
    __shared__ int smod[kDlRows];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ar = lane & 15, kg = lane >> 4;
    const int64_t row0 = static_cast<int64_t>(tile) * kDlRows;
    const int npairs = K >> 6;                      // 64-column quarters of the row

    if (tid < kDlRows) {
        const int64_t t = row0 + tid;
        smod[tid] = t < T ? sane_mod(mod[t], n_mod) : 0;
    }
    __syncthreads();
    unsigned pres = 0;
    for (int m = 1; m < n_mod; ++m) {
        bool any = false;
        for (int k = lane; k < kDlRows; k += 64) any = any || smod[k] == m;
        if (__ballot(any) != 0ull) pres |= 1u << m;
    }
    const unsigned present = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<int>(pres)));
    if (present == 0) return;                      // uniform over the workgroup
    int mods[3] = {0, 0, 0};
    int np = 0;
    for (int m = 1; m < n_mod; ++m)
        if (present & (1u << m)) mods[np++] = m;
    const int ncb = r >> 4;
    const int nsl = min(np, 2);                     // modalities staged in LDS
    const int64_t trow = row0 + 16 * wave + ar;
    const bool valid = trow < T;
    const int mrow = smod[16 * wave + ar];
    const int qb = s * nchunk * (kDlCols / 64);     // first quarter of the slice
    const int nq = min(nchunk * (kDlCols / 64), npairs - qb);   // its quarters, >= 1
    const int g = 2 + kDlFragOps * nsl + (wave == 0 ? 1 : 0);   // DMA instructions per quarter, this wave

    // quarter h into buffer h % kDlBufs: (wave 0) the factors, lane i those
    // of modality i / 16 (the last one past n_mod), columns 4 (i % 16) ..;
    // rows 8 (2 w + j) .. + 7 of X (rows past T repeat row T - 1, their
    // results unused); rank rows 8 w .. + 7 of each staged modality (rows
    // past r repeat row r - 1)
    auto issue = [&](int h) __attribute__((always_inline)) {
        const int col = 64 * (qb + h);
        const uint32_t base = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(
            static_cast<int>(reinterpret_cast<uintptr_t>(&sb[h % kDlBufs]))));
        if (wave == 0) {
            const int m = min(lane >> 4, n_mod - 1);
            lds_dma16(inv_s + static_cast<int64_t>(m) * K + col + 4 * (lane & 15),
                      base + static_cast<uint32_t>(offsetof(DlQuarter, s)));
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int row = 8 * (2 * wave + j) + (lane >> 3);
            const int64_t t = min(row0 + row, T - 1);
            lds_dma16(x + t * K + col + 8 * ((lane & 7) ^ dl_swz(row)),
                      base + static_cast<uint32_t>(offsetof(DlQuarter, x)) + 1024u * (2 * wave + j));
        }
        for (int j = 0; j < nsl; ++j)
#pragma unroll
            for (int o = 0; o < kDlFragOps; ++o) {
                const int blk = kDlFragOps * wave + o;             // 8 rank rows a block
                const int rr = 8 * blk + (lane >> 3);
                lds_dma16(l_down + (static_cast<int64_t>(mods[j] - 1) * r + min(rr, r - 1)) * K + col +
                              8 * ((lane & 7) ^ dl_swz(rr)),
                          base + static_cast<uint32_t>(offsetof(DlQuarter, f)) + 8192u * j + 1024u * blk);
            }
    };

    const v4i zero = {0, 0, 0, 0};
    v4f acc[4];
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) acc[jb] = v4f{0.f, 0.f, 0.f, 0.f};
    // one k step: the smoothed row piece as bf16 hi + lo against the four
    // N blocks of fragments
    auto step = [&](v4i raw, v4f s0, v4f s1, const v4i (&fb)[4], bool ok) __attribute__((always_inline)) {
        const float sm[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        float xs[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            xs[2 * j] = __uint_as_float(static_cast<uint32_t>(raw[j]) << 16) * sm[2 * j];
            xs[2 * j + 1] = __uint_as_float(static_cast<uint32_t>(raw[j]) & 0xFFFF0000u) * sm[2 * j + 1];
        }
        v4i hi, lo;
        split_bf16x8(xs, hi, lo);
        const v4i hh = ok ? hi : zero, ll = ok ? lo : zero;
#pragma unroll
        for (int jb = 0; jb < 4; ++jb)
            acc[jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(v8bf, hh), __builtin_bit_cast(v8bf, fb[jb]), acc[jb], 0, 0, 0);
#pragma unroll
        for (int jb = 0; jb < 4; ++jb)
            acc[jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(v8bf, ll), __builtin_bit_cast(v8bf, fb[jb]), acc[jb], 0, 0, 0);
    };

    for (int h = 0; h < kDlAhead && h < nq; ++h) issue(h);
    const int xrow = 16 * wave + ar;
    for (int h = 0; h < nq; ++h) {
        // quarter h has landed once at most the younger quarters' DMA is in
        // flight; the barrier also retires every read of the buffer the next
        // issue refills (quarter h - 1's)
        dl_wait(min(nq - 1 - h, kDlAhead - 1) * g);
        __syncthreads();
        if (h + kDlAhead < nq) issue(h + kDlAhead);
        const DlQuarter& q = sb[h % kDlBufs];
        const float* sq = reinterpret_cast<const float*>(q.s);
        for (int mi = 0; mi < nsl; ++mi) {
            const bool mine = valid && mrow == mods[mi];
            if (__ballot(mine) == 0ull) continue;  // uniform over the wave
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                const int pc = 4 * st + kg;
                const float* sp = sq + mrow * 64 + 8 * pc;
                v4i fb[4];
#pragma unroll
                for (int jb = 0; jb < 4; ++jb) {
                    const int rr = 16 * min(jb, ncb - 1) + ar;
                    fb[jb] = q.f[mi][rr * 8 + (pc ^ dl_swz(rr))];
                }
                step(q.x[xrow * 8 + (pc ^ dl_swz(xrow))], *reinterpret_cast<const v4f*>(sp),
                     *reinterpret_cast<const v4f*>(sp + 4), fb, mine);
            }
        }
    }
    if (np == 3) {
        // rows of a third non-text modality in the tile: their quarters in
        // turn, operands straight from global memory
        const int m = mods[2];
        const bool mine = valid && mrow == m;
        if (__ballot(mine) != 0ull) {
            const bf16_t* xr = x + (valid ? trow : row0) * static_cast<int64_t>(K) + 8 * kg;
            const float* srow = inv_s + static_cast<int64_t>(m) * K + 8 * kg;
            for (int h = 0; h < nq; ++h) {
#pragma unroll
                for (int st = 0; st < 2; ++st) {
                    const int c = 64 * (qb + h) + 32 * st;
                    v4i fb[4];
#pragma unroll
                    for (int jb = 0; jb < 4; ++jb)
                        fb[jb] = *reinterpret_cast<const v4i*>(
                            l_down + (static_cast<int64_t>(m - 1) * r + 16 * min(jb, ncb - 1) + ar) * K + c +
                            8 * kg);
                    step(*reinterpret_cast<const v4i*>(xr + c), *reinterpret_cast<const v4f*>(srow + c),
                         *reinterpret_cast<const v4f*>(srow + c + 4), fb, mine);
                }
            }
        }
    }
    // partials of the wave's rows: lane holds rows 4 (l / 16) + i, column
    // 16 jb + l % 16
    float* pp = part + static_cast<int64_t>(s) * T * r;
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
        if (jb >= ncb) break;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t t = row0 + 16 * wave + 4 * kg + i;
            if (t < T) pp[t * r + 16 * jb + ar] = acc[jb][i];
        }
    }
}

__global__ __launch_bounds__(64 * kDlWaves) void k_down_lds(
    const bf16_t* __restrict__ x, const int32_t* __restrict__ mod, const float* __restrict__ inv_s,
    const bf16_t* __restrict__ l_down, int64_t T, int K, int r, int n_mod, int nchunk,
    float* __restrict__ part) {
    down_lds_tile(x, mod, inv_s, l_down, T, K, r, n_mod, nchunk, part, blockIdx.x, blockIdx.y);
}

// ---------------------------------------------------------------- fused stage 1, rows in registers
// Stage 1 for bf16 activations (stage1_fr_ok shapes): a workgroup of
// kFrWaves waves owns 16 RG rows, each wave a slice of the row in 64-column
// pairs.  Every lane issues all of its slice's loads at once (one instruction
// reads 16 rows x 64 bytes) and keeps the raw bf16 values in registers, so
// each row comes from HBM once and the second pass (the codes) reads nothing.
// Lane l covers row l % 16 of each row group and, in pair p, the columns
// 64 p + 16 (l / 16) .. + 15 as two 8-column halves, each one k group of
// v_mfma_f32_16x16x32_bf16; the L1 fragments are read in the same column
// order, so the MFMA's k order is a permutation of the row's (which changes
// only the fp32 rounding order of u).  The fragments come from L2 and are
// shared by the RG row groups; their L2 traffic (|L1^m| per 16 RG rows) is
// what bounds the down-projection.  The waves' u partials are added in LDS in
// a fixed order.
constexpr int kFrLook = 2;          // k steps of L1 fragments in flight ahead of their MFMAs
constexpr int kFrRedPitch = 68;     // floats per row of the u partials in LDS

template <int P, int RG>
__global__ __launch_bounds__(64 * kFrWaves) void k_stage1_fr(
    const bf16_t* __restrict__ x, const int32_t* __restrict__ mod, const float* __restrict__ inv_s,
    const bf16_t* __restrict__ l_down, int64_t T, int K, int r, int n_mod,
    int8_t* __restrict__ q, float* __restrict__ x_scale, float* __restrict__ u,
    uint8_t* __restrict__ u_hl, int* __restrict__ zero_ints, int n_zero, UFinish fin,
    bool pair) {
    constexpr int kRows = 16 * RG;
    if (blockIdx.x == 0)                           // arrival counters of stage 2
        for (int i = threadIdx.x; i < n_zero; i += blockDim.x) zero_ints[i] = 0;

    __shared__ __attribute__((aligned(16))) float s_inv[kFrInvFloats];
    // u partials of the second half of the waves; rows padded to 68 floats so
    // that the four row groups a wave writes at once (rows 4 kg + i) fall on
    // different banks
    __shared__ __attribute__((aligned(16))) float red[kFrWaves / 2][kRows][kFrRedPitch];
    __shared__ int smod[kRows];
    __shared__ float samax[kFrWaves][kRows];
    __shared__ float srq[kRows];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kRows;
    const int ar = lane & 15, kg = lane >> 4;
    const int npairs = K >> 6;
    const int pb = wave * P;                       // this wave's first pair

    // the smoothing factors of every modality into LDS, modality m's row at
    // m * istride floats (1 KB DMA blocks; a row's last block repeats its last
    // piece past the row's end, inside the row's whole blocks; the host checks
    // the fit), then this lane's share of its rows, every load in flight
    const int istride = static_cast<int>(fr_inv_stride(K));
    {
        const int rpieces = K / 4;                             // 16-byte pieces of a row
        const int rblocks = (rpieces + 63) / 64;
        const uint32_t b0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(s_inv));
        for (int i = wave; i < n_mod * rblocks; i += kFrWaves) {
            const int m = i / rblocks, bi = i - m * rblocks;
            lds_dma16(inv_s + static_cast<int64_t>(m) * K + 4 * min(bi * 64 + lane, rpieces - 1),
                      b0 + static_cast<uint32_t>(m * istride * 4 + bi * 1024));
        }
    }
    int mymod = 0;
    if (tid < kRows) {
        const int64_t t = row0 + tid;
        mymod = t < T ? sane_mod(mod[t], n_mod) : 0;
    }
    bool valid[RG];
    const bf16_t* xr[RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        const int64_t t = row0 + 16 * g + ar;
        valid[g] = t < T;
        xr[g] = x + (valid[g] ? t : row0) * static_cast<int64_t>(K) + 16 * kg;
    }
    v4i xa[RG][P], xb[RG][P];
    asm volatile("" ::: "memory");
#pragma unroll
    for (int p = 0; p < P; ++p) {
        const int gp = min(pb + p, npairs - 1);
#pragma unroll
        for (int g = 0; g < RG; ++g) {
            xa[g][p] = *reinterpret_cast<const v4i*>(xr[g] + 64 * gp);
            xb[g][p] = *reinterpret_cast<const v4i*>(xr[g] + 64 * gp + 8);
        }
    }
    asm volatile("" ::: "memory");
    if (tid < kRows) smod[tid] = mymod;
    // the DMA and the id loads are older than this lane's 2 P RG row loads
    MASQ_WAIT_VMCNT_LGKM0(2 * P * RG);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (fin.part != nullptr) {
        // u of the tile's rows from the down-projection's slice partials, while
        // the rows are still arriving (wave w finishes rows w, w + kFrWaves, ..)
        for (int i = wave; i < kRows; i += kFrWaves) {
            const int64_t t = row0 + i;
            if (t < T)
                finish_u_row(t, T, smod[i] == 0, fin.part, fin.slices, fin.r, fin.u, fin.u_hl, lane);
        }
    }

    unsigned pres = 0;
#pragma unroll
    for (int i = 0; i < kRows; ++i)
        if (smod[i] > 0) pres |= 1u << smod[i];
    const unsigned present = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<int>(pres)));
    int mods[3] = {0, 0, 0};
    int np = 0;
    if (r > 0)                                     // rank 0: quantisation only
        for (int m = 1; m < n_mod; ++m)
            if (present & (1u << m)) mods[np++] = m;
    const int ncb = r >> 4;                        // 16-column MFMA blocks (<= 4)
    int mrow[RG];
    const float* srow[RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        mrow[g] = smod[16 * g + ar];
        srow[g] = s_inv + mrow[g] * istride + 16 * kg;
    }

    // xs of half h of pair p of row group g (8 values) from the registers
    // and the factors
    auto smoothed = [&](int g, int p, int h, float (&xs)[8]) __attribute__((always_inline)) {
        const int gp = min(pb + p, npairs - 1);
        const v4i raw = h ? xb[g][p] : xa[g][p];
        const float* sp = srow[g] + 64 * gp + 8 * h;
        const v4f s0 = *reinterpret_cast<const v4f*>(sp);
        const v4f s1 = *reinterpret_cast<const v4f*>(sp + 4);
        const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            xs[2 * j] = __uint_as_float(static_cast<uint32_t>(raw[j]) << 16) * sv[2 * j];
            xs[2 * j + 1] = __uint_as_float(static_cast<uint32_t>(raw[j]) & 0xFFFF0000u) * sv[2 * j + 1];
        }
    };

    // pass 1: the rows' absmax and, for non-text rows, u = xs L1^m
    float amax[RG];
    v4f acc[RG][4];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        amax[g] = 0.f;
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) acc[g][jb] = v4f{0.f, 0.f, 0.f, 0.f};
    }
    const v4i zero = {0, 0, 0, 0};
    if (np == 0) {
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
            for (int g = 0; g < RG; ++g)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    float xs[8];
                    smoothed(g, p, h, xs);
                    if (valid[g] && pb + p < npairs)
#pragma unroll
                        for (int e = 0; e < 8; ++e) amax[g] = fmaxf(amax[g], fabsf(xs[e]));
                }
    } else {
        // L1 fragments of k step s2 = 2 p + h: rows 16 jb + (l % 16) of
        // (L1^m)^T for the four N blocks jb (blocks past r repeat the last
        // one; their sums are never stored), the step's columns of this
        // lane's group
        const int64_t rowK = static_cast<int64_t>(K);
        auto step_off = [&](int s2) __attribute__((always_inline)) {
            return 64 * min(pb + (s2 >> 1), npairs - 1) + 8 * (s2 & 1);
        };
        // one modality's MFMAs over the wave's k steps, its fragments kFrLook
        // steps ahead; rows of other modalities enter as zeros
        auto project = [&](int m, bool first) __attribute__((always_inline)) {
            const bf16_t* fp[4];
#pragma unroll
            for (int jb = 0; jb < 4; ++jb)
                fp[jb] = l_down + (static_cast<int64_t>(m - 1) * r + 16 * min(jb, ncb - 1) + ar) * rowK +
                         16 * kg;
            v4i fb[2 * P][4];
#pragma unroll
            for (int s2 = 0; s2 < kFrLook && s2 < 2 * P; ++s2)
#pragma unroll
                for (int jb = 0; jb < 4; ++jb)
                    fb[s2][jb] = *reinterpret_cast<const v4i*>(fp[jb] + step_off(s2));
#pragma unroll
            for (int s2 = 0; s2 < 2 * P; ++s2) {
                if (s2 + kFrLook < 2 * P) {
#pragma unroll
                    for (int jb = 0; jb < 4; ++jb)
                        fb[s2 + kFrLook][jb] =
                            *reinterpret_cast<const v4i*>(fp[jb] + step_off(s2 + kFrLook));
                }
                const int p = s2 >> 1, h = s2 & 1;
#pragma unroll
                for (int g = 0; g < RG; ++g) {
                    const bool ok = valid[g] && pb + p < npairs;
                    float xs[8];
                    smoothed(g, p, h, xs);
                    if (first && ok)
#pragma unroll
                        for (int e = 0; e < 8; ++e) amax[g] = fmaxf(amax[g], fabsf(xs[e]));
                    v4i hi, lo;
                    split_bf16x8(xs, hi, lo);
                    const bool use = ok && mrow[g] == m;
                    const v4i hh = use ? hi : zero, ll = use ? lo : zero;
#pragma unroll
                    for (int jb = 0; jb < 4; ++jb)
                        acc[g][jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(v8bf, hh), __builtin_bit_cast(v8bf, fb[s2][jb]),
                            acc[g][jb], 0, 0, 0);
#pragma unroll
                    for (int jb = 0; jb < 4; ++jb)
                        acc[g][jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(v8bf, ll), __builtin_bit_cast(v8bf, fb[s2][jb]),
                            acc[g][jb], 0, 0, 0);
                }
            }
        };
        project(mods[0], true);
        // tiles that hold a second or third non-text modality (run borders)
        for (int mi = 1; mi < np; ++mi) project(mods[mi], false);
    }
    // the four lanes of a row (lane % 16) hold its four column groups
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        float a = amax[g];
        a = fmaxf(a, __shfl_xor(a, 16));
        a = fmaxf(a, __shfl_xor(a, 32));
        if (lane < 16) samax[wave][16 * g + lane] = a;
    }
    // u partials: waves kFrWaves / 2 .. hand theirs to the first half,
    // which add them
    constexpr int half = kFrWaves / 2;
    if (np > 0 && wave >= half) {
#pragma unroll
        for (int g = 0; g < RG; ++g)
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) {
                if (jb >= ncb) break;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    red[wave - half][16 * g + 4 * kg + i][16 * jb + ar] = acc[g][jb][i];
            }
    }
    __syncthreads();
    if (tid < kRows) {
        float a = samax[0][tid];
#pragma unroll
        for (int w = 1; w < kFrWaves; ++w) a = fmaxf(a, samax[w][tid]);
        const bool nz = a > 0.f;
        srq[tid] = nz ? 127.0f / a : 0.f;                     // correctly rounded
        if (row0 + tid < T) x_scale[row0 + tid] = nz ? a / 127.0f : 0.f;
    }
    if (np > 0 && wave < half) {
#pragma unroll
        for (int g = 0; g < RG; ++g)
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) {
                if (jb >= ncb) break;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float& slot = red[wave][16 * g + 4 * kg + i][16 * jb + ar];
                    slot = acc[g][jb][i] + slot;
                }
            }
    }
    __syncthreads();
    // u (fp32, written when the tile has non-text rows) and its bf16 hi/lo
    // rows [hi 64 | lo 64] for the GEMM epilogue (text rows and columns past
    // r zero there): thread (row, c) adds columns 8 c .. 8 c + 7 of the
    // partials in a fixed order
    static_assert(kRows * 8 <= 64 * kFrWaves, "one thread per (row, 8 columns)");
    if (tid < kRows * 8 && (np > 0 || u_hl != nullptr)) {
        const int row = tid >> 3, c = tid & 7;
        const int64_t t = row0 + row;
        if (t < T) {
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = 0.f;
            if (np > 0 && 8 * c < r) {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    v4f a = *reinterpret_cast<const v4f*>(&red[0][row][8 * c + 4 * h]);
#pragma unroll
                    for (int w = 1; w < half; ++w)
                        a += *reinterpret_cast<const v4f*>(&red[w][row][8 * c + 4 * h]);
                    v[4 * h] = a.x; v[4 * h + 1] = a.y; v[4 * h + 2] = a.z; v[4 * h + 3] = a.w;
                    *reinterpret_cast<v4f*>(u + t * r + 8 * c + 4 * h) = a;
                }
            }
            if (u_hl != nullptr) {
                v4i hi, lo;
                split_bf16x8(v, hi, lo);
                const bool live = smod[row] > 0;
                *reinterpret_cast<v4i*>(u_hl + t * 256 + 16 * c) = live ? hi : zero;
                *reinterpret_cast<v4i*>(u_hl + t * 256 + 128 + 16 * c) = live ? lo : zero;
            }
        }
    }

    // pass 2: the codes of this lane's 16 columns of each pair, one 16-byte
    // store each, from the registers
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        const float rq = srq[16 * g + ar];
        int8_t* qr = q + code_row(valid[g] ? row0 + 16 * g + ar : row0, K, pair) + 16 * kg;
#pragma unroll
        for (int p = 0; p < P; ++p) {
            uint32_t w[4];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                float xs[8];
                smoothed(g, p, h, xs);
                uint32_t w0 = 0u, w1 = 0u;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    float c = rintf(xs[e] * rq);
                    c = fminf(fmaxf(c, -127.0f), 127.0f);
                    const uint32_t b = (static_cast<uint32_t>(static_cast<int32_t>(c)) & 0xFFu)
                                       << (8 * (e & 3));
                    if (e < 4) w0 |= b; else w1 |= b;
                }
                w[2 * h] = w0;
                w[2 * h + 1] = w1;
            }
            if (valid[g] && pb + p < npairs)
                *reinterpret_cast<v4i*>(qr + code_col(64 * (pb + p), pair)) =
                    v4i{static_cast<int32_t>(w[0]), static_cast<int32_t>(w[1]),
                        static_cast<int32_t>(w[2]), static_cast<int32_t>(w[3])};
        }
    }
}

// ================================================================ standalone CMC
template <typename XT, typename LT, typename YT>
__global__ __launch_bounds__(256) void k_lowrank_comp(const XT* __restrict__ x,
                                                      const int32_t* __restrict__ mod,
                                                      const float* __restrict__ inv_s,
                                                      const LT* __restrict__ l_down,
                                                      const LT* __restrict__ r_up, int64_t T,
                                                      int K, int N, int r, int n_mod,
                                                      YT* __restrict__ y) {
    __shared__ int smod[kRowsDown];
    __shared__ float red[4][kRowsDown][64];
    __shared__ float su[kRowsDown][kMaxRank];
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kRowsDown;
    if (threadIdx.x < kRowsDown) {
        const int64_t t = row0 + threadIdx.x;
        smod[threadIdx.x] = t < T ? sane_mod(mod[t], n_mod) : 0;
    }
    __syncthreads();
    const unsigned present = tile_presence(smod);
    if (!present) return;
    for (int c0 = 0; c0 < r; c0 += 64)
        down_group<4, XT, LT>(x, inv_s, l_down, row0, T, K, r, n_mod, 0, K, c0, smod, present, red,
                              [&](int row, int col, float v) { su[row][col] = v; });
    for (int o = threadIdx.x; o < N; o += 256) {
        for (int i = 0; i < kRowsDown; ++i) {
            const int m = smod[i];
            const int64_t t = row0 + i;
            if (t >= T || m == 0) continue;
            const LT* rr = r_up + (static_cast<int64_t>(m - 1) * N + o) * r;
            float c = 0.f;
            for (int k = 0; k < r; ++k) c = fmaf(su[i][k], Elem<LT>::load1(rr + k), c);
            YT* yp = y + t * N + o;
            Elem<YT>::store1(yp, Elem<YT>::load1(yp) + c);
        }
    }
}

// ================================================================ int8 GEMM
// Output coordinates of accumulator element e of a 32 x 32 MFMA block.
__device__ __forceinline__ int acc_row(int e, int lane) {
    return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
}

// Cross-Modal Compensation inside the GEMM epilogue.  Per chunk of up to 64
// rank columns, the tile's u rows (each row's own modality; text rows zero)
// and, for every modality m present, the matching rows of (L2^m)^T are staged
// in LDS.  Each 32 x 32 output block then accumulates u L2^m onto its
// dequantised fp32 values with MFMA, the A operand masked to the rows of
// modality m.  With bf16 factors u enters as a hi + lo pair of bf16 terms
// (about 16 significant bits).  Tiles whose pieces do not fit in the 128 KB of
// LDS read u and L2^T straight from global memory instead.
template <typename LT> struct Cmc;

template <> struct Cmc<bf16_t> {          // bf16 operands, v_mfma_f32_32x32x16_bf16
    static constexpr int kUBytes = 2 * kTileM * 128;   // u hi + u lo, 128-byte rows
    static constexpr int kRBytes = kTileM * 128;       // one modality's L2^T rows

    // All of a thread's global loads are issued before any is consumed (from
    // clamped, always valid addresses; unused values are replaced by zeros),
    // so the staging pays the memory latency once rather than per row.
    template <int NT>
    static __device__ __forceinline__ void stage_u(uint8_t* su, const int* s_mod, const float* u,
                                                   int64_t row0, int64_t T, int r, int c0,
                                                   int tid) {
        constexpr int kIt = 8 * 256 / NT, kRowStep = NT / 8;
        const int nch = min(64, r - c0) >> 3;
        const int ch = tid & 7;
        const int chc = min(ch, nch - 1);
        v4f va[kIt], vb[kIt];
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int row = (tid >> 3) + kRowStep * it;
            const int64_t t = min(row0 + row, T - 1);
            const float* src = u + t * r + c0 + 8 * chc;
            va[it] = *reinterpret_cast<const v4f*>(src);
            vb[it] = *reinterpret_cast<const v4f*>(src + 4);
        }
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int row = (tid >> 3) + kRowStep * it;
            const bool live = ch < nch && (row0 + row) < T && s_mod[row] > 0;
            const float uv[8] = {va[it].x, va[it].y, va[it].z, va[it].w,
                                 vb[it].x, vb[it].y, vb[it].z, vb[it].w};
            v4i hi, lo;
            split_bf16x8(uv, hi, lo);
            const v4i zero = {0, 0, 0, 0};
            const int off = row * 128 + ((ch ^ swz(row)) << 4);
            *reinterpret_cast<v4i*>(su + off) = live ? hi : zero;
            *reinterpret_cast<v4i*>(su + kTileM * 128 + off) = live ? lo : zero;
        }
    }

    template <int NT>
    static __device__ __forceinline__ void stage_r(uint8_t* sr, const bf16_t* rm, int col0, int N,
                                                   int r, int c0, int tid) {
        constexpr int kIt = 8 * 256 / NT, kRowStep = NT / 8;
        const int nch = min(64, r - c0) >> 3;
        const int ch = tid & 7;
        const int chc = min(ch, nch - 1);
        v4i pr[kIt];
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int col = min(col0 + (tid >> 3) + kRowStep * it, N - 1);
            pr[it] = *reinterpret_cast<const v4i*>(rm + static_cast<int64_t>(col) * r + c0 + 8 * chc);
        }
        const v4i zero = {0, 0, 0, 0};
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int row = (tid >> 3) + kRowStep * it;
            *reinterpret_cast<v4i*>(sr + row * 128 + ((ch ^ swz(row)) << 4)) = ch < nch ? pr[it] : zero;
        }
    }

    // yb += [rows of modality m] u . L2^T over this chunk's rc columns.
    static __device__ __forceinline__ v16f from_lds(const uint8_t* su, const uint8_t* sr, int rc,
                                                    int arow, int brow, bool live, int lane,
                                                    v16f yb) {
        const v4i zero = {0, 0, 0, 0};
        for (int ks = 0; ks < (rc >> 4); ++ks) {
            const int c = 2 * ks + (lane >> 5);
            const int offa = arow * 128 + ((c ^ swz(arow)) << 4);
            v4i hi = *reinterpret_cast<const v4i*>(su + offa);
            v4i lo = *reinterpret_cast<const v4i*>(su + kTileM * 128 + offa);
            hi = live ? hi : zero;
            lo = live ? lo : zero;
            const v8bf b = __builtin_bit_cast(
                v8bf, *reinterpret_cast<const v4i*>(sr + brow * 128 + ((c ^ swz(brow)) << 4)));
            yb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, __builtin_bit_cast(v8bf, hi), yb, 0, 0, 0);
            yb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, __builtin_bit_cast(v8bf, lo), yb, 0, 0, 0);
        }
        return yb;
    }

    static __device__ __forceinline__ v16f from_global(const float* u, const bf16_t* rm, bool live,
                                                       int64_t t, int col, int r, int c0,
                                                       int lane, v16f yb) {
        const int rc = min(64, r - c0);
        for (int ks = 0; ks < (rc >> 4); ++ks) {
            const int k = c0 + 16 * ks + 8 * (lane >> 5);
            v4i hi = {0, 0, 0, 0}, lo = {0, 0, 0, 0};
            if (live) {
                float uv[8];
                load8_f32(u + t * r + k, uv);
                split_bf16x8(uv, hi, lo);
            }
            const v8bf b = __builtin_bit_cast(
                v8bf, *reinterpret_cast<const v4i*>(rm + static_cast<int64_t>(col) * r + k));
            yb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, __builtin_bit_cast(v8bf, hi), yb, 0, 0, 0);
            yb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, __builtin_bit_cast(v8bf, lo), yb, 0, 0, 0);
        }
        return yb;
    }
};

template <> struct Cmc<float> {           // fp32 operands, v_mfma_f32_32x32x2f32
    static constexpr int kUBytes = kTileM * 256;       // 64 floats per row
    static constexpr int kRBytes = kTileN * 256;

    // 16-byte pieces, 8 per thread in flight: slot idx -> row idx / 16,
    // piece idx % 16 (pieces past the chunk's rc / 4 are skipped)
    template <int NT>
    static __device__ __forceinline__ void stage_u(uint8_t* base, const int* s_mod, const float* u,
                                                   int64_t row0, int64_t T, int r, int c0,
                                                   int tid) {
        float* su = reinterpret_cast<float*>(base);
        const int nq = min(64, r - c0) >> 2;
        for (int b = 0; b < kTileM * 16; b += NT * 8) {
            v4f v[8];
#pragma unroll
            for (int it = 0; it < 8; ++it) {
                const int idx = b + tid + NT * it, row = idx >> 4, pc = min(idx & 15, nq - 1);
                const int64_t t = min(row0 + row, T - 1);
                v[it] = *reinterpret_cast<const v4f*>(u + t * r + c0 + 4 * pc);
            }
#pragma unroll
            for (int it = 0; it < 8; ++it) {
                const int idx = b + tid + NT * it, row = idx >> 4, pc = idx & 15;
                if (pc >= nq) continue;
                const bool live = row0 + row < T && s_mod[row] > 0;
                *reinterpret_cast<v4f*>(su + row * 64 + 4 * pc) = live ? v[it] : v4f{0.f, 0.f, 0.f, 0.f};
            }
        }
    }

    template <int NT>
    static __device__ __forceinline__ void stage_r(uint8_t* base, const float* rm, int col0, int N,
                                                   int r, int c0, int tid) {
        float* sr = reinterpret_cast<float*>(base);
        const int nq = min(64, r - c0) >> 2;
        for (int b = 0; b < kTileN * 16; b += NT * 8) {
            v4f v[8];
#pragma unroll
            for (int it = 0; it < 8; ++it) {
                const int idx = b + tid + NT * it, row = idx >> 4, pc = min(idx & 15, nq - 1);
                const int col = min(col0 + row, N - 1);
                v[it] = *reinterpret_cast<const v4f*>(rm + static_cast<int64_t>(col) * r + c0 + 4 * pc);
            }
#pragma unroll
            for (int it = 0; it < 8; ++it) {
                const int idx = b + tid + NT * it, row = idx >> 4, pc = idx & 15;
                if (pc < nq) *reinterpret_cast<v4f*>(sr + row * 64 + 4 * pc) = v[it];
            }
        }
    }

    static __device__ __forceinline__ v16f from_lds(const uint8_t* su_, const uint8_t* sr_, int rc,
                                                    int arow, int brow, bool live, int lane,
                                                    v16f yb) {
        const float* su = reinterpret_cast<const float*>(su_);
        const float* sr = reinterpret_cast<const float*>(sr_);
        for (int ks = 0; ks < (rc >> 1); ++ks) {
            const int k = 2 * ks + (lane >> 5);
            const float a = live ? su[arow * 64 + k] : 0.f;
            yb = __builtin_amdgcn_mfma_f32_32x32x2f32(sr[brow * 64 + k], a, yb, 0, 0, 0);
        }
        return yb;
    }

    // the same for NJ channel blocks at once (rows brow[j] of the staged L2),
    // reads of 8 k steps batched ahead of their MFMAs and the NJ independent
    // accumulation chains interleaved
    template <int NJ>
    static __device__ __forceinline__ void from_lds_multi(const uint8_t* base_u, const uint8_t* base_r,
                                                          int rc, int arow, const int (&brow)[NJ],
                                                          bool live, int lane, v16f (&yb)[NJ]) {
        const float* su = reinterpret_cast<const float*>(base_u);
        const float* sr = reinterpret_cast<const float*>(base_r);
        for (int k0 = 0; k0 < rc; k0 += 16) {                 // rc % 16 == 0
            float av[8], bv[NJ][8];
#pragma unroll
            for (int st = 0; st < 8; ++st) {
                const int k = k0 + 2 * st + (lane >> 5);
                av[st] = live ? su[arow * 64 + k] : 0.f;
#pragma unroll
                for (int j = 0; j < NJ; ++j) bv[j][st] = sr[brow[j] * 64 + k];
            }
#pragma unroll
            for (int st = 0; st < 8; ++st)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    yb[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(bv[j][st], av[st], yb[j], 0, 0, 0);
        }
    }

    static __device__ __forceinline__ v16f from_global(const float* u, const float* rm, bool live,
                                                       int64_t t, int col, int r, int c0,
                                                       int lane, v16f yb) {
        const int rc = min(64, r - c0);
        for (int ks = 0; ks < (rc >> 1); ++ks) {
            const int k = c0 + 2 * ks + (lane >> 5);
            const float a = live ? u[t * r + k] : 0.f;
            yb = __builtin_amdgcn_mfma_f32_32x32x2f32(rm[static_cast<int64_t>(col) * r + k], a, yb, 0, 0, 0);
        }
        return yb;
    }
};

// Workgroups are dealt round-robin to the 8 XCDs; give each XCD a contiguous
// range of tiles, ordered in groups of 8 tile-rows, so that tiles running
// together on one XCD share A and B stages in its L2.  Returns false for the
// padding workgroups of the last XCD range.
__device__ __forceinline__ bool tile_coords_at(int b, int tiles_m, int tiles_n, int& tm, int& tn) {
    const int nt = tiles_m * tiles_n;
    const int per_xcd = (nt + 7) >> 3;
    if ((b >> 3) >= per_xcd) return false;
    const int L = (b & 7) * per_xcd + (b >> 3);
    if (L >= nt) return false;
    constexpr int GM = 8;
    const int gsize = GM * tiles_n;
    const int g = L / gsize;
    const int first_m = g * GM;
    const int gm = min(GM, tiles_m - first_m);
    const int li = L - g * gsize;
    tm = first_m + li % gm;
    tn = li / gm;
    return true;
}
__device__ __forceinline__ bool tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
    return tile_coords_at(static_cast<int>(blockIdx.x), tiles_m, tiles_n, tm, tn);
}

// Shared LDS of both GEMM kernels: the K stages during the main loop, then
// the compensation pieces in the epilogue.
// Per-wave output transpose buffer: 32 rows of TW bf16 channels (TW = 64
// with 4 waves, 32 with 8), rows padded by 16 bytes (16-byte aligned rows
// for the reads; the column writes, one row per lane, hit distinct banks).
constexpr int tr_pitch(int tw) { return 2 * tw + 16; }
constexpr int kTrBytes = 20480;       // max(4 x 32 x pitch(64), 8 x 32 x pitch(32))

// Per-row and per-channel epilogue operands of a tile.
struct RowOps {
    float dx[kTileM];
    float ws[kTileN];
    int mod[kTileM];          // modality of each row (invalid ids read as text)
    int rawmod[kTileM];       // modality ids as given (LDS-DMA target)
};
struct GemmSmem {
    uint8_t buf[2 * 65536];
    RowOps ro[2];             // the tile's set and (persistent grid) the next tile's
    unsigned wpresent[8];     // per wave: bit m set if a row of modality m is in its rows
    uint8_t tr[kTrBytes];     // 16-byte aligned (the transposes use 16-byte LDS accesses)
    int last;                 // split K: this workgroup is the last slice of its tile to arrive
};
static_assert(offsetof(GemmSmem, tr) % 16 == 0, "tr alignment");
static_assert(4 * 32 * tr_pitch(64) <= kTrBytes && 8 * 32 * tr_pitch(32) <= kTrBytes, "tr");

// Epilogue of a 256 x 256 tile whose int32 accumulators are in acc (this
// wave's 128 x 128 quarter as 4 x 4 blocks of 32 x 32): optional int32 store,
// dequantisation, Cross-Modal Compensation on non-text rows, cast and store.
// Per-thread epilogue operands (thread t: token row0 + t, channel col0 + t),
// loaded at the start of the kernel so that their latency hides behind the
// main loop.
struct EpiPrefetch {
    float dx, ws;
    int mod;
};

__device__ __forceinline__ EpiPrefetch epi_prefetch(const float* __restrict__ x_scale,
                                                    const float* __restrict__ w_scale,
                                                    const int32_t* __restrict__ mod, bool cmc,
                                                    int64_t T, int N, int64_t row0, int col0,
                                                    int n_mod) {
    const int tid = threadIdx.x;
    const int64_t t = row0 + tid;
    EpiPrefetch e;
    e.dx = t < T ? x_scale[t] : 0.f;
    e.ws = (col0 + tid) < N ? w_scale[col0 + tid] : 0.f;
    e.mod = (cmc && t < T) ? sane_mod(mod[t], n_mod) : 0;
    return e;
}

// State handed over by the DMA kernel: the per-row operands are in LDS
// already, the modalities present are known, and with pre the fast-path
// compensation operands sit at the given byte offsets of the K buffers.
struct EpiDma {
    unsigned present;
    bool pre;
    int off_uh, off_ul, off_r[2];
    int grp_rows;      // grouped tile (GRP): its valid rows; the rawmod operands hold their token indices
};

// NWN waves along the channels (2: four waves of 128 x 128, 4: eight waves of
// 128 x 64); NJ = 8 / NWN channel blocks of 32 per wave.  DMA: called from
// the DMA kernel (state in ed; pf unused), else the per-thread operands pf
// are written to LDS here.
template <typename YT, typename LT, bool CMC, bool ACC, int NWN = 2, bool DMA = false,
          bool GRP = false>
__device__ __forceinline__ void gemm_epilogue(
    v16i (&acc)[4][8 / NWN], GemmSmem& sm, const EpiPrefetch& pf, int64_t T, int N, int64_t row0,
    int col0, const float* __restrict__ u, int r, int n_mod, const LT* __restrict__ r_up,
    int32_t* __restrict__ acc_out, YT* __restrict__ y, const EpiDma& ed = EpiDma{}, int rb = 0,
    int tid_in = -1) {
    constexpr int NJ = 8 / NWN, NW = 2 * NWN, NT = 64 * NW;
    constexpr int kWaveCols = 32 * NJ;                 // channels per wave
    constexpr int TW = NJ == 4 ? 64 : 32;              // transpose unit width (channels)
    constexpr int kPitch = tr_pitch(TW);
    const int tid = tid_in >= 0 ? tid_in : static_cast<int>(threadIdx.x);
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / NWN, wn = wave % NWN;
    RowOps& ro = sm.ro[rb];
    // dx, ws, mod and wpresent lie outside the K-stage buffers, so they can be
    // written before the barrier; after it every wave is also done with the
    // K stages
    if constexpr (!DMA) {
        if (tid < kTileM) {                    // threads past 256 carry no prefetch
            ro.dx[tid] = pf.dx;
            ro.ws[tid] = pf.ws;
        }
        if constexpr (CMC) {
            if (tid < kTileM) ro.mod[tid] = pf.mod;
            unsigned wp = 0;
            for (int m = 1; m < n_mod; ++m)
                if (__ballot(tid < kTileM && pf.mod == m) != 0ull) wp |= 1u << m;
            if (lane == 0) sm.wpresent[wave] = wp;
        }
    }
    __syncthreads();

    // ---- compensation: modalities present in the tile, LDS plan per 64-column chunk.
    // Every quantity that selects a code path is wave-uniform (scalar registers).
    int n_present = 0;
    bool staged = false;
    unsigned present = 0;
    const int n_chunks = (r + 63) >> 6;
    constexpr int kChunkBase = CMC ? Cmc<LT>::kUBytes : 0;
    // LDS byte offsets of the fast path's u hi, u lo and L2 pieces
    int off_uh = 0, off_ul = kTileM * 128, off_r0 = kChunkBase, off_r1 = kChunkBase + (CMC ? Cmc<LT>::kRBytes : 0);
    if constexpr (CMC) {
        if constexpr (DMA) {
            present = ed.present;
        } else {
            unsigned pa = 0;
#pragma unroll
            for (int w = 0; w < NW; ++w) pa |= sm.wpresent[w];
            present = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<int>(pa)));
        }
        n_present = __builtin_popcount(present);
        const int chunk_bytes = Cmc<LT>::kUBytes + n_present * Cmc<LT>::kRBytes;
        staged = n_chunks * chunk_bytes <= static_cast<int>(sizeof(sm.buf));
        if (DMA && ed.pre) {
            staged = true;
            off_uh = ed.off_uh;
            off_ul = ed.off_ul;
            off_r0 = ed.off_r[0];
            off_r1 = ed.off_r[1];
        } else if (n_present > 0 && staged && y != nullptr) {
            for (int c = 0; c < n_chunks; ++c) {
                uint8_t* base = sm.buf + c * chunk_bytes;
                Cmc<LT>::template stage_u<NT>(base, ro.mod, u, row0, T, r, 64 * c, tid);
                int p = 0;
                for (int m = 1; m < n_mod; ++m) {
                    if (!(present & (1u << m))) continue;
                    Cmc<LT>::template stage_r<NT>(base + kChunkBase + p * Cmc<LT>::kRBytes,
                                     r_up + static_cast<int64_t>(m - 1) * N * r, col0, N, r,
                                     64 * c, tid);
                    ++p;
                }
            }
            __syncthreads();
        }
    }

    // ---- accumulator layout: register e of a lane in block (i, j) holds token
    // wm*128 + 32 i + (lane % 32) and channel wn*kWaveCols + 32 j + 8 (e / 4) +
    // 4 (lane / 32) + e % 4.  Loops over blocks are fully unrolled: the
    // accumulators are registers and must be indexed by constants.
    static_assert(!GRP || (DMA && !CMC && !ACC), "grouped tiles: plain product, DMA kernel");
    // GRP: local row l of the tile is token ro.rawmod[l], valid for l < ed.grp_rows
    const bool interior = GRP ? (ed.grp_rows == kTileM && col0 + kTileN <= N)
                              : (row0 + kTileM <= T) && (col0 + kTileN <= N);
    auto row_ok = [&](int local) __attribute__((always_inline)) {
        return GRP ? local < ed.grp_rows : row0 + local < T;
    };
    auto out_row = [&](int local) __attribute__((always_inline)) -> int64_t {
        return GRP ? static_cast<int64_t>(ro.rawmod[local]) : row0 + local;
    };
    auto tok_of = [&](int i) { return wm * 128 + i * 32 + (lane & 31); };
    auto ch_of = [&](int j, int g) { return wn * kWaveCols + j * 32 + 8 * g + 4 * (lane >> 5); };

    if constexpr (ACC) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t tok = row0 + tok_of(i);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int ch = col0 + ch_of(j, g);
                    if (interior || (tok < T && ch < N)) {
                        const v4i w = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                       acc[i][j][4 * g + 3]};
                        *reinterpret_cast<v4i*>(acc_out + tok * N + ch) = w;
                    }
                }
        }
    }
    if (y == nullptr) return;

    // ---- per 32 x 32 block: dequantise, compensate, cast and store.  The
    // tile takes one of three wave-uniform paths: no compensation (text-only
    // tiles), the fast compensation (bf16 factors, rank <= 64, at most two
    // non-text modalities present, all staged), or the general one.
    // dequantisation of block (i, j) with the channel scales ws[g] of its
    // four 4-channel groups
    auto dequant_with = [&](const int i, const int j, const v4f (&ws)[4]) __attribute__((always_inline)) {
        const float dx = ro.dx[tok_of(i)];
        const v16i a = acc[i][j];
        v16f yb;
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                yb[4 * g + e] = (static_cast<float>(a[4 * g + e]) * dx) * ws[g][e];
        return yb;
    };
    auto load_ws = [&](const int j, v4f (&ws)[4]) __attribute__((always_inline)) {
#pragma unroll
        for (int g = 0; g < 4; ++g) ws[g] = *reinterpret_cast<const v4f*>(&ro.ws[ch_of(j, g)]);
    };
    auto dequant = [&](const int i, const int j) __attribute__((always_inline)) {
        v4f ws[4];
        load_ws(j, ws);
        return dequant_with(i, j, ws);
    };
    // Stores of one token block (32 rows x kWaveCols channels of this wave).
    // bf16 output goes through a small per-wave LDS transpose, TW channels
    // at a time, so that every store instruction writes whole row pieces of
    // 2 TW bytes (the MFMA layout would give 32 rows x 16 bytes per
    // instruction); LDS operations of one wave execute in order, so the
    // buffer needs no further synchronisation.
    auto store_rowblock = [&](const int i, const v16f (&ybs)[NJ]) __attribute__((always_inline)) {
        const int loc0 = wm * 128 + i * 32;
        if constexpr (sizeof(YT) == 2) {
            uint8_t* scr = sm.tr + wave * 32 * kPitch;
            const int rw = lane & 31, h = lane >> 5;
            constexpr int kJper = TW / 32;                 // channel blocks per unit
            constexpr int kLanesPerRow = TW / 8;           // 16-byte pieces per row
            constexpr int kRowsPerRead = 64 / kLanesPerRow;
#pragma unroll
            for (int jp = 0; jp < NJ / kJper; ++jp) {
#pragma unroll
                for (int jj = 0; jj < kJper; ++jj)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const v16f& yb = ybs[kJper * jp + jj];
                        v2i w;
                        w.x = static_cast<int32_t>(pack_bf16x2(yb[4 * g], yb[4 * g + 1]));
                        w.y = static_cast<int32_t>(pack_bf16x2(yb[4 * g + 2], yb[4 * g + 3]));
                        *reinterpret_cast<v2i*>(scr + rw * kPitch + (jj * 32 + 8 * g + 4 * h) * 2) = w;
                    }
                const int ch = col0 + wn * kWaveCols + jp * TW + (lane % kLanesPerRow) * 8;
#pragma unroll
                for (int k = 0; k < 32 / kRowsPerRead; ++k) {
                    const int rr = k * kRowsPerRead + lane / kLanesPerRow;
                    const v4i d = *reinterpret_cast<const v4i*>(scr + rr * kPitch + (lane % kLanesPerRow) * 16);
                    if (interior || (row_ok(loc0 + rr) && ch < N))
                        *reinterpret_cast<v4i*>(y + out_row(loc0 + rr) * N + ch) = d;
                }
            }
        } else {
            const int loc = loc0 + (lane & 31);
            const bool ok = row_ok(loc);
            const int64_t tok = out_row(loc);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int ch = col0 + ch_of(j, g);
                    if (interior || (ok && ch < N)) {
                        const v4f w = {ybs[j][4 * g], ybs[j][4 * g + 1], ybs[j][4 * g + 2], ybs[j][4 * g + 3]};
                        *reinterpret_cast<v4f*>(y + tok * N + ch) = w;
                    }
                }
        }
    };

    if (!CMC || n_present == 0) {
        v4f wsv[NJ][4];                      // the wave's channel scales, read once
#pragma unroll
        for (int j = 0; j < NJ; ++j) load_ws(j, wsv[j]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v16f ybs[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j) ybs[j] = dequant_with(i, j, wsv[j]);
            store_rowblock(i, ybs);
        }
        return;
    }

    if constexpr (CMC && sizeof(LT) == 2) {
        if (n_present <= 2 && staged && n_chunks == 1) {
            // Fast path: the present modalities lie side by side along the
            // rank dimension (slot p holds modality mods[p], r / 16 k steps
            // of 16 each).  Per token block, the compensation of its four
            // channel blocks runs as four independent MFMA chains that
            // accumulate onto the dequantised values.
            int mods[2] = {0, 0};
            {
                int p = 0;
                for (int m = 1; m < n_mod && p < 2; ++m)
                    if (present & (1u << m)) mods[p++] = m;
            }
            const int nks = r >> 4;
            const v4i zero4 = {0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int trow = tok_of(i);
                const int tm_ = ro.mod[trow];
                v16f ybs[NJ];
#pragma unroll
                for (int j = 0; j < NJ; ++j) ybs[j] = dequant(i, j);
#pragma unroll
                for (int kk = 0; kk < 8; ++kk) {
                    const int p = kk >> 2, ks = kk & 3;
                    if (p >= n_present || ks >= nks) continue;
                    const int cc = 2 * ks + (lane >> 5);
                    const int off = trow * 128 + ((cc ^ swz(trow)) << 4);
                    // text rows are zero in the staged u; a second modality
                    // present needs each slot masked to its own rows
                    v4i h = *reinterpret_cast<const v4i*>(sm.buf + off_uh + off);
                    v4i l = *reinterpret_cast<const v4i*>(sm.buf + off_ul + off);
                    if (n_present > 1) {
                        const bool live = tm_ == mods[p];
                        h = live ? h : zero4;
                        l = live ? l : zero4;
                    }
                    const uint8_t* sr = sm.buf + (p == 0 ? off_r0 : off_r1);
#pragma unroll
                    for (int j = 0; j < NJ; ++j) {
                        const int crow = wn * kWaveCols + j * 32 + (lane & 31);
                        const v8bf bj = __builtin_bit_cast(
                            v8bf, *reinterpret_cast<const v4i*>(sr + crow * 128 + ((cc ^ swz(crow)) << 4)));
                        ybs[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bj, __builtin_bit_cast(v8bf, h), ybs[j], 0, 0, 0);
                        ybs[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bj, __builtin_bit_cast(v8bf, l), ybs[j], 0, 0, 0);
                    }
                }
                store_rowblock(i, ybs);
            }
            return;
        }
    }

    // fp32 factors, all pieces staged: the channel blocks of a token block
    // advance together (independent MFMA chains, batched LDS reads)
    if constexpr (CMC && sizeof(LT) == 4) {
        if (staged) {
            const int chunk_bytes = Cmc<LT>::kUBytes + n_present * Cmc<LT>::kRBytes;
            int brow[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j) brow[j] = wn * kWaveCols + j * 32 + (lane & 31);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int trow = tok_of(i);
                const int tm_ = ro.mod[trow];
                v16f ybs[NJ];
#pragma unroll
                for (int j = 0; j < NJ; ++j) ybs[j] = dequant(i, j);
                for (int c = 0; c < n_chunks; ++c) {
                    int p = 0;
                    for (int m = 1; m < n_mod; ++m) {
                        if (!(present & (1u << m))) continue;
                        const uint8_t* base = sm.buf + c * chunk_bytes;
                        Cmc<LT>::template from_lds_multi<NJ>(base, base + kChunkBase + p * Cmc<LT>::kRBytes,
                                                             min(64, r - 64 * c), trow, brow,
                                                             tm_ == m, lane, ybs);
                        ++p;
                    }
                }
                store_rowblock(i, ybs);
            }
            return;
        }
    }

    // General compensation of one block: any rank, any number of modalities,
    // staged pieces or global memory.
    if constexpr (CMC) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int trow = tok_of(i);
            const int tm_ = ro.mod[trow];
            v16f ybs[NJ];
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                v16f& yb = ybs[j];
                yb = dequant(i, j);
                const int crow = wn * kWaveCols + j * 32 + (lane & 31);
                const int chunk_bytes = Cmc<LT>::kUBytes + n_present * Cmc<LT>::kRBytes;
                for (int c = 0; c < n_chunks; ++c) {
                    int p = 0;
                    for (int m = 1; m < n_mod; ++m) {
                        if (!(present & (1u << m))) continue;
                        const bool live = tm_ == m;
                        if (staged) {
                            const uint8_t* base = sm.buf + c * chunk_bytes;
                            yb = Cmc<LT>::from_lds(base, base + kChunkBase + p * Cmc<LT>::kRBytes,
                                                   min(64, r - 64 * c), trow, crow, live, lane, yb);
                        } else {
                            yb = Cmc<LT>::from_global(u, r_up + static_cast<int64_t>(m - 1) * N * r,
                                                      live && (row0 + trow) < T, row0 + trow,
                                                      min(col0 + crow, N - 1), r, 64 * c, lane, yb);
                        }
                        ++p;
                    }
                }
            }
            store_rowblock(i, ybs);
        }
    }
}

// 16 x 32 x 32 MFMA steps of one wave's 128 x 128 quarter: fragments of the
// 4 token blocks (q rows) and 4 channel blocks (Wq rows) for k chunk c (lane
// group l / 32 selects the chunk), read through the row swizzle `sw`.  The
// product is formed transposed, channels x tokens, so that each lane ends up
// holding one token and 4 consecutive output channels per register group.
template <int kRowBytes, typename Swz>
__device__ __forceinline__ void mfma_kstep(const uint8_t* sa, const uint8_t* sb, int c, int wm,
                                           int wn, int lane, Swz sw, v16i (&acc)[4][4]) {
    v4i fa[4], fb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = wm * 128 + i * 32 + (lane & 31);
        fa[i] = *reinterpret_cast<const v4i*>(sa + row * kRowBytes + ((c ^ sw(row)) << 4));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int row = wn * 128 + j * 32 + (lane & 31);
        fb[j] = *reinterpret_cast<const v4i*>(sb + row * kRowBytes + ((c ^ sw(row)) << 4));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fb[j], fa[i], acc[i][j], 0, 0, 0);
}

// ---------------------------------------------------------------- GEMM, general K
// K stages of 128 bytes go global -> registers -> LDS, double-buffered; any
// c_in that is a multiple of 16 (chunks past K are zero-filled).
template <typename YT, typename LT, bool CMC, bool ACC>
__global__ __launch_bounds__(256, 1) void k_gemm(
    const int8_t* __restrict__ A, const int8_t* __restrict__ B, const float* __restrict__ x_scale,
    const float* __restrict__ w_scale, int64_t T, int K, int N, int tiles_m, int tiles_n,
    const int32_t* __restrict__ mod, const float* __restrict__ u, int r, int n_mod,
    const LT* __restrict__ r_up, int32_t* __restrict__ acc_out, YT* __restrict__ y) {
    __shared__ __attribute__((aligned(16))) GemmSmem sm;
    int tm, tn;
    if (!tile_coords(tiles_m, tiles_n, tm, tn)) return;
    const int64_t row0 = static_cast<int64_t>(tm) * kTileM;
    const int col0 = tn * kTileN;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lc = tid & 7;      // 16-byte chunk of a 128-byte stage row
    const int lr = tid >> 3;     // first row this thread loads (+32 j)

    v16i acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = v16i{0};

    const EpiPrefetch pf = epi_prefetch(x_scale, w_scale, mod, CMC, T, N, row0, col0, n_mod);
    v4i ra[8], rb[8];
    // Row indices are clamped into the matrix (rows past T or N are computed
    // and discarded); chunks past K are loaded from a clamped in-bounds
    // address and replaced by zeros at the LDS store.
    int64_t a_off[8], b_off[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        a_off[j] = min(row0 + lr + 32 * j, T - 1) * K;
        b_off[j] = static_cast<int64_t>(min(col0 + lr + 32 * j, N - 1)) * K;
    }
    bool kin = true;          // this thread's chunk of the stage lies inside K
    auto gload = [&](int k0) {
        const int kraw = k0 + lc * 16;
        kin = kraw < K;
        const int kk = kin ? kraw : K - 16;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            ra[j] = *reinterpret_cast<const v4i*>(A + a_off[j] + kk);
            rb[j] = *reinterpret_cast<const v4i*>(B + b_off[j] + kk);
        }
    };
    auto sstore = [&](int buf) {
        uint8_t* sa = sm.buf + buf * 65536;
        uint8_t* sb = sa + 32768;
        const v4i zero = {0, 0, 0, 0};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int row = lr + 32 * j;
            const int off = row * 128 + ((lc ^ swz(row)) << 4);
            *reinterpret_cast<v4i*>(sa + off) = kin ? ra[j] : zero;
            *reinterpret_cast<v4i*>(sb + off) = kin ? rb[j] : zero;
        }
    };
    auto sw8 = [](int row) { return swz(row); };

    const int nk = (K + kTileK - 1) / kTileK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * kTileK);
        const uint8_t* sa = sm.buf + cur * 65536;
        const uint8_t* sb = sa + 32768;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            mfma_kstep<128>(sa, sb, 2 * ks + (lane >> 5), wm, wn, lane, sw8, acc);
        if (kt + 1 < nk) sstore(cur ^ 1);
        __syncthreads();
    }
    gemm_epilogue<YT, LT, CMC, ACC>(acc, sm, pf, T, N, row0, col0, u, r, n_mod, r_up, acc_out, y);
}

// ---------------------------------------------------------------- GEMM, K % 64 == 0
// Direct-to-LDS pipeline: 64-byte K stages (A and B tiles 256 x 64 each) go
// from global memory straight into one of 4 LDS buffers with
// global_load_lds_dwordx4, three stages ahead of the MFMAs.  Each wave waits
// for its own loads of a stage (s_waitcnt vmcnt) before the barrier that
// publishes the stage to the other waves.
constexpr int kDmaStageK = 64;
constexpr int kDmaStages = 4;
constexpr int kDmaStageBytes = 2 * kTileM * kDmaStageK;     // A + B

// 4-chunk swizzle of a 64-byte row.  Measured on gfx950 with a ds_read_b128
// microbenchmark (SQ_LDS_BANK_CONFLICT = 0): 32 lanes reading one logical
// chunk of 32 consecutive rows hit distinct banks.  (The LDS behaves as 64
// four-byte banks served 16 lanes at a time: rows r..r+15 occupy distinct
// 16-byte slots (r % 4) * 4 + (chunk ^ (r / 4 % 4)).)
__device__ __forceinline__ int swz4(int row) { return (row >> 2) & 3; }


// NWN waves along the channels: 2 (four waves of 128 x 128, one per SIMD)
// or 4 (eight waves of 128 x 64, two per SIMD).
//
// The per-row and per-channel epilogue operands (x scales, channel scales,
// modality ids) reach LDS by DMA ahead of the first K stage.  When the
// compensation takes the fast path (bf16 factors, rank <= 64, one or two
// non-text modalities in the tile, u given as bf16 hi/lo rows in u_hl), its
// LDS operands -- u hi, u lo and the L2 rows of each modality present, 32 KB
// each -- are copied by DMA into the K buffers after the loop, with no
// conversion in the epilogue.
//
// W4: Wq holds packed 4-bit codes.  A stage's B tile is then 256 rows of 32
// bytes (two 16-byte halves, the half at position p of row r holding
// logical half p ^ ((r / 8) % 2), so that a wave's 8-byte fragment reads
// spread over the banks); lane group h of a wave takes the codes of half h
// (k chunks 2h and 2h + 1 of the stage, one per k step), and the q
// fragments follow the same k order.
//
// GRP (the MAS-only comparator, a weight per modality): tile row tm is entry
// tm of a table built on the device, {first, count, modality}: its rows are
// tokens grows[first .. first + count) (one modality, in token order), its
// weight and channel scales those of that modality (B + modality b_stride,
// w_scale + modality N).  A rows and their scales are gathered by the DMA,
// outputs are written to the tokens' own rows; table entries past *gtab_n
// (the grid is sized for the largest possible table) exit at once.
//
// PERSIST (whole tiles of one weight, no split): a grid of at most one
// workgroup per compute unit walks the tiles blockIdx.x, + gridDim.x, ...
// (gridDim.x a multiple of 8, so every tile keeps its XCD).  While a tile's
// epilogue runs, the next tile's per-row operands go to the other of two
// LDS sets and its first stages into the K buffers the epilogue leaves free
// (all three with no compensation operands staged, one with a single
// non-text modality's), the ring of K buffers then starting at that buffer.
template <typename YT, typename LT, bool CMC, bool ACC, int NWN = 2, bool SPLIT = false,
          bool W4 = false, bool GRP = false, bool PERSIST = false>
__global__ __launch_bounds__(128 * NWN, 1) void k_gemm_dma(
    const int8_t* __restrict__ A, const int8_t* __restrict__ B, const float* __restrict__ x_scale,
    const float* __restrict__ w_scale, int64_t T, int K, int N, int tiles_m, int tiles_n,
    const int32_t* __restrict__ mod, const float* __restrict__ u, const uint8_t* __restrict__ u_hl,
    int r, int n_mod, const LT* __restrict__ r_up, int32_t* __restrict__ acc_out,
    YT* __restrict__ y, int S, int32_t* __restrict__ part, int* __restrict__ tickets,
    const int32_t* __restrict__ grows, const v4i* __restrict__ gtab,
    const int* __restrict__ gtab_n, int64_t b_stride, bool a_pair) {
    __shared__ __attribute__((aligned(16))) GemmSmem sm;
    static_assert(kDmaStages * kDmaStageBytes <= static_cast<int>(sizeof(GemmSmem::buf)), "LDS");
    static_assert(kDmaStageBytes == kTileM * 128, "an epilogue operand fills one K stage buffer");
    static_assert(!PERSIST || (!SPLIT && !GRP), "persistent grid: whole tiles, one weight");
    if constexpr (!SPLIT) S = 1;
    constexpr int NJ = 8 / NWN, NW = 2 * NWN;
    constexpr int kRowsPerWave = kTileM / NW;           // DMA rows of A and of B per wave
    constexpr int kStepB = W4 ? kDmaStageK / 2 : kDmaStageK;   // B bytes per row and stage
    constexpr int kDmaA = kRowsPerWave / 16;            // DMA instructions per thread per stage:
    constexpr int kDmaB = kRowsPerWave * kStepB / 1024; //   A rows, B rows
    constexpr int kDmaPerStage = kDmaA + kDmaB;
    constexpr int kDmaExtra = kRowsPerWave / 8;         // per epilogue operand (128-byte rows)
    static_assert(kDmaB >= 1 && kRowsPerWave * kStepB % 1024 == 0, "B rows per DMA");
    using BRaw = std::conditional_t<W4, v2i, v4i>;      // a lane's B bytes of one k step
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(sm.buf));
    // per-row operand pieces: 64 entries per instruction, piece c (x scales,
    // channel scales, modality ids; 4 each) issued by wave c % NW
    constexpr int kPieces = (CMC || GRP) ? 12 : 8;
    constexpr int kPiecesMin = kPieces / NW;            // the fewest a wave issues
    const int nk_all = K / kDmaStageK;
    const int a_step = a_pair ? 2 * kDmaStageK : kDmaStageK;   // A bytes between stages
    // carried from one tile to the next (PERSIST)
    int ring = 0;        // K buffer of the tile's stage 0
    int rb = 0;          // LDS set of the tile's per-row operands
    int pf = 0;          // the tile's stages already queued
    for (int vb = static_cast<int>(blockIdx.x);; vb += static_cast<int>(gridDim.x)) {
    // the thread index through an opaque copy, so that no per-lane address of
    // a tile's loop or epilogue is hoisted out of the tile loop (where it would
    // stay live across the main loop)
    int tid = static_cast<int>(threadIdx.x);
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / NWN, wn = wave % NWN;
    int tm, tn;
    if (!tile_coords_at(vb, tiles_m, tiles_n * S, tm, tn)) break;
    // split K: slice sl of S covers stages [kst0, kst0 + nk) of the tile
    int sl = 0;
    if constexpr (SPLIT) {
        sl = tn % S;
        tn /= S;
    }
    const int nk_slice = SPLIT ? (nk_all + S - 1) / S : nk_all;
    const int kst0 = sl * nk_slice;
    const int64_t row0 = GRP ? 0 : static_cast<int64_t>(tm) * kTileM;
    const int col0 = tn * kTileN;
    // GRP: the tile's rows grows[gfirst .. gfirst + grows_n), modality gmod
    int gfirst = 0, grows_n = kTileM, gmod = 0;
    if constexpr (GRP) {
        if (tm >= *gtab_n) break;                       // wave-uniform (one tile per workgroup)
        const v4i e = gtab[tm];
        gfirst = e.x;
        grows_n = e.y;
        gmod = e.z;
        B += gmod * b_stride;
        w_scale += static_cast<int64_t>(gmod) * N;
    }
    // token of the tile's local row l (rows past the tile's end repeat its
    // last row; their results are discarded)
    auto a_row = [&](int l) __attribute__((always_inline)) -> int64_t {
        if constexpr (GRP) return grows[gfirst + min(l, grows_n - 1)];
        else return min(row0 + l, T - 1);
    };
    RowOps& ro = sm.ro[rb];

    v16i acc[4][NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = v16i{0};

    // per-row operands of the tile at rows r0.., channels c0.. into set `o`:
    // indices past T or N are clamped (their results are discarded)
    auto issue_rowops = [&](RowOps& o, int64_t r0, int c0) __attribute__((always_inline)) {
        // (GRP: the third group is the tiles' token indices, the output rows)
        for (int c = wave; c < kPieces; c += NW) {
            const int part = c & 3, e = 64 * part + lane;
            const void* src;
            uint32_t dst;
            if (c < 4) {
                src = x_scale + (GRP ? a_row(e) : min(r0 + e, T - 1));
                dst = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&o.dx[64 * part]));
            } else if (c < 8) {
                src = w_scale + min(c0 + e, N - 1);
                dst = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&o.ws[64 * part]));
            } else {
                src = GRP ? static_cast<const void*>(grows + gfirst + min(e, grows_n - 1))
                          : static_cast<const void*>(mod + min(r0 + e, T - 1));
                dst = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&o.rawmod[64 * part]));
            }
            lds_dma4(src, static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(dst))));
        }
    };
    if (vb == static_cast<int>(blockIdx.x)) issue_rowops(ro, row0, col0);   // later tiles: queued ahead

    // Wave w loads rows [w R, w R + R) of the A and of the B tile (R =
    // kRowsPerWave), 16 rows per instruction; lane i covers row 16 j + i / 4
    // at LDS chunk i % 4, which holds logical chunk (i % 4) ^ swz4(row).
    // (W4 B rows: 32 rows per instruction, lane i covers row 32 j + i / 2 at
    // half i % 2.)  Rows past T or N are clamped into the matrix; their
    // results are discarded.
    // (Row-paired A, code_row / code_col: a stage of a row pair is one
    // 128-byte line, the next stage 128 bytes on.)
    // (The stage st of a tile goes to K buffer (ring + st) % kDmaStages.)
    const int8_t* src[kDmaPerStage];      // [0, kDmaA): A rows, then B rows
    uint32_t dst_off[kDmaPerStage];
    // sources of the tile at rows r0.., channels c0.. (PERSIST: also the next tile's)
    auto set_src = [&](const int8_t* (&sp)[kDmaPerStage], int64_t r0, int c0) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < kDmaA; ++j) {
            const int row = wave * kRowsPerWave + 16 * j + (lane >> 2);
            const int chunk = (lane & 3) ^ swz4(row);
            const int64_t tok = GRP ? a_row(row) : min(r0 + row, T - 1);
            sp[j] = A + code_row(tok, K, a_pair) + kst0 * a_step + 16 * chunk;
        }
#pragma unroll
        for (int j = 0; j < kDmaB; ++j) {
            constexpr int kRowsPerDma = 1024 / kStepB;
            const int lanes_per_row = kStepB / 16;
            const int row = wave * kRowsPerWave + kRowsPerDma * j + lane / lanes_per_row;
            const int piece = W4 ? ((lane & 1) ^ ((row >> 3) & 1)) : ((lane & 3) ^ swz4(row));
            sp[kDmaA + j] = B + static_cast<int64_t>(min(c0 + row, N - 1)) * (W4 ? K / 2 : K) +
                            kst0 * kStepB + 16 * piece;
        }
    };
    set_src(src, row0, col0);
#pragma unroll
    for (int j = 0; j < kDmaA; ++j)
        dst_off[j] = static_cast<uint32_t>(
            __builtin_amdgcn_readfirstlane((wave * kRowsPerWave + 16 * j) * kDmaStageK));
#pragma unroll
    for (int j = 0; j < kDmaB; ++j) {
        constexpr int kRowsPerDma = 1024 / kStepB;
        dst_off[kDmaA + j] = kTileM * kDmaStageK + static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(
                                 (wave * kRowsPerWave + kRowsPerDma * j) * kStepB));
    }
    auto issue_from = [&](const int8_t* const (&sp)[kDmaPerStage], int st, int q, int rg)
                          __attribute__((always_inline)) {
        const uint32_t sbase = lds0 + ((rg + st) % kDmaStages) * kDmaStageBytes;
        lds_dma16(sp[q] + st * (q < kDmaA ? a_step : kStepB), sbase + dst_off[q]);
    };
    auto issue_one = [&](int st, int q) __attribute__((always_inline)) { issue_from(src, st, q, ring); };
    auto issue = [&](int st) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < kDmaPerStage; ++q) issue_one(st, q);
    };
    // fragment f of one 32-byte k step (f < 4: token block f of the q rows,
    // f >= 4: channel block f - 4 of the Wq rows)
    auto read_frag = [&](int st, int ks, int f, v4i (&fa)[4], BRaw (&fb)[NJ]) __attribute__((always_inline)) {
        const uint8_t* sa = sm.buf + ((ring + st) % kDmaStages) * kDmaStageBytes;
        const int c = W4 ? 2 * (lane >> 5) + ks : 2 * ks + (lane >> 5);
        if (f < 4) {
            const int row = wm * 128 + f * 32 + (lane & 31);
            fa[f] = *reinterpret_cast<const v4i*>(sa + row * kDmaStageK + ((c ^ swz4(row)) << 4));
        } else {
            const int row = wn * 32 * NJ + (f - 4) * 32 + (lane & 31);
            const uint8_t* sb = sa + kTileM * kDmaStageK;
            if constexpr (W4)
                fb[f - 4] = *reinterpret_cast<const v2i*>(
                    sb + row * kStepB + 16 * ((lane >> 5) ^ ((row >> 3) & 1)) + 8 * ks);
            else
                fb[f - 4] = *reinterpret_cast<const v4i*>(sb + row * kDmaStageK +
                                                          ((c ^ swz4(row)) << 4));
        }
    };
    // The 4 NJ MFMAs of one k step.  Interleaved with them, in a fixed order
    // (each step is fenced against compiler reordering): two fragment reads
    // of the next k step (st_next, ks_next) after each of the first MFMAs,
    // and with DMA one of stage dma_st's loads after every second MFMA, so
    // the LDS and vector-memory pipelines work while the matrix cores do.
    constexpr int kFrags = 4 + NJ;
    auto mfma_group = [&](const v4i (&fa)[4], const BRaw (&fb)[NJ], auto with_reads, int st_next,
                          int ks_next, v4i (&na)[4], BRaw (&nb)[NJ], auto with_dma, int dma_st)
                          __attribute__((always_inline)) {
        v4i ub[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            if constexpr (W4) ub[j] = w4_operand(fb[j]);
            else ub[j] = fb[j];
        }
#pragma unroll
        for (int q = 0; q < 4 * NJ; ++q) {
            acc[q / NJ][q % NJ] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ub[q % NJ], fa[q / NJ],
                                                                        acc[q / NJ][q % NJ], 0, 0, 0);
            if constexpr (decltype(with_reads)::value)
                if (2 * q < kFrags) {
                    read_frag(st_next, ks_next, 2 * q, na, nb);
                    read_frag(st_next, ks_next, 2 * q + 1, na, nb);
                }
            if constexpr (decltype(with_dma)::value)
                if ((q & 1) && (q >> 1) < kDmaPerStage) issue_one(dma_st, q >> 1);
            MASQ_SCHED_FENCE();
        }
    };
    // publish stage st to all waves: this wave's loads of st are complete
    // once at most those of the `younger` later stages are in flight, and its
    // LDS reads of the buffer about to be refilled are complete
    auto publish = [&](int younger) __attribute__((always_inline)) {
        if (younger >= 2) MASQ_WAIT_VMCNT_LGKM0(2 * kDmaPerStage);
        else if (younger == 1) MASQ_WAIT_VMCNT_LGKM0(kDmaPerStage);
        else MASQ_WAIT_VMCNT_LGKM0(0);
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };

    // Pipeline: stage kt is consumed as two 32-byte k steps.  The fragments of
    // each k step are read during the MFMAs of the previous one; the barrier
    // that publishes stage kt + 1 sits between the two MFMA groups of stage
    // kt.  The DMA of stage kt + 3 refills the buffer of stage kt - 1, which
    // every wave finished reading before the previous barrier.  The loop is
    // split into uniform phases (DMA still to issue / none / last stage) so
    // that each body has a single shape.
    using yes = std::true_type;
    using no = std::false_type;
    const int nk = min(nk_slice, nk_all - kst0);             // >= 1 (plan_gemm_splits)
    // (PERSIST) the previous tile's epilogue is done with the K buffers
    if (PERSIST && vb != static_cast<int>(blockIdx.x)) __syncthreads();
    for (int st = pf; st < kDmaStages - 1 && st < nk; ++st) issue(st);
    v4i fa0[4], fa1[4];
    BRaw fb0[NJ], fb1[NJ];
    publish(min(nk - 1, 2));

    // The per-row operands have landed (they precede stage 0 in every wave's
    // queue).  Modalities present in the tile, as scalars.
    unsigned present = 0;
    int mod0 = 0, mod1 = 0;                 // the first two non-text modalities present
    bool pre = false;
    if constexpr (CMC) {
        if (tid < kTileM) ro.mod[tid] = sane_mod(ro.rawmod[tid], n_mod);   // read after a barrier
        const v4i m4 = *reinterpret_cast<const v4i*>(&ro.rawmod[4 * lane]);
        const int s0 = sane_mod(m4.x, n_mod), s1 = sane_mod(m4.y, n_mod);
        const int s2 = sane_mod(m4.z, n_mod), s3 = sane_mod(m4.w, n_mod);
        for (int m = 1; m < n_mod; ++m)
            if (__ballot(s0 == m || s1 == m || s2 == m || s3 == m) != 0ull) present |= 1u << m;
        present = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(static_cast<int>(present)));
        const unsigned rest = present & (present - 1u);       // bit 0 (text) is never set
        mod0 = present ? __builtin_ctz(present) : 0;
        mod1 = rest ? __builtin_ctz(rest) : 0;
        const int np = __builtin_popcount(present);
        pre = sizeof(LT) == 2 && u_hl != nullptr && r <= 64 && np >= 1 && np <= 2 && y != nullptr;
    }
    // compensation operand v (0: u hi, 1: u lo, 2: L2 rows of mod0, 3: of mod1)
    // into K buffer v, 128-byte rows: lane i covers row 8 q + i / 8 of this
    // wave's share at LDS chunk i % 8, which holds logical chunk
    // (i % 8) ^ swz(row)
    auto issue_extra = [&](int v) __attribute__((always_inline)) {
        const uint32_t sbase = lds0 + v * kDmaStageBytes;
        const LT* rm = r_up + static_cast<int64_t>(max((v == 2 ? mod0 : mod1) - 1, 0)) * N * r;
#pragma unroll
        for (int q = 0; q < kDmaExtra; ++q) {
            const int rw = wave * kRowsPerWave + 8 * q;
            const int row = rw + (lane >> 3);
            const int lc = (lane & 7) ^ swz(row);
            const uint8_t* sp =
                v < 2 ? u_hl + min(row0 + row, T - 1) * 256 + 128 * v + 16 * lc
                      : reinterpret_cast<const uint8_t*>(
                            rm + static_cast<int64_t>(min(col0 + row, N - 1)) * r) +
                            16 * min(lc, (r >> 3) - 1);
            lds_dma16(sp, sbase + static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(rw * 128)));
        }
    };

#pragma unroll
    for (int f = 0; f < kFrags; ++f) read_frag(0, 0, f, fa0, fb0);
    auto body = [&](int kt, auto with_dma, auto with_next) __attribute__((always_inline)) {
        MASQ_SCHED_FENCE();
        mfma_group(fa0, fb0, yes{}, kt, 1, fa1, fb1, with_dma, kt + kDmaStages - 1);
        if constexpr (decltype(with_next)::value) {
            publish(min(nk - 2 - kt, 2));
            MASQ_SCHED_FENCE();
            mfma_group(fa1, fb1, yes{}, kt + 1, 0, fa0, fb0, no{}, 0);
        } else {
            mfma_group(fa1, fb1, no{}, 0, 0, fa0, fb0, no{}, 0);
        }
    };
    int kt = 0;
    for (; kt + kDmaStages - 1 < nk; ++kt) body(kt, yes{}, yes{});
    for (; kt + 1 < nk; ++kt) body(kt, no{}, yes{});
    body(kt, no{}, no{});
    if constexpr (W4) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[i][j][e] >>= 4;     // exact: 16 x the sum
    }

    if constexpr (SPLIT) {
        // Every slice writes its accumulators to its slot of the tile's
        // workspace (value-major: each 16-byte store instruction covers 1 KB
        // of consecutive bytes) with the agent-coherent cache policy (sc1),
        // so the XCD-local L2 does not hold them back, and counts its arrival
        // once the stores have completed; the last slice to arrive reads the
        // others' slots with the same policy and adds them (exact in any
        // order) before the epilogue.  No fence, no waiting on other
        // workgroups.  Accesses go through a buffer descriptor that covers
        // exactly the tile's S slots (raw, untyped: descriptor word 3 =
        // 0x00020000 on this architecture).
        constexpr int NT = 64 * NW, kV4 = 4 * NJ * 4;          // v4 groups per thread
        constexpr int kSlot = kTileM * kTileN * 4;            // bytes per slice slot
        constexpr int kPolicy = 16;                           // sc1
        const int tile = tm * tiles_n + tn;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            part + static_cast<int64_t>(tile) * S * (kTileM * kTileN), 0, S * kSlot, 0x00020000);
#pragma unroll
        for (int c = 0; c < kV4; ++c) {
            const v16i& blk = acc[c / (4 * NJ)][(c / 4) % NJ];
            const v4i v = {blk[4 * (c % 4)], blk[4 * (c % 4) + 1], blk[4 * (c % 4) + 2],
                           blk[4 * (c % 4) + 3]};
            __builtin_amdgcn_raw_buffer_store_b128(v, rs, sl * kSlot + (c * NT + tid) * 16, 0, kPolicy);
        }
        MASQ_WAIT_VMCNT_LGKM0(0);
        __syncthreads();
        if (tid == 0)
            sm.last = __hip_atomic_fetch_add(&tickets[tile], 1, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT) == S - 1;
        __syncthreads();
        if (!sm.last) return;
        if (tid == 0) __hip_atomic_store(&tickets[tile], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (int s2 = 0; s2 < S; ++s2) {
            if (s2 == sl) continue;
#pragma unroll
            for (int c = 0; c < kV4; ++c) {
                const v4i v = __builtin_amdgcn_raw_buffer_load_b128(
                    rs, s2 * kSlot + (c * NT + tid) * 16, 0, kPolicy);
                v16i& blk = acc[c / (4 * NJ)][(c / 4) % NJ];
#pragma unroll
                for (int e = 0; e < 4; ++e) blk[4 * (c % 4) + e] += v[e];
            }
        }
    }

    EpiDma ed{};
    ed.present = present;
    ed.pre = pre;
    ed.grp_rows = grows_n;
    bool synced = false;
    if constexpr (CMC) {
        if (pre) {
            // the K buffers are free once every wave is past its last reads
            __syncthreads();
            synced = true;
            issue_extra(0);
            issue_extra(1);
            issue_extra(2);
            if (mod1 != 0) issue_extra(3);
            ed.off_uh = 0;
            ed.off_ul = kDmaStageBytes;
            ed.off_r[0] = 2 * kDmaStageBytes;
            ed.off_r[1] = 3 * kDmaStageBytes;
        }
    }
    // PERSIST: the next tile's per-row operands (the other LDS set) and its
    // first stages, into the K buffers this epilogue leaves free: stages 0-2
    // into buffers 0-2 when it stages no compensation operands, stage 0 into
    // buffer 3 when they are one modality's (buffers 0-2), none with two
    int npf = -1, nring = 0;                 // npf < 0: no next tile
    if constexpr (PERSIST) {
        int tmn, tnn;
        if (tile_coords_at(vb + static_cast<int>(gridDim.x), tiles_m, tiles_n, tmn, tnn)) {
            const int64_t r0n = static_cast<int64_t>(tmn) * kTileM;
            const int c0n = tnn * kTileN;
            issue_rowops(sm.ro[rb ^ 1], r0n, c0n);
            npf = 0;
            if (!CMC || present == 0) {
                npf = min(kDmaStages - 1, nk_all);
            } else if (pre && mod1 == 0) {
                npf = 1;
                nring = 3;
            }
            if (npf > 0) {
                if (!synced) __syncthreads();    // every wave is past its reads of the last stages
                const int8_t* srcn[kDmaPerStage];
                set_src(srcn, r0n, c0n);
                for (int st = 0; st < npf; ++st)
#pragma unroll
                    for (int q = 0; q < kDmaPerStage; ++q) issue_from(srcn, st, q, nring);
            }
        }
    }
    // this tile's operands have landed once at most the next tile's (younger)
    // loads are in flight; a wave queued kPiecesMin or kPiecesMin + 1 pieces
    if (npf < 0) MASQ_WAIT_VMCNT_LGKM0(0);
    else if (npf == 0) MASQ_WAIT_VMCNT_LGKM0(kPiecesMin);
    else if (npf == 1) MASQ_WAIT_VMCNT_LGKM0(kPiecesMin + kDmaPerStage);
    else if (npf == 2) MASQ_WAIT_VMCNT_LGKM0(kPiecesMin + 2 * kDmaPerStage);
    else MASQ_WAIT_VMCNT_LGKM0(kPiecesMin + 3 * kDmaPerStage);
    gemm_epilogue<YT, LT, CMC, ACC, NWN, true, GRP>(acc, sm, EpiPrefetch{}, T, N, row0, col0, u, r, n_mod,
                                               r_up, acc_out, y, ed, rb, tid);
    if constexpr (!PERSIST) break;
    ring = nring;
    pf = max(npf, 0);
    rb ^= 1;
    }
}

// ================================================================ small-batch GEMM
// For batches of at most 16 tokens (decoding) the layer is bound by
// streaming Wq from HBM.  A workgroup owns 16 output channels; its four
// waves split K and keep kSmallDepth 64-byte k steps of Wq and q loads in
// flight, feeding v_mfma_i32_16x16x64_i8 (tokens as the 16 rows).  The
// per-wave int32 partials are added in a fixed order in LDS (exact), then
// each thread finishes one (token, channel): dequantisation, the rank-r
// compensation u L2^m in fp32 for non-text tokens, and the store.
constexpr int kSmallDepth = 16;

// u of a small batch's rows into LDS (256 threads), adding the k-slice
// partials in slice order when the down-projection left them separate.
__device__ __forceinline__ void small_u_rows(float (&su)[kSmallMaxT][kMaxRank],
                                             const float* __restrict__ u,
                                             const float* __restrict__ u_part, int n_kslices,
                                             int T, int r, int tid) {
    const bool parts = u_part != nullptr && n_kslices > 1;
    const float* src = parts ? u_part : u;
    const int slices = parts ? n_kslices : 1;
    for (int idx = 4 * tid; idx < T * r; idx += 4 * 256) {       // T r % 16 == 0
        v4f v = {0.f, 0.f, 0.f, 0.f};
        for (int q0 = 0; q0 < slices; q0 += kUBatch) {
            v4f p[kUBatch];
#pragma unroll
            for (int q = 0; q < kUBatch; ++q)                        // a batch in flight
                p[q] = *reinterpret_cast<const v4f*>(
                    src + static_cast<int64_t>(min(q0 + q, slices - 1)) * T * r + idx);
#pragma unroll
            for (int q = 0; q < kUBatch; ++q)
                if (q0 + q < slices) v = (q0 + q == 0) ? p[q] : v + p[q];   // slice order
        }
        const int tt = idx / r, c = idx - tt * r;
        *reinterpret_cast<v4f*>(&su[tt][c]) = v;
    }
}

// Dequantisation, compensation (u rows in su) and store of one output of a
// small batch: token t, channel ch, int32 accumulator a.
template <typename YT, typename LT>
__device__ __forceinline__ void small_output(const float (&su)[kSmallMaxT][kMaxRank], int a, int t,
                                             int ch, int N, const float* __restrict__ x_scale,
                                             const float* __restrict__ w_scale,
                                             const int32_t* __restrict__ mod, bool cmc, int r,
                                             int n_mod, const LT* __restrict__ r_up,
                                             YT* __restrict__ y) {
    float v = (static_cast<float>(a) * x_scale[t]) * w_scale[ch];
    const int m = cmc ? sane_mod(mod[t], n_mod) : 0;
    if (m > 0) {
        const LT* rr = r_up + (static_cast<int64_t>(m - 1) * N + ch) * r;
        float c = 0.f;
        for (int k0 = 0; k0 < r; k0 += 8) {
            float uv[8], rv[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) uv[k] = su[t][k0 + k];
            Elem<LT>::load8(rr + k0, rv);
#pragma unroll
            for (int k = 0; k < 8; ++k) c = fmaf(uv[k], rv[k], c);
        }
        v += c;
    }
    Elem<YT>::store1(y + static_cast<int64_t>(t) * N + ch, v);
}

template <typename YT, typename LT, bool W4>
__global__ __launch_bounds__(256) void k_gemm_small(
    const int8_t* __restrict__ A, const int8_t* __restrict__ B, const float* __restrict__ x_scale,
    const float* __restrict__ w_scale, int T, int K, int N, const int32_t* __restrict__ mod,
    const float* __restrict__ u, const float* __restrict__ u_part, int n_kslices, int r,
    int n_mod, const LT* __restrict__ r_up, int32_t* __restrict__ acc_out, YT* __restrict__ y) {
    __shared__ int part[4][16][16];
    __shared__ float su[kSmallMaxT][kMaxRank];     // u rows of the batch
    const int tid = threadIdx.x, lane = tid & 63;
    // wave-uniform k range (scalar registers), so the loop below branches on
    // it: MFMA instructions ignore EXEC and must not sit under a lane mask
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col0 = blockIdx.x * 16;
    const int nsteps = K >> 6;
    const int per = (nsteps + 3) >> 2;
    const int sb = min(nsteps, wave * per);
    const int se = min(nsteps, sb + per);
    // lane: row (token / channel) lane % 16, 16-byte k group lane / 16
    // (W4: Wq rows of K / 2 packed bytes, 8 bytes a lane a step)
    using BRaw = std::conditional_t<W4, v2i, v4i>;
    constexpr int kStepB = W4 ? 32 : 64;
    const int8_t* ap = A + static_cast<int64_t>(min(lane & 15, T - 1)) * K + 16 * (lane >> 4);
    const int8_t* bp = B + static_cast<int64_t>(col0 + (lane & 15)) * (W4 ? K / 2 : K) +
                       (kStepB / 4) * (lane >> 4);
    auto step_addr = [&](int st) { return static_cast<int64_t>(min(st, nsteps - 1)) * 64; };
    auto step_addr_b = [&](int st) { return static_cast<int64_t>(min(st, nsteps - 1)) * kStepB; };
    v4i acc = {0, 0, 0, 0};
    v4i fa[kSmallDepth];
    BRaw fb[kSmallDepth];
#pragma unroll
    for (int d = 0; d < kSmallDepth; ++d) {
        fa[d] = *reinterpret_cast<const v4i*>(ap + step_addr(sb + d));
        fb[d] = *reinterpret_cast<const BRaw*>(bp + step_addr_b(sb + d));
    }
    const v4i zero = {0, 0, 0, 0};
    for (int st0 = sb; st0 < se; st0 += kSmallDepth) {
#pragma unroll
        for (int d = 0; d < kSmallDepth; ++d) {
            // steps past the wave's range (last round) contribute zeros
            const bool in = st0 + d < se;
            v4i b;
            if constexpr (W4) b = w4_operand(fb[d]);
            else b = fb[d];
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(in ? fa[d] : zero, b, acc, 0, 0, 0);
            fa[d] = *reinterpret_cast<const v4i*>(ap + step_addr(st0 + d + kSmallDepth));
            fb[d] = *reinterpret_cast<const BRaw*>(bp + step_addr_b(st0 + d + kSmallDepth));
        }
    }
    if constexpr (W4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] >>= 4;                   // exact: 16 x the sum
    }
    // acc[e]: token 4 (lane / 16) + e, channel col0 + lane % 16
#pragma unroll
    for (int e = 0; e < 4; ++e) part[wave][4 * (lane >> 4) + e][lane & 15] = acc[e];
    if (u != nullptr) small_u_rows(su, u, u_part, n_kslices, T, r, tid);
    __syncthreads();
    const int t = tid >> 4, o = tid & 15;
    if (t >= T) return;
    const int a = ((part[0][t][o] + part[1][t][o]) + part[2][t][o]) + part[3][t][o];
    const int ch = col0 + o;
    if (acc_out != nullptr) acc_out[static_cast<int64_t>(t) * N + ch] = a;
    if (y == nullptr) return;
    small_output<YT, LT>(su, a, t, ch, N, x_scale, w_scale, mod, u != nullptr, r, n_mod, r_up, y);
}

// ---------------------------------------------------------------- decode GEMM
// The fused layer's small-batch GEMM.  At most 16 tokens make the layer a
// stream of Wq from HBM, so the kernel is shaped to keep as many Wq bytes in
// flight as it can: a workgroup covers kDecCh output channels (16 per wave)
// and one k slice of sp <= kDecSteps 64-byte steps, and each wave issues all
// of its slice's Wq loads at once into registers.  The slice of q goes to
// LDS by DMA queued ahead of those loads (vector-memory loads complete in
// issue order, so waiting for q does not wait for Wq).  The int32 partial
// sums of each slice go to the workspace; the last workgroup of a channel
// group to arrive adds the slices in slice order and finishes the outputs
// like the single-pass kernel (dequantisation, compensation, store).
// The compensation term of the group's outputs is computed off that tail
// when its operands fit in LDS: workgroup (g, s) takes the tokens t with
// t % ns == s.  The u partials of those tokens and the L2 rows of the
// group's channels are queued by DMA with the q slice, ahead of the Wq
// loads, so they have landed long before Wq has; the workgroup adds the
// partials (slice order), forms (x S^-1 L1) L2 for its tokens while its Wq
// loads are still in flight (each thread sums over the rank in 8-column
// chunks, starting at a lane-dependent chunk), and hands the fp32 terms over
// beside the int32 partials.  The last workgroup then only adds.
// W4: Wq holds packed 4-bit codes (K / 2 bytes a row, 8 bytes a lane a step,
// unpacked into the MFMA operand in registers).
// only_mod >= 0 (the MAS-only comparator, one launch per modality's weight):
// only the outputs of tokens of that modality are stored.
template <typename YT, typename LT, bool W4>
__global__ __launch_bounds__(256, 2) void k_gemm_decode(
    const int8_t* __restrict__ A, const int8_t* __restrict__ B, const float* __restrict__ x_scale,
    const float* __restrict__ w_scale, int T, int K, int N, int ns, int sp,
    const int32_t* __restrict__ mod, const float* __restrict__ u,
    const float* __restrict__ u_part, int n_kslices, int r, int n_mod,
    const LT* __restrict__ r_up, int32_t* __restrict__ part, int* __restrict__ tickets,
    YT* __restrict__ y, int only_mod) {
    __shared__ __attribute__((aligned(16))) uint8_t sq[kDecSteps * 1024];
    // compensation operands (u partials of the token share, then L2 rows of
    // the group's channels) or, when they do not fit, the u rows of the batch
    __shared__ __attribute__((aligned(16))) uint8_t scm[kDecCmcBytes];
    static_assert(sizeof(float) * kSmallMaxT * kMaxRank <= kDecCmcBytes, "u rows fit scm");
    auto& su = *reinterpret_cast<float (*)[kSmallMaxT][kMaxRank]>(scm);
    __shared__ int s_last;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = blockIdx.x / ns, sl = blockIdx.x - g * ns;        // channel group, k slice
    const int st0 = sl * sp;
    const int S = min(sp, (K >> 6) - st0);                         // steps of this slice, >= 1
    const int cb = g * kDecCh + 16 * wave;                         // the wave's first channel
    const bool active = cb < N;

    // q slice into LDS: step j as 16 rows x 64 bytes, row t's piece p at
    // position p ^ swz4(t); rows past T repeat row T - 1 (results discarded)
    const uint32_t sq0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(sq));
    {
        const int t = lane >> 2, p = (lane & 3) ^ swz4(lane >> 2);
        const int8_t* qa = A + static_cast<int64_t>(min(t, T - 1)) * K +
                           static_cast<int64_t>(st0) * 64 + 16 * p;
        for (int j = wave; j < S; j += 4) lds_dma16(qa + 64 * j, sq0 + j * 1024);
    }
    // compensation operands of the token share, when they fit: the u slice
    // partials as rows [slice][share token][r] fp32, then the L2 rows
    // [modality - 1][channel of the group][r]; both padded to whole 1 KB
    // DMA blocks (a block's pieces past the end repeat the last piece)
    const bool cmc = u != nullptr;
    const int uslices = (u_part != nullptr && n_kslices > 1) ? n_kslices : 1;
    const float* usrc = uslices > 1 ? u_part : u;
    const int nts = (T + ns - 1) / ns;                              // share tokens, at most
    const int own = sl < T ? (T - sl + ns - 1) / ns : 0;            // this workgroup's
    const int up_pieces = uslices * nts * (r >> 2);                 // 16-byte pieces
    const int up_bytes = ((up_pieces * 16 + 1023) >> 10) << 10;
    const int rrow = r * static_cast<int>(sizeof(LT));              // bytes of one L2 row
    const int rp_pieces = cmc ? (n_mod - 1) * kDecCh * (rrow >> 4) : 0;
    const bool early = cmc && nts <= 4 && up_bytes + rp_pieces * 16 <= kDecCmcBytes;
    const uint32_t scm0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(scm));
    int tmod = 0;                                   // modality of the thread's share output
    if (early) {
        const int ti = tid >> 6;
        if (ti < own) tmod = sane_mod(mod[sl + ti * ns], n_mod);
        const int upr = r >> 2;                                     // pieces per u row
        for (int i = wave; i * 64 < up_pieces; i += 4) {
            const int pc = min(i * 64 + lane, up_pieces - 1);
            const int row = pc / upr, c = pc - row * upr;
            const int s = row / nts, tt = min(sl + (row - s * nts) * ns, T - 1);
            lds_dma16(usrc + (static_cast<int64_t>(s) * T + tt) * r + 4 * c, scm0 + i * 1024);
        }
        const int rpr = rrow >> 4;                                  // pieces per L2 row
        for (int i = wave; i * 64 < rp_pieces; i += 4) {
            const int pc = i * 64 + lane;                           // rp_pieces % 64 == 0
            const int row = pc / rpr, c = pc - row * rpr;
            const int mm = row / kDecCh, ch = min(g * kDecCh + (row - mm * kDecCh), N - 1);
            lds_dma16(reinterpret_cast<const uint8_t*>(r_up + (static_cast<int64_t>(mm) * N + ch) * r) +
                          16 * c,
                      scm0 + up_bytes + i * 1024);
        }
    }
    // every Wq step of the slice (steps past S repeat step S - 1 and are not
    // used; a wave past N reads the last channel block and stores nothing)
    using BRaw = std::conditional_t<W4, v2i, v4i>;
    constexpr int kStepB = W4 ? 32 : 64;                           // Wq bytes per row and step
    BRaw fb[kDecSteps];
    {
        const int64_t pitch = W4 ? K / 2 : K;                      // bytes per Wq row
        const int8_t* bp = B + (min(cb, N - 16) + (lane & 15)) * pitch +
                           static_cast<int64_t>(st0) * kStepB + (kStepB / 4) * (lane >> 4);
        asm volatile("" ::: "memory");
#pragma unroll
        for (int j = 0; j < kDecSteps; ++j)
            fb[j] = *reinterpret_cast<const BRaw*>(bp + kStepB * min(j, S - 1));
        asm volatile("" ::: "memory");
    }
    // this wave's q loads are the ones older than its kDecSteps Wq loads;
    // the barrier publishes every wave's share
    MASQ_WAIT_VMCNT_LGKM0(kDecSteps);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    // while Wq streams in: u rows of the share (slice partials added in
    // slice order, into slice 0's rows), then one compensation term per
    // thread (share token tid / 64, channel tid % 64), k in order
    float cterm = 0.f;
    if (early) {
        float* up = reinterpret_cast<float*>(scm);
        const int stride = nts * r;                                 // floats per slice
        for (int idx = 4 * tid; idx < stride; idx += 4 * 256) {
            v4f v = *reinterpret_cast<const v4f*>(up + idx);
            for (int s = 1; s < uslices; ++s) v = v + *reinterpret_cast<const v4f*>(up + s * stride + idx);
            *reinterpret_cast<v4f*>(up + idx) = v;
        }
        __syncthreads();
        if (tmod > 0) {
            // lane l starts at 8-column chunk l % (r / 8) of its L2 row (the
            // rows lie 128 or 256 bytes apart, so reading the chunks in the
            // same order would put every lane on the same banks)
            const float* ur = up + (tid >> 6) * r;
            const LT* rr = reinterpret_cast<const LT*>(scm + up_bytes +
                                                       ((tmod - 1) * kDecCh + (tid & 63)) * rrow);
            const int nch = r >> 3;
            for (int j = 0; j < nch; ++j) {
                const int k0 = 8 * ((j + lane) % nch);
                float rv[8];
                Elem<LT>::load8(rr + k0, rv);
#pragma unroll
                for (int k = 0; k < 8; ++k) cterm = fmaf(ur[k0 + k], rv[k], cterm);
            }
        }
    }
    MASQ_SCHED_FENCE();
    v4i acc = {0, 0, 0, 0};
    {
        const int rt = lane & 15;
        const uint8_t* rd = sq + rt * 64 + (((lane >> 4) ^ swz4(rt)) << 4);
        const v4i zero = {0, 0, 0, 0};
#pragma unroll
        for (int j = 0; j < kDecSteps; ++j) {
            // steps past S multiply zeros (MFMA does not branch on lanes)
            v4i fa = *reinterpret_cast<const v4i*>(rd + min(j, S - 1) * 1024);
            fa = j < S ? fa : zero;
            if constexpr (W4)
                acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa, w4_operand(fb[j]), acc, 0, 0, 0);
            else
                acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa, fb[j], acc, 0, 0, 0);
        }
        if constexpr (W4) {
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] >>= 4;               // exact: 16 x the sum
        }
    }
    // Hand-over of the partials without cache maintenance: they are written
    // and read only by agent-scope atomic accesses, which the XCD-local L2
    // does not hold back, and every store has completed (vmcnt 0) before the
    // workgroup's arrival is counted.  (A device-scope fence would write
    // back the whole L2 of the XCD, once per workgroup.)
    // acc[e]: token 4 (lane / 16) + e, channel cb + lane % 16
    if (active) {
        int32_t* pp = part + static_cast<int64_t>(sl) * kSmallMaxT * N + cb + (lane & 15);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t = 4 * (lane >> 4) + e;
            if (t < T)
                __hip_atomic_store(pp + static_cast<int64_t>(t) * N, acc[e], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    // the share's compensation terms: fp32 bits in slot ns of the partials
    if (tmod > 0 && g * kDecCh + (tid & 63) < N)
        __hip_atomic_store(part + static_cast<int64_t>(ns) * kSmallMaxT * N +
                               static_cast<int64_t>(sl + (tid >> 6) * ns) * N + g * kDecCh + (tid & 63),
                           __float_as_int(cterm), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    MASQ_WAIT_VMCNT_LGKM0(0);
    __syncthreads();
    if (tid == 0)
        s_last = __hip_atomic_fetch_add(&tickets[g], 1, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT) == ns - 1;
    __syncthreads();
    if (!s_last) return;
    if (tid == 0)                       // ready for the next launch
        __hip_atomic_store(&tickets[g], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    // Everything the outputs need is loaded before any of it is used: the
    // slice partials of the thread's outputs (slices past ns re-read slice
    // ns - 1 and are not added), their scales and modality ids, the L2 rows
    // of the group's channels for every non-text modality (into the q
    // buffer, free now, slot (m - 1) kDecCh + o, when they fit in
    // kRStage bytes) and the u rows of the batch; or, when the slices have
    // formed the compensation terms, those terms.
    constexpr int kOut = kSmallMaxT * kDecCh / 256;
    constexpr int kRStage = 16384;
    constexpr int kRPieces = kRStage / 16 / 256;                       // per thread
    int pv[kOut][kDecMaxSlices], mv[kOut], om[kOut];
    float dxv[kOut], dwv[kOut], cv[kOut];
#pragma unroll
    for (int i = 0; i < kOut; ++i) {
        const int idx = tid + 256 * i;
        const int t = min(idx / kDecCh, T - 1), ch = min(g * kDecCh + idx % kDecCh, N - 1);
        int32_t* pa = part + static_cast<int64_t>(t) * N + ch;
#pragma unroll
        for (int q = 0; q < kDecMaxSlices; ++q)
            pv[i][q] = __hip_atomic_load(pa + static_cast<int64_t>(min(q, ns - 1)) * kSmallMaxT * N,
                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        cv[i] = early ? __int_as_float(__hip_atomic_load(pa + static_cast<int64_t>(ns) * kSmallMaxT * N,
                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                      : 0.f;
        dxv[i] = x_scale[t];
        dwv[i] = w_scale[ch];
        mv[i] = cmc ? sane_mod(mod[t], n_mod) : 0;
        om[i] = only_mod >= 0 ? sane_mod(mod[t], n_mod) : -1;
    }
    const int row_bytes = r * static_cast<int>(sizeof(LT));
    const bool staged = cmc && !early && (n_mod - 1) * kDecCh * row_bytes <= kRStage;
    const int per_row = row_bytes >> 4;                                // 16-byte pieces per row
    const int pieces = staged ? (n_mod - 1) * kDecCh * per_row : 0;
    v4i rpc[kRPieces];
#pragma unroll
    for (int k = 0; k < kRPieces; ++k) {
        const int i = min(tid + 256 * k, max(pieces - 1, 0));
        const int row = i / max(per_row, 1), pc = i - row * max(per_row, 1);
        const int mm = row / kDecCh, o = row - mm * kDecCh;
        const int ch = min(g * kDecCh + o, N - 1);
        if (tid + 256 * k < pieces)
            rpc[k] = *reinterpret_cast<const v4i*>(
                reinterpret_cast<const uint8_t*>(r_up + (static_cast<int64_t>(mm) * N + ch) * r) +
                16 * pc);
    }
    // u rows: one v4f of T x r per thread, the k slices in batches of kUB
    // (the first issued with the loads above), when the batch is small
    // enough; else the general loop
    const bool u_fast = cmc && !early && T * r <= 4 * 256;
    constexpr int kUB = kUBatch;
    v4f up[kUB];
    if (u_fast && 4 * tid < T * r) {
#pragma unroll
        for (int q = 0; q < kUB; ++q)
            if (q < uslices)
                up[q] = *reinterpret_cast<const v4f*>(usrc + static_cast<int64_t>(q) * T * r + 4 * tid);
    }
#pragma unroll
    for (int k = 0; k < kRPieces; ++k) {
        const int i = tid + 256 * k;
        if (i < pieces) {
            const int row = i / per_row, pc = i - row * per_row;
            *reinterpret_cast<v4i*>(sq + row * row_bytes + 16 * pc) = rpc[k];
        }
    }
    if (u_fast) {
        if (4 * tid < T * r) {
            v4f v = up[0];
#pragma unroll
            for (int q = 1; q < kUB; ++q)
                if (q < uslices) v = v + up[q];                     // slice order
            for (int q0 = kUB; q0 < uslices; q0 += kUB) {
#pragma unroll
                for (int q = 0; q < kUB; ++q)
                    if (q0 + q < uslices)
                        up[q] = *reinterpret_cast<const v4f*>(
                            usrc + static_cast<int64_t>(q0 + q) * T * r + 4 * tid);
#pragma unroll
                for (int q = 0; q < kUB; ++q)
                    if (q0 + q < uslices) v = v + up[q];
            }
            const int tt = (4 * tid) / r, c = 4 * tid - tt * r;
            *reinterpret_cast<v4f*>(&su[tt][c]) = v;
        }
    } else if (cmc && !early) {
        small_u_rows(su, u, u_part, n_kslices, T, r, tid);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kOut; ++i) {
        const int idx = tid + 256 * i;
        const int t = idx / kDecCh, o = idx % kDecCh, ch = g * kDecCh + o;
        if (t >= T || ch >= N || om[i] != only_mod) continue;
        int a = pv[i][0];
#pragma unroll
        for (int q = 1; q < kDecMaxSlices; ++q) a += q < ns ? pv[i][q] : 0;
        float v = (static_cast<float>(a) * dxv[i]) * dwv[i];
        const int m = mv[i];
        if (m > 0 && early) {
            v += cv[i];
        } else if (m > 0) {
            float c = 0.f;
            if (staged) {
                const LT* rr = reinterpret_cast<const LT*>(sq + ((m - 1) * kDecCh + o) * row_bytes);
                for (int k0 = 0; k0 < r; k0 += 8) {
                    float rv[8];
                    Elem<LT>::load8(rr + k0, rv);
#pragma unroll
                    for (int k = 0; k < 8; ++k) c = fmaf(su[t][k0 + k], rv[k], c);
                }
            } else {
                const LT* rr = r_up + (static_cast<int64_t>(m - 1) * N + ch) * r;
                for (int k0 = 0; k0 < r; k0 += 8) {
                    float rv[8];
                    Elem<LT>::load8(rr + k0, rv);
#pragma unroll
                    for (int k = 0; k < 8; ++k) c = fmaf(su[t][k0 + k], rv[k], c);
                }
            }
            v += c;
        }
        Elem<YT>::store1(y + static_cast<int64_t>(t) * N + ch, v);
    }
}

// ================================================================ MAS-only routing
// Rows grouped by modality (the MAS-only comparator, whose tiles each take
// one modality's weight): a stable counting sort of the token ids (ids
// outside [0, n_mod) read as text) by one workgroup.  rows[T]: token
// indices, modality 0's first, each modality's in token order.  tab: one
// entry {first, count, modality, 0} per 256-row tile of a modality's rows
// (count <= 256), modality by modality; *tab_n: the number of entries.
// Also clears n_zero ints at zero_ints (the grouped GEMM's arrival counters).
constexpr int kGrpThreads = 1024;

__global__ __launch_bounds__(kGrpThreads) void k_group_rows(
    const int32_t* __restrict__ mod, int64_t T, int n_mod, int32_t* __restrict__ rows,
    v4i* __restrict__ tab, int* __restrict__ tab_n, int* __restrict__ zero_ints, int n_zero) {
    __shared__ v4i scan[2][kGrpThreads];
    __shared__ int base[4];
    const int tid = threadIdx.x;
    for (int i = tid; i < n_zero; i += kGrpThreads) zero_ints[i] = 0;
    const int64_t per = (T + kGrpThreads - 1) / kGrpThreads;
    const int64_t t0 = min(T, tid * per), t1 = min(T, t0 + per);
    v4i c = {0, 0, 0, 0};
    for (int64_t t = t0; t < t1; ++t) {
        const int m = sane_mod(mod[t], n_mod);
        c[0] += m == 0; c[1] += m == 1; c[2] += m == 2; c[3] += m == 3;
    }
    // inclusive scan over the threads (Hillis-Steele, double-buffered)
    int cur = 0;
    scan[0][tid] = c;
    __syncthreads();
    for (int off = 1; off < kGrpThreads; off <<= 1) {
        v4i v = scan[cur][tid];
        if (tid >= off) v += scan[cur][tid - off];
        scan[cur ^ 1][tid] = v;
        cur ^= 1;
        __syncthreads();
    }
    const v4i incl = scan[cur][tid];
    const v4i total = scan[cur][kGrpThreads - 1];
    if (tid == 0) {
        base[0] = 0;
        base[1] = total[0];
        base[2] = total[0] + total[1];
        base[3] = total[0] + total[1] + total[2];
    }
    __syncthreads();
    int pos[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) pos[m] = base[m] + incl[m] - c[m];
    for (int64_t t = t0; t < t1; ++t) {
        const int m = sane_mod(mod[t], n_mod);
        const int at = m == 0 ? pos[0]++ : m == 1 ? pos[1]++ : m == 2 ? pos[2]++ : pos[3]++;
        rows[at] = static_cast<int32_t>(t);
    }
    if (tid == 0) {
        int k = 0;
        for (int m = 0; m < n_mod; ++m)
            for (int off = 0; off < total[m]; off += kTileM)
                tab[k++] = v4i{base[m] + off, min(kTileM, total[m] - off), m, 0};
        *tab_n = k;
    }
}

}  // namespace

// ================================================================ launchers
// Workgroups of the persistent GEMM grid: the current device's compute units
// (one 256 x 256 tile's workgroup fills a unit's LDS), a multiple of 8 so
// that every tile keeps its XCD.  Looked up once per device.
static int persistent_blocks() {
    static int cached[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
    if (cached[dev] == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus < 8)
            cus = 8;
        cached[dev] = cus / 8 * 8;
    }
    return cached[dev];
}

// Waves along the channels of the 256 x 256 GEMM workgroup (2: four waves of
// 128 x 128; 4: eight waves of 128 x 64, two per SIMD).
constexpr int kGemmWavesN = 4;

// The register-resident stage 1 (stage1_fr_ok shapes): rank 0 (or no
// factors) quantises only.
static hipError_t launch_stage1_fr(const void* x, const int32_t* mod, const float* inv_s,
                                   const void* l_down, int64_t T, int64_t K, int rank, int n_mod,
                                   int8_t* q, float* x_scale, float* u, uint8_t* u_hl,
                                   int* zero_ints, int n_zero, hipStream_t s, bool pair,
                                   const UFinish& fin = UFinish{nullptr, 0, 0, nullptr, nullptr}) {
    const int P = static_cast<int>(((K / 64) + kFrWaves - 1) / kFrWaves);
    // one row group: two (sharing each L1 fragment) need more than a lane's
    // 256 registers from 4 pairs a wave on
    const dim3 grid(static_cast<unsigned>((T + 15) / 16)), block(64 * kFrWaves);
#define MASQ_FR(PP) case PP: hipLaunchKernelGGL((k_stage1_fr<PP, 1>), grid, block, 0, s, \
        static_cast<const bf16_t*>(x), mod, inv_s, static_cast<const bf16_t*>(l_down), T, \
        static_cast<int>(K), rank, n_mod, q, x_scale, u, u_hl, zero_ints, n_zero, fin, pair); break;
    switch (P) {
        MASQ_FR(1) MASQ_FR(2) MASQ_FR(3) MASQ_FR(4) MASQ_FR(5) MASQ_FR(6) MASQ_FR(7) MASQ_FR(8)
        default: return hipErrorInvalidValue;
    }
#undef MASQ_FR
    static_assert(kFrMaxPairs == 8, "one case per pair count");
    return hipGetLastError();
}

hipError_t launch_smooth_quant(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               int64_t T, int64_t K, int n_mod, int8_t* q, float* x_scale,
                               int* zero_ints, int n_zero, hipStream_t s, const UFinish* fin_in,
                               bool pair) {
    const UFinish fin = fin_in ? *fin_in : UFinish{nullptr, 0, 0, nullptr, nullptr};
    if (pair && K % 64 != 0) return hipErrorInvalidValue;
    // (after a split down-projection, fin: the row kernels, whose more
    // numerous workgroups add the slice partials faster)
    if (T > kSmallMaxT && stage1_fr_ok(x_dt, K, n_mod) && fin.part == nullptr)
        return launch_stage1_fr(x, mod, inv_s, nullptr, T, K, 0, n_mod, q, x_scale, nullptr,
                                nullptr, zero_ints, n_zero, s, pair, fin);
    // a wave per row for large batches whose rows fit its register cache
    if (T >= kRowsPerWaveMinT && K <= 64 * 8 * 8) {
        const dim3 grid(static_cast<unsigned>((T + 3) / 4)), block(256);
        if (x_dt == DT::BF16)
            hipLaunchKernelGGL((k_smooth_quant_rows<bf16_t, 8>), grid, block, 0, s,
                               static_cast<const bf16_t*>(x), mod, inv_s, T, static_cast<int>(K),
                               n_mod, q, x_scale, zero_ints, n_zero, fin, pair);
        else
            hipLaunchKernelGGL((k_smooth_quant_rows<float, 8>), grid, block, 0, s,
                               static_cast<const float*>(x), mod, inv_s, T, static_cast<int>(K),
                               n_mod, q, x_scale, zero_ints, n_zero, fin, pair);
        return hipGetLastError();
    }
    const dim3 grid(static_cast<unsigned>(T)), block(256);
    if (x_dt == DT::BF16)
        hipLaunchKernelGGL(k_smooth_quant<bf16_t>, grid, block, 0, s,
                           static_cast<const bf16_t*>(x), mod, inv_s, static_cast<int>(K), n_mod,
                           q, x_scale, zero_ints, n_zero, T, fin, pair);
    else
        hipLaunchKernelGGL(k_smooth_quant<float>, grid, block, 0, s,
                           static_cast<const float*>(x), mod, inv_s, static_cast<int>(K), n_mod,
                           q, x_scale, zero_ints, n_zero, T, fin, pair);
    return hipGetLastError();
}

template <typename XT, typename LT>
static void launch_down_t(const void* x, const int32_t* mod, const float* inv_s, const void* ld,
                          int64_t T, int64_t K, int rank, int n_mod, const Workspace& w,
                          hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((T + kDownRows - 1) / kDownRows),
                    static_cast<unsigned>(w.n_kslices)), block(64 * kDownWaves);
    hipLaunchKernelGGL((k_lowrank_down<XT, LT>), grid, block, 0, s, static_cast<const XT*>(x),
                       mod, inv_s, static_cast<const LT*>(ld), T, static_cast<int>(K), rank,
                       n_mod, w.kslice, w.n_kslices, w.u, w.u_part, w.tickets);
}

hipError_t launch_lowrank_down(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, DT lr_dt, int64_t T, int64_t K, int rank,
                               int n_mod, const Workspace& w, hipStream_t s) {
    if (x_dt == DT::BF16) {
        if (lr_dt == DT::BF16) launch_down_t<bf16_t, bf16_t>(x, mod, inv_s, l_down, T, K, rank, n_mod, w, s);
        else launch_down_t<bf16_t, float>(x, mod, inv_s, l_down, T, K, rank, n_mod, w, s);
    } else {
        if (lr_dt == DT::BF16) launch_down_t<float, bf16_t>(x, mod, inv_s, l_down, T, K, rank, n_mod, w, s);
        else launch_down_t<float, float>(x, mod, inv_s, l_down, T, K, rank, n_mod, w, s);
    }
    return hipGetLastError();
}

hipError_t launch_down_wide(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                            const void* l_down, int64_t T, int64_t K, int rank, int n_mod,
                            const Workspace& w, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((T + kDownWideRows - 1) / kDownWideRows),
                    static_cast<unsigned>(w.dw_slices)), block(256);
    if (x_dt == DT::BF16)
        hipLaunchKernelGGL((k_down_wide<bf16_t>), grid, block, 0, s, static_cast<const bf16_t*>(x),
                           mod, inv_s, static_cast<const bf16_t*>(l_down), T, static_cast<int>(K),
                           rank, n_mod, w.dw_kslice, w.dw_part);
    else
        hipLaunchKernelGGL((k_down_wide<float>), grid, block, 0, s, static_cast<const float*>(x),
                           mod, inv_s, static_cast<const bf16_t*>(l_down), T, static_cast<int>(K),
                           rank, n_mod, w.dw_kslice, w.dw_part);
    return hipGetLastError();
}

hipError_t launch_stage1_fused(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, int64_t T, int64_t K, int rank, int n_mod,
                               int8_t* q, float* x_scale, float* u, uint8_t* u_hl,
                               int* zero_ints, int n_zero, hipStream_t s, bool pair) {
    if (pair && K % 64 != 0) return hipErrorInvalidValue;
    if (stage1_fr_ok(x_dt, K, n_mod))
        return launch_stage1_fr(x, mod, inv_s, l_down, T, K, rank, n_mod, q, x_scale, u, u_hl,
                                zero_ints, n_zero, s, pair);
    // 32 rows per workgroup halve the L1 re-reads once the batch fills the
    // chip at that size; smaller batches keep 16 rows for more workgroups
    const bool wide = T >= kFuseWideMinT;
    const int rows = wide ? 32 : 16;
    const dim3 grid(static_cast<unsigned>((T + rows - 1) / rows)), block(64 * kFuseWaves);
#define MASQ_F1(XT, RG, SL) hipLaunchKernelGGL((k_stage1_fused<XT, RG, SL>), grid, block, 0, s, \
        static_cast<const XT*>(x), mod, inv_s, static_cast<const bf16_t*>(l_down), T, \
        static_cast<int>(K), rank, n_mod, q, x_scale, u, u_hl, zero_ints, n_zero, pair)
    // 32 rows: smoothing factors from LDS when all modalities' fit (bf16
    // activations); 16 rows keep them in registers (their pass 1 was no
    // faster with them in LDS and a deeper load pipeline)
    const bool sl = wide &&
                    ((static_cast<int64_t>(n_mod) * K * 4 + 1023) / 1024) * 1024 <= kFuseInvBytes;
    if (x_dt == DT::BF16) {
        if (sl) MASQ_F1(bf16_t, 2, true);
        else if (wide) MASQ_F1(bf16_t, 2, false);
        else MASQ_F1(bf16_t, 1, false);
    } else {
        if (wide) MASQ_F1(float, 2, false); else MASQ_F1(float, 1, false);
    }
#undef MASQ_F1
    return hipGetLastError();
}

hipError_t launch_down_lds(const void* x, const int32_t* mod, const float* inv_s,
                           const void* l_down, int64_t T, int64_t K, int rank, int n_mod,
                           float* part, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((T + kDlRows - 1) / kDlRows),
                    static_cast<unsigned>(down_lds_slices(T, K))),
        block(64 * kDlWaves);
    hipLaunchKernelGGL(k_down_lds, grid, block, 0, s, static_cast<const bf16_t*>(x), mod, inv_s,
                       static_cast<const bf16_t*>(l_down), T, static_cast<int>(K), rank, n_mod,
                       down_lds_chunks(T, K), part);
    return hipGetLastError();
}

template <typename XT, typename LT>
static void launch_stage1_small_t(const void* x, const int32_t* mod, const float* inv_s,
                                  const void* ld, int64_t T, int64_t K, int rank, int n_mod,
                                  bool cmc, const Workspace& w, hipStream_t s) {
    const unsigned blocks = static_cast<unsigned>(T + (cmc ? w.n_kslices : 0));
    hipLaunchKernelGGL((k_stage1_small<XT, LT>), dim3(blocks), dim3(256), 0, s,
                       static_cast<const XT*>(x), mod, inv_s, cmc ? static_cast<const LT*>(ld) : nullptr,
                       static_cast<int>(T), static_cast<int>(K), rank, n_mod, w.kslice, w.n_kslices,
                       w.q, w.x_scale, w.u, w.u_part, w.dec_tickets,
                       w.dec_tickets ? w.dec_groups : 0);
}

hipError_t launch_stage1_small(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, DT lr_dt, int64_t T, int64_t K, int rank,
                               int n_mod, bool cmc, const Workspace& w, hipStream_t s) {
    if (x_dt == DT::BF16) {
        if (lr_dt == DT::BF16) launch_stage1_small_t<bf16_t, bf16_t>(x, mod, inv_s, l_down, T, K, rank, n_mod, cmc, w, s);
        else launch_stage1_small_t<bf16_t, float>(x, mod, inv_s, l_down, T, K, rank, n_mod, cmc, w, s);
    } else {
        if (lr_dt == DT::BF16) launch_stage1_small_t<float, bf16_t>(x, mod, inv_s, l_down, T, K, rank, n_mod, cmc, w, s);
        else launch_stage1_small_t<float, float>(x, mod, inv_s, l_down, T, K, rank, n_mod, cmc, w, s);
    }
    return hipGetLastError();
}

template <typename YT, typename LT, bool W4>
static void launch_gemm_decode_t(const int8_t* q, const float* x_scale, const int8_t* wq,
                                 const float* w_scale, int64_t T, int64_t K, int64_t N,
                                 const int32_t* mod, const float* u, const float* u_part,
                                 int n_kslices, int rank, int n_mod, const void* r_up,
                                 int32_t* part, int* tickets, void* y, hipStream_t s,
                                 int only_mod = -1) {
    int ns, sp, ngroups;
    plan_decode(K, N, ns, sp, ngroups);
    hipLaunchKernelGGL((k_gemm_decode<YT, LT, W4>), dim3(static_cast<unsigned>(ngroups * ns)), dim3(256),
                       0, s, q, wq, x_scale, w_scale, static_cast<int>(T), static_cast<int>(K),
                       static_cast<int>(N), ns, sp, mod, u, u_part, n_kslices, rank, n_mod,
                       static_cast<const LT*>(r_up), part, tickets, static_cast<YT*>(y), only_mod);
}

hipError_t launch_gemm_decode_mas(const int8_t* q, const float* x_scale, const int8_t* wq,
                                  const float* w_scale, int64_t T, int64_t K, int64_t N,
                                  const int32_t* mod, int n_mod, int32_t* part, int* tickets,
                                  void* y, DT y_dt, hipStream_t s) {
    int ns = 0, sp = 0, ng = 0;
    if (!small_path(T, K)) return hipErrorInvalidValue;
    plan_decode(K, N, ns, sp, ng);
    if (ns > kDecMaxSlices) return hipErrorInvalidValue;
    for (int m = 0; m < n_mod; ++m) {
        const int8_t* wm = wq + static_cast<int64_t>(m) * N * K;
        const float* sm = w_scale + static_cast<int64_t>(m) * N;
        if (y_dt == DT::BF16)
            launch_gemm_decode_t<bf16_t, bf16_t, false>(q, x_scale, wm, sm, T, K, N, mod, nullptr,
                                                         nullptr, 1, 0, n_mod, nullptr, part,
                                                         tickets, y, s, m);
        else
            launch_gemm_decode_t<float, bf16_t, false>(q, x_scale, wm, sm, T, K, N, mod, nullptr,
                                                        nullptr, 1, 0, n_mod, nullptr, part,
                                                        tickets, y, s, m);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <typename YT, typename LT, bool W4>
static void launch_gemm_small_t(const int8_t* q, const float* x_scale, const int8_t* wq,
                                const float* w_scale, int64_t T, int64_t K, int64_t N,
                                const int32_t* mod, const float* u, const float* u_part,
                                int n_kslices, int rank, int n_mod, const void* r_up, int32_t* acc,
                                void* y, hipStream_t s) {
    hipLaunchKernelGGL((k_gemm_small<YT, LT, W4>), dim3(static_cast<unsigned>(N / 16)), dim3(256), 0, s,
                       q, wq, x_scale, w_scale, static_cast<int>(T), static_cast<int>(K),
                       static_cast<int>(N), mod, u, u_part, n_kslices, rank, n_mod,
                       static_cast<const LT*>(r_up), acc, static_cast<YT*>(y));
}

template <typename YT, typename LT, bool CMC, bool ACC, bool W4>
static void launch_gemm_t(const int8_t* q, const float* x_scale, const int8_t* wq,
                          const float* w_scale, int64_t T, int64_t K, int64_t N,
                          const int32_t* mod, const float* u, const uint8_t* u_hl, int rank,
                          int n_mod, const void* r_up, int32_t* acc, void* y, int S,
                          int32_t* part, int* tickets, hipStream_t s, bool a_pair) {
    const int tiles_m = static_cast<int>((T + kTileM - 1) / kTileM);
    const int tiles_n = static_cast<int>((N + kTileN - 1) / kTileN);
    const int nt = tiles_m * tiles_n;
    const dim3 grid(8 * ((nt + 7) / 8)), block(256);
    if (K % kDmaStageK == 0) {
        if (part == nullptr || tickets == nullptr) S = 1;
        const dim3 gridk(8 * ((nt * S + 7) / 8));
        // whole tiles: a persistent grid of at most one workgroup per compute unit
        const dim3 gridp(static_cast<unsigned>(min(8 * ((nt + 7) / 8), persistent_blocks())));
        if (S > 1)
            hipLaunchKernelGGL((k_gemm_dma<YT, LT, CMC, ACC, kGemmWavesN, true, W4>), gridk,
                               dim3(128 * kGemmWavesN), 0, s, q, wq, x_scale, w_scale, T,
                               static_cast<int>(K), static_cast<int>(N), tiles_m, tiles_n, mod, u,
                               u_hl, rank, n_mod, static_cast<const LT*>(r_up), acc,
                               static_cast<YT*>(y), S, part, tickets, nullptr, nullptr, nullptr, 0,
                               a_pair);
        else
            hipLaunchKernelGGL((k_gemm_dma<YT, LT, CMC, ACC, kGemmWavesN, false, W4, false, true>), gridp,
                               dim3(128 * kGemmWavesN), 0, s, q, wq, x_scale, w_scale, T,
                               static_cast<int>(K), static_cast<int>(N), tiles_m, tiles_n, mod, u,
                               u_hl, rank, n_mod, static_cast<const LT*>(r_up), acc,
                               static_cast<YT*>(y), 1, nullptr, nullptr, nullptr, nullptr, nullptr, 0,
                               a_pair);
    } else if constexpr (!W4)
        hipLaunchKernelGGL((k_gemm<YT, LT, CMC, ACC>), grid, block, 0, s, q, wq, x_scale, w_scale, T,
                           static_cast<int>(K), static_cast<int>(N), tiles_m, tiles_n, mod, u,
                           rank, n_mod, static_cast<const LT*>(r_up), acc, static_cast<YT*>(y));
}

hipError_t launch_group_rows(const int32_t* mod, int64_t T, int n_mod, int32_t* rows,
                             int32_t* tab, int* tab_n, int* zero_ints, int n_zero, hipStream_t s) {
    hipLaunchKernelGGL(k_group_rows, dim3(1), dim3(kGrpThreads), 0, s, mod, T, n_mod, rows,
                       reinterpret_cast<v4i*>(tab), tab_n, zero_ints, n_zero);
    return hipGetLastError();
}

template <typename YT>
static void launch_gemm_grouped_t(const int8_t* q, const float* x_scale, const int8_t* wq,
                                  const float* w_scale, int64_t T, int64_t K, int64_t N,
                                  int n_mod, const int32_t* rows, const int32_t* tab,
                                  const int* tab_n, void* y, int S, int32_t* part, int* tickets,
                                  hipStream_t s) {
    const int tiles_m = grouped_tab_max(T, n_mod);
    const int tiles_n = static_cast<int>((N + kTileN - 1) / kTileN);
    const dim3 grid(8 * ((tiles_m * tiles_n * S + 7) / 8)), block(128 * kGemmWavesN);
    const v4i* tb = reinterpret_cast<const v4i*>(tab);
    if (S > 1)
        hipLaunchKernelGGL((k_gemm_dma<YT, bf16_t, false, false, kGemmWavesN, true, false, true>), grid,
                           block, 0, s, q, wq, x_scale, w_scale, T, static_cast<int>(K),
                           static_cast<int>(N), tiles_m, tiles_n, nullptr, nullptr, nullptr, 0, n_mod,
                           nullptr, nullptr, static_cast<YT*>(y), S, part, tickets, rows, tb, tab_n,
                           N * K, true);
    else
        hipLaunchKernelGGL((k_gemm_dma<YT, bf16_t, false, false, kGemmWavesN, false, false, true>), grid,
                           block, 0, s, q, wq, x_scale, w_scale, T, static_cast<int>(K),
                           static_cast<int>(N), tiles_m, tiles_n, nullptr, nullptr, nullptr, 0, n_mod,
                           nullptr, nullptr, static_cast<YT*>(y), 1, nullptr, nullptr, rows, tb,
                           tab_n, N * K, true);
}

hipError_t launch_gemm_grouped(const int8_t* q, const float* x_scale, const int8_t* wq,
                               const float* w_scale, int64_t T, int64_t K, int64_t N, int n_mod,
                               const int32_t* rows, const int32_t* tab, const int* tab_n, void* y,
                               DT y_dt, int S, int32_t* part, int* tickets, hipStream_t s) {
    if (K % kDmaStageK != 0) return hipErrorInvalidValue;
    if (part == nullptr || tickets == nullptr) S = 1;
    if (y_dt == DT::BF16)
        launch_gemm_grouped_t<bf16_t>(q, x_scale, wq, w_scale, T, K, N, n_mod, rows, tab, tab_n, y,
                                      S, part, tickets, s);
    else
        launch_gemm_grouped_t<float>(q, x_scale, wq, w_scale, T, K, N, n_mod, rows, tab, tab_n, y,
                                     S, part, tickets, s);
    return hipGetLastError();
}

hipError_t launch_gemm(const int8_t* q, const float* x_scale, const int8_t* wq,
                       const float* w_scale, int64_t T, int64_t K, int64_t N,
                       const int32_t* mod, const float* u, const uint8_t* u_hl,
                       int32_t* dec_part, int* dec_tickets, int gk_splits, int32_t* gk_part,
                       int* gk_tickets, const float* u_part, int n_kslices,
                       int rank, int n_mod, const void* r_up, DT lr_dt, bool cmc, int32_t* acc,
                       void* y, DT y_dt, hipStream_t s, bool w4, bool a_pair) {
    // packed 4-bit Wq: K % 64 == 0 (checked by the caller), so every batch
    // takes the decode, small-batch or direct-to-LDS kernel
    if (w4 && K % 64 != 0) return hipErrorInvalidValue;
    // row-paired codes are read by the direct-to-LDS GEMM only
    if (a_pair && !paired_codes(T, K)) return hipErrorInvalidValue;
    int dns = 0, dsp = 0, dng = 0;
    if (small_path(T, K)) plan_decode(K, N, dns, dsp, dng);
    if (small_path(T, K) && dec_part != nullptr && dec_tickets != nullptr && acc == nullptr &&
        dns <= kDecMaxSlices) {
        const float* uu = cmc ? u : nullptr;
#define MASQ_DEC(YT, LT) (w4 ? launch_gemm_decode_t<YT, LT, true> : launch_gemm_decode_t<YT, LT, false>)(q, x_scale, wq, w_scale, T, K, N, mod, uu, u_part, n_kslices, rank, n_mod, r_up, dec_part, dec_tickets, y, s, -1)
        if (y_dt == DT::BF16) {
            if (lr_dt == DT::BF16) MASQ_DEC(bf16_t, bf16_t);
            else MASQ_DEC(bf16_t, float);
        } else {
            if (lr_dt == DT::BF16) MASQ_DEC(float, bf16_t);
            else MASQ_DEC(float, float);
        }
#undef MASQ_DEC
        return hipGetLastError();
    }
    if (small_path(T, K)) {
        const float* uu = cmc ? u : nullptr;
#define MASQ_SMALL(YT, LT) (w4 ? launch_gemm_small_t<YT, LT, true> : launch_gemm_small_t<YT, LT, false>)(q, x_scale, wq, w_scale, T, K, N, mod, uu, u_part, n_kslices, rank, n_mod, r_up, acc, y, s)
        if (y_dt == DT::BF16) {
            if (lr_dt == DT::BF16) MASQ_SMALL(bf16_t, bf16_t);
            else MASQ_SMALL(bf16_t, float);
        } else {
            if (lr_dt == DT::BF16) MASQ_SMALL(float, bf16_t);
            else MASQ_SMALL(float, float);
        }
#undef MASQ_SMALL
        return hipGetLastError();
    }
#define MASQ_GEMM(YT, LT, C, A) (w4 ? launch_gemm_t<YT, LT, C, A, true> : launch_gemm_t<YT, LT, C, A, false>)(q, x_scale, wq, w_scale, T, K, N, mod, u, u_hl, rank, n_mod, r_up, acc, y, gk_splits, gk_part, gk_tickets, s, a_pair)
    // the int32 accumulator output exists only for the plain product (no
    // compensation); it is a separate instantiation because storing the
    // accumulators as well raises the epilogue's register pressure
    if (!cmc) {
        if (acc != nullptr) {
            if (y_dt == DT::BF16) MASQ_GEMM(bf16_t, bf16_t, false, true);
            else MASQ_GEMM(float, bf16_t, false, true);
        } else {
            if (y_dt == DT::BF16) MASQ_GEMM(bf16_t, bf16_t, false, false);
            else MASQ_GEMM(float, bf16_t, false, false);
        }
    } else if (y_dt == DT::BF16) {
        if (lr_dt == DT::BF16) MASQ_GEMM(bf16_t, bf16_t, true, false);
        else MASQ_GEMM(bf16_t, float, true, false);
    } else {
        if (lr_dt == DT::BF16) MASQ_GEMM(float, bf16_t, true, false);
        else MASQ_GEMM(float, float, true, false);
    }
#undef MASQ_GEMM
    return hipGetLastError();
}

template <typename XT, typename LT, typename YT>
static void launch_comp_t(const void* x, const int32_t* mod, const float* inv_s, const void* ld,
                          const void* ru, int64_t T, int64_t K, int64_t N, int rank, int n_mod,
                          void* y, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((T + kRowsDown - 1) / kRowsDown)), block(256);
    hipLaunchKernelGGL((k_lowrank_comp<XT, LT, YT>), grid, block, 0, s,
                       static_cast<const XT*>(x), mod, inv_s, static_cast<const LT*>(ld),
                       static_cast<const LT*>(ru), T, static_cast<int>(K), static_cast<int>(N),
                       rank, n_mod, static_cast<YT*>(y));
}

hipError_t launch_lowrank_comp(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, const void* r_up, DT lr_dt, int64_t T,
                               int64_t K, int64_t N, int rank, int n_mod, void* y, DT y_dt,
                               hipStream_t s) {
#define MASQ_COMP(XT, LT, YT) launch_comp_t<XT, LT, YT>(x, mod, inv_s, l_down, r_up, T, K, N, rank, n_mod, y, s)
    const int key = (x_dt == DT::BF16 ? 4 : 0) | (lr_dt == DT::BF16 ? 2 : 0) | (y_dt == DT::BF16 ? 1 : 0);
    switch (key) {
        case 0: MASQ_COMP(float, float, float); break;
        case 1: MASQ_COMP(float, float, bf16_t); break;
        case 2: MASQ_COMP(float, bf16_t, float); break;
        case 3: MASQ_COMP(float, bf16_t, bf16_t); break;
        case 4: MASQ_COMP(bf16_t, float, float); break;
        case 5: MASQ_COMP(bf16_t, float, bf16_t); break;
        case 6: MASQ_COMP(bf16_t, bf16_t, float); break;
        default: MASQ_COMP(bf16_t, bf16_t, bf16_t); break;
    }
#undef MASQ_COMP
    return hipGetLastError();
}

}  // namespace masq
