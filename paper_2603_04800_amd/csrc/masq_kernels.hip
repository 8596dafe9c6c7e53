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

// Round-to-nearest-even narrowing of a finite fp32 value to bf16 bits.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

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

// ================================================================ smoothing + quant
template <typename XT>
__global__ __launch_bounds__(256) void k_smooth_quant(const XT* __restrict__ x,
                                                      const int32_t* __restrict__ mod,
                                                      const float* __restrict__ inv_s, int K,
                                                      int n_mod, int8_t* __restrict__ q,
                                                      float* __restrict__ x_scale) {
    __shared__ float red[4];
    const int64_t t = blockIdx.x;
    const int m = sane_mod(mod[t], n_mod);
    const XT* xr = x + t * static_cast<int64_t>(K);
    const float* sr = inv_s + static_cast<int64_t>(m) * K;
    const int nv = K >> 3;

    float amax = 0.f;
    for (int v = threadIdx.x; v < nv; v += 256) {
        float xv[8], sv[8];
        Elem<XT>::load8(xr + 8 * v, xv);
        load8_f32(sr + 8 * v, sv);
#pragma unroll
        for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(xv[j] * sv[j]));
    }
    amax = wave_max(amax);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
    __syncthreads();
    amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));

    const bool nz = amax > 0.f;
    const float dx = nz ? amax / 127.0f : 0.f;     // correctly rounded
    const float rq = nz ? 127.0f / amax : 0.f;
    if (threadIdx.x == 0) x_scale[t] = dx;

    int8_t* qr = q + t * static_cast<int64_t>(K);
    for (int v = threadIdx.x; v < nv; v += 256) {
        float xv[8], sv[8];
        Elem<XT>::load8(xr + 8 * v, xv);
        load8_f32(sr + 8 * v, sv);
        uint32_t w[2] = {0u, 0u};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float xs = xv[j] * sv[j];
            float c = rintf(xs * rq);
            c = fminf(fmaxf(c, -127.0f), 127.0f);
            w[j >> 2] |= (static_cast<uint32_t>(static_cast<int32_t>(c)) & 0xFFu) << (8 * (j & 3));
        }
        v2i out;
        out.x = static_cast<int32_t>(w[0]);
        out.y = static_cast<int32_t>(w[1]);
        *reinterpret_cast<v2i*>(qr + 8 * v) = out;
    }
}

// ================================================================ down-projection
// One 16 x 16 block of u = (x S_m^-1) L1^m over k in [kb, ke): 16 token rows
// (row0..row0+15) times 16 rank columns (c0..c0+15).  Rows whose modality is
// not m contribute zeros.  MFMA operand layout: lane l holds row/column
// (l % 16) and the k group (l / 16); A and B use the same k assignment.
template <typename XT, typename LT> struct Down;

template <typename XT> struct Down<XT, bf16_t> {   // bf16 factors: bf16 MFMA
    static __device__ __forceinline__ v4f block(const XT* x, const float* inv_s_m,
                                                const bf16_t* ld_m, int64_t row0, int64_t T,
                                                int K, int kb, int ke, int c0, const int* smod,
                                                int m, v4f acc, int lane) {
        const int ar = lane & 15, kg = lane >> 4;
        const int64_t t = row0 + ar;
        const bool live = (t < T) && (smod[ar] == m);
        const XT* xrow = x + (live ? t : row0) * static_cast<int64_t>(K);
        const bf16_t* lrow = ld_m + static_cast<int64_t>(c0 + ar) * K;
        for (int k0 = kb; k0 < ke; k0 += 32) {
            const int k = k0 + 8 * kg;
            v4i av = {0, 0, 0, 0};
            v4i bv = {0, 0, 0, 0};
            if (k < ke) {
                bv = *reinterpret_cast<const v4i*>(lrow + k);
                if (live) {
                    float xv[8], sv[8];
                    Elem<XT>::load8(xrow + k, xv);
                    load8_f32(inv_s_m + k, sv);
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const uint32_t lo = f32_to_bf16(xv[2 * j] * sv[2 * j]);
                        const uint32_t hi = f32_to_bf16(xv[2 * j + 1] * sv[2 * j + 1]);
                        av[j] = static_cast<int32_t>(lo | (hi << 16));
                    }
                }
            }
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, av),
                                                          __builtin_bit_cast(v8bf, bv), acc, 0, 0, 0);
        }
        return acc;
    }
};

template <typename XT> struct Down<XT, float> {    // fp32 factors: fp32 MFMA
    static __device__ __forceinline__ v4f block(const XT* x, const float* inv_s_m,
                                                const float* ld_m, int64_t row0, int64_t T,
                                                int K, int kb, int ke, int c0, const int* smod,
                                                int m, v4f acc, int lane) {
        const int ar = lane & 15, kg = lane >> 4;
        const int64_t t = row0 + ar;
        const bool live = (t < T) && (smod[ar] == m);
        const XT* xrow = x + (live ? t : row0) * static_cast<int64_t>(K);
        const float* lrow = ld_m + static_cast<int64_t>(c0 + ar) * K;
        for (int k0 = kb; k0 < ke; k0 += 4) {
            const int k = k0 + kg;
            float a = 0.f, b = 0.f;
            if (k < ke) {
                b = lrow[k];
                if (live) a = Elem<XT>::load1(xrow + k) * inv_s_m[k];
            }
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
        }
        return acc;
    }
};

// Sum over the modalities present in the tile of one 16 x 16 block of u.
template <typename XT, typename LT>
__device__ __forceinline__ v4f down_tile(const XT* x, const float* inv_s, const LT* l_down,
                                         int64_t row0, int64_t T, int K, int r, int n_mod,
                                         int kb, int ke, int c0, const int* smod,
                                         unsigned present, int lane) {
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    for (int m = 1; m < n_mod; ++m) {
        if (!(present & (1u << m))) continue;
        acc = Down<XT, LT>::block(x, inv_s + static_cast<int64_t>(m) * K,
                                  l_down + static_cast<int64_t>(m - 1) * r * K, row0, T, K, kb,
                                  ke, c0, smod, m, acc, lane);
    }
    return acc;
}

__device__ __forceinline__ unsigned tile_presence(const int* smod) {
    unsigned present = 0;
#pragma unroll
    for (int i = 0; i < kRowsDown; ++i)
        if (smod[i] > 0) present |= 1u << smod[i];
    return present;
}

// grid: (ceil(T / 16), n_kslices); u[s][t][c] partial over k-slice s.
template <typename XT, typename LT>
__global__ __launch_bounds__(256) void k_lowrank_down(const XT* __restrict__ x,
                                                      const int32_t* __restrict__ mod,
                                                      const float* __restrict__ inv_s,
                                                      const LT* __restrict__ l_down, int64_t T,
                                                      int K, int r, int n_mod, int kslice,
                                                      float* __restrict__ u) {
    __shared__ int smod[kRowsDown];
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kRowsDown;
    const int s = blockIdx.y;
    const int kb = s * kslice;
    const int ke = min(K, kb + kslice);
    if (threadIdx.x < kRowsDown) {
        const int64_t t = row0 + threadIdx.x;
        smod[threadIdx.x] = t < T ? sane_mod(mod[t], n_mod) : 0;
    }
    __syncthreads();
    const unsigned present = tile_presence(smod);
    if (!present) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int c0 = wave * 16; c0 < r; c0 += 64) {
        const v4f acc = down_tile<XT, LT>(x, inv_s, l_down, row0, T, K, r, n_mod, kb, ke, c0,
                                          smod, present, lane);
        const int col = c0 + (lane & 15);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t t = row0 + 4 * (lane >> 4) + i;
            if (t < T) u[(static_cast<int64_t>(s) * T + t) * r + col] = acc[i];
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
    __shared__ float su[kRowsDown][kMaxRank];
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kRowsDown;
    if (threadIdx.x < kRowsDown) {
        const int64_t t = row0 + threadIdx.x;
        smod[threadIdx.x] = t < T ? sane_mod(mod[t], n_mod) : 0;
    }
    __syncthreads();
    const unsigned present = tile_presence(smod);
    if (!present) return;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int c0 = wave * 16; c0 < r; c0 += 64) {
        const v4f acc = down_tile<XT, LT>(x, inv_s, l_down, row0, T, K, r, n_mod, 0, K, c0,
                                          smod, present, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i) su[4 * (lane >> 4) + i][c0 + (lane & 15)] = acc[i];
    }
    __syncthreads();
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

// Cross-Modal Compensation inside the GEMM epilogue.  For each modality m
// present in the tile and each chunk of up to 64 rank columns ("piece"), the
// u rows of that modality (others zero) and the matching rows of L2^T are
// staged in LDS; each 32 x 32 output block then accumulates u L2 onto its
// dequantised fp32 values with MFMA.  Pieces that do not fit in the 128 KB of
// LDS are read straight from global memory instead.
template <typename LT> struct Cmc;

template <> struct Cmc<bf16_t> {          // bf16 operands, v_mfma_f32_32x32x16_bf16
    static constexpr int kPieceBytes = 2 * kTileM * 128;    // u + L2^T, 128-byte rows

    static __device__ __forceinline__ void stage(uint8_t* piece, const int* s_mod, int m,
                                                 const float* u, const bf16_t* rm, int64_t row0,
                                                 int64_t T, int col0, int N, int r, int c0,
                                                 int tid) {
        uint8_t* su = piece;
        uint8_t* sr = piece + kTileM * 128;
        const int nch = min(64, r - c0) >> 3;
        for (int idx = tid; idx < kTileM * 8; idx += 256) {
            const int row = idx >> 3, ch = idx & 7;
            const int64_t t = row0 + row;
            v4i pk = {0, 0, 0, 0}, pr = {0, 0, 0, 0};
            if (ch < nch) {
                if (t < T && s_mod[row] == m) {
                    float uv[8];
                    load8_f32(u + t * r + c0 + 8 * ch, uv);
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        pk[j] = static_cast<int32_t>(f32_to_bf16(uv[2 * j]) |
                                                     (f32_to_bf16(uv[2 * j + 1]) << 16));
                }
                const int col = min(col0 + row, N - 1);
                pr = *reinterpret_cast<const v4i*>(rm + static_cast<int64_t>(col) * r + c0 + 8 * ch);
            }
            const int off = row * 128 + ((ch ^ swz(row)) << 4);
            *reinterpret_cast<v4i*>(su + off) = pk;
            *reinterpret_cast<v4i*>(sr + off) = pr;
        }
    }

    // yb += u[rows of block i] . L2^T[cols of block j] over this piece's columns.
    static __device__ __forceinline__ v16f from_lds(const uint8_t* piece, int rc, int arow,
                                                    int brow, int lane, v16f yb) {
        const uint8_t* su = piece;
        const uint8_t* sr = piece + kTileM * 128;
        for (int ks = 0; ks < (rc >> 4); ++ks) {
            const int c = 2 * ks + (lane >> 5);
            const v4i fa = *reinterpret_cast<const v4i*>(su + arow * 128 + ((c ^ swz(arow)) << 4));
            const v4i fb = *reinterpret_cast<const v4i*>(sr + brow * 128 + ((c ^ swz(brow)) << 4));
            yb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, fa),
                                                         __builtin_bit_cast(v8bf, fb), yb, 0, 0, 0);
        }
        return yb;
    }

    static __device__ __forceinline__ v16f from_global(const float* u, const bf16_t* rm, int m,
                                                       int smod_row, int64_t t, int64_t T,
                                                       int col, int r, int c0, int lane, v16f yb) {
        const int rc = min(64, r - c0);
        const bool live = t < T && smod_row == m;
        for (int ks = 0; ks < (rc >> 4); ++ks) {
            const int k = c0 + 16 * ks + 8 * (lane >> 5);
            v4i fa = {0, 0, 0, 0};
            if (live) {
                float uv[8];
                load8_f32(u + t * r + k, uv);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    fa[j] = static_cast<int32_t>(f32_to_bf16(uv[2 * j]) | (f32_to_bf16(uv[2 * j + 1]) << 16));
            }
            const v4i fb = *reinterpret_cast<const v4i*>(rm + static_cast<int64_t>(col) * r + k);
            yb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, fa),
                                                         __builtin_bit_cast(v8bf, fb), yb, 0, 0, 0);
        }
        return yb;
    }
};

template <> struct Cmc<float> {           // fp32 operands, v_mfma_f32_32x32x2f32
    static constexpr int kPieceBytes = 2 * kTileM * 256;    // u + L2^T, 64 floats per row

    static __device__ __forceinline__ void stage(uint8_t* piece, const int* s_mod, int m,
                                                 const float* u, const float* rm, int64_t row0,
                                                 int64_t T, int col0, int N, int r, int c0,
                                                 int tid) {
        float* su = reinterpret_cast<float*>(piece);
        float* sr = reinterpret_cast<float*>(piece + kTileM * 256);
        const int rc = min(64, r - c0);
        for (int idx = tid; idx < kTileM * rc; idx += 256) {
            const int row = idx / rc, k = idx - row * rc;
            const int64_t t = row0 + row;
            su[row * 64 + k] = (t < T && s_mod[row] == m) ? u[t * r + c0 + k] : 0.f;
            const int col = min(col0 + row, N - 1);
            sr[row * 64 + k] = rm[static_cast<int64_t>(col) * r + c0 + k];
        }
    }

    static __device__ __forceinline__ v16f from_lds(const uint8_t* piece, int rc, int arow,
                                                    int brow, int lane, v16f yb) {
        const float* su = reinterpret_cast<const float*>(piece);
        const float* sr = reinterpret_cast<const float*>(piece + kTileM * 256);
        for (int ks = 0; ks < (rc >> 1); ++ks) {
            const int k = 2 * ks + (lane >> 5);
            yb = __builtin_amdgcn_mfma_f32_32x32x2f32(su[arow * 64 + k], sr[brow * 64 + k], yb, 0, 0, 0);
        }
        return yb;
    }

    static __device__ __forceinline__ v16f from_global(const float* u, const float* rm, int m,
                                                       int smod_row, int64_t t, int64_t T,
                                                       int col, int r, int c0, int lane, v16f yb) {
        const int rc = min(64, r - c0);
        const bool live = t < T && smod_row == m;
        for (int ks = 0; ks < (rc >> 1); ++ks) {
            const int k = c0 + 2 * ks + (lane >> 5);
            const float a = live ? u[t * r + k] : 0.f;
            yb = __builtin_amdgcn_mfma_f32_32x32x2f32(a, rm[static_cast<int64_t>(col) * r + k], yb, 0, 0, 0);
        }
        return yb;
    }
};

template <typename YT, typename LT, bool CMC>
__global__ __launch_bounds__(256, 1) void k_gemm(
    const int8_t* __restrict__ A, const int8_t* __restrict__ B, const float* __restrict__ x_scale,
    const float* __restrict__ w_scale, int64_t T, int K, int N, int tiles_m, int tiles_n,
    const int32_t* __restrict__ mod, const float* __restrict__ u, int r, int n_mod,
    const LT* __restrict__ r_up, int32_t* __restrict__ acc_out, YT* __restrict__ y) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * 65536];
    __shared__ float s_dx[kTileM];
    __shared__ float s_ws[kTileN];
    __shared__ int s_mod[kTileM];
    __shared__ unsigned s_present;

    // Workgroups are dealt round-robin to the 8 XCDs; give each XCD a
    // contiguous range of tiles, ordered in groups of 8 tile-rows, so that
    // tiles running together on one XCD share A and B stages in its L2.
    const int nt = tiles_m * tiles_n;
    const int per_xcd = (nt + 7) >> 3;
    const int L = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (L >= nt) return;
    constexpr int GM = 8;
    const int gsize = GM * tiles_n;
    const int g = L / gsize;
    const int first_m = g * GM;
    const int gm = min(GM, tiles_m - first_m);
    const int li = L - g * gsize;
    const int tm = first_m + li % gm;
    const int tn = li / gm;
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

    v4i ra[8], rb[8];
    // Row indices are clamped into the matrix (rows past T or N are computed
    // and discarded); chunks past K are loaded from a clamped in-bounds
    // address and replaced by zeros, so every load is unconditional.
    int64_t a_off[8], b_off[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        a_off[j] = min(row0 + lr + 32 * j, T - 1) * K;
        b_off[j] = static_cast<int64_t>(min(col0 + lr + 32 * j, N - 1)) * K;
    }
    auto gload = [&](int k0) {
        const int kraw = k0 + lc * 16;
        const bool kin = kraw < K;
        const int kk = kin ? kraw : K - 16;
        const v4i zero = {0, 0, 0, 0};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const v4i va = *reinterpret_cast<const v4i*>(A + a_off[j] + kk);
            const v4i vb = *reinterpret_cast<const v4i*>(B + b_off[j] + kk);
            ra[j] = kin ? va : zero;
            rb[j] = kin ? vb : zero;
        }
    };
    auto sstore = [&](int buf) {
        uint8_t* sa = smem + buf * 65536;
        uint8_t* sb = sa + 32768;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int row = lr + 32 * j;
            const int off = row * 128 + ((lc ^ swz(row)) << 4);
            *reinterpret_cast<v4i*>(sa + off) = ra[j];
            *reinterpret_cast<v4i*>(sb + off) = rb[j];
        }
    };

    const int nk = (K + kTileK - 1) / kTileK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * kTileK);
        const uint8_t* sa = smem + cur * 65536;
        const uint8_t* sb = sa + 32768;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int c = 2 * ks + (lane >> 5);
            v4i fa[4], fb[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = wm * 128 + i * 32 + (lane & 31);
                fa[i] = *reinterpret_cast<const v4i*>(sa + row * 128 + ((c ^ swz(row)) << 4));
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = wn * 128 + j * 32 + (lane & 31);
                fb[j] = *reinterpret_cast<const v4i*>(sb + row * 128 + ((c ^ swz(row)) << 4));
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) sstore(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue: scales and modalities of this tile
    {
        const int64_t t = row0 + tid;
        s_dx[tid] = t < T ? x_scale[t] : 0.f;
        s_ws[tid] = (col0 + tid) < N ? w_scale[col0 + tid] : 0.f;
        if (CMC) s_mod[tid] = t < T ? sane_mod(mod[t], n_mod) : 0;
        if (tid == 0) s_present = 0u;
    }
    __syncthreads();

    // ---- compensation pieces: (modality, 64-column chunk) pairs present here
    int n_pieces = 0;
    bool staged = false;
    unsigned present = 0;
    const int n_chunks = (r + 63) >> 6;
    if constexpr (CMC) {
        if (s_mod[tid] > 0) atomicOr(&s_present, 1u << s_mod[tid]);
        __syncthreads();
        present = s_present;
        n_pieces = __builtin_popcount(present) * n_chunks;
        staged = n_pieces * Cmc<LT>::kPieceBytes <= static_cast<int>(sizeof(smem));
        if (n_pieces > 0 && staged && y != nullptr) {
            int p = 0;
            for (int m = 1; m < n_mod; ++m) {
                if (!(present & (1u << m))) continue;
                const LT* rm = r_up + static_cast<int64_t>(m - 1) * N * r;
                for (int c = 0; c < n_chunks; ++c, ++p)
                    Cmc<LT>::stage(smem + p * Cmc<LT>::kPieceBytes, s_mod, m, u, rm, row0, T,
                                   col0, N, r, 64 * c, tid);
            }
            __syncthreads();
        }
    }

    // ---- per 32 x 32 block: (int32 store), dequantise, compensate, cast, store.
    // Invoked with constant block indices so the accumulators stay in registers.
    const bool interior = (row0 + kTileM <= T) && (col0 + kTileN <= N);
    auto epilogue_block = [&](const int i, const int j, const v16i a) __attribute__((always_inline)) {
        const int arow = wm * 128 + i * 32 + (lane & 31);   // A-operand row of this lane
        const int bcol = wn * 128 + j * 32 + (lane & 31);
        const int col = col0 + bcol;
        if (acc_out != nullptr) {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t row = row0 + wm * 128 + i * 32 + acc_row(e, lane);
                if (interior || (row < T && col < N)) acc_out[row * N + col] = a[e];
            }
        }
        if (y == nullptr) return;
        const float ws = s_ws[bcol];
        v16f yb;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const float dx = s_dx[wm * 128 + i * 32 + acc_row(e, lane)];
            yb[e] = (static_cast<float>(a[e]) * dx) * ws;
        }
        if constexpr (CMC) {
            if (n_pieces > 0) {
                int p = 0;
                for (int m = 1; m < n_mod; ++m) {
                    if (!(present & (1u << m))) continue;
                    const LT* rm = r_up + static_cast<int64_t>(m - 1) * N * r;
                    for (int c = 0; c < n_chunks; ++c, ++p) {
                        if (staged)
                            yb = Cmc<LT>::from_lds(smem + p * Cmc<LT>::kPieceBytes,
                                                   min(64, r - 64 * c), arow, bcol, lane, yb);
                        else
                            yb = Cmc<LT>::from_global(u, rm, m, s_mod[arow], row0 + arow, T,
                                                      min(col, N - 1), r, 64 * c, lane, yb);
                    }
                }
            }
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int64_t row = row0 + wm * 128 + i * 32 + acc_row(e, lane);
            if (interior || (row < T && col < N)) Elem<YT>::store1(y + row * N + col, yb[e]);
        }
    };
#define MASQ_EPI_ROW(I) epilogue_block(I, 0, acc[I][0]); epilogue_block(I, 1, acc[I][1]); \
                        epilogue_block(I, 2, acc[I][2]); epilogue_block(I, 3, acc[I][3]);
    MASQ_EPI_ROW(0) MASQ_EPI_ROW(1) MASQ_EPI_ROW(2) MASQ_EPI_ROW(3)
#undef MASQ_EPI_ROW
}

}  // namespace

// ================================================================ launchers
hipError_t launch_smooth_quant(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               int64_t T, int64_t K, int n_mod, int8_t* q, float* x_scale,
                               hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(T)), block(256);
    if (x_dt == DT::BF16)
        hipLaunchKernelGGL(k_smooth_quant<bf16_t>, grid, block, 0, s,
                           static_cast<const bf16_t*>(x), mod, inv_s, static_cast<int>(K), n_mod,
                           q, x_scale);
    else
        hipLaunchKernelGGL(k_smooth_quant<float>, grid, block, 0, s,
                           static_cast<const float*>(x), mod, inv_s, static_cast<int>(K), n_mod,
                           q, x_scale);
    return hipGetLastError();
}

template <typename XT, typename LT>
static void launch_down_t(const void* x, const int32_t* mod, const float* inv_s, const void* ld,
                          int64_t T, int64_t K, int rank, int n_mod, int kslice, int nks,
                          float* u, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((T + kRowsDown - 1) / kRowsDown), nks), block(256);
    hipLaunchKernelGGL((k_lowrank_down<XT, LT>), grid, block, 0, s, static_cast<const XT*>(x),
                       mod, inv_s, static_cast<const LT*>(ld), T, static_cast<int>(K), rank,
                       n_mod, kslice, u);
}

hipError_t launch_lowrank_down(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, DT lr_dt, int64_t T, int64_t K, int rank,
                               int n_mod, int kslice, int n_kslices, float* u, hipStream_t s) {
    if (x_dt == DT::BF16) {
        if (lr_dt == DT::BF16) launch_down_t<bf16_t, bf16_t>(x, mod, inv_s, l_down, T, K, rank, n_mod, kslice, n_kslices, u, s);
        else launch_down_t<bf16_t, float>(x, mod, inv_s, l_down, T, K, rank, n_mod, kslice, n_kslices, u, s);
    } else {
        if (lr_dt == DT::BF16) launch_down_t<float, bf16_t>(x, mod, inv_s, l_down, T, K, rank, n_mod, kslice, n_kslices, u, s);
        else launch_down_t<float, float>(x, mod, inv_s, l_down, T, K, rank, n_mod, kslice, n_kslices, u, s);
    }
    return hipGetLastError();
}

template <typename YT, typename LT, bool CMC>
static void launch_gemm_t(const int8_t* q, const float* x_scale, const int8_t* wq,
                          const float* w_scale, int64_t T, int64_t K, int64_t N,
                          const int32_t* mod, const float* u, int rank, int n_mod,
                          const void* r_up, int32_t* acc, void* y, hipStream_t s) {
    const int tiles_m = static_cast<int>((T + kTileM - 1) / kTileM);
    const int tiles_n = static_cast<int>((N + kTileN - 1) / kTileN);
    const int nt = tiles_m * tiles_n;
    const dim3 grid(8 * ((nt + 7) / 8)), block(256);
    hipLaunchKernelGGL((k_gemm<YT, LT, CMC>), grid, block, 0, s, q, wq, x_scale, w_scale, T,
                       static_cast<int>(K), static_cast<int>(N), tiles_m, tiles_n, mod, u, rank,
                       n_mod, static_cast<const LT*>(r_up), acc, static_cast<YT*>(y));
}

hipError_t launch_gemm(const int8_t* q, const float* x_scale, const int8_t* wq,
                       const float* w_scale, int64_t T, int64_t K, int64_t N,
                       const int32_t* mod, const float* u, int rank, int n_mod,
                       const void* r_up, DT lr_dt, bool cmc, int32_t* acc, void* y, DT y_dt,
                       hipStream_t s) {
#define MASQ_GEMM(YT, LT, C) launch_gemm_t<YT, LT, C>(q, x_scale, wq, w_scale, T, K, N, mod, u, rank, n_mod, r_up, acc, y, s)
    if (!cmc) {
        if (y_dt == DT::BF16) MASQ_GEMM(bf16_t, bf16_t, false);
        else MASQ_GEMM(float, bf16_t, false);
    } else if (y_dt == DT::BF16) {
        if (lr_dt == DT::BF16) MASQ_GEMM(bf16_t, bf16_t, true);
        else MASQ_GEMM(bf16_t, float, true);
    } else {
        if (lr_dt == DT::BF16) MASQ_GEMM(float, bf16_t, true);
        else MASQ_GEMM(float, float, true);
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
