// Calibration on the GPU: the exact, non-iterative part of the offline
// calibration that produces the layer's smoothing factors and shared weight.
//
//   R^m_i   = max over the tokens of modality m of |x_ti|         (Sec. 4.1)
//   s^m_i   = sqrt(max(R^m_i, 1e-5) / max(w_i, 1e-5)),            (Sec. 4.2,
//             w_i = max_j |w_ij| over the output channels           alpha = 1/2)
//   Q(S_t W): per output channel o, step d_o = max_i |s^t_i w_io| / qmax and
//             codes rint((s^t_i w_io) / d_o) clamped to [-qmax, qmax]  (eq. PTQ)
//
// and the inputs and products of the compensation factors' calibration:
// the smoothed rows Z_m = X_m S_m^-1 of one modality, the weight difference
// dW_m = S_m W - Q(S_t W), and an fp64 GEMM for the Gram matrix, the
// whitening and the randomized truncated SVD (Sec. 3.2, 4.3).
//
// Every quantity that decides a value is computed in the same precision as
// the definition's host implementation (fp64 for the factor and the weight
// step, one rounding to fp32 at the end), so the results are bit-exact.
// The C ABI of these calls is declared in masq.h.

#include <hip/hip_runtime.h>
#include <math.h>

#include "masq.h"

namespace {

using bf16_t = unsigned short;

__device__ __forceinline__ float load_abs(const float* p) { return fabsf(*p); }
__device__ __forceinline__ float load_abs(const bf16_t* p) {
    return fabsf(__uint_as_float(static_cast<uint32_t>(*p) << 16));
}

// range [n_mod][K] := 0 (the maxima below are taken with integer atomics on
// the bits of non-negative floats, which order like the values).
__global__ __launch_bounds__(256) void k_zero_f32(float* __restrict__ p, int64_t n) {
    for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n; i += gridDim.x * 256ll) p[i] = 0.f;
}

// grid (ceil(K / 256), row chunks): thread = column i, rows of its chunk;
// per-modality maxima in registers, then one atomic max per modality.
// Tokens whose id is outside [0, n_mod) belong to no modality.
template <typename XT>
__global__ __launch_bounds__(256) void k_channel_range(const XT* __restrict__ x,
                                                       const int32_t* __restrict__ mod,
                                                       int64_t T, int K, int n_mod,
                                                       int rows_per_chunk,
                                                       float* __restrict__ range) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= K) return;
    const int64_t t0 = static_cast<int64_t>(blockIdx.y) * rows_per_chunk;
    const int64_t t1 = t0 + rows_per_chunk < T ? t0 + rows_per_chunk : T;
    float m[4] = {0.f, 0.f, 0.f, 0.f};
    for (int64_t t = t0; t < t1; ++t) {
        const int mm = mod[t];                                 // uniform across the block
        const float a = load_abs(x + t * K + i);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (mm == k) m[k] = fmaxf(m[k], a);
    }
    for (int k = 0; k < n_mod; ++k)
        if (m[k] > 0.f)
            atomicMax(reinterpret_cast<int*>(range + static_cast<int64_t>(k) * K + i),
                      __float_as_int(m[k]));
}

// One wave per input channel i: w_i = max_j |w_ij| over its row of W
// [K][N], then s^m_i = fl32(sqrt(max(R, 1e-5) / max(w_i, 1e-5))) in fp64 for
// every modality and inv = fl32(1 / s) (correctly rounded).
__global__ __launch_bounds__(256) void k_smoothing_factors(const float* __restrict__ range,
                                                           const float* __restrict__ w, int K,
                                                           int N, int n_mod,
                                                           float* __restrict__ s,
                                                           float* __restrict__ inv_s) {
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (i >= K) return;
    const float* row = w + static_cast<int64_t>(i) * N;
    float a = 0.f;
    for (int j = lane; j < N; j += 64) a = fmaxf(a, fabsf(row[j]));
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) a = fmaxf(a, __shfl_xor(a, o));
    if (lane < n_mod) {
        const double r = static_cast<double>(range[static_cast<int64_t>(lane) * K + i]);
        const double v = sqrt(fmax(r, 1e-5) / fmax(static_cast<double>(a), 1e-5));
        const float s32 = static_cast<float>(v);
        s[static_cast<int64_t>(lane) * K + i] = s32;
        inv_s[static_cast<int64_t>(lane) * K + i] = 1.0f / s32;
    }
}

// Q(S_t W) for 64 output channels per workgroup (W [K][N] fp32, paper layout;
// codes written as wq [N][K]).  Pass 1: step d_o = max_i |s_i w_io| / qmax in
// fp64 (s_i w_io is exact in fp64).  Pass 2: 64 x 64 blocks of codes
// rint(s_i w_io / d_o) (fp64 division, round half to even), transposed
// through LDS so both the reads (along o) and the writes (along i) are
// contiguous.
__global__ __launch_bounds__(256) void k_quantize_weight(const float* __restrict__ w,
                                                         const float* __restrict__ s_text,
                                                         int K, int N, int qmax,
                                                         int8_t* __restrict__ wq,
                                                         float* __restrict__ w_scale) {
    __shared__ double smax[4][64];
    __shared__ double sdelta[64];
    __shared__ int8_t tile[64][65];
    const int tid = threadIdx.x, ol = tid & 63, part = tid >> 6;
    const int o0 = blockIdx.x * 64;
    const int o = o0 + ol;
    double a = 0.0;
    if (o < N)
        for (int i = part; i < K; i += 4)
            a = fmax(a, fabs(static_cast<double>(s_text[i]) * static_cast<double>(w[static_cast<int64_t>(i) * N + o])));
    smax[part][ol] = a;
    __syncthreads();
    if (tid < 64) {
        const double m = fmax(fmax(smax[0][tid], smax[1][tid]), fmax(smax[2][tid], smax[3][tid]));
        const double d = m / qmax;
        sdelta[tid] = d;
        if (o0 + tid < N) w_scale[o0 + tid] = static_cast<float>(d);
    }
    __syncthreads();
    const double d = sdelta[ol];
    for (int i0 = 0; i0 < K; i0 += 64) {
        // read: thread (ol, part) takes rows i0 + part + 4 k of channel o
        for (int k = 0; k < 16; ++k) {
            const int il = part + 4 * k, i = i0 + il;
            int c = 0;
            if (o < N && i < K && d > 0.0) {
                const double v = static_cast<double>(s_text[i]) * static_cast<double>(w[static_cast<int64_t>(i) * N + o]);
                const double r = rint(v / d);
                c = static_cast<int>(fmin(fmax(r, static_cast<double>(-qmax)), static_cast<double>(qmax)));
            }
            tile[ol][il] = static_cast<int8_t>(c);
        }
        __syncthreads();
        // write: thread (ol', part) writes 16 consecutive codes of channel o0 + ol' ... as
        // row (tid / 4) of the block, 16 bytes at 16 (tid % 4)
        {
            const int orow = tid >> 2, seg = (tid & 3) * 16;
            const int oo = o0 + orow;
            if (oo < N) {
                int8_t* dst = wq + static_cast<int64_t>(oo) * K + i0 + seg;
                for (int e = 0; e < 16; ++e)
                    if (i0 + seg + e < K) dst[e] = tile[orow][seg + e];
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ CMC inputs
// The compensation factors (Sec. 3.2, 4.3; eq. l1l2) come from the smoothed
// calibration rows Z_m = X_m S_m^-1 of one modality, their Gram matrix, and
// the weight difference dW_m = S_m W - Q(S_t W); the products below are the
// heavy part of that calibration at full layer sizes.

__device__ __forceinline__ double load_f64(const float* p) { return static_cast<double>(*p); }
__device__ __forceinline__ double load_f64(const bf16_t* p) {
    return static_cast<double>(__uint_as_float(static_cast<uint32_t>(*p) << 16));
}

// z [n][K]: z_ic = x[rows[i]][c] / s_c in fp64 (exact operands, one
// correctly rounded division); a row index outside [0, T) gives a zero row.
// grid (ceil(K / 256), row chunks).
template <typename XT>
__global__ __launch_bounds__(256) void k_gather_smoothed(const XT* __restrict__ x, int64_t T, int K,
                                                         const int32_t* __restrict__ rows,
                                                         int64_t n, const float* __restrict__ s,
                                                         double* __restrict__ z) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= K) return;
    const double sc = static_cast<double>(s[c]);
    for (int64_t i = blockIdx.y; i < n; i += gridDim.y) {
        const int64_t r = rows[i];
        double v = 0.0;
        if (r >= 0 && r < T) v = load_f64(x + r * K + c) / sc;
        z[i * K + c] = v;
    }
}

// dw [K][N] = s_i w_io - wq_oi d_o in fp64: both products are exact (24 x 24
// and 8 x 24 significant bits), so the one subtraction is the only rounding.
// 64 x 64 blocks: the codes wq [N][K] are read along i and transposed
// through LDS, w and dw are read and written along o.
__global__ __launch_bounds__(256) void k_weight_difference(const float* __restrict__ w,
                                                           const float* __restrict__ s,
                                                           const int8_t* __restrict__ wq,
                                                           const float* __restrict__ w_scale,
                                                           int K, int N, double* __restrict__ dw) {
    __shared__ int8_t tile[64][65];                         // [o][i]
    const int tid = threadIdx.x;
    const int o0 = blockIdx.x * 64, i0 = blockIdx.y * 64;
    {
        const int orow = tid >> 2, seg = (tid & 3) * 16, o = o0 + orow;
        for (int e = 0; e < 16; ++e) {
            const int i = i0 + seg + e;
            tile[orow][seg + e] = (o < N && i < K) ? wq[static_cast<int64_t>(o) * K + i] : int8_t(0);
        }
    }
    __syncthreads();
    const int ol = tid & 63, o = o0 + ol;
    if (o >= N) return;
    const double d = static_cast<double>(w_scale[o]);
    for (int il = tid >> 6; il < 64; il += 4) {
        const int i = i0 + il;
        if (i >= K) break;
        const int64_t at = static_cast<int64_t>(i) * N + o;
        const double a = static_cast<double>(s[i]) * static_cast<double>(w[at]);
        const double b = static_cast<double>(tile[ol][il]) * d;
        dw[at] = a - b;
    }
}

// C (i, j) at c[i * crs + j * ccs] = alpha A B (+ beta C), fp64, with A (i,
// k) at a[i * ars + k * acs] and B (k, j) at b[k * brs + j * bcs], so
// transposed operands are strides, not copies.  TL x TL tiles (128, or 64
// when the 128-tiles would not give every CU one), 256 threads of TL/16 x
// TL/16 outputs (rows ty + 16 u, columns tx + 16 v), k in steps of 16 staged
// through LDS with the next step's loads in flight.  Every element is summed
// in increasing k by fused multiply-adds, whatever the tile size; the sum is
// then multiplied by alpha (exact for alpha = +-1) and beta C added.  With
// lower, tiles wholly above the diagonal (every j > i) are skipped.
constexpr int kDgTile = 128;
constexpr int kDgStep = 16;
template <int TL>
__global__ __launch_bounds__(256) void k_dgemm(int64_t M, int64_t N, int64_t K,
                                               const double* __restrict__ a, int64_t ars,
                                               int64_t acs, const double* __restrict__ b,
                                               int64_t brs, int64_t bcs, double alpha, double beta,
                                               double* __restrict__ c, int64_t crs, int64_t ccs,
                                               int lower) {
    constexpr int NU = TL / 16, NQ = TL * kDgStep / 256;     // outputs a row, loads per operand
    constexpr int LT = TL == 128 ? 7 : 6;                    // log2(TL)
    __shared__ double as[kDgStep][TL + 1];
    __shared__ double bs[kDgStep][TL + 1];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int64_t i0 = static_cast<int64_t>(blockIdx.y) * TL;
    const int64_t j0 = static_cast<int64_t>(blockIdx.x) * TL;
    if (lower && j0 > i0 + TL - 1) return;                   // block-uniform
    // staging: element e = tid + 256 q of each TL x 16 operand block; the
    // fastest-moving index follows the operand's unit-stride direction
    const bool a_k_fast = acs == 1, b_k_fast = bcs != 1;
    double ra[NQ], rb[NQ];
    auto load = [&](int64_t k0) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int e = tid + 256 * q;
            const int kk = a_k_fast ? (e & 15) : (e >> LT);
            const int ii = a_k_fast ? (e >> 4) : (e & (TL - 1));
            const int64_t i = i0 + ii, k = k0 + kk;
            ra[q] = (i < M && k < K) ? a[i * ars + k * acs] : 0.0;
        }
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int e = tid + 256 * q;
            const int kk = b_k_fast ? (e & 15) : (e >> LT);
            const int jj = b_k_fast ? (e >> 4) : (e & (TL - 1));
            const int64_t j = j0 + jj, k = k0 + kk;
            rb[q] = (j < N && k < K) ? b[k * brs + j * bcs] : 0.0;
        }
    };
    auto stash = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int e = tid + 256 * q;
            as[a_k_fast ? (e & 15) : (e >> LT)][a_k_fast ? (e >> 4) : (e & (TL - 1))] = ra[q];
            bs[b_k_fast ? (e & 15) : (e >> LT)][b_k_fast ? (e >> 4) : (e & (TL - 1))] = rb[q];
        }
    };
    double acc[NU][NU];
#pragma unroll
    for (int u = 0; u < NU; ++u)
#pragma unroll
        for (int v = 0; v < NU; ++v) acc[u][v] = 0.0;
    if (K > 0) load(0);
    for (int64_t k0 = 0; k0 < K; k0 += kDgStep) {
        __syncthreads();
        stash();
        __syncthreads();
        if (k0 + kDgStep < K) load(k0 + kDgStep);
#pragma unroll 4
        for (int kk = 0; kk < kDgStep; ++kk) {
            double av[NU], bv[NU];
#pragma unroll
            for (int u = 0; u < NU; ++u) av[u] = as[kk][ty + 16 * u];
#pragma unroll
            for (int v = 0; v < NU; ++v) bv[v] = bs[kk][tx + 16 * v];
#pragma unroll
            for (int u = 0; u < NU; ++u)
#pragma unroll
                for (int v = 0; v < NU; ++v) acc[u][v] = fma(av[u], bv[v], acc[u][v]);
        }
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        const int64_t i = i0 + ty + 16 * u;
        if (i >= M) break;
#pragma unroll
        for (int v = 0; v < NU; ++v) {
            const int64_t j = j0 + tx + 16 * v;
            if (j < N) {
                double r = alpha * acc[u][v];
                if (beta != 0.0) r = r + beta * c[i * crs + j * ccs];
                c[i * crs + j * ccs] = r;
            }
        }
    }
}

// ------------------------------------------------------- MAS optimisation
// The per-modality objective mean |Q(X S^-1) Q(S W) - X W| (Sec. 4.2, eq.
// mas_quant) and its straight-through gradient: the quantizers are the
// inference ones above; these kernels dequantize their codes, take the
// residual's sign and assemble dL/ds from the two products of the backward
// pass (formed with k_dgemm).

// out [R][C] fp64 = codes [R][C] * scale[r] (exact: 8 x 24 significant bits).
__global__ __launch_bounds__(256) void k_dequantize_rows(const int8_t* __restrict__ codes,
                                                         const float* __restrict__ scale,
                                                         int64_t R, int64_t C,
                                                         double* __restrict__ out) {
    const int64_t n = R * C;
    for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < n; e += gridDim.x * 256ll)
        out[e] = static_cast<double>(codes[e]) * static_cast<double>(scale[e / C]);
}

// g_e = sign(y_e - ref_e) * inv_count; partial[b] = the sum of |y_e - ref_e|
// over block b's kMaeChunk elements (a fixed tree order, so the loss the
// caller adds up is reproducible).
constexpr int kMaeChunk = 4096;
__global__ __launch_bounds__(256) void k_mae_sign(const double* __restrict__ y,
                                                  const double* __restrict__ ref, int64_t n,
                                                  double inv_count, double* __restrict__ g,
                                                  double* __restrict__ partial) {
    __shared__ double red[4];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kMaeChunk;
    double acc = 0.0;
    for (int j = threadIdx.x; j < kMaeChunk; j += 256) {
        const int64_t e = base + j;
        if (e >= n) break;
        const double r = y[e] - ref[e];
        g[e] = r > 0.0 ? inv_count : (r < 0.0 ? -inv_count : 0.0);
        acc += fabs(r);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) partial[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// loss[0] = (partial[0] + partial[1] + ... + partial[nparts - 1]) / count,
// in that order (one thread: a few thousand block sums at most).
__global__ void k_mae_loss(const double* __restrict__ partial, int64_t nparts, double count,
                           double* __restrict__ loss) {
    double s = 0.0;
    for (int64_t b = 0; b < nparts; ++b) s += partial[b];
    *loss = s / count;
}

// Adam on theta = ln s (Kingma and Ba 2015), one element a thread, each
// operation rounded as written (the build disables contraction):
//   g  = lam * s * grad                (d/dtheta of the objective)
//   m1 = b1 m1 + (1 - b1) g,  m2 = b2 m2 + ((1 - b2) g) g
//   theta -= (lr (m1 / c1)) / (sqrt(m2 / c2) + eps),  c_i = 1 - b_i^step
//   s := fl32(exp(theta)),  inv_s := fl32(1 / s)
__global__ __launch_bounds__(256) void k_adam_log(double* __restrict__ theta, double* __restrict__ m1,
                                                  double* __restrict__ m2,
                                                  const double* __restrict__ grad,
                                                  float* __restrict__ s, float* __restrict__ inv_s,
                                                  int64_t K, double lam, double lr, double b1,
                                                  double omb1, double b2, double omb2, double c1,
                                                  double c2, double eps) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= K) return;
    const double g = (lam * static_cast<double>(s[i])) * grad[i];
    const double a = b1 * m1[i] + omb1 * g;
    const double v = b2 * m2[i] + (omb2 * g) * g;
    const double th = theta[i] - (lr * (a / c1)) / (sqrt(v / c2) + eps);
    m1[i] = a;
    m2[i] = v;
    theta[i] = th;
    const float sn = static_cast<float>(exp(th));
    s[i] = sn;
    inv_s[i] = 1.0f / sn;
}

// theta = ln s, m1 = m2 = 0, then s := fl32(exp(theta)), inv_s := fl32(1 / s)
// (the factors the first step's forward pass uses).
__global__ __launch_bounds__(256) void k_adam_log_init(double* __restrict__ theta,
                                                       double* __restrict__ m1,
                                                       double* __restrict__ m2,
                                                       float* __restrict__ s,
                                                       float* __restrict__ inv_s, int64_t K) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= K) return;
    const double th = log(static_cast<double>(s[i]));
    theta[i] = th;
    m1[i] = 0.0;
    m2[i] = 0.0;
    const float sn = static_cast<float>(exp(th));
    s[i] = sn;
    inv_s[i] = 1.0f / sn;
}

// colpart[i] = sum_t x[t][i] a[t][i] (thread per column, t in order).
__global__ __launch_bounds__(256) void k_column_dot(const double* __restrict__ x,
                                                    const double* __restrict__ a, int64_t T,
                                                    int64_t K, double* __restrict__ out) {
    const int64_t i = blockIdx.x * 256ll + threadIdx.x;
    if (i >= K) return;
    double acc = 0.0;
    for (int64_t t = 0; t < T; ++t) acc = fma(x[t * K + i], a[t * K + i], acc);
    out[i] = acc;
}

// grad[i] = -colpart[i] / (s_i s_i) + sum_o w[i][o] b[i][o] (a wave per row i).
__global__ __launch_bounds__(256) void k_mas_grad(const double* __restrict__ colpart,
                                                  const double* __restrict__ w,
                                                  const double* __restrict__ b,
                                                  const float* __restrict__ s, int64_t K,
                                                  int64_t N, double* __restrict__ grad) {
    const int lane = threadIdx.x & 63;
    const int64_t i = blockIdx.x * 4ll + (threadIdx.x >> 6);
    if (i >= K) return;
    double acc = 0.0;
    for (int64_t o = lane; o < N; o += 64) acc = fma(w[i * N + o], b[i * N + o], acc);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane == 0) {
        const double si = static_cast<double>(s[i]);
        grad[i] = -colpart[i] / (si * si) + acc;
    }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

}  // namespace

namespace masq {

hipError_t launch_dgemm(int64_t m, int64_t n, int64_t k, const double* a, int64_t ars,
                        int64_t acs, const double* b, int64_t brs, int64_t bcs, double alpha,
                        double beta, double* c, int64_t crs, int64_t ccs, bool lower,
                        hipStream_t s) {
    if (m <= 0 || n <= 0) return hipSuccess;
    const int64_t tiles = ((n + kDgTile - 1) / kDgTile) * ((m + kDgTile - 1) / kDgTile);
    const int tl = (tiles < 256 && (m + 63) / 64 <= 65535) ? 64 : kDgTile;
    const dim3 grid(static_cast<unsigned>((n + tl - 1) / tl), static_cast<unsigned>((m + tl - 1) / tl));
    if (tl == 64)
        hipLaunchKernelGGL(k_dgemm<64>, grid, dim3(256), 0, s, m, n, k, a, ars, acs, b, brs, bcs,
                           alpha, beta, c, crs, ccs, lower ? 1 : 0);
    else
        hipLaunchKernelGGL(k_dgemm<kDgTile>, grid, dim3(256), 0, s, m, n, k, a, ars, acs, b, brs,
                           bcs, alpha, beta, c, crs, ccs, lower ? 1 : 0);
    return hipGetLastError();
}

}  // namespace masq

extern "C" {

masq_status masq_channel_range(const void* x, masq_dtype x_dt, const int32_t* modality,
                               int64_t T, int64_t c_in, int32_t n_mod, float* range,
                               void* stream) {
    if (x_dt != MASQ_F32 && x_dt != MASQ_BF16) return MASQ_ERR_DTYPE;
    if (T < 0 || c_in <= 0 || c_in % 16 != 0 || c_in > (1LL << 30) || n_mod < 1 || n_mod > 4)
        return MASQ_ERR_SHAPE;
    if (!range || (T > 0 && (!x || !modality))) return MASQ_ERR_NULL;
    if (!aligned16(range) || (T > 0 && (!aligned16(x) || !aligned16(modality))))
        return MASQ_ERR_ALIGN;
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    const int64_t n = static_cast<int64_t>(n_mod) * c_in;
    hipLaunchKernelGGL(k_zero_f32, dim3(static_cast<unsigned>((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024)),
                       dim3(256), 0, s, range, n);
    if (T > 0) {
        const int K = static_cast<int>(c_in);
        const int64_t col_blocks = (K + 255) / 256;
        int64_t chunks = (2048 + col_blocks - 1) / col_blocks;          // about 2048 workgroups
        if (chunks > T) chunks = T;
        const int rows = static_cast<int>((T + chunks - 1) / chunks);
        chunks = (T + rows - 1) / rows;
        const dim3 grid(static_cast<unsigned>(col_blocks), static_cast<unsigned>(chunks));
        if (x_dt == MASQ_BF16)
            hipLaunchKernelGGL(k_channel_range<bf16_t>, grid, dim3(256), 0, s,
                               static_cast<const bf16_t*>(x), modality, T, K, n_mod, rows, range);
        else
            hipLaunchKernelGGL(k_channel_range<float>, grid, dim3(256), 0, s,
                               static_cast<const float*>(x), modality, T, K, n_mod, rows, range);
    }
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_smoothing_factors(const float* range, const float* w, int64_t c_in,
                                   int64_t c_out, int32_t n_mod, float* smooth,
                                   float* inv_smooth, void* stream) {
    if (c_in <= 0 || c_in % 16 != 0 || c_out <= 0 || c_out % 16 != 0 || c_in > (1LL << 30) ||
        c_out > (1LL << 30) || n_mod < 1 || n_mod > 4)
        return MASQ_ERR_SHAPE;
    if (!range || !w || !smooth || !inv_smooth) return MASQ_ERR_NULL;
    if (!aligned16(range) || !aligned16(w) || !aligned16(smooth) || !aligned16(inv_smooth))
        return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_smoothing_factors, dim3(static_cast<unsigned>((c_in + 3) / 4)), dim3(256),
                       0, static_cast<hipStream_t>(stream), range, w, static_cast<int>(c_in),
                       static_cast<int>(c_out), n_mod, smooth, inv_smooth);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_quantize_weight(const float* w, const float* smooth_text, int64_t c_in,
                                 int64_t c_out, int32_t bits, int8_t* wq, float* w_scale,
                                 void* stream) {
    if (c_in <= 0 || c_in % 16 != 0 || c_out <= 0 || c_out % 16 != 0 || c_in > (1LL << 30) ||
        c_out > (1LL << 30) || (bits != 8 && bits != 4))
        return MASQ_ERR_SHAPE;
    if (!w || !smooth_text || !wq || !w_scale) return MASQ_ERR_NULL;
    if (!aligned16(w) || !aligned16(smooth_text) || !aligned16(wq) || !aligned16(w_scale))
        return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_quantize_weight, dim3(static_cast<unsigned>((c_out + 63) / 64)), dim3(256),
                       0, static_cast<hipStream_t>(stream), w, smooth_text, static_cast<int>(c_in),
                       static_cast<int>(c_out), (1 << (bits - 1)) - 1, wq, w_scale);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_gather_smoothed(const void* x, masq_dtype x_dt, int64_t T, int64_t c_in,
                                 const int32_t* rows, int64_t n_rows, const float* smooth,
                                 double* z, void* stream) {
    if (x_dt != MASQ_F32 && x_dt != MASQ_BF16) return MASQ_ERR_DTYPE;
    if (T < 0 || n_rows < 0 || c_in <= 0 || c_in % 16 != 0 || c_in > (1LL << 30))
        return MASQ_ERR_SHAPE;
    if (n_rows == 0) return MASQ_OK;
    if (!rows || !smooth || !z || (T > 0 && !x)) return MASQ_ERR_NULL;
    if (!aligned16(rows) || !aligned16(smooth) || !aligned16(z) || (T > 0 && !aligned16(x)))
        return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    const int K = static_cast<int>(c_in);
    const int64_t col_blocks = (K + 255) / 256;
    int64_t chunks = (2048 + col_blocks - 1) / col_blocks;
    if (chunks > n_rows) chunks = n_rows;
    if (chunks > 65535) chunks = 65535;
    const dim3 grid(static_cast<unsigned>(col_blocks), static_cast<unsigned>(chunks));
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (x_dt == MASQ_BF16)
        hipLaunchKernelGGL(k_gather_smoothed<bf16_t>, grid, dim3(256), 0, s,
                           static_cast<const bf16_t*>(x), T, K, rows, n_rows, smooth, z);
    else
        hipLaunchKernelGGL(k_gather_smoothed<float>, grid, dim3(256), 0, s,
                           static_cast<const float*>(x), T, K, rows, n_rows, smooth, z);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_weight_difference(const float* w, const float* smooth, const int8_t* wq,
                                   const float* w_scale, int64_t c_in, int64_t c_out,
                                   double* dw, void* stream) {
    if (c_in <= 0 || c_in % 16 != 0 || c_out <= 0 || c_out % 16 != 0 || c_in > (1LL << 30) ||
        c_out > (1LL << 30) || (c_in + 63) / 64 > 65535)
        return MASQ_ERR_SHAPE;
    if (!w || !smooth || !wq || !w_scale || !dw) return MASQ_ERR_NULL;
    if (!aligned16(w) || !aligned16(smooth) || !aligned16(wq) || !aligned16(w_scale) ||
        !aligned16(dw))
        return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    const dim3 grid(static_cast<unsigned>((c_out + 63) / 64), static_cast<unsigned>((c_in + 63) / 64));
    hipLaunchKernelGGL(k_weight_difference, grid, dim3(256), 0, static_cast<hipStream_t>(stream),
                       w, smooth, wq, w_scale, static_cast<int>(c_in), static_cast<int>(c_out), dw);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_dgemm(int64_t m, int64_t n, int64_t k, const double* a, int64_t a_row_stride,
                       int64_t a_col_stride, const double* b, int64_t b_row_stride,
                       int64_t b_col_stride, double beta, double* c, int64_t ldc, void* stream) {
    if (m < 0 || n < 0 || k < 0 || a_row_stride < 0 || a_col_stride < 0 || b_row_stride < 0 ||
        b_col_stride < 0 || (m + kDgTile - 1) / kDgTile > 65535 ||
        (n + kDgTile - 1) / kDgTile > 0x7fffffffLL || (m > 0 && n > 0 && ldc < n))
        return MASQ_ERR_SHAPE;
    if (m == 0 || n == 0) return MASQ_OK;
    if (!c || (k > 0 && (!a || !b))) return MASQ_ERR_NULL;
    if (!aligned8(c) || (k > 0 && (!aligned8(a) || !aligned8(b)))) return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    return masq::launch_dgemm(m, n, k, a, a_row_stride, a_col_stride, b, b_row_stride,
                              b_col_stride, 1.0, beta, c, ldc, 1, false,
                              static_cast<hipStream_t>(stream)) == hipSuccess
               ? MASQ_OK
               : MASQ_ERR_HIP;
}

masq_status masq_dequantize_rows(const int8_t* codes, const float* scale, int64_t rows,
                                 int64_t cols, double* out, void* stream) {
    if (rows < 0 || cols < 0 || (cols > 0 && rows > (1LL << 40) / cols)) return MASQ_ERR_SHAPE;
    if (rows == 0 || cols == 0) return MASQ_OK;
    if (!codes || !scale || !out) return MASQ_ERR_NULL;
    if (!aligned16(codes) || !aligned16(scale) || !aligned16(out)) return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    const int64_t n = rows * cols;
    const int64_t blocks = (n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192;
    hipLaunchKernelGGL(k_dequantize_rows, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), codes, scale, rows, cols, out);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

int64_t masq_mae_partials(int64_t count) {
    return count <= 0 ? 0 : (count + kMaeChunk - 1) / kMaeChunk;
}

masq_status masq_mae_sign(const double* y, const double* ref, int64_t count, double* g,
                          double* partial, void* stream) {
    if (count < 0 || masq_mae_partials(count) > 0x7fffffffLL) return MASQ_ERR_SHAPE;
    if (count == 0) return MASQ_OK;
    if (!y || !ref || !g || !partial) return MASQ_ERR_NULL;
    if (!aligned8(y) || !aligned8(ref) || !aligned8(g) || !aligned8(partial)) return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_mae_sign, dim3(static_cast<unsigned>(masq_mae_partials(count))), dim3(256),
                       0, static_cast<hipStream_t>(stream), y, ref, count,
                       1.0 / static_cast<double>(count), g, partial);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_mae_loss(const double* partial, int64_t count, double* loss, void* stream) {
    if (count < 0 || masq_mae_partials(count) > 0x7fffffffLL) return MASQ_ERR_SHAPE;
    if (!loss || (count > 0 && !partial)) return MASQ_ERR_NULL;
    if (!aligned8(loss) || (count > 0 && !aligned8(partial))) return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_mae_loss, dim3(1), dim3(1), 0, static_cast<hipStream_t>(stream), partial,
                       masq_mae_partials(count), count > 0 ? static_cast<double>(count) : 1.0, loss);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_adam_log_step(double* theta, double* m1, double* m2, const double* grad,
                               float* smooth, float* inv_smooth, int64_t c_in, double lam,
                               double lr, double b1, double b2, double eps, int64_t step,
                               void* stream) {
    if (c_in < 0 || c_in > (1LL << 30) || step < 0 || !(lr >= 0.0) || !(b1 >= 0.0 && b1 < 1.0) ||
        !(b2 >= 0.0 && b2 < 1.0) || !(eps > 0.0) || !isfinite(lam) || !isfinite(lr))
        return MASQ_ERR_SHAPE;
    if (c_in == 0) return MASQ_OK;
    if (!theta || !m1 || !m2 || !smooth || !inv_smooth || (step > 0 && !grad))
        return MASQ_ERR_NULL;
    if (!aligned8(theta) || !aligned8(m1) || !aligned8(m2) || (step > 0 && !aligned8(grad)) ||
        (reinterpret_cast<uintptr_t>(smooth) & 3u) != 0 ||
        (reinterpret_cast<uintptr_t>(inv_smooth) & 3u) != 0)
        return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    hipStream_t st = static_cast<hipStream_t>(stream);
    const dim3 grid(static_cast<unsigned>((c_in + 255) / 256));
    if (step == 0) {
        hipLaunchKernelGGL(k_adam_log_init, grid, dim3(256), 0, st, theta, m1, m2, smooth,
                           inv_smooth, c_in);
    } else {
        const double sd = static_cast<double>(step);
        hipLaunchKernelGGL(k_adam_log, grid, dim3(256), 0, st, theta, m1, m2, grad, smooth,
                           inv_smooth, c_in, lam, lr, b1, 1.0 - b1, b2, 1.0 - b2,
                           1.0 - pow(b1, sd), 1.0 - pow(b2, sd), eps);
    }
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_mas_gradient(const double* x, const double* a, const double* w, const double* b,
                              const float* smooth, int64_t T, int64_t c_in, int64_t c_out,
                              double* colpart, double* grad, void* stream) {
    if (T < 0 || c_in <= 0 || c_out <= 0 || c_in > (1LL << 30) || c_out > (1LL << 30))
        return MASQ_ERR_SHAPE;
    if (!w || !b || !smooth || !colpart || !grad || (T > 0 && (!x || !a))) return MASQ_ERR_NULL;
    if (!aligned8(w) || !aligned8(b) || !aligned8(smooth) || !aligned8(colpart) ||
        !aligned8(grad) || (T > 0 && (!aligned8(x) || !aligned8(a))))
        return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k_column_dot, dim3(static_cast<unsigned>((c_in + 255) / 256)), dim3(256), 0,
                       st, x, a, T, c_in, colpart);
    hipLaunchKernelGGL(k_mas_grad, dim3(static_cast<unsigned>((c_in + 3) / 4)), dim3(256), 0, st,
                       colpart, w, b, smooth, c_in, c_out, grad);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

}  // extern "C"
