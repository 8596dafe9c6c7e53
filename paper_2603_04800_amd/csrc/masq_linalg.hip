// Dense fp64 factorisations of the compensation factors' calibration
// (Sec. 3.2 and 4.3; eq. l1l2), so that no decomposition runs on the host:
//
//   masq_cholesky    C + eps I = L L^T (blocked, lower).  The whitening only
//                    has to satisfy T^T T = C + eps I: T = L^T serves as well
//                    as the symmetric root, and the truncated SVD of T dW
//                    then gives the same L1 = T^-1 U_r and L2 = Sigma_r V_r^T
//                    (a T' = Q T with Q orthogonal rotates the left singular
//                    vectors by Q and leaves T'^-1 U' and Sigma V^T as they
//                    were).
//   masq_trsm_right  X L^T = Y or X L = Y with that factor: T^-1 applied to
//                    the left singular vectors, and the solves of CholeskyQR
//                    (the range finder's orthogonalisations).
//   masq_jacobi_svd  one-sided Jacobi SVD of the projected matrix (one launch
//                    per round of disjoint column pairs; this call waits for
//                    the stream once per sweep to test for convergence).
//
// The blocked routines run the diagonal blocks in one workgroup each and the
// updates on the fp64 GEMM (masq::launch_dgemm).  The C ABI is declared in
// masq.h.

#include <hip/hip_runtime.h>
#include <math.h>

#include "masq.h"
#include "masq_linalg.h"

namespace {

constexpr int kNb = 64;          // block size of the factorisation and the solves
constexpr int kJacobiMaxN = 1024;

bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

// a := a + (ridge * tr(a) / n) I, with tr(a) (taken before the shift)
// written to trace when given, and info := 0.  One workgroup; the trace is
// summed in a fixed order.
__global__ __launch_bounds__(1024) void k_add_ridge(double* __restrict__ a, int64_t n,
                                                    int64_t lda, double ridge,
                                                    double* __restrict__ trace,
                                                    int32_t* __restrict__ info) {
    __shared__ double red[1024];
    const int tid = threadIdx.x;
    double s = 0.0;
    for (int64_t i = tid; i < n; i += 1024) s += a[i * lda + i];
    red[tid] = s;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (tid < w) red[tid] += red[tid + w];
        __syncthreads();
    }
    const double tr = red[0];
    if (tid == 0) {
        if (trace != nullptr) *trace = tr;
        *info = 0;
    }
    const double eps = ridge * tr / static_cast<double>(n);
    if (eps != 0.0)
        for (int64_t i = tid; i < n; i += 1024) a[i * lda + i] += eps;
}

// Cholesky factor of the jb x jb diagonal block at a (row stride lda), in
// place: the lower triangle becomes L with L L^T = the block, the strict
// upper triangle zero.  One workgroup, the block in LDS, right-looking.  A
// pivot that is not positive (or NaN) is recorded in info as j0 + k + 1
// (the first over the whole factorisation wins) and replaced by 1, so the
// factorisation runs to its end.
__global__ __launch_bounds__(256) void k_potf2(double* __restrict__ a, int64_t lda, int jb,
                                               int64_t j0, int32_t* __restrict__ info) {
    __shared__ double s[kNb][kNb + 1];
    const int tid = threadIdx.x;
    for (int e = tid; e < kNb * kNb; e += 256) {
        const int i = e / kNb, j = e % kNb;
        s[i][j] = (i < jb && j <= i) ? a[i * lda + j] : 0.0;
    }
    __syncthreads();
    for (int k = 0; k < jb; ++k) {
        const double d = s[k][k];
        const bool ok = d > 0.0;
        const double piv = ok ? sqrt(d) : 1.0;
        __syncthreads();                                  // every thread has read s[k][k]
        if (tid == 0) {
            s[k][k] = piv;
            if (!ok) atomicCAS(reinterpret_cast<int*>(info), 0, static_cast<int>(j0 + k + 1));
        }
        if (tid > k && tid < jb) s[tid][k] /= piv;
        __syncthreads();
        for (int e = tid; e < kNb * kNb; e += 256) {
            const int i = e / kNb, j = e % kNb;
            if (j > k && i >= j && i < jb) s[i][j] = fma(-s[i][k], s[j][k], s[i][j]);
        }
        __syncthreads();
    }
    for (int e = tid; e < kNb * kNb; e += 256) {
        const int i = e / kNb, j = e % kNb;
        if (i < jb && j < jb) a[i * lda + j] = j <= i ? s[i][j] : 0.0;
    }
}

// Row-wise solves with a jb x jb lower-triangular block L (jb <= 64, at l,
// row stride ldl): each of the `rows` rows y of Y (row stride ldy, jb
// entries) is replaced by the x with
//   FWD: x L^T = y  (x_k = (y_k - sum_{m<k} x_m L_km) / L_kk, k ascending)
//   BWD: x L   = y  (x_k = (y_k - sum_{m>k} x_m L_mk) / L_kk, k descending);
// the sums are accumulated term by term, in the order of k, into the entries
// still open.  A wave takes a row at a time, lane j holding x_j; L is in LDS.
template <bool FWD>
__global__ __launch_bounds__(256) void k_trsm_rows(double* __restrict__ y, int64_t rows,
                                                   int64_t ldy, const double* __restrict__ l,
                                                   int64_t ldl, int jb) {
    __shared__ double s[kNb][kNb + 1];
    const int tid = threadIdx.x, lane = tid & 63;
    for (int e = tid; e < kNb * kNb; e += 256) {
        const int i = e / kNb, j = e % kNb;
        s[i][j] = (i < jb && j <= i) ? l[i * ldl + j] : 0.0;
    }
    __syncthreads();
    for (int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (tid >> 6); r < rows;
         r += static_cast<int64_t>(gridDim.x) * 4) {
        double* yr = y + r * ldy;
        double x = lane < jb ? yr[lane] : 0.0;
        if constexpr (FWD) {
            for (int k = 0; k < jb; ++k) {
                if (lane == k) x = x / s[k][k];
                const double xk = __shfl(x, k);
                if (lane > k) x = fma(-xk, s[lane][k], x);
            }
        } else {
            for (int k = jb - 1; k >= 0; --k) {
                if (lane == k) x = x / s[k][k];
                const double xk = __shfl(x, k);
                if (lane < k) x = fma(-xk, s[k][lane], x);
            }
        }
        if (lane < jb) yr[lane] = x;
    }
}

// Workgroups of k_trsm_rows for `rows` rows: one row a wave, at most 1024.
unsigned trsm_grid(int64_t rows) {
    const int64_t g = (rows + 3) / 4;
    return static_cast<unsigned>(g < 1024 ? (g > 0 ? g : 1) : 1024);
}

// a := 0 above the diagonal (row stride lda, n x n).
__global__ __launch_bounds__(256) void k_zero_upper(double* __restrict__ a, int64_t n, int64_t lda) {
    const int64_t i = blockIdx.y;
    for (int64_t j = i + 1 + static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; j < n;
         j += static_cast<int64_t>(gridDim.x) * 256)
        a[i * lda + j] = 0.0;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;                    // the same value in every lane (each step is commutative)
}

// Player at position p of round t of the round-robin pairing of np players
// (np even): position 0 stays, the others rotate.
__device__ __forceinline__ int rr_player(int p, int t, int np) {
    return p == 0 ? 0 : (p - 1 + t) % (np - 1) + 1;
}

// One-sided Jacobi SVD (Hestenes) of an m x n matrix A given by its columns
// (column j at a + j m, overwritten), n <= kJacobiMaxN.  A sweep is the
// np - 1 rounds of the round-robin pairing (np = n rounded up to even; pairs
// with the padding player are skipped); the np / 2 pairs of a round are
// disjoint, so a round is one launch of k_jacobi_round with a workgroup a
// pair.  A pair p < q is rotated in the plane that makes the columns
// orthogonal (alpha = |a_p|^2, beta = |a_q|^2, gamma = a_p . a_q; zeta =
// (beta - alpha) / (2 gamma), t = sign(zeta) / (|zeta| + sqrt(1 + zeta^2)),
// c = 1 / sqrt(1 + t^2), s = c t), and the same rotation is applied to the
// columns of V (vw, n x n by columns, I at the start).  A pair is left alone
// when |gamma| <= 1e-15 sqrt(alpha beta), or when either column's squared
// norm is at most 1e-28 |A|_F^2 (a numerically zero column: those of a
// rank-deficient A converge to such).  Sweeps end after one that rotated
// nothing, or after max_sweeps.  Then A V = U Sigma, sigma_j = |a_j|.

// V := I, fro2[0] := |A|_F^2 (one workgroup, fixed summation order).
__global__ __launch_bounds__(1024) void k_jacobi_init(const double* __restrict__ a, int m, int n,
                                                      double* __restrict__ vw,
                                                      double* __restrict__ fro2) {
    __shared__ double part[16];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int64_t e = tid; e < static_cast<int64_t>(n) * n; e += 1024)
        vw[e] = (e / n == e % n) ? 1.0 : 0.0;
    double ss = 0.0;
    for (int j = wave; j < n; j += 16) {
        const double* aj = a + static_cast<int64_t>(j) * m;
        for (int i = lane; i < m; i += 64) ss = fma(aj[i], aj[i], ss);
    }
    ss = wave_sum(ss);
    if (lane == 0) part[wave] = ss;
    __syncthreads();
    if (tid == 0) {
        double f = 0.0;
        for (int w = 0; w < 16; ++w) f += part[w];
        *fro2 = f;
    }
}

__global__ void k_set_int(int32_t* __restrict__ p, int v) { *p = v; }

// One round: workgroup b rotates pair b (256 threads along the columns).
// rotated := 1 when any pair of the round was rotated.
__global__ __launch_bounds__(256) void k_jacobi_round(double* __restrict__ a, int m, int n,
                                                      double* __restrict__ vw, int t, int np,
                                                      const double* __restrict__ fro2,
                                                      int32_t* __restrict__ rotated) {
    __shared__ double red[3][4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int pi = blockIdx.x;
    int p = rr_player(pi, t, np), q = rr_player(np - 1 - pi, t, np);
    if (p >= n || q >= n) return;                              // workgroup-uniform
    if (p > q) {
        const int tmp = p;
        p = q;
        q = tmp;
    }
    double* ap = a + static_cast<int64_t>(p) * m;
    double* aq = a + static_cast<int64_t>(q) * m;
    double al = 0.0, be = 0.0, ga = 0.0;
    for (int i = tid; i < m; i += 256) {
        const double x = ap[i], y = aq[i];
        al = fma(x, x, al);
        be = fma(y, y, be);
        ga = fma(x, y, ga);
    }
    al = wave_sum(al);
    be = wave_sum(be);
    ga = wave_sum(ga);
    if (lane == 0) {
        red[0][wave] = al;
        red[1][wave] = be;
        red[2][wave] = ga;
    }
    __syncthreads();
    al = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
    be = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
    ga = ((red[2][0] + red[2][1]) + red[2][2]) + red[2][3];
    constexpr double kTol = 1e-15, kTiny = 1e-28;
    if (!(fabs(ga) > kTol * sqrt(al * be)) || fmin(al, be) <= kTiny * *fro2) return;
    const double zeta = (be - al) / (2.0 * ga);
    const double az = fabs(zeta);
    const double tt = (az > 1e150 ? 0.5 / az : 1.0 / (az + sqrt(1.0 + zeta * zeta))) *
                      (zeta < 0.0 ? -1.0 : 1.0);
    const double c = 1.0 / sqrt(1.0 + tt * tt), sn = c * tt;
    for (int i = tid; i < m; i += 256) {
        const double x = ap[i], y = aq[i];
        ap[i] = c * x - sn * y;
        aq[i] = sn * x + c * y;
    }
    double* vp = vw + static_cast<int64_t>(p) * n;
    double* vq = vw + static_cast<int64_t>(q) * n;
    for (int i = tid; i < n; i += 256) {
        const double x = vp[i], y = vq[i];
        vp[i] = c * x - sn * y;
        vq[i] = sn * x + c * y;
    }
    if (tid == 0) __hip_atomic_store(rotated, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// sigma_j = |a_j|; the columns go out in decreasing sigma (ties in index
// order): u_j = a_j / sigma_j (0 when sigma_j = 0), or a_j itself with flag
// bit 0; v_j, times sigma_j with flag bit 1.  sweeps := nsweeps.  One
// workgroup.
__global__ __launch_bounds__(1024) void k_jacobi_finish(const double* __restrict__ a, int m, int n,
                                                        const double* __restrict__ vw,
                                                        double* __restrict__ sigma,
                                                        double* __restrict__ u_out,
                                                        double* __restrict__ v_out, int flags,
                                                        int nsweeps, int32_t* __restrict__ sweeps) {
    __shared__ double sig[kJacobiMaxN];
    __shared__ int rnk[kJacobiMaxN];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int j = wave; j < n; j += 16) {
        const double* aj = a + static_cast<int64_t>(j) * m;
        double ss = 0.0;
        for (int i = lane; i < m; i += 64) ss = fma(aj[i], aj[i], ss);
        ss = wave_sum(ss);
        if (lane == 0) sig[j] = sqrt(ss);
    }
    __syncthreads();
    for (int j = tid; j < n; j += 1024) {
        const double sj = sig[j];
        int rk = 0;
        for (int i = 0; i < n; ++i) rk += (sig[i] > sj || (sig[i] == sj && i < j)) ? 1 : 0;
        rnk[j] = rk;
    }
    __syncthreads();
    for (int j = wave; j < n; j += 16) {
        const int rj = rnk[j];
        const double sj = sig[j];
        if (lane == 0) sigma[rj] = sj;
        const double* aj = a + static_cast<int64_t>(j) * m;
        double* uo = u_out + static_cast<int64_t>(rj) * m;
        for (int i = lane; i < m; i += 64)
            uo[i] = (flags & 1) ? aj[i] : (sj > 0.0 ? aj[i] / sj : 0.0);
        const double* vj = vw + static_cast<int64_t>(j) * n;
        double* vo = v_out + static_cast<int64_t>(rj) * n;
        for (int i = lane; i < n; i += 64) vo[i] = (flags & 2) ? vj[i] * sj : vj[i];
    }
    if (tid == 0) *sweeps = nsweeps;
}

// X L^T = Y (trans) or X L = Y, in place on Y [m][n] (row stride ldy), L
// lower [n][n] (row stride ldl), by column blocks of kNb: the block's rows
// solved with k_trsm_rows, the remaining columns updated on the GEMM.
hipError_t trsm_right(int64_t m, int64_t n, const double* l, int64_t ldl, bool trans, double* y,
                      int64_t ldy, hipStream_t s) {
    const unsigned grid = trsm_grid(m);
    if (trans) {
        for (int64_t j0 = 0; j0 < n; j0 += kNb) {
            const int jb = static_cast<int>(n - j0 < kNb ? n - j0 : kNb);
            const int64_t j1 = j0 + jb;
            hipLaunchKernelGGL(k_trsm_rows<true>, dim3(grid), dim3(256), 0, s, y + j0, m, ldy,
                               l + j0 * ldl + j0, ldl, jb);
            if (j1 < n) {
                // Y[:, j1:] -= X[:, j0:j1] L[j1:, j0:j1]^T
                const hipError_t e = masq::launch_dgemm(m, n - j1, jb, y + j0, ldy, 1,
                                                        l + j1 * ldl + j0, 1, ldl, -1.0, 1.0,
                                                        y + j1, ldy, 1, false, s);
                if (e != hipSuccess) return e;
            }
        }
    } else {
        const int64_t nblk = (n + kNb - 1) / kNb;
        for (int64_t b = nblk - 1; b >= 0; --b) {
            const int64_t j0 = b * kNb;
            const int jb = static_cast<int>(n - j0 < kNb ? n - j0 : kNb);
            hipLaunchKernelGGL(k_trsm_rows<false>, dim3(grid), dim3(256), 0, s, y + j0, m, ldy,
                               l + j0 * ldl + j0, ldl, jb);
            if (j0 > 0) {
                // Y[:, :j0] -= X[:, j0:j1] L[j0:j1, :j0]
                const hipError_t e = masq::launch_dgemm(m, j0, jb, y + j0, ldy, 1, l + j0 * ldl, ldl,
                                                        1, -1.0, 1.0, y, ldy, 1, false, s);
                if (e != hipSuccess) return e;
            }
        }
    }
    return hipGetLastError();
}

}  // namespace

extern "C" {

masq_status masq_cholesky(int64_t n, double* a, int64_t lda, double ridge, int32_t* info,
                          double* trace, void* stream) {
    if (n < 0 || lda < n || n > 65535 || !(ridge >= 0.0) || !isfinite(ridge))
        return MASQ_ERR_SHAPE;
    if (!info || (n > 0 && !a)) return MASQ_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(info) & 3u) != 0 || (n > 0 && !aligned8(a)) ||
        (trace && !aligned8(trace)))
        return MASQ_ERR_ALIGN;
    if (n == 0) return MASQ_OK;                            // nothing enqueued
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_add_ridge, dim3(1), dim3(1024), 0, s, a, n, lda, ridge, trace, info);
    for (int64_t j0 = 0; j0 < n; j0 += kNb) {
        const int jb = static_cast<int>(n - j0 < kNb ? n - j0 : kNb);
        const int64_t j1 = j0 + jb;
        hipLaunchKernelGGL(k_potf2, dim3(1), dim3(256), 0, s, a + j0 * lda + j0, lda, jb, j0, info);
        if (j1 < n) {
            // L21 = A21 L11^-T, then A22 -= L21 L21^T (lower triangle)
            hipLaunchKernelGGL(k_trsm_rows<true>, dim3(trsm_grid(n - j1)), dim3(256), 0, s,
                               a + j1 * lda + j0, n - j1, lda, a + j0 * lda + j0, lda, jb);
            if (masq::launch_dgemm(n - j1, n - j1, jb, a + j1 * lda + j0, lda, 1, a + j1 * lda + j0,
                                   1, lda, -1.0, 1.0, a + j1 * lda + j1, lda, 1, true, s) !=
                hipSuccess)
                return MASQ_ERR_HIP;
        }
    }
    const unsigned gx = static_cast<unsigned>((n + 255) / 256 < 64 ? (n + 255) / 256 : 64);
    hipLaunchKernelGGL(k_zero_upper, dim3(gx, static_cast<unsigned>(n)), dim3(256), 0, s, a, n, lda);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

masq_status masq_trsm_right(int64_t m, int64_t n, const double* l, int64_t ldl, int32_t trans,
                            double* y, int64_t ldy, void* stream) {
    if (m < 0 || n < 0 || ldl < n || ldy < n || (trans != 0 && trans != 1) ||
        m > (1LL << 38) || n > (1LL << 24))
        return MASQ_ERR_SHAPE;
    if (m == 0 || n == 0) return MASQ_OK;
    if (!l || !y) return MASQ_ERR_NULL;
    if (!aligned8(l) || !aligned8(y)) return MASQ_ERR_ALIGN;
    (void)hipGetLastError();
    return trsm_right(m, n, l, ldl, trans == 1, y, ldy, static_cast<hipStream_t>(stream)) ==
                   hipSuccess
               ? MASQ_OK
               : MASQ_ERR_HIP;
}

masq_status masq_jacobi_svd(int64_t m, int64_t n, double* a, double* v_work, double* sigma,
                            double* u, double* v, int32_t flags, int32_t max_sweeps,
                            int32_t* sweeps, void* stream) {
    if (m < 1 || n < 1 || n > kJacobiMaxN || m > (1LL << 31) - 1 || flags < 0 || flags > 3 ||
        max_sweeps < 1 || max_sweeps > 1000)
        return MASQ_ERR_SHAPE;
    if (!a || !v_work || !sigma || !u || !v || !sweeps) return MASQ_ERR_NULL;
    if (!aligned8(a) || !aligned8(v_work) || !aligned8(sigma) || !aligned8(u) || !aligned8(v) ||
        (reinterpret_cast<uintptr_t>(sweeps) & 3u) != 0)
        return MASQ_ERR_ALIGN;
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    const int mi = static_cast<int>(m), ni = static_cast<int>(n), np = ni + (ni & 1);
    // |A|_F^2 is kept in sigma[0] until the end (k_jacobi_finish overwrites it);
    // *sweeps serves as the sweep's rotation flag
    hipLaunchKernelGGL(k_jacobi_init, dim3(1), dim3(1024), 0, s, a, mi, ni, v_work, sigma);
    int done = 0;
    for (; done < max_sweeps;) {
        hipLaunchKernelGGL(k_set_int, dim3(1), dim3(1), 0, s, sweeps, 0);
        for (int t = 0; t < np - 1; ++t)
            hipLaunchKernelGGL(k_jacobi_round, dim3(static_cast<unsigned>(np / 2)), dim3(256), 0, s,
                               a, mi, ni, v_work, t, np, sigma, sweeps);
        ++done;
        int32_t rotated = 1;
        if (hipGetLastError() != hipSuccess ||
            hipMemcpyAsync(&rotated, sweeps, sizeof(rotated), hipMemcpyDeviceToHost, s) !=
                hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess)
            return MASQ_ERR_HIP;
        if (rotated == 0) break;
    }
    hipLaunchKernelGGL(k_jacobi_finish, dim3(1), dim3(1024), 0, s, a, mi, ni, v_work, sigma, u, v,
                       static_cast<int>(flags), done, sweeps);
    return hipGetLastError() == hipSuccess ? MASQ_OK : MASQ_ERR_HIP;
}

}  // extern "C"
