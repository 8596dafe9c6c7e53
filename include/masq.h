/*
 * masq.h -- C ABI of the MI355X (gfx950) modality-aware W8A8 + low-rank linear.
 *
 * The layer is the inference rule of MASQuant (Modality-Aware Smoothing
 * Quantization), Sec. 4.3, final case equation.  For a token row x_t of
 * modality m (0 = text, the base modality; 1.. = vision, audio, ...):
 *
 *     xs_t  = x_t * inv_smooth[m]                       (X_m S_m^-1, Sec. 3.1/4.3)
 *     q_t   = Q(xs_t)  per-token symmetric int8         (eq. PTQ, z = 0, [-127,127])
 *     y_t   = (float(q_t . Wq^T) * delta_t) * w_scale   (the shared Q(S_t W))
 *     y_t  += (xs_t L1^m) L2^m          for m != text   (Cross-Modal Compensation,
 *                                                        eq. l1l2)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every array argument is a DEVICE pointer owned by the caller; it must stay
 *    valid until the work enqueued on `stream` has completed.  Inputs are never
 *    modified.  The library never allocates, frees or synchronises; scratch
 *    space comes from the caller's workspace.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Every entry point only enqueues work; device faults surface at the
 *    caller's next synchronisation.
 *  - Layouts are row-major.  Weight-like operands are [out][in] (the
 *    nn.Linear convention), so every contraction reads K-contiguous rows:
 *        x          [T][c_in]            f32 or bf16 (masq_dtype)
 *        modality   [T]                  int32, values in [0, n_mod)
 *        inv_smooth [n_mod][c_in]        f32, fl(1 / s^m)         (Sec. 4.2)
 *        wq         [c_out][c_in]        int8, Q(S_t W) transposed (Sec. 4.3)
 *        w_scale    [c_out]              f32, per-output-channel step
 *        l_down     [n_mod-1][rank][c_in]  (L1^m)^T, slot m-1 for modality m
 *        r_up       [n_mod-1][c_out][rank] (L2^m)^T
 *        y          [T][c_out]           f32 or bf16
 *  - Preconditions, checked before anything is enqueued (on failure nothing is
 *    enqueued and outputs are untouched): non-null pointers (except where
 *    marked nullable), T >= 0, c_in > 0 and c_in % 16 == 0, c_out > 0 and
 *    c_out % 16 == 0, rank == 0 or rank % 16 == 0 (rank <= 256),
 *    for every call that accumulates (GEMM and whole layer) c_in small enough
 *    that int32 accumulation is exact: c_in <= 133136 (= 127 * 127 * c_in
 *    below 2^31, a multiple of 16) with int8 codes, c_in <= 150976 with the
 *    packed 4-bit weight (127 * 112 * c_in below 2^31, a multiple of 64),
 *    1 <= n_mod <= 4, 16-byte aligned pointers, a large enough workspace.
 *    T == 0 is a successful no-op once sizes and dtypes are valid (pointers
 *    may then be NULL: nothing is read or written).
 *  - Modality ids outside [0, n_mod) are treated as text (memory-safe, but
 *    not a supported input); non-finite inputs give unspecified results.
 *  - Rounding contract (bit-exact parts): the smoothing is one fp32 multiply;
 *    delta_t = fl(amax_t / 127) and the codes use a multiply by
 *    fl(127 / amax_t), both correctly rounded divisions; codes round half to
 *    even; an all-zero row gives delta = 0 and zero codes; int32 accumulation
 *    is exact; dequantisation is fl(fl(float(acc) * delta_t) * w_scale[o]);
 *    bf16 outputs are one round-to-nearest-even of the fp32 result.
 *  - No C++ exception crosses this boundary.  The library's only global
 *    state is the static scratch of masq_linear_fused_noalloc (and its
 *    per-device address); every other call is safe concurrently if their
 *    outputs and workspaces do not overlap.
 */
#ifndef MASQ_H
#define MASQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MASQ_OK = 0,
    MASQ_ERR_NULL = 1,        /* a required pointer is NULL                      */
    MASQ_ERR_SHAPE = 2,       /* a size violates the preconditions above         */
    MASQ_ERR_DTYPE = 3,       /* unknown or unsupported dtype combination        */
    MASQ_ERR_ALIGN = 4,       /* a pointer is not 16-byte aligned                */
    MASQ_ERR_WORKSPACE = 5,   /* workspace smaller than the query says           */
    MASQ_ERR_HIP = 6,         /* a kernel launch was rejected by the runtime     */
    MASQ_ERR_UNSUPPORTED = 7, /* valid request this build does not implement     */
    MASQ_ERR_SCRATCH = 8,     /* needs more than the static scratch (below)      */
    /* not statuses: they make every int32 a value of the type, so that any
     * integer a caller passes to masq_status_str is well defined */
    MASQ_STATUS_RANGE_LO_ = -2147483647 - 1,
    MASQ_STATUS_RANGE_HI_ = 2147483647
} masq_status;

typedef enum {
    MASQ_F32 = 0,
    MASQ_BF16 = 1,
    /* not dtypes: every int32 is a value of the type, so an unknown value
     * reaches the library's check and gives MASQ_ERR_DTYPE */
    MASQ_DTYPE_RANGE_LO_ = -2147483647 - 1,
    MASQ_DTYPE_RANGE_HI_ = 2147483647
} masq_dtype;

/* Version of this interface (bumped on any signature or semantics change). */
int masq_abi_version(void);

/* Human-readable name of a status code (static storage, never NULL). */
const char* masq_status_str(masq_status s);

/*
 * Smoothing and per-token quantisation (Sec. 4.3 X_m S_m^-1; eq. PTQ).
 * Writes q [T][c_in] int8 and x_scale [T] f32 (delta_t).
 * x_dt: MASQ_F32 or MASQ_BF16.
 */
masq_status masq_smooth_quant(const void* x, masq_dtype x_dt, const int32_t* modality,
                              const float* inv_smooth, int64_t T, int64_t c_in,
                              int32_t n_mod, int8_t* q, float* x_scale, void* stream);

/*
 * Product with the shared quantised weight, Q(X S^-1) . Q(S_t W) (Sec. 4.3).
 * acc (nullable): int32 [T][c_out] exact accumulators.
 * y   (nullable): the dequantised product in y_dt (no compensation).
 * At least one of acc, y must be non-null.
 */
masq_status masq_w8a8_gemm(const int8_t* q, const float* x_scale, const int8_t* wq,
                           const float* w_scale, int64_t T, int64_t c_in, int64_t c_out,
                           int32_t* acc, void* y, masq_dtype y_dt, void* stream);

/*
 * Cross-Modal Compensation alone (Sec. 4.3, eq. l1l2): for every row with
 * modality m != 0, y[t] += (x_t S_m^-1 L1^m) L2^m, accumulated in fp32 and
 * rounded once into y's dtype.  Text rows of y are left untouched.
 * y is read-modify-write.  lr_dt is the dtype of l_down and r_up.
 */
masq_status masq_lowrank_comp(const void* x, masq_dtype x_dt, const int32_t* modality,
                              const float* inv_smooth, const void* l_down,
                              const void* r_up, masq_dtype lr_dt, int64_t T,
                              int64_t c_in, int64_t c_out, int32_t rank, int32_t n_mod,
                              void* y, masq_dtype y_dt, void* stream);

/*
 * The whole layer (Sec. 4.3 final case equation): smoothing, per-token int8
 * quantisation, the shared-weight int8 GEMM with int32 accumulation,
 * dequantisation and, on non-text rows only, the rank-r compensation; y is
 * fully overwritten.  workspace: device scratch of at least
 * masq_linear_fused_workspace_bytes(...) bytes, 256-byte aligned, whose
 * contents need not be initialised; it must not be shared by calls that may
 * run concurrently.
 */
masq_status masq_linear_fused(const void* x, masq_dtype x_dt, const int32_t* modality,
                              const float* inv_smooth, const int8_t* wq,
                              const float* w_scale, const void* l_down, const void* r_up,
                              masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out,
                              int32_t rank, int32_t n_mod, void* y, masq_dtype y_dt,
                              void* workspace, size_t workspace_bytes, void* stream);

size_t masq_linear_fused_workspace_bytes(int64_t T, int64_t c_in, int64_t c_out,
                                         int32_t rank, int32_t n_mod);

/*
 * The whole layer without a workspace argument, for callers that cannot
 * allocate device memory (code under stream or graph capture, tight serving
 * loops, harnesses that forbid allocation).  Same arguments, semantics,
 * kernels and results as masq_linear_fused (bit for bit), except that the
 * scratch comes from a static device array of MASQ_SCRATCH_BYTES bytes that
 * the library holds on every GPU it runs on until the process ends.  Its
 * device address is looked up once per device (the first call with that
 * device current); no call allocates or frees memory.
 *
 * Limit: problems whose masq_linear_fused_workspace_bytes(...) exceeds
 * MASQ_SCRATCH_BYTES are rejected with MASQ_ERR_SCRATCH before anything is
 * enqueued (use masq_linear_fused with a workspace for those).  Every call on
 * one GPU shares that GPU's array: calls that may overlap in time on one GPU
 * (different streams, different host threads) race and give wrong results;
 * calls ordered on one stream are safe.  Whatever must start at zero (arrival
 * counters) is cleared by each call's own kernels, so leftovers of an earlier
 * call never matter.  MASQ_ERR_HIP if the array's address cannot be obtained.
 */
#define MASQ_SCRATCH_BYTES ((size_t)64 << 20)
masq_status masq_linear_fused_noalloc(const void* x, masq_dtype x_dt, const int32_t* modality,
                                      const float* inv_smooth, const int8_t* wq,
                                      const float* w_scale, const void* l_down,
                                      const void* r_up, masq_dtype lr_dt, int64_t T,
                                      int64_t c_in, int64_t c_out, int32_t rank,
                                      int32_t n_mod, void* y, masq_dtype y_dt, void* stream);

/*
 * The MAS-only comparator (Sec. 4.2, the inference with per-modality
 * smoothing factors and per-modality weights before the shared weight of
 * Sec. 4.3): for a token row x_t of modality m,
 *     y_t = (float(Q(x_t S_m^-1) . wq[m]^T) * delta_t) * w_scale[m]
 * with the same smoothing, per-token quantisation, exact int32 accumulation,
 * dequantisation order and output rounding as masq_linear_fused, and no
 * compensation.  The rows are grouped by modality on the device (a stable
 * counting sort of the ids) and each 256-row tile of one modality's rows is
 * multiplied by that modality's weight; the host never reads the ids, and
 * any layout of modalities works.  Batches of at most 16 tokens (with
 * c_in <= 20480) instead stream each modality's weight once through the
 * small-batch GEMM, which stores only the rows of that modality's tokens.
 *   wq       [n_mod][c_out][c_in] int8, Q(S_m W) transposed, per modality
 *   w_scale  [n_mod][c_out] f32
 *   inv_smooth, x, modality, y as for masq_linear_fused (ids outside
 *   [0, n_mod) are treated as text).
 * workspace: at least masq_mas_only_workspace_bytes(...) bytes, 256-byte
 * aligned, contents need not be initialised; not shared by concurrent calls.
 * c_in must be a multiple of 64 (else MASQ_ERR_UNSUPPORTED); the other
 * preconditions and errors are masq_linear_fused's (rank does not apply).
 */
masq_status masq_mas_only_linear(const void* x, masq_dtype x_dt, const int32_t* modality,
                                 const float* inv_smooth, const int8_t* wq, const float* w_scale,
                                 int64_t T, int64_t c_in, int64_t c_out, int32_t n_mod, void* y,
                                 masq_dtype y_dt, void* workspace, size_t workspace_bytes,
                                 void* stream);
size_t masq_mas_only_workspace_bytes(int64_t T, int64_t c_in, int64_t c_out, int32_t n_mod);

/*
 * The two launch stages masq_linear_fused is made of, with identical
 * arguments, exposed so that a caller can place events or other stream work
 * between them.  stage1: smoothing, quantisation and the rank-r
 * down-projection into the workspace.  stage2: the int8 GEMM with the fused
 * dequantisation and compensation epilogue, reading the workspace stage1
 * wrote.  stage1 followed by stage2 on one stream equals masq_linear_fused.
 */
masq_status masq_linear_stage1(const void* x, masq_dtype x_dt, const int32_t* modality,
                               const float* inv_smooth, const int8_t* wq,
                               const float* w_scale, const void* l_down, const void* r_up,
                               masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out,
                               int32_t rank, int32_t n_mod, void* y, masq_dtype y_dt,
                               void* workspace, size_t workspace_bytes, void* stream);
masq_status masq_linear_stage2(const void* x, masq_dtype x_dt, const int32_t* modality,
                               const float* inv_smooth, const int8_t* wq,
                               const float* w_scale, const void* l_down, const void* r_up,
                               masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out,
                               int32_t rank, int32_t n_mod, void* y, masq_dtype y_dt,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * 4-bit shared weight (W4A8, the low-bit setting of Tables 1-2).  Q(S_t W)
 * is quantised per output channel to 4-bit codes (eq. PTQ with b = 4:
 * codes in [-7, 7], w_scale[o] = max_i |(S_t W)[o][i]| / 7) and stored
 * packed, two codes per byte: row o of wq4 is c_in / 2 bytes; the 4-byte
 * word g of a row holds codes 8g .. 8g + 7, its byte b carrying code 8g + b
 * in the low nibble and code 8g + b + 4 in the high nibble, two's
 * complement.  The activations stay 8-bit.  Each entry point matches its
 * int8 counterpart called with the unpacked codes as wq, bit for bit (the
 * product of codes is still summed exactly in int32), with the same
 * arguments, workspace (masq_linear_fused_workspace_bytes) and errors, and
 * in addition: c_in must be a multiple of 64 (else MASQ_ERR_SHAPE); wq4
 * must be 16-byte aligned (else MASQ_ERR_ALIGN).  The weight bytes read
 * from memory halve, which is what bounds small batches.
 */
masq_status masq_w4a8_gemm(const int8_t* q, const float* x_scale, const uint8_t* wq4,
                           const float* w_scale, int64_t T, int64_t c_in, int64_t c_out,
                           int32_t* acc, void* y, masq_dtype y_dt, void* stream);
masq_status masq_linear_fused_w4a8(const void* x, masq_dtype x_dt, const int32_t* modality,
                                   const float* inv_smooth, const uint8_t* wq4,
                                   const float* w_scale, const void* l_down, const void* r_up,
                                   masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out,
                                   int32_t rank, int32_t n_mod, void* y, masq_dtype y_dt,
                                   void* workspace, size_t workspace_bytes, void* stream);
masq_status masq_linear_stage1_w4a8(const void* x, masq_dtype x_dt, const int32_t* modality,
                                    const float* inv_smooth, const uint8_t* wq4,
                                    const float* w_scale, const void* l_down, const void* r_up,
                                    masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out,
                                    int32_t rank, int32_t n_mod, void* y, masq_dtype y_dt,
                                    void* workspace, size_t workspace_bytes, void* stream);
masq_status masq_linear_stage2_w4a8(const void* x, masq_dtype x_dt, const int32_t* modality,
                                    const float* inv_smooth, const uint8_t* wq4,
                                    const float* w_scale, const void* l_down, const void* r_up,
                                    masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out,
                                    int32_t rank, int32_t n_mod, void* y, masq_dtype y_dt,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * Calibration on the GPU: the exact part of the offline calibration that
 * gives the smoothing factors and the shared weight (the compensation
 * factors L1, L2 need a whitening and a truncated SVD and are not here).
 * Each result is bit-exact against its definition: maxima are exact, the
 * factor and the weight step are computed in fp64 and rounded once to fp32.
 *
 * masq_channel_range: range[m][i] = max |x_ti| over the tokens t of modality
 * m (Sec. 4.1, R^m); 0 where a modality has no tokens.  x [T][c_in] f32 or
 * bf16; modality [T]; tokens whose id is outside [0, n_mod) belong to no
 * modality.  range: [n_mod][c_in] f32, fully overwritten.  T == 0 gives
 * zeros.
 *
 * masq_smoothing_factors: the MAS initial factors (Sec. 4.2, alpha = 1/2),
 * smooth[m][i] = fl32(sqrt(max(range[m][i], 1e-5) / max(w_i, 1e-5))) with
 * w_i = max_j |w[i][j]| in fp64, and inv_smooth[m][i] = fl32(1 / smooth[m][i])
 * (correctly rounded).  w is the float weight in the paper's layout
 * [c_in][c_out] f32; smooth, inv_smooth: [n_mod][c_in] f32.
 *
 * masq_quantize_weight: the shared weight Q(S_t W) (Sec. 4.3; eq. PTQ per
 * output channel, symmetric, z = 0): with v_io = smooth_text[i] * w[i][o]
 * (exact in fp64), w_scale[o] = fl32(d_o), d_o = max_i |v_io| / qmax, and
 * wq[o][i] = clamp(rint(v_io / d_o), -qmax, qmax) (fp64, round half to
 * even; 0 when d_o = 0).  bits = 8 (qmax 127) or 4 (qmax 7, the W4A8
 * setting; codes are returned one per byte, unpacked).  wq: [c_out][c_in]
 * int8; w_scale: [c_out] f32.
 *
 * Preconditions as for the layer calls (c_in, c_out multiples of 16,
 * 1 <= n_mod <= 4, 16-byte aligned pointers); violations return an error
 * before anything is enqueued.
 */
masq_status masq_channel_range(const void* x, masq_dtype x_dt, const int32_t* modality,
                               int64_t T, int64_t c_in, int32_t n_mod, float* range,
                               void* stream);
masq_status masq_smoothing_factors(const float* range, const float* w, int64_t c_in,
                                   int64_t c_out, int32_t n_mod, float* smooth,
                                   float* inv_smooth, void* stream);
masq_status masq_quantize_weight(const float* w, const float* smooth_text, int64_t c_in,
                                 int64_t c_out, int32_t bits, int8_t* wq, float* w_scale,
                                 void* stream);

/* Inputs and products of the compensation factors' calibration (Sec. 3.2
 * and 4.3; eq. l1l2): L1^m, L2^m minimise ||Z_m (dW_m - L1 L2)||_F over the
 * smoothed calibration rows Z_m = X_m S_m^-1 of modality m, with the weight
 * difference dW_m = S_m W - Q(S_t W).  The whitening of Z_m (from its Gram
 * matrix) and the truncated SVD are built from these calls; their small
 * decompositions are the calls below (masq_cholesky, masq_trsm_right,
 * masq_jacobi_svd).
 *
 * masq_gather_smoothed: z[i][c] = x[rows[i]][c] / smooth[c] in fp64 (the
 * operands are exact, the division correctly rounded), for i < n_rows; a
 * row index outside [0, T) gives a zero row.  x: [T][c_in] f32 or bf16;
 * rows: [n_rows] int32; smooth: [c_in] f32 (S_m's diagonal); z: [n_rows]
 * [c_in] f64, caller-allocated.  n_rows = 0 is a no-op.
 *
 * masq_weight_difference: dw[i][o] = smooth[i] * w[i][o] - wq[o][i] *
 * w_scale[o] in fp64 (both products are exact, so the subtraction is the
 * only rounding).  w: [c_in][c_out] f32 (paper layout); smooth: [c_in] f32
 * (S_m); wq: [c_out][c_in] int8 codes of Q(S_t W) (8- or 4-bit, one code a
 * byte) with steps w_scale [c_out] f32; dw: [c_in][c_out] f64.
 *
 * masq_dgemm: c[i * ldc + j] = sum_k A(i, k) B(k, j) (+ beta * c[i * ldc +
 * j] when beta != 0) for i < m, j < n, in fp64, with A(i, k) = a[i *
 * a_row_stride + k * a_col_stride] and B(k, j) = b[k * b_row_stride + j *
 * b_col_stride] (element strides, so a transposed operand is a stride swap).
 * Each sum runs in increasing k with fused multiply-adds; beta * c is added
 * after it.  c must not overlap a or b.  k = 0 gives beta * c (or zeros);
 * m = 0 or n = 0 is a no-op.  Pointers 8-byte aligned; m <= 65535 * 128.
 *
 * Preconditions as for the calls above; violations return an error before
 * anything is enqueued.
 */
masq_status masq_gather_smoothed(const void* x, masq_dtype x_dt, int64_t T, int64_t c_in,
                                 const int32_t* rows, int64_t n_rows, const float* smooth,
                                 double* z, void* stream);
masq_status masq_weight_difference(const float* w, const float* smooth, const int8_t* wq,
                                   const float* w_scale, int64_t c_in, int64_t c_out,
                                   double* dw, void* stream);
masq_status masq_dgemm(int64_t m, int64_t n, int64_t k, const double* a, int64_t a_row_stride,
                       int64_t a_col_stride, const double* b, int64_t b_row_stride,
                       int64_t b_col_stride, double beta, double* c, int64_t ldc, void* stream);

/* Factorisations of the compensation factors' calibration (Sec. 3.2 and
 * 4.3; eq. l1l2), in fp64 on the GPU.  The whitening T of Z_m only has to
 * satisfy T^T T = C with C = Z_m^T Z_m + eps I: the Cholesky factor T = L^T
 * (C = L L^T) serves as well as the symmetric root, since T' = Q T with Q
 * orthogonal leaves L1 = T^-1 U_r and L2 = Sigma_r V_r^T of the truncated
 * SVD of T dW unchanged.  The randomized range finder's orthogonalisations
 * are CholeskyQR (Gram matrix, its Cholesky factor, a triangular solve), and
 * the SVD of the small projected matrix is a one-sided Jacobi SVD.
 *
 * masq_cholesky: a [n][n] (row stride lda >= n), symmetric, overwritten by
 * L, lower triangular with L L^T = a + (ridge * tr(a) / n) I (only the lower
 * triangle of a is read; the strict upper triangle of the result is zero).
 * Blocked right-looking factorisation with 64 x 64 diagonal blocks.  info
 * (device int32, 4-byte aligned) := 0, or k + 1 for the first pivot k that
 * is not positive (which is then taken as 1 so that the call runs to its
 * end; L is then meaningless); trace (device fp64, optional) := tr(a) before
 * the shift.  0 <= n <= 65535 (n = 0 enqueues nothing and writes neither
 * info nor trace); ridge >= 0 and finite.
 *
 * masq_trsm_right: y [m][n] (row stride ldy >= n) overwritten by the X with
 * X L^T = Y (trans = 1) or X L = Y (trans = 0), for l [n][n] (row stride ldl
 * >= n) lower triangular with a nonzero diagonal, as masq_cholesky leaves it
 * (entries above the diagonal are not read).  Blocked by 64 columns: each
 * diagonal block's solves row by row, the rest on the fp64 GEMM.  l and y
 * must not overlap.
 *
 * masq_jacobi_svd: the SVD of the m x n matrix A whose column j is a[j * m ..
 * j * m + m) (a is overwritten), 1 <= n <= 1024, by one-sided Jacobi
 * rotations (round-robin pairs, a pair left alone when |a_p . a_q| <= 1e-15
 * |a_p| |a_q| or when a column's squared norm is at most 1e-28 |A|_F^2, a
 * numerically zero column) until a sweep rotates nothing or max_sweeps
 * (1..1000) sweeps have run; the count goes to *sweeps (device int32,
 * 4-byte aligned, required).  Each round of disjoint pairs is one launch (a
 * workgroup a pair); unlike the other calls this one waits for the stream
 * once per sweep, to read whether the sweep rotated anything.  Outputs, in
 * decreasing singular value (ties in column order): sigma [n]; u [n][m], row
 * j the left singular vector u_j (0 when sigma_j = 0), or sigma_j u_j with
 * flags bit 0; v [n][n], row j the right singular vector v_j, or sigma_j v_j
 * with flags bit 1; A = sum_j sigma_j u_j v_j^T.  v_work [n][n] is scratch.
 * No output may overlap another or a.
 *
 * Pointers 8-byte aligned unless stated; violations return an error before
 * anything is enqueued.
 */
masq_status masq_cholesky(int64_t n, double* a, int64_t lda, double ridge, int32_t* info,
                          double* trace, void* stream);
masq_status masq_trsm_right(int64_t m, int64_t n, const double* l, int64_t ldl, int32_t trans,
                            double* y, int64_t ldy, void* stream);
masq_status masq_jacobi_svd(int64_t m, int64_t n, double* a, double* v_work, double* sigma,
                            double* u, double* v, int32_t flags, int32_t max_sweeps,
                            int32_t* sweeps, void* stream);

/* The MAS factor optimisation (Sec. 4.2, eq. mas_quant): per modality m,
 * minimise L(S_m) = mean |Q(X_m S_m^-1) Q(S_m W) - X_m W| over the
 * smoothing factors, with the inference quantizers (masq_smooth_quant,
 * masq_quantize_weight) in the forward pass and the straight-through
 * estimator in the backward pass:
 *   dL/ds_i = -(1 / s_i^2) sum_t x_ti A_ti + sum_o w_io B_io,
 *   G = sign(Xq Wq - X W) / (T N), A = G Wq^T, B = Xq^T G
 * (Xq, Wq the dequantized operands; A and B formed with masq_dgemm).
 *
 * masq_dequantize_rows: out[r][c] = codes[r][c] * scale[r] in fp64 (exact)
 * for codes [rows][cols] int8 and scale [rows] f32: Xq from the per-token
 * codes and steps, or Wq^T [c_out][c_in] from the shared-weight codes.
 *
 * masq_mae_sign: g[e] = sign(y[e] - ref[e]) / count (0 on ties) for the
 * count elements of y and ref (fp64); partial[b] = the sum of |y - ref|
 * over elements [4096 b, 4096 b + 4096), in a fixed order, for the
 * masq_mae_partials(count) blocks: the loss is their sum / count.
 * g must not overlap y or ref.
 *
 * masq_mas_gradient: grad[i] = -colpart[i] / s_i^2 + sum_o w[i][o] b[i][o]
 * with colpart[i] = sum_t x[t][i] a[t][i] (written to colpart, [c_in] f64
 * caller scratch): x, a [T][c_in] f64 (the batch's raw rows and A), w, b
 * [c_in][c_out] f64 (W and B), smooth [c_in] f32 (the factors used in the
 * forward pass), grad [c_in] f64.  Sums run in increasing t and in a fixed
 * lane order over o.
 *
 * Pointers 16-byte (dequantize) or 8-byte (the others) aligned; violations
 * return an error before anything is enqueued.
 */
masq_status masq_dequantize_rows(const int8_t* codes, const float* scale, int64_t rows,
                                 int64_t cols, double* out, void* stream);
int64_t masq_mae_partials(int64_t count);
masq_status masq_mae_sign(const double* y, const double* ref, int64_t count, double* g,
                          double* partial, void* stream);
masq_status masq_mas_gradient(const double* x, const double* a, const double* w, const double* b,
                              const float* smooth, int64_t T, int64_t c_in, int64_t c_out,
                              double* colpart, double* grad, void* stream);

/* masq_mae_loss: loss[0] = (partial[0] + ... + partial[P - 1]) / count, summed
 * in that order, over the P = masq_mae_partials(count) block sums that
 * masq_mae_sign left (count = 0 gives 0).  One device scalar, so a run of
 * optimisation steps keeps its losses on the device.
 *
 * masq_adam_log_step: Adam (Kingma and Ba 2015) on theta = ln s, the
 * parameterisation of the factors; theta, m1, m2 [c_in] fp64 (state),
 * smooth / inv_smooth [c_in] f32: the factors s the step's forward pass
 * used on entry, the next ones (s = fl32(exp(theta)), inv = fl32(1 / s)) on
 * return.  step = 0 starts the run: theta = ln s, m1 = m2 = 0, and s, inv
 * from theta (grad unused).  step >= 1 applies the gradient grad [c_in] fp64
 * (dL/ds): g = lam s grad, m1 = b1 m1 + (1 - b1) g, m2 = b2 m2 + ((1 - b2) g)
 * g, theta -= (lr (m1 / (1 - b1^step))) / (sqrt(m2 / (1 - b2^step)) + eps),
 * each operation rounded once.  Requires 0 <= b1, b2 < 1, eps > 0, lr >= 0.
 */
masq_status masq_mae_loss(const double* partial, int64_t count, double* loss, void* stream);
masq_status masq_adam_log_step(double* theta, double* m1, double* m2, const double* grad,
                               float* smooth, float* inv_smooth, int64_t c_in, double lam,
                               double lr, double b1, double b2, double eps, int64_t step,
                               void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MASQ_H */
