// Internal declarations shared by the kernel and C-ABI translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace masq {

// Tile shape of the int8 GEMM: 256 x 256 output tile per workgroup of four
// wave64s (2 x 2, each wave 128 x 128), 128-byte K stages, double-buffered.
constexpr int kTileM = 256;
constexpr int kTileN = 256;
constexpr int kTileK = 128;
constexpr int kRowsDown = 16;     // rows per down-projection tile
constexpr int kDownRows = kRowsDown;
constexpr int kDownStep = 512;    // k granularity of a down-projection slice (128 per wave)
constexpr int kMaxRank = 256;
constexpr int kSmallMaxT = 16;    // batches this small use the Wq-streaming GEMM
constexpr int kSmallSlices = 64;  // down-projection k slices (at most; >= 512 columns each) summed by that GEMM
constexpr int kUBatch = 16;        // slice partials of u a thread keeps in flight when adding them

// The small-batch path: the Wq-streaming GEMM, which also adds the
// down-projection's k-slice partials itself.
inline bool small_path(int64_t T, int64_t K) { return T <= kSmallMaxT && K % 64 == 0; }

// Layout of the fused layer's int8 activation codes in its workspace.  Plain:
// code (t, k) at byte t K + k.  Row-paired (paired_codes: K % 64 == 0 and a
// batch past the small path, whose GEMM takes its A operand by LDS DMA): rows
// 2i and 2i + 1 interleave in 64-byte pieces, code (t, k) at byte
// (t / 2) 2K + (k / 64) 128 + (t % 2) 64 + k % 64, so that the two rows'
// 64-column pieces of one K stage are a single 128-byte line (one L2 request
// where the plain rows take two 64-byte ones).  An odd batch's last pair has
// an unused second row (the workspace holds T rounded up to even rows).
inline bool paired_codes(int64_t T, int64_t K) { return !small_path(T, K) && K % 64 == 0; }
__host__ __device__ inline int64_t code_row(int64_t t, int64_t K, bool pair) {
    return pair ? (t >> 1) * 2 * K + (t & 1) * 64 : t * K;
}
__host__ __device__ inline int code_col(int k, bool pair) { return pair ? k + (k & ~63) : k; }

// Stage 1 of large batches with bf16 factors, rank <= 64 (fused_stage1_ok),
// in its wide form: the down-projection runs over 128-row tiles and S k
// slices of kslice columns (about 512 workgroups, slices of at least 256
// columns); the quantisation kernel then adds the slices' partials into u.
// The fused stage 1 walks each 16-row tile along its whole row, so its time
// grows with K and hardly with T until its T / 16 workgroups reach one per
// compute unit (4096 tokens); it keeps rows shorter than 2048 columns (too
// few k slices for the wide form) and, from 4096 tokens on, rows shorter
// than 8192 columns (where reading each row once, not twice, wins).
constexpr int64_t kDownWideMinK = 2048;
constexpr int64_t kFusedFullT = 4096;
constexpr int64_t kDownWideLongK = 8192;
constexpr int kDownWideRows = 128;
inline bool down_wide(int64_t T, int64_t K) {
    return K >= kDownWideMinK && (T < kFusedFullT || K >= kDownWideLongK);
}
inline void plan_down_wide(int64_t T, int64_t K, int& S, int& kslice) {
    const int64_t tiles = (T + kDownWideRows - 1) / kDownWideRows;
    int64_t want = (512 + tiles - 1) / tiles;
    const int64_t most = (K + 255) / 256;
    if (want > most) want = most;
    if (want < 1) want = 1;
    kslice = static_cast<int>(((K + want - 1) / want + 63) / 64 * 64);
    S = static_cast<int>((K + kslice - 1) / kslice);
}

// K split of the 256 x 256 tile GEMM for grids with few tiles (fused layer,
// K % 64 == 0): S slices of at least 8 64-byte stages; each slice's int32
// accumulators go to the workspace and the last slice of a tile to arrive
// adds them and finishes the tile.
constexpr int kSplitMaxTiles = 128;   // grids with at least this many tiles are not split
constexpr int kSplitMax = 4;
inline int plan_gemm_splits(int64_t T, int64_t K, int64_t N) {
    if (T <= 0 || N <= 0 || small_path(T, K) || K % 64 != 0) return 1;
    const int64_t tiles = ((T + kTileM - 1) / kTileM) * ((N + kTileN - 1) / kTileN);
    if (tiles >= kSplitMaxTiles) return 1;
    int64_t S = 256 / tiles;
    if (S > kSplitMax) S = kSplitMax;
    if (S > (K / 64) / 8) S = (K / 64) / 8;
    return S < 1 ? 1 : static_cast<int>(S);
}

// Decode GEMM of the fused small-batch path: a workgroup covers kDecCh output
// channels and one k slice of at most kDecSteps 64-byte steps (its waves hold
// every Wq step of the slice in registers).  ns slices of sp steps (the last
// may be shorter, none is empty), ngroups channel groups.
constexpr int kDecSteps = 40;
constexpr int kDecCh = 64;
constexpr int kDecMaxSlices = 8;    // longer rows (K > 8 * 40 * 64) take the single-pass GEMM
constexpr int kDecCmcBytes = 32768;  // LDS for the compensation operands of a k-slice workgroup
inline void plan_decode(int64_t K, int64_t N, int& ns, int& sp, int& ngroups) {
    const int64_t nsteps = K / 64;
    const int64_t ns0 = (nsteps + kDecSteps - 1) / kDecSteps;
    sp = static_cast<int>((nsteps + ns0 - 1) / ns0);
    ns = static_cast<int>((nsteps + sp - 1) / sp);
    ngroups = static_cast<int>((N + kDecCh - 1) / kDecCh);
}
constexpr int64_t kRowsPerWaveMinT = 256;   // batches this large quantise one row per wave

enum class DT : int { F32 = 0, BF16 = 1 };

struct LinearArgs {
    const void* x;
    DT x_dt;
    const int32_t* modality;
    const float* inv_smooth;
    const int8_t* wq;
    const float* w_scale;
    const void* l_down;
    const void* r_up;
    DT lr_dt;
    int64_t T, K, N;
    int rank, n_mod;
    void* y;
    DT y_dt;
};

// Workspace carve-up of the fused layer.
struct Workspace {
    int8_t* q;         // codes, row-paired when `pair` (code_row / code_col)
    bool pair;         // paired_codes(T, K)
    float* x_scale;
    float* u;          // [T][rank] fp32 down-projection u = (x S^-1) L1
    uint8_t* u_hl;     // [T][256 B] u as bf16 hi | lo rows (rank <= 64, large batches)
    float* u_part;     // [n_kslices][T][rank] fp32 partial sums over k slices (n_kslices > 1)
    int* tickets;      // [ceil(T / kDownRows)] arrival counters of the slice workgroups
    int32_t* dec_part; // small-batch path: [ns][kSmallMaxT][N] int32 partial sums per k slice,
                       // then [kSmallMaxT][N] fp32 compensation terms
    int* dec_tickets;  // small-batch path: [ngroups] arrival counters (zeroed by stage 1)
    int dec_ns, dec_sp, dec_groups;   // plan_decode of the small-batch path
    int gk_splits;     // plan_gemm_splits
    int32_t* gk_part;  // [tiles][gk_splits][256 * 256] int32 slice accumulators (gk_splits > 1)
    int* gk_tickets;   // [tiles] arrival counters (gk_splits > 1); follow `tickets` when both exist
    int n_zero;        // ints from zero_base that stage 1 clears
    int* zero_base;
    int dw_slices, dw_kslice;   // plan_down_wide (dw_part != nullptr)
    float* dw_part;    // [dw_slices][T][rank] fp32 partials of the wide down-projection
    float* dl_part;    // [down_lds_slices(T, K)][T][rank] fp32 partials of k_down_lds
    int n_kslices;
    int kslice;
    size_t bytes;
};

Workspace plan_workspace(void* base, int64_t T, int64_t K, int64_t N, int rank, int n_mod);

// zero_ints / n_zero: optional array the kernel clears on the way (the
// down-projection's tickets, which must start at zero).
// fin (optional): add the wide down-projection's slice partials into u (and
// its bf16 hi/lo rows) while quantising.  pair: write the codes row-paired
// (code_row / code_col; K % 64 == 0).
struct UFinish {
    const float* part;   // [slices][T][r]
    int slices, r;
    float* u;
    uint8_t* u_hl;       // may be null
};
hipError_t launch_smooth_quant(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               int64_t T, int64_t K, int n_mod, int8_t* q, float* x_scale,
                               int* zero_ints, int n_zero, hipStream_t s,
                               const UFinish* fin = nullptr, bool pair = false);

hipError_t launch_down_wide(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                            const void* l_down, int64_t T, int64_t K, int rank, int n_mod,
                            const Workspace& w, hipStream_t s);

hipError_t launch_lowrank_down(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, DT lr_dt, int64_t T, int64_t K, int rank,
                               int n_mod, const Workspace& w, hipStream_t s);

// Stage 1 in one kernel for bf16 factors and rank <= 64 (fused_stage1_ok):
// smoothing, quantisation and the down-projection, reading each row once.
inline bool fused_stage1_ok(int64_t T, int64_t K, int rank, DT lr_dt) {
    return !small_path(T, K) && lr_dt == DT::BF16 && rank > 0 && rank <= 64;
}
// The register-resident form of stage 1 (smoothing, quantisation and, for
// bf16 factors of rank <= 64, the down-projection): bf16 activations, 16 rows
// per workgroup of kFrWaves waves, rows of a multiple of 64 columns up to
// kFrWaves x kFrMaxPairs x 64 (each wave holds at most kFrMaxPairs 64-column
// pairs of its 16 rows in registers), and the smoothing factors of every
// modality within kFrInvFloats floats of LDS, each modality's row at a
// stride of fr_inv_stride(K) floats (whole 1 KB blocks plus 16 bytes, so that
// lanes reading different modalities' factors hit different banks).
constexpr int kFrWaves = 8;
constexpr int kFrMaxPairs = 8;
constexpr int kFrInvFloats = 12304;
__host__ __device__ inline int64_t fr_inv_stride(int64_t K) { return (K + 255) / 256 * 256 + 4; }
inline bool stage1_fr_ok(DT x_dt, int64_t K, int n_mod) {
    return x_dt == DT::BF16 && K % 64 == 0 && K <= int64_t{kFrWaves} * kFrMaxPairs * 64 &&
           static_cast<int64_t>(n_mod) * fr_inv_stride(K) <= kFrInvFloats;
}
// Down-projection with the L1 fragments staged in LDS (k_down_lds): bf16
// activations and factors, rank <= 64, K % 64 == 0; slice partials
// [down_lds_slices(T, K)][T][rank] for the quantisation kernel to add.
constexpr int64_t kDownLdsCols = 256;    // columns staged in LDS at a time (a chunk)
constexpr int64_t kDownLdsRows = 128;    // rows of a workgroup's tile
// Chunks per k slice: the workgroups (two per CU: 66 KB of LDS each) stream
// the chunks of their slice through a software pipeline, so the slices are
// made as long as a grid of about kDownLdsWgs workgroups (one round) allows:
// fewer partials to write and to add.
constexpr int64_t kDownLdsWgs = 512;
inline int down_lds_chunks(int64_t T, int64_t K) {
    const int64_t chunks = (K + kDownLdsCols - 1) / kDownLdsCols;
    const int64_t tiles = (T + kDownLdsRows - 1) / kDownLdsRows;
    const int64_t n = (tiles * chunks + kDownLdsWgs - 1) / kDownLdsWgs;
    return static_cast<int>(n < 1 ? 1 : (n > chunks ? chunks : n));
}
inline int down_lds_slices(int64_t T, int64_t K) {
    const int64_t chunks = (K + kDownLdsCols - 1) / kDownLdsCols;
    const int n = down_lds_chunks(T, K);
    return static_cast<int>((chunks + n - 1) / n);
}
inline bool down_lds_ok(DT x_dt, int64_t K) { return x_dt == DT::BF16 && K % 64 == 0; }
// Stage 1 of the fused layer for rows that k_stage1_fr cannot hold: k_down_lds,
// then the quantisation adding its partials.
constexpr bool kStage1SplitDown = true;
// Rows that k_stage1_fr can hold take it only for batches of kFusedFullT
// tokens and more with at most one non-text modality; other batches take
// the split form as well.  k_stage1_fr reads the whole of L1 for every
// non-text modality present in each 16-row group, k_down_lds once per
// 128-row tile and k slice; below kFusedFullT tokens k_stage1_fr's T / 16
// workgroups leave compute units idle, and with two non-text modalities
// more of its groups read two L1s.  (Measured, rank 64, 3584 columns:
// 2048 tokens 22.2 -> 17.7 us with one non-text modality, 33.3 -> 19.4 us
// with two; 4096 tokens 24.1 -> 25.9 us with one, 35.4 -> 31.2 us with two;
// 8192 tokens 47.7 -> 51.9 us with one, 60.1 -> 57.9 us with two.)
inline bool stage1_fr_first(int64_t T, int n_mod) { return T >= kFusedFullT && n_mod <= 2; }
hipError_t launch_down_lds(const void* x, const int32_t* mod, const float* inv_s,
                           const void* l_down, int64_t T, int64_t K, int rank, int n_mod,
                           float* part, hipStream_t s);

hipError_t launch_stage1_fused(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, int64_t T, int64_t K, int rank, int n_mod,
                               int8_t* q, float* x_scale, float* u, uint8_t* u_hl,
                               int* zero_ints, int n_zero, hipStream_t s, bool pair = false);

// Stage 1 of the small-batch path (small_path): quantisation of every row
// and the k-sliced down-projection (partials) in one launch.
hipError_t launch_stage1_small(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, DT lr_dt, int64_t T, int64_t K, int rank,
                               int n_mod, bool cmc, const Workspace& w, hipStream_t s);

// u: the down-projection; on the small-batch path (small_path) with
// n_kslices > 1 the GEMM adds the slice partials u_part itself.  u_hl
// (optional): u as bf16 hi/lo rows, written by the fused stage 1.  dec_part /
// dec_tickets (optional, small-batch path): workspace of the k-sliced decode
// GEMM; without them the single-pass small-batch GEMM runs.  w4: wq holds
// packed 4-bit codes ([N][K / 2] bytes, K % 64 == 0).  a_pair: q is
// row-paired (code_row / code_col), which only the LDS-DMA GEMM reads
// (K % 64 == 0, batches past the small path).
hipError_t launch_gemm(const int8_t* q, const float* x_scale, const int8_t* wq,
                       const float* w_scale, int64_t T, int64_t K, int64_t N,
                       const int32_t* mod, const float* u, const uint8_t* u_hl,
                       int32_t* dec_part, int* dec_tickets, int gk_splits, int32_t* gk_part,
                       int* gk_tickets, const float* u_part, int n_kslices,
                       int rank, int n_mod, const void* r_up, DT lr_dt, bool cmc, int32_t* acc,
                       void* y, DT y_dt, hipStream_t s, bool w4 = false,
                       bool a_pair = false);

// MAS-only comparator (a weight per modality, no compensation): rows grouped
// by modality on the device, then the direct-to-LDS GEMM over tiles of one
// modality each (K % 64 == 0).  The tile table holds at most
// grouped_tab_max entries {first row, rows, modality, 0}.  The codes q are
// row-paired (code_row / code_col), the quantiser's pair layout.
inline int grouped_tab_max(int64_t T, int n_mod) {
    return static_cast<int>((T + kTileM - 1) / kTileM) + n_mod - 1;
}
hipError_t launch_group_rows(const int32_t* mod, int64_t T, int n_mod, int32_t* rows,
                             int32_t* tab, int* tab_n, int* zero_ints, int n_zero, hipStream_t s);
// MAS-only at small batches (small_path, plan_decode's slices within
// kDecMaxSlices): the decode GEMM once per modality's weight (wq
// [n_mod][N][K], w_scale [n_mod][N]), each launch storing the outputs of its
// modality's tokens only; plain codes.  part / tickets: the decode GEMM's
// workspace (tickets zero before the first launch; each launch leaves them
// zero).
hipError_t launch_gemm_decode_mas(const int8_t* q, const float* x_scale, const int8_t* wq,
                                  const float* w_scale, int64_t T, int64_t K, int64_t N,
                                  const int32_t* mod, int n_mod, int32_t* part, int* tickets,
                                  void* y, DT y_dt, hipStream_t s);
hipError_t launch_gemm_grouped(const int8_t* q, const float* x_scale, const int8_t* wq,
                               const float* w_scale, int64_t T, int64_t K, int64_t N, int n_mod,
                               const int32_t* rows, const int32_t* tab, const int* tab_n, void* y,
                               DT y_dt, int S, int32_t* part, int* tickets, hipStream_t s);

hipError_t launch_lowrank_comp(const void* x, DT x_dt, const int32_t* mod, const float* inv_s,
                               const void* l_down, const void* r_up, DT lr_dt, int64_t T,
                               int64_t K, int64_t N, int rank, int n_mod, void* y, DT y_dt,
                               hipStream_t s);

}  // namespace masq
