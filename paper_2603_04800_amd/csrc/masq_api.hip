// C ABI of the modality-aware W8A8 + low-rank linear: argument validation,
// workspace planning and stream-ordered kernel dispatch.  Every check runs
// before any HIP call, so a rejected call enqueues nothing and touches no
// output.  The semantics of each entry point are documented in masq.h.

#include "masq.h"
#include "masq_common.h"

#include <algorithm>
#include <mutex>

// Scratch of masq_linear_fused_noalloc: a file-scope device array, one copy
// per GPU at its own address.  In host code `scratch` is only a handle for
// hipGetSymbolAddress; kernels receive the per-device address obtained from it.
static __device__ __align__(256) uint8_t scratch[MASQ_SCRATCH_BYTES];

namespace masq {

static size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// Number of k slices of the down-projection.  Small batches (at most 16 row
// tiles) are split along k so that enough workgroups run; slices are
// multiples of kDownStep.  Larger batches keep one slice: the cross-XCD
// visibility that combining slices needs (a device-scope fence per
// workgroup) costs more there than the extra parallelism gains.
static void plan_kslices(int64_t T, int64_t K, int& n_kslices, int& kslice) {
    const int64_t tiles = T > 0 ? (T + kDownRows - 1) / kDownRows : 1;
    const int64_t steps = (K + kDownStep - 1) / kDownStep;
    int64_t want = small_path(T, K) ? kSmallSlices
                                    : (tiles <= 16 ? (512 + tiles - 1) / tiles : 1);
    want = want < 1 ? 1 : (want > steps ? steps : want);
    const int64_t per = (steps + want - 1) / want;          // steps per slice
    kslice = static_cast<int>(per * kDownStep);
    n_kslices = static_cast<int>((K + kslice - 1) / kslice);
}

Workspace plan_workspace(void* base, int64_t T, int64_t K, int64_t N, int rank, int n_mod) {
    Workspace w{};
    w.kslice = static_cast<int>(K);
    w.n_kslices = 1;
    size_t off = 0;
    uint8_t* b = static_cast<uint8_t*>(base);
    auto carve = [&](size_t bytes) {
        uint8_t* p = b ? b + off : nullptr;
        off += align256(bytes);
        return p;
    };
    w.pair = paired_codes(T, K);
    const int64_t q_rows = w.pair ? (T + 1) / 2 * 2 : T;    // whole row pairs
    w.q = reinterpret_cast<int8_t*>(carve(static_cast<size_t>(q_rows) * static_cast<size_t>(K)));
    w.x_scale = reinterpret_cast<float*>(carve(static_cast<size_t>(T) * sizeof(float)));
    w.u = nullptr;
    w.u_hl = nullptr;
    w.u_part = nullptr;
    w.tickets = nullptr;
    w.dec_part = nullptr;
    w.dec_tickets = nullptr;
    w.dec_ns = w.dec_sp = w.dec_groups = 0;
    if (small_path(T, K) && T > 0 && N > 0) {
        plan_decode(K, N, w.dec_ns, w.dec_sp, w.dec_groups);
        w.dec_part = reinterpret_cast<int32_t*>(carve(static_cast<size_t>(w.dec_ns + 1) * kSmallMaxT *
                                                      static_cast<size_t>(N) * sizeof(int32_t)));
        w.dec_tickets = reinterpret_cast<int*>(carve(static_cast<size_t>(w.dec_groups) * sizeof(int)));
    }
    int n_down_tickets = 0;
    if (rank > 0 && n_mod > 1) {
        plan_kslices(T, K, w.n_kslices, w.kslice);
        const size_t ur = static_cast<size_t>(T) * static_cast<size_t>(rank) * sizeof(float);
        w.u = reinterpret_cast<float*>(carve(ur));
        if (rank <= 64 && !small_path(T, K))
            w.u_hl = carve(static_cast<size_t>(T) * 256);
        if (w.n_kslices > 1) {
            w.u_part = reinterpret_cast<float*>(carve(ur * static_cast<size_t>(w.n_kslices)));
            if (!small_path(T, K))    // the small-batch GEMM adds the partials itself
                n_down_tickets = static_cast<int>((T + kDownRows - 1) / kDownRows);
        }
    }
    w.gk_splits = plan_gemm_splits(T, K, N);
    const int n_gk_tickets = w.gk_splits > 1 ? static_cast<int>(((T + kTileM - 1) / kTileM) *
                                                                 ((N + kTileN - 1) / kTileN))
                                             : 0;
    // the arrival counters of the down-projection and of the split GEMM lie
    // side by side, so that stage 1 clears them in one go
    w.tickets = nullptr;
    w.gk_tickets = nullptr;
    w.zero_base = nullptr;
    w.n_zero = n_down_tickets + n_gk_tickets;
    if (w.n_zero > 0) {
        w.zero_base = reinterpret_cast<int*>(carve(static_cast<size_t>(w.n_zero) * sizeof(int)));
        if (n_down_tickets > 0) w.tickets = w.zero_base;
        if (n_gk_tickets > 0) w.gk_tickets = w.zero_base ? w.zero_base + n_down_tickets : nullptr;
    }
    // the slice partials of the wide down-projection (any activation dtype)
    // and of k_down_lds (bf16 activations) are never needed by one call:
    // they share one region, as large as the larger of the two
    w.dw_slices = w.dw_kslice = 0;
    w.dw_part = nullptr;
    w.dl_part = nullptr;
    const bool cmc64 = rank > 0 && rank <= 64 && n_mod > 1 && !small_path(T, K);
    const bool dw = cmc64 && down_wide(T, K);
    const bool dl = kStage1SplitDown && cmc64 && K % 64 == 0;
    if (dw) plan_down_wide(T, K, w.dw_slices, w.dw_kslice);
    const size_t row_bytes = static_cast<size_t>(T) * static_cast<size_t>(rank) * sizeof(float);
    const size_t part_bytes = std::max(dw ? w.dw_slices * row_bytes : 0,
                                       dl ? down_lds_slices(T, K) * row_bytes : 0);
    if (part_bytes > 0) {
        float* p = reinterpret_cast<float*>(carve(part_bytes));
        if (dw) w.dw_part = p;
        if (dl) w.dl_part = p;
    }
    w.gk_part = nullptr;
    if (n_gk_tickets > 0)
        w.gk_part = reinterpret_cast<int32_t*>(carve(static_cast<size_t>(n_gk_tickets) * w.gk_splits *
                                                     kTileM * kTileN * sizeof(int32_t)));
    w.bytes = off;
    return w;
}

// Workspace of the MAS-only comparator: codes, scales, the rows grouped by
// modality, the tile table and its length, and (K split over few tiles)
// arrival counters and slice accumulators; for small batches (the decode
// GEMM per modality) codes, scales and the decode GEMM's partials and
// counters.
struct MasOnlyWs {
    bool decode;       // small batch: the decode GEMM once per modality, plain codes
    int32_t* dec_part; // its partial sums [ns + 1][kSmallMaxT][N]
    int* dec_tickets;  // and arrival counters [groups]
    int dec_groups;
    int8_t* q;         // codes: plain when `decode`, else row-paired (code_row / code_col)
    float* x_scale;
    int32_t* rows;
    int32_t* tab;
    int* tab_n;
    int* tickets;
    int n_tickets;
    int32_t* part;
    int S;
    size_t bytes;
};

MasOnlyWs plan_mas_only(void* base, int64_t T, int64_t K, int64_t N, int n_mod) {
    MasOnlyWs w{};
    size_t off = 0;
    uint8_t* b = static_cast<uint8_t*>(base);
    auto carve = [&](size_t bytes) {
        uint8_t* p = b ? b + off : nullptr;
        off += align256(bytes);
        return p;
    };
    int ns = 0, sp = 0;
    w.decode = T > 0 && N > 0 && small_path(T, K);
    if (w.decode) {
        plan_decode(K, N, ns, sp, w.dec_groups);
        w.decode = ns <= kDecMaxSlices;
    }
    if (w.decode) {
        w.q = reinterpret_cast<int8_t*>(carve(static_cast<size_t>(T) * static_cast<size_t>(K)));
        w.x_scale = reinterpret_cast<float*>(carve(static_cast<size_t>(T) * sizeof(float)));
        w.dec_part = reinterpret_cast<int32_t*>(carve(static_cast<size_t>(ns + 1) * kSmallMaxT *
                                                      static_cast<size_t>(N) * sizeof(int32_t)));
        w.dec_tickets = reinterpret_cast<int*>(carve(static_cast<size_t>(w.dec_groups) * sizeof(int)));
        w.bytes = off;
        return w;
    }
    const int tab_max = grouped_tab_max(T, n_mod);
    const int64_t tiles = static_cast<int64_t>(tab_max) * ((N + kTileN - 1) / kTileN);
    // codes row-paired (code_row / code_col; K % 64 == 0), whole row pairs
    w.q = reinterpret_cast<int8_t*>(carve(static_cast<size_t>((T + 1) / 2 * 2) * static_cast<size_t>(K)));
    w.x_scale = reinterpret_cast<float*>(carve(static_cast<size_t>(T) * sizeof(float)));
    w.rows = reinterpret_cast<int32_t*>(carve(static_cast<size_t>(T) * sizeof(int32_t)));
    w.tab = reinterpret_cast<int32_t*>(carve(static_cast<size_t>(tab_max) * 4 * sizeof(int32_t)));
    w.tab_n = reinterpret_cast<int*>(carve(sizeof(int)));
    w.S = plan_gemm_splits(static_cast<int64_t>(tab_max) * kTileM, K, N);
    w.n_tickets = w.S > 1 ? static_cast<int>(tiles) : 0;
    w.tickets = w.S > 1 ? reinterpret_cast<int*>(carve(static_cast<size_t>(tiles) * sizeof(int))) : nullptr;
    w.part = w.S > 1 ? reinterpret_cast<int32_t*>(carve(static_cast<size_t>(tiles) * w.S * kTileM *
                                                        kTileN * sizeof(int32_t)))
                     : nullptr;
    w.bytes = off;
    return w;
}

}  // namespace masq

using masq::DT;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_dt(masq_dtype d) { return d == MASQ_F32 || d == MASQ_BF16; }

DT to_dt(masq_dtype d) { return d == MASQ_BF16 ? DT::BF16 : DT::F32; }

masq_status check_dims(int64_t T, int64_t c_in, int64_t c_out, bool need_out) {
    if (T < 0 || c_in <= 0 || (c_in % 16) != 0) return MASQ_ERR_SHAPE;
    if (need_out && (c_out <= 0 || (c_out % 16) != 0)) return MASQ_ERR_SHAPE;
    // 32-bit indexing inside a row and a 2^31 bound on the grid
    if (c_in > (1LL << 30) || c_out > (1LL << 30) || T > (1LL << 31) - 1) return MASQ_ERR_SHAPE;
    return MASQ_OK;
}

// Longest rows whose int32 accumulation stays exact: |acc| <= 127 * 127 * c_in
// for int8 codes, and 127 * 112 * c_in for the 4-bit weight (its codes enter
// the MFMA as 16 x code, |16 x code| <= 112, and the sum is shifted back by 4),
// each below 2^31 and rounded down to the width granularity of its path.
constexpr int64_t kMaxCinW8 = ((((1LL << 31) - 1) / (127 * 127)) / 16) * 16;   // 133136
constexpr int64_t kMaxCinW4 = ((((1LL << 31) - 1) / (127 * 112)) / 64) * 64;   // 150976
static_assert(kMaxCinW8 * 127 * 127 < (1LL << 31) && kMaxCinW4 * 127 * 112 < (1LL << 31), "");

masq_status check_exact_acc(int64_t c_in, bool w4) {
    return c_in > (w4 ? kMaxCinW4 : kMaxCinW8) ? MASQ_ERR_SHAPE : MASQ_OK;
}

masq_status check_rank(int32_t rank, int32_t n_mod) {
    if (n_mod < 1 || n_mod > 4) return MASQ_ERR_SHAPE;
    if (rank < 0 || rank > masq::kMaxRank || (rank % 16) != 0) return MASQ_ERR_SHAPE;
    return MASQ_OK;
}

masq_status from_hip(hipError_t e) { return e == hipSuccess ? MASQ_OK : MASQ_ERR_HIP; }

struct Fused {
    const void* x; masq_dtype x_dt; const int32_t* modality; const float* inv_smooth;
    const int8_t* wq; const float* w_scale; const void* l_down; const void* r_up;
    masq_dtype lr_dt; int64_t T, c_in, c_out; int32_t rank, n_mod; void* y; masq_dtype y_dt;
    void* workspace; size_t workspace_bytes; void* stream;
    bool w4;      // wq: packed 4-bit codes, [c_out][c_in / 2] bytes
};

masq_status validate_fused(const Fused& a) {
    masq_status st = check_dims(a.T, a.c_in, a.c_out, true);
    if (st != MASQ_OK) return st;
    if (a.w4 && a.c_in % 64 != 0) return MASQ_ERR_SHAPE;
    if ((st = check_exact_acc(a.c_in, a.w4)) != MASQ_OK) return st;
    if ((st = check_rank(a.rank, a.n_mod)) != MASQ_OK) return st;
    if (!valid_dt(a.x_dt) || !valid_dt(a.y_dt) || !valid_dt(a.lr_dt)) return MASQ_ERR_DTYPE;
    if (a.T == 0) return MASQ_OK;      // empty batch: nothing is read or written
    const bool cmc = a.rank > 0 && a.n_mod > 1;
    if (!a.x || !a.modality || !a.inv_smooth || !a.wq || !a.w_scale || !a.y) return MASQ_ERR_NULL;
    if (cmc && (!a.l_down || !a.r_up)) return MASQ_ERR_NULL;
    if (a.T > 0 && !a.workspace) return MASQ_ERR_NULL;
    if (!aligned16(a.x) || !aligned16(a.modality) || !aligned16(a.inv_smooth) ||
        !aligned16(a.wq) || !aligned16(a.w_scale) || !aligned16(a.y))
        return MASQ_ERR_ALIGN;
    if (cmc && (!aligned16(a.l_down) || !aligned16(a.r_up))) return MASQ_ERR_ALIGN;
    if (a.workspace && (reinterpret_cast<uintptr_t>(a.workspace) & 255u) != 0) return MASQ_ERR_ALIGN;
    const masq::Workspace w = masq::plan_workspace(nullptr, a.T, a.c_in, a.c_out, a.rank, a.n_mod);
    if (a.T > 0 && a.workspace_bytes < w.bytes) return MASQ_ERR_WORKSPACE;
    return MASQ_OK;
}

masq_status fused_stage(const Fused& a, int stage) {
    masq_status st = validate_fused(a);
    if (st != MASQ_OK || a.T == 0) return st;
    const bool cmc = a.rank > 0 && a.n_mod > 1;
    const masq::Workspace w =
        masq::plan_workspace(a.workspace, a.T, a.c_in, a.c_out, a.rank, a.n_mod);
    hipStream_t s = static_cast<hipStream_t>(a.stream);
    (void)hipGetLastError();
    if ((stage & 1) && masq::small_path(a.T, a.c_in)) {
        st = from_hip(masq::launch_stage1_small(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth,
                                                a.l_down, to_dt(a.lr_dt), a.T, a.c_in, a.rank,
                                                a.n_mod, cmc, w, s));
        if (st != MASQ_OK) return st;
    } else if ((stage & 1) && cmc && masq::fused_stage1_ok(a.T, a.c_in, a.rank, to_dt(a.lr_dt)) &&
               masq::stage1_fr_ok(to_dt(a.x_dt), a.c_in, a.n_mod) &&
               (masq::stage1_fr_first(a.T, a.n_mod) || w.dl_part == nullptr)) {
        // rows held in registers: one kernel, each row read once
        st = from_hip(masq::launch_stage1_fused(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth,
                                                a.l_down, a.T, a.c_in, a.rank, a.n_mod, w.q,
                                                w.x_scale, w.u, w.u_hl, w.zero_base, w.n_zero, s,
                                                w.pair));
        if (st != MASQ_OK) return st;
    } else if ((stage & 1) && cmc && masq::fused_stage1_ok(a.T, a.c_in, a.rank, to_dt(a.lr_dt)) &&
               masq::down_lds_ok(to_dt(a.x_dt), a.c_in) && w.dl_part != nullptr) {
        // rows too long for the registers: down-projection over 128-row
        // tiles, then the quantisation adding its slice partials into u (and
        // its bf16 hi/lo rows)
        st = from_hip(masq::launch_down_lds(a.x, a.modality, a.inv_smooth, a.l_down, a.T, a.c_in,
                                            a.rank, a.n_mod, w.dl_part, s));
        if (st != MASQ_OK) return st;
        const masq::UFinish fin{w.dl_part, masq::down_lds_slices(a.T, a.c_in), a.rank, w.u, w.u_hl};
        st = from_hip(masq::launch_smooth_quant(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth,
                                                a.T, a.c_in, a.n_mod, w.q, w.x_scale,
                                                w.zero_base, w.n_zero, s, &fin, w.pair));
        if (st != MASQ_OK) return st;
    } else if ((stage & 1) && cmc && masq::fused_stage1_ok(a.T, a.c_in, a.rank, to_dt(a.lr_dt)) &&
               w.dw_part != nullptr) {
        // large batch: wide down-projection, then quantisation adding its partials
        st = from_hip(masq::launch_down_wide(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth, a.l_down,
                                             a.T, a.c_in, a.rank, a.n_mod, w, s));
        if (st != MASQ_OK) return st;
        const masq::UFinish fin{w.dw_part, w.dw_slices, a.rank, w.u, w.u_hl};
        st = from_hip(masq::launch_smooth_quant(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth,
                                                a.T, a.c_in, a.n_mod, w.q, w.x_scale,
                                                w.zero_base, w.n_zero, s, &fin, w.pair));
        if (st != MASQ_OK) return st;
    } else if ((stage & 1) && cmc && masq::fused_stage1_ok(a.T, a.c_in, a.rank, to_dt(a.lr_dt))) {
        st = from_hip(masq::launch_stage1_fused(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth,
                                                a.l_down, a.T, a.c_in, a.rank, a.n_mod, w.q,
                                                w.x_scale, w.u, w.u_hl, w.zero_base, w.n_zero, s,
                                                w.pair));
        if (st != MASQ_OK) return st;
    } else if (stage & 1) {
        st = from_hip(masq::launch_smooth_quant(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth,
                                                a.T, a.c_in, a.n_mod, w.q, w.x_scale,
                                                w.zero_base, w.n_zero, s, nullptr, w.pair));
        if (st != MASQ_OK) return st;
        if (cmc) {
            st = from_hip(masq::launch_lowrank_down(a.x, to_dt(a.x_dt), a.modality, a.inv_smooth,
                                                    a.l_down, to_dt(a.lr_dt), a.T, a.c_in,
                                                    a.rank, a.n_mod, w, s));
            if (st != MASQ_OK) return st;
        }
    }
    if (stage & 2) {
        // the hi/lo rows of u exist when the fused stage 1 wrote them
        const bool hl = cmc && !masq::small_path(a.T, a.c_in) &&
                        masq::fused_stage1_ok(a.T, a.c_in, a.rank, to_dt(a.lr_dt));
        st = from_hip(masq::launch_gemm(w.q, w.x_scale, a.wq, a.w_scale, a.T, a.c_in, a.c_out,
                                        a.modality, w.u, hl ? w.u_hl : nullptr, w.dec_part,
                                        w.dec_tickets, w.gk_splits, w.gk_part, w.gk_tickets,
                                        w.u_part,
                                        w.n_kslices, a.rank, a.n_mod,
                                        a.r_up, to_dt(a.lr_dt), cmc, nullptr, a.y, to_dt(a.y_dt),
                                        s, a.w4, w.pair));
    }
    return st;
}

// Device address of `scratch` on each device, looked up on the first
// allocation-free call made with that device current.
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};

masq_status scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return MASQ_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return MASQ_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return MASQ_OK;
}

}  // namespace

extern "C" {

int masq_abi_version(void) { return 1; }

const char* masq_status_str(masq_status s) {
    switch (s) {
        case MASQ_OK: return "MASQ_OK";
        case MASQ_ERR_NULL: return "MASQ_ERR_NULL: a required pointer is NULL";
        case MASQ_ERR_SHAPE: return "MASQ_ERR_SHAPE: a size violates the preconditions";
        case MASQ_ERR_DTYPE: return "MASQ_ERR_DTYPE: unsupported dtype";
        case MASQ_ERR_ALIGN: return "MASQ_ERR_ALIGN: a pointer is not suitably aligned";
        case MASQ_ERR_WORKSPACE: return "MASQ_ERR_WORKSPACE: workspace too small";
        case MASQ_ERR_HIP: return "MASQ_ERR_HIP: kernel launch failed";
        case MASQ_ERR_UNSUPPORTED: return "MASQ_ERR_UNSUPPORTED: not implemented by this build";
        case MASQ_ERR_SCRATCH:
            return "MASQ_ERR_SCRATCH: the problem needs more than the static scratch "
                   "(MASQ_SCRATCH_BYTES); use masq_linear_fused with a workspace";
        default: break;
    }
    return "MASQ_ERR_UNKNOWN";
}

masq_status masq_smooth_quant(const void* x, masq_dtype x_dt, const int32_t* modality,
                              const float* inv_smooth, int64_t T, int64_t c_in, int32_t n_mod,
                              int8_t* q, float* x_scale, void* stream) {
    masq_status st = check_dims(T, c_in, 16, false);
    if (st != MASQ_OK) return st;
    if (n_mod < 1 || n_mod > 4) return MASQ_ERR_SHAPE;
    if (!valid_dt(x_dt)) return MASQ_ERR_DTYPE;
    if (T == 0) return MASQ_OK;
    if (!x || !modality || !inv_smooth || !q || !x_scale) return MASQ_ERR_NULL;
    if (!aligned16(x) || !aligned16(modality) || !aligned16(inv_smooth) || !aligned16(q) ||
        !aligned16(x_scale))
        return MASQ_ERR_ALIGN;
    if (T == 0) return MASQ_OK;
    (void)hipGetLastError();
    return from_hip(masq::launch_smooth_quant(x, to_dt(x_dt), modality, inv_smooth, T, c_in,
                                              n_mod, q, x_scale, nullptr, 0,
                                              static_cast<hipStream_t>(stream)));
}

static masq_status gemm_call(const int8_t* q, const float* x_scale, const int8_t* wq,
                             const float* w_scale, int64_t T, int64_t c_in, int64_t c_out,
                             int32_t* acc, void* y, masq_dtype y_dt, void* stream, bool w4) {
    masq_status st = check_dims(T, c_in, c_out, true);
    if (st != MASQ_OK) return st;
    if (w4 && c_in % 64 != 0) return MASQ_ERR_SHAPE;
    if ((st = check_exact_acc(c_in, w4)) != MASQ_OK) return st;
    if (!valid_dt(y_dt)) return MASQ_ERR_DTYPE;
    if (T == 0) return MASQ_OK;
    if (!q || !x_scale || !wq || !w_scale || (!acc && !y)) return MASQ_ERR_NULL;
    if (!aligned16(q) || !aligned16(x_scale) || !aligned16(wq) || !aligned16(w_scale) ||
        (acc && !aligned16(acc)) || (y && !aligned16(y)))
        return MASQ_ERR_ALIGN;
    if (T == 0) return MASQ_OK;
    (void)hipGetLastError();
    return from_hip(masq::launch_gemm(q, x_scale, wq, w_scale, T, c_in, c_out, nullptr, nullptr,
                                      nullptr, nullptr, nullptr, 1, nullptr, nullptr, nullptr, 1, 0,
                                      1, nullptr, DT::BF16, false, acc, y, to_dt(y_dt),
                                      static_cast<hipStream_t>(stream), w4));
}

masq_status masq_w8a8_gemm(const int8_t* q, const float* x_scale, const int8_t* wq,
                           const float* w_scale, int64_t T, int64_t c_in, int64_t c_out,
                           int32_t* acc, void* y, masq_dtype y_dt, void* stream) {
    return gemm_call(q, x_scale, wq, w_scale, T, c_in, c_out, acc, y, y_dt, stream, false);
}

masq_status masq_w4a8_gemm(const int8_t* q, const float* x_scale, const uint8_t* wq4,
                           const float* w_scale, int64_t T, int64_t c_in, int64_t c_out,
                           int32_t* acc, void* y, masq_dtype y_dt, void* stream) {
    return gemm_call(q, x_scale, reinterpret_cast<const int8_t*>(wq4), w_scale, T, c_in, c_out,
                     acc, y, y_dt, stream, true);
}

masq_status masq_lowrank_comp(const void* x, masq_dtype x_dt, const int32_t* modality,
                              const float* inv_smooth, const void* l_down, const void* r_up,
                              masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out,
                              int32_t rank, int32_t n_mod, void* y, masq_dtype y_dt,
                              void* stream) {
    masq_status st = check_dims(T, c_in, c_out, true);
    if (st != MASQ_OK) return st;
    if ((st = check_rank(rank, n_mod)) != MASQ_OK) return st;
    if (!valid_dt(x_dt) || !valid_dt(lr_dt) || !valid_dt(y_dt)) return MASQ_ERR_DTYPE;
    if (T == 0) return MASQ_OK;
    const bool cmc = rank > 0 && n_mod > 1;
    if (!x || !modality || !inv_smooth || !y) return MASQ_ERR_NULL;
    if (cmc && (!l_down || !r_up)) return MASQ_ERR_NULL;
    if (!aligned16(x) || !aligned16(modality) || !aligned16(inv_smooth) || !aligned16(y))
        return MASQ_ERR_ALIGN;
    if (cmc && (!aligned16(l_down) || !aligned16(r_up))) return MASQ_ERR_ALIGN;
    if (T == 0 || !cmc) return MASQ_OK;
    (void)hipGetLastError();
    return from_hip(masq::launch_lowrank_comp(x, to_dt(x_dt), modality, inv_smooth, l_down, r_up,
                                              to_dt(lr_dt), T, c_in, c_out, rank, n_mod, y,
                                              to_dt(y_dt), static_cast<hipStream_t>(stream)));
}

size_t masq_mas_only_workspace_bytes(int64_t T, int64_t c_in, int64_t c_out, int32_t n_mod) {
    if (T < 0 || c_in <= 0 || c_out <= 0 || n_mod < 1 || n_mod > 4) return 0;
    return masq::plan_mas_only(nullptr, T, c_in, c_out, n_mod).bytes;
}

masq_status masq_mas_only_linear(const void* x, masq_dtype x_dt, const int32_t* modality,
                                 const float* inv_smooth, const int8_t* wq, const float* w_scale,
                                 int64_t T, int64_t c_in, int64_t c_out, int32_t n_mod, void* y,
                                 masq_dtype y_dt, void* workspace, size_t workspace_bytes,
                                 void* stream) {
    masq_status st = check_dims(T, c_in, c_out, true);
    if (st != MASQ_OK) return st;
    if ((st = check_exact_acc(c_in, false)) != MASQ_OK) return st;
    if (n_mod < 1 || n_mod > 4) return MASQ_ERR_SHAPE;
    if (!valid_dt(x_dt) || !valid_dt(y_dt)) return MASQ_ERR_DTYPE;
    if (c_in % 64 != 0) return MASQ_ERR_UNSUPPORTED;
    if (T == 0) return MASQ_OK;
    if (!x || !modality || !inv_smooth || !wq || !w_scale || !y || !workspace) return MASQ_ERR_NULL;
    if (!aligned16(x) || !aligned16(modality) || !aligned16(inv_smooth) || !aligned16(wq) ||
        !aligned16(w_scale) || !aligned16(y))
        return MASQ_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return MASQ_ERR_ALIGN;
    const masq::MasOnlyWs w = masq::plan_mas_only(workspace, T, c_in, c_out, n_mod);
    if (workspace_bytes < w.bytes) return MASQ_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    if (w.decode) {
        // a small batch streams each modality's weight once: the decode GEMM
        // per weight, storing its own tokens' rows (the quantiser clears the
        // arrival counters)
        st = from_hip(masq::launch_smooth_quant(x, to_dt(x_dt), modality, inv_smooth, T, c_in,
                                                n_mod, w.q, w.x_scale, w.dec_tickets,
                                                w.dec_groups, s));
        if (st != MASQ_OK) return st;
        return from_hip(masq::launch_gemm_decode_mas(w.q, w.x_scale, wq, w_scale, T, c_in, c_out,
                                                     modality, n_mod, w.dec_part, w.dec_tickets,
                                                     y, to_dt(y_dt), s));
    }
    st = from_hip(masq::launch_group_rows(modality, T, n_mod, w.rows, w.tab, w.tab_n, w.tickets,
                                          w.n_tickets, s));
    if (st != MASQ_OK) return st;
    st = from_hip(masq::launch_smooth_quant(x, to_dt(x_dt), modality, inv_smooth, T, c_in, n_mod,
                                            w.q, w.x_scale, nullptr, 0, s, nullptr, true));
    if (st != MASQ_OK) return st;
    return from_hip(masq::launch_gemm_grouped(w.q, w.x_scale, wq, w_scale, T, c_in, c_out, n_mod,
                                              w.rows, w.tab, w.tab_n, y, to_dt(y_dt), w.S, w.part,
                                              w.tickets, s));
}

size_t masq_linear_fused_workspace_bytes(int64_t T, int64_t c_in, int64_t c_out, int32_t rank,
                                         int32_t n_mod) {
    if (T < 0 || c_in <= 0 || c_out <= 0 || rank < 0) return 0;
    return masq::plan_workspace(nullptr, T, c_in, c_out, rank, n_mod).bytes;
}

#define MASQ_FUSED_ARGS                                                                      \
    const void *x, masq_dtype x_dt, const int32_t *modality, const float *inv_smooth,        \
        const int8_t *wq, const float *w_scale, const void *l_down, const void *r_up,        \
        masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out, int32_t rank, int32_t n_mod, \
        void *y, masq_dtype y_dt, void *workspace, size_t workspace_bytes, void *stream
#define MASQ_FUSED_ARGS_W4                                                                     \
    const void *x, masq_dtype x_dt, const int32_t *modality, const float *inv_smooth,        \
        const uint8_t *wq4, const float *w_scale, const void *l_down, const void *r_up,      \
        masq_dtype lr_dt, int64_t T, int64_t c_in, int64_t c_out, int32_t rank, int32_t n_mod, \
        void *y, masq_dtype y_dt, void *workspace, size_t workspace_bytes, void *stream
#define MASQ_FUSED_PACK(W, FOUR)                                                             \
    Fused { x, x_dt, modality, inv_smooth, W, w_scale, l_down, r_up, lr_dt, T, c_in, c_out,  \
            rank, n_mod, y, y_dt, workspace, workspace_bytes, stream, FOUR }
#define MASQ_W4 reinterpret_cast<const int8_t*>(wq4)

masq_status masq_linear_fused(MASQ_FUSED_ARGS) { return fused_stage(MASQ_FUSED_PACK(wq, false), 3); }

masq_status masq_linear_fused_noalloc(const void* x, masq_dtype x_dt, const int32_t* modality,
                                      const float* inv_smooth, const int8_t* wq,
                                      const float* w_scale, const void* l_down,
                                      const void* r_up, masq_dtype lr_dt, int64_t T,
                                      int64_t c_in, int64_t c_out, int32_t rank,
                                      int32_t n_mod, void* y, masq_dtype y_dt, void* stream) {
    // every argument is checked against a stand-in workspace of the scratch's
    // size first (host arithmetic only), then the array's address is fetched
    Fused a{x, x_dt, modality, inv_smooth, wq, w_scale, l_down, r_up, lr_dt, T, c_in, c_out,
            rank, n_mod, y, y_dt, reinterpret_cast<void*>(static_cast<uintptr_t>(256)),
            MASQ_SCRATCH_BYTES, stream, false};
    masq_status st = validate_fused(a);
    if (st == MASQ_ERR_WORKSPACE) return MASQ_ERR_SCRATCH;
    if (st != MASQ_OK || T == 0) return st;
    void* p = nullptr;
    if ((st = scratch_address(&p)) != MASQ_OK) return st;
    a.workspace = p;
    return fused_stage(a, 3);
}
masq_status masq_linear_stage1(MASQ_FUSED_ARGS) { return fused_stage(MASQ_FUSED_PACK(wq, false), 1); }
masq_status masq_linear_stage2(MASQ_FUSED_ARGS) { return fused_stage(MASQ_FUSED_PACK(wq, false), 2); }
masq_status masq_linear_fused_w4a8(MASQ_FUSED_ARGS_W4) {
    return fused_stage(MASQ_FUSED_PACK(MASQ_W4, true), 3);
}
masq_status masq_linear_stage1_w4a8(MASQ_FUSED_ARGS_W4) {
    return fused_stage(MASQ_FUSED_PACK(MASQ_W4, true), 1);
}
masq_status masq_linear_stage2_w4a8(MASQ_FUSED_ARGS_W4) {
    return fused_stage(MASQ_FUSED_PACK(MASQ_W4, true), 2);
}

}  // extern "C"
