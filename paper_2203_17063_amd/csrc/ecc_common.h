// Internal definitions shared by the libecc translation units (HIP, gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "libecc.h"

namespace ecc {

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

#define ECC_HIP(expr)                                                                   \
    do {                                                                                \
        hipError_t e_ = (expr);                                                         \
        if (e_ != hipSuccess) {                                                         \
            ::ecc::set_error("%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_),     \
                             __FILE__, __LINE__);                                       \
            return ECC_ERR_DEVICE;                                                      \
        }                                                                               \
    } while (0)

#define ECC_LAUNCH_CHECK()                                                              \
    do {                                                                                \
        hipError_t e_ = hipGetLastError();                                              \
        if (e_ != hipSuccess) {                                                         \
            ::ecc::set_error("kernel launch failed: %s (%s:%d)", hipGetErrorString(e_), \
                             __FILE__, __LINE__);                                       \
            return ECC_ERR_DEVICE;                                                      \
        }                                                                               \
    } while (0)

#define ECC_ARG(cond, ...)                                                              \
    do {                                                                                \
        if (!(cond)) {                                                                  \
            ::ecc::set_error(__VA_ARGS__);                                              \
            return ECC_ERR_ARG;                                                         \
        }                                                                               \
    } while (0)

// ---------------------------------------------------------------------------
// layouts shared by host and device
// ---------------------------------------------------------------------------
constexpr int kAssembleThreads = 256;
constexpr int kAssembleTile = 2048;      // elements copied by one workgroup
// Partial allreduce block shape: 1,024 threads x 16 elements, so that a
// workgroup streams 128 KB of each rank's vector at a time (measured on
// MI355X: 5.45 TB/s at 256 ranks x 4M, against 4.89 TB/s with 256 x 4).
constexpr int kReduceThreads = 1024;
constexpr int kReduceElems = 16;  // elements per thread per rank (pairs of 16 B)
constexpr int kReduceU = 1;       // ranks whose loads are in flight together
constexpr int kSweepThreads = 256;
constexpr int kStreamCap = 2048;         // nonzeros staged in LDS by a stream item
constexpr int kStreamRows = 256;         // rows of one stream item at most
constexpr int kVectorCap = 16384;        // nonzeros of one vector item / piece
constexpr int kMaxSweepBlocks = 8192;    // workgroups of one sweep launch at most
constexpr int kFusedMaxP = 1024;         // ranks whose state a fused sweep stages in LDS
constexpr int kNormThreads = 256;        // threads of every norm reduction

// Diagonal form of a short-row matrix: the offsets col - row its entries
// lie on (at most kDiagMax, ascending).
constexpr int kDiagMax = ECC_MAX_DIAGONALS;
struct DiagOffsets {
    int32_t v[kDiagMax];
};

// One assembly tile: `len` elements of rank `rank` starting `off` elements
// into its block.
struct Tile {
    int64_t off;
    int32_t rank;
    int32_t len;
};

// One sweep work item: rows [row0, row0 + nrows) of rank `rank`, whose block
// is [lo, hi), touching nonzeros [k0, k1).  kind: stream (many short rows
// staged in LDS), vector (one long row, whole workgroup) or piece (slice
// [k0, k1) of a very long row; its partial sum goes to piece slot `slot`).
// In the sorted layout, row0 of a stream item and [k0, k1) of every item
// refer to the sorted copy of the matrix; row0 of a vector item or a piece
// is the row itself.
enum { kItemStream = 0, kItemVector = 1, kItemPiece = 2 };
// Sweep layouts of a matrix: stream items staged through LDS; the same over
// a copy whose rows are sorted by decreasing length within each rank (very
// uneven rows); short-row items, one lane per row read directly (every row
// holds at most kShortRow entries); very uneven rows over a large vector cut
// by column range into sub-rows, summed per range and then per row.
enum { kLayStream = 0, kLaySorted = 1, kLayShort = 2, kLayRanges = 3 };
constexpr int kMaxRanges = 16;              // column ranges of the range layout at most
constexpr int64_t kRangeBytes = 8 << 20;    // bytes of the vector per column range
constexpr int64_t kRangeBytesColumns = 16 << 20;  // the same for a column-value matrix
constexpr int32_t kHotCols = 1024;  // column values, range layout: columns held in LDS
// Plane tiling of the short-row layout: applied when one plane of rows
// streams more than kTileMinBytes (the rows one plane apart no longer meet
// in an XCD's 4 MB L2); tiles of kTileNearFactor times the largest in-plane
// column offset, at least kTileMinRows rows.
constexpr int64_t kTileMinBytes = 4 << 20;
constexpr int64_t kTileNearFactor = 64;
constexpr int64_t kTileMinRows = 4096;
// Item queue of a short-layout sweep (see sweep.hip): one ticket counter per
// XCD range of items, 256 bytes apart, then the count of workgroups done.
// Taken when a workgroup would otherwise walk at least kQueueMinItems items.
constexpr int kQueueRanges = 8;
constexpr int kQueueStride = 64;
constexpr int64_t kQueueMinItems = 16;
// Single-launch solve of a small short-row problem (tiny.hip): one workgroup
// of kTinyThreads holds x, the next iterate and the assembled vector in LDS.
constexpr int kTinyThreads = 1024;
constexpr int kTinyMaxRows = 4096;
constexpr int kTinyMaxItems = 64;
constexpr int kTinyMaxP = 1024;
// Does a short-row problem fit the single launch: up to 2,048 rows with up to
// 8 entries each, or up to 4,096 rows with up to 3 (the rows' entries are
// held in registers), at most kTinyMaxItems items and kTinyMaxP ranks?
inline bool tiny_fits(int64_t n, int32_t max_row, int64_t n_items, int32_t P) {
    const bool rows = n <= 2 * kTinyThreads || (n <= kTinyMaxRows && max_row <= 3);
    return n > 0 && rows && n_items <= kTinyMaxItems && P <= kTinyMaxP;
}
constexpr int kShortRow = 8;
static_assert(kShortRow <= 8, "a short row is summed from eight registers");
static_assert(kStreamRows <= 256 && kStreamRows <= kSweepThreads, "one lane per short row");
struct WorkItem {
    int32_t row0;
    int32_t nrows;
    int32_t k0, k1;
    int32_t lo, hi;
    int32_t kind;
    int32_t rank;
    int32_t slot;
    int32_t pad[3];
};
static_assert(sizeof(WorkItem) == 48, "work item layout");

// A row split into pieces, recombined by the last workgroup in piece order.
struct Fixup {
    int32_t row;
    int32_t slot0;
    int32_t npieces;
    int32_t rank;
};

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

// Staleness decision of Algorithm 1 for one rank at clock step t: the data
// last received (version) is used unless it is older than S steps, in which
// case the caller waits for an update (a forced arrival); never-received
// blocks arrive with the initial exchange.
__device__ __forceinline__ bool stale_select(int32_t version, uint8_t arrived, int64_t t,
                                             int32_t S) {
    return version < 0 || arrived != 0 || (t - (int64_t)version) > (int64_t)S;
}

// 64-bit lane exchange through two 32-bit DPP moves.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), CTRL, 0xf, 0xf, false);
    return __hiloint2double(hi, lo);
}

constexpr int kDppQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowBcast15 = 0x142;  // lane 15 of each row to the next row
constexpr int kDppRowBcast31 = 0x143;  // lane 31 to rows 2 and 3

// Sum over aligned groups of G lanes (G a power of two <= 64); every lane of
// the group receives the group's sum.  The pairing is fixed, so the result is
// deterministic.  All lanes of a group must be active.
template <int G>
__device__ __forceinline__ double group_sum(double v) {
    if constexpr (G >= 2) v += dpp_f64<kDppQuadXor1>(v);
    if constexpr (G >= 4) v += dpp_f64<kDppQuadXor2>(v);
    if constexpr (G >= 8) v += dpp_f64<kDppRowHalfMirror>(v);
    if constexpr (G >= 16) v += dpp_f64<kDppRowMirror>(v);
    if constexpr (G >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (G >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// The sum of a wave's 64 values, in lane 63 (other lanes hold partial sums):
// group_sum<64>'s pairing -- quads, eights, rows of 16, then the four rows
// pairwise -- with the last two steps done by the DPP row broadcasts 15 and
// 31 instead of two shuffles through LDS.  Lane 63 adds (R3 + R2) + (R1 + R0)
// where group_sum adds (R0 + R1) + (R2 + R3); IEEE addition is commutative,
// so the two are bitwise equal.  All lanes must be active.
__device__ __forceinline__ double wave_sum_lane63(double v) {
    v += dpp_f64<kDppQuadXor1>(v);
    v += dpp_f64<kDppQuadXor2>(v);
    v += dpp_f64<kDppRowHalfMirror>(v);
    v += dpp_f64<kDppRowMirror>(v);
    v += dpp_f64<kDppRowBcast15>(v);
    v += dpp_f64<kDppRowBcast31>(v);
    return v;
}

// Runtime group size version (g in {1,2,4,...,64}).
__device__ __forceinline__ double group_sum_dyn(double v, int g) {
    if (g >= 2) v += dpp_f64<kDppQuadXor1>(v);
    if (g >= 4) v += dpp_f64<kDppQuadXor2>(v);
    if (g >= 8) v += dpp_f64<kDppRowHalfMirror>(v);
    if (g >= 16) v += dpp_f64<kDppRowMirror>(v);
    if (g >= 32) v += __shfl_xor(v, 16, 64);
    if (g >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// Deterministic workgroup sum (NT threads, a multiple of 64).  Returns the
// total in thread 0.  `scratch` holds NT/64 doubles of LDS.
template <int NT>
__device__ __forceinline__ double block_sum(double v, double *scratch) {
    v = group_sum<64>(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) scratch[wave] = v;
    __syncthreads();
    double total = 0.0;
    if (threadIdx.x == 0) {
        total = scratch[0];
        for (int w = 1; w < NT / 64; ++w) total += scratch[w];
    }
    __syncthreads();
    return total;
}

// Bookkeeping of one clock step (run by one whole workgroup): new versions
// and ages, the eff flags, the forced-arrival count and the minimum version
// (the clock of a reduced result).  Returns nothing; thread 0 writes.
// record_step keeps one count per wave of the calling block: at most 16.
static_assert(kAssembleThreads <= 1024 && kReduceThreads <= 1024 && kSweepThreads <= 1024,
              "record_step holds 16 wave slots");
__device__ __forceinline__ void record_step(int32_t P, int32_t S, int64_t t,
                                            const uint8_t *__restrict__ arrived,
                                            const int32_t *__restrict__ ver_in,
                                            int32_t *__restrict__ ver_out,
                                            int32_t *__restrict__ age_state,
                                            uint8_t *__restrict__ eff_state,
                                            unsigned long long *__restrict__ forced,
                                            uint8_t *__restrict__ eff_user,
                                            int32_t *__restrict__ age_user,
                                            int32_t *__restrict__ result_clock) {
    __shared__ int s_cnt[16];
    __shared__ int s_min[16];
    int cnt = 0, mn = 0x7fffffff;
    for (int32_t p = threadIdx.x; p < P; p += blockDim.x) {
        const int32_t v = ver_in[p];
        const uint8_t a = arrived[p];
        const bool e = stale_select(v, a, t, S);
        if (e && a == 0 && v >= 0) ++cnt;
        const int32_t nv = e ? (int32_t)t : v;
        const int32_t age = (int32_t)(t - nv);
        ver_out[p] = nv;
        age_state[p] = age;
        eff_state[p] = e ? 1 : 0;
        if (eff_user) eff_user[p] = e ? 1 : 0;
        if (age_user) age_user[p] = age;
        mn = min(mn, nv);
    }
    for (int off = 32; off >= 1; off >>= 1) {
        cnt += __shfl_xor(cnt, off, 64);
        mn = min(mn, __shfl_xor(mn, off, 64));
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_cnt[wave] = cnt;
        s_min[wave] = mn;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long total = 0;
        int m = 0x7fffffff;
        for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
            total += (unsigned long long)s_cnt[w];
            m = min(m, s_min[w]);
        }
        *forced = *forced + total;
        if (result_clock) *result_clock = m;
    }
    __syncthreads();
}

// Row epilogue of the block-row iterations; returns the row's contribution
// to the norm (r_i^2 for Jacobi, |x_next_j - x_own_j| for the power step).
template <int KIND>
__device__ __forceinline__ double row_finish(int32_t i, double s, double dg, double bi,
                                             double xo, double alpha, double beta,
                                             double *__restrict__ x_next) {
    if constexpr (KIND == ECC_KIND_JACOBI) {
        const double bs = bi - s;
        const double xn = bs / dg;
        x_next[i] = xn;
        const double r = bs - dg * xo;
        return r * r;
    } else {
        const double xn = alpha * s + beta;
        x_next[i] = xn;
        return fabs(xn - xo);
    }
}

// Rows of a short-layout item padded to a multiple of 32 in the item-major
// copy of its entries.
__device__ __forceinline__ int32_t sell_pad(int32_t nrows) { return (nrows + 31) & ~31; }

// The sum of 8 values as a pairwise tree: ((0+1)+(2+3))+((4+5)+(6+7)).
__device__ __forceinline__ double tree8(const double *t) {
    return ((t[0] + t[1]) + (t[2] + t[3])) + ((t[4] + t[5]) + (t[6] + t[7]));
}

// Deterministic reduction of n values to their sum by kNormThreads threads:
// thread j takes values j, j + kNormThreads, ... eight at a time, adds each
// full group of eight as a pairwise tree (tree8) to its running sum, then the
// remaining values one by one, in index order; then a fixed tree over the
// threads (block_sum).  The value at index `n - 1` may be supplied in a
// register (`last`, used when `use_last`) instead of being read, with the
// same order of operations.
__device__ __forceinline__ double reduce_values(const double *__restrict__ v, int64_t n,
                                                bool use_last, double last, double *scratch) {
    double acc = 0.0;
    int64_t k = threadIdx.x;
    for (; k + 7 * kNormThreads < n; k += 8 * kNormThreads) {
        double t[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t q = k + (int64_t)j * kNormThreads;
            t[j] = (use_last && q == n - 1) ? last : v[q];
        }
        acc += tree8(t);
    }
    for (; k < n; k += kNormThreads) acc += (use_last && k == n - 1) ? last : v[k];
    return block_sum<kNormThreads>(acc, scratch);
}

}  // namespace ecc

// ---------------------------------------------------------------------------
// opaque handles
// ---------------------------------------------------------------------------
struct ecc_plan_s {
    int32_t P = 0;
    int32_t S = 0;
    int device = 0;
    hipStream_t stream = nullptr;
    int64_t clock = 0;

    bool has_layout = false;
    bool tiles_rows = false;  // displs = exclusive scan of counts
    std::vector<int64_t> counts, displs;
    int64_t extent = 0;       // max(displs + counts)

    // device state (owned)
    int32_t *d_version = nullptr;   // [2][P], buffer (clock & 1) holds the current versions
    int32_t *d_age = nullptr;       // [P]
    uint8_t *d_eff = nullptr;       // [P] eff of the last call
    unsigned long long *d_forced = nullptr;  // total forced arrivals
    int64_t *d_displs = nullptr;    // [P]
    int32_t *d_block_start = nullptr;  // [P+1] when tiles_rows and extent < 2^31
    ecc::Tile *d_tiles = nullptr;   // assembly tiles (packed layout)
    int64_t n_tiles = 0;
    int32_t *d_ctrl = nullptr;      // [0] done flag, [1] iterations run (loop control)
    int32_t *h_ctrl = nullptr;      // pinned host copy of d_ctrl[0..1], written by the
                                    // single-launch solve (no copy back to the host)
    double *d_scalar = nullptr;     // scratch result of ecc_residual

    // optional event timing per kernel kind
    bool timing = false;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> pending[ECC_TIMING_KINDS];
    std::vector<hipEvent_t> event_pool;
    double timed_ms[ECC_TIMING_KINDS] = {};
    int64_t timed_launches[ECC_TIMING_KINDS] = {};
};

struct ecc_matrix_s {
    ecc_plan_t plan = nullptr;
    ecc_csr_t A{};
    int32_t kind = 0;
    ecc::WorkItem *d_items = nullptr;
    int64_t n_items = 0;
    ecc::Fixup *d_fixups = nullptr;
    int64_t n_fixups = 0;
    double2 *d_pieces = nullptr;    // (partial sum, diagonal) per piece
    int64_t n_pieces = 0;
    int32_t grid = 1;               // workgroups of a sweep launch
    bool irregular = false;         // row lengths vary widely: sorted layout, items dealt round-robin
    int layout = 0;                 // kLayStream, kLaySorted or kLayShort
    int32_t short_r = ecc::kShortRow;  // short layout: entries per row the kernel holds (>= longest row)
    int64_t bandwidth = 0;          // max |col - row|
    int32_t *d_order = nullptr;     // sorted layout: the row at each sorted position, [n]
    int32_t *d_srow_ptr = nullptr;  // sorted layout: row pointers of the sorted copy, [n + 1]
    int32_t *d_scol = nullptr;      // sorted layout: its column indices, [nnz]
    double *d_sval = nullptr;       // sorted layout: its values, [nnz]
    // range layout (the sorted copy above holds the sub-rows, range by range)
    int32_t n_ranges = 0;           // column ranges
    int64_t n_sub = 0;              // sub-rows
    int2 *d_sinfo = nullptr;        // [n_sub] (row, rank) of each sub-row
    double *d_rpart = nullptr;      // [n_ranges][n] sums of each row's sub-rows
    uint16_t *d_rmask = nullptr;    // [n] the ranges in which each row has entries
    double *d_diag = nullptr;       // [n] Jacobi: each row's diagonal entry
    ecc::Fixup *d_rfix = nullptr;   // split sub-rows: (row, first piece, pieces, range)
    int64_t n_rfix = 0;
    int32_t *d_ell_col = nullptr;   // short layout: entries item by item, entry-major (-1: padding)
    uint8_t *d_ell_mask = nullptr;  // short layout, diagonal form: the diagonals each row holds
    bool dia = false;               // short layout in diagonal form (d_ell_mask, no d_ell_col)
    int32_t n_dia = 0;              // its diagonals
    ecc::DiagOffsets dia_off{};     // their offsets, ascending
    double *d_ell_val = nullptr;    // short layout: their values
    int64_t tile_plane = 0;         // short layout: plane rows of the tiled item order (0: row order)
    int64_t tile_rows = 0;          // short layout: rows per tile
    double *d_partials = nullptr;   // internal partials of ecc_solve: 2 x n_part
    int64_t n_part = 1;             // partial sums a sweep writes: grid + 1, or n_items + 1 (queue)
    bool queue = false;             // short layout: items claimed from a run-time queue
    bool tiny = false;              // short layout: ecc_solve runs as one single-workgroup launch;
                                    // sweeps write one partial per row (n_part = n + 1)
    unsigned *d_queue = nullptr;    // its ticket counters, (kQueueRanges + 1) x kQueueStride
    // power kind, sorted or range layout: every column's entries hold one
    // value; the copy keeps no values, and sweeps gather z = c * x instead
    bool colscale = false;
    double *d_cscale = nullptr;     // [n] the value of each column (0 for empty ones)
    double *d_zown = nullptr;       // [n] c * x_own of the current sweep
    double *d_zhat = nullptr;       // [n] c * x_hat of the current sweep
    // column values in the range layout: the most gathered columns, whose
    // gathers from outside their own rank block read an LDS copy instead
    int32_t n_hot = 0;              // such columns (at most kHotCols)
    int32_t *d_hot_col = nullptr;   // [n_hot] the columns, ascending
    int32_t *d_hot_rank = nullptr;  // [n_hot] the rank whose block holds each
    double *d_hot = nullptr;        // [n_hot] c * x_hat at those columns, this sweep
};

namespace ecc {
// kernels and launchers implemented in the .hip files
ecc_status_t launch_assemble(ecc_plan_t plan, const double *const *d_send,
                             const double *d_send_base, double *d_recv,
                             const uint8_t *d_arrived, uint8_t *d_eff_out, int32_t *d_age_out,
                             const int32_t *d_done);
// One sweep launch.  With `arrived` non-NULL it is a whole loop iteration:
// staleness decision, assembly of the arrived blocks into x_hat and the sweep
// on the assembled view, on the plan's next clock.  Workgroup 0 also reduces
// `prev_partials` (if given) into *prev_rho with `norm`.
struct SweepLaunch {
    const double *b = nullptr;
    double alpha = 0.0, beta = 0.0;
    const double *x_own = nullptr;
    double *x_hat = nullptr;
    double *x_next = nullptr;
    double *partials = nullptr;
    const uint8_t *arrived = nullptr;
    uint8_t *eff_user = nullptr;
    int32_t *age_user = nullptr;
    const double *prev_partials = nullptr;
    double *prev_rho = nullptr;
    int32_t norm = 0;
    const int32_t *done = nullptr;
    // column-value matrix: the scaled views are already formed (by the
    // assembly of the same loop iteration)
    bool scaled = false;
};
ecc_status_t launch_sweep(ecc_matrix_t M, const SweepLaunch &L);
// Column-value matrix: the staleness decision and assembly of one loop
// iteration (as launch_assemble, from x_own into x_hat) that also forms the
// scaled views M->d_zown and M->d_zhat for the sweep that follows.
ecc_status_t launch_assemble_scaled(ecc_matrix_t M, const double *x_own, double *x_hat,
                                    const uint8_t *d_arrived, uint8_t *d_eff_out,
                                    int32_t *d_age_out, const int32_t *d_done);
// Second pass: split rows (their contribution -> partial G) and, with
// norm != 0, the norm into *rho_out and the loop control block.
struct Pass2Launch {
    double *partials = nullptr;
    const double *b = nullptr;
    double alpha = 0.0, beta = 0.0;
    const double *x_own = nullptr;
    double *x_next = nullptr;
    double *x_hat = nullptr;
    bool step = false;  // loop iteration: also assemble arrived split rows
    int32_t norm = 0;
    double *rho_out = nullptr;
    double tol = 0.0;
    int32_t *ctrl = nullptr;
    int64_t t = 0;
    const int32_t *done = nullptr;
};
ecc_status_t launch_pass2(ecc_matrix_t M, const Pass2Launch &L);
// The whole loop of ecc_solve as one single-workgroup launch (M->tiny).
ecc_status_t launch_solve_tiny(ecc_matrix_t M, const double *d_b, double alpha, double beta,
                               double *d_x, double *d_x_hat, const uint8_t *d_mask, int32_t T,
                               double tol, double *d_rho, uint8_t *d_eff_hist,
                               int32_t *d_age_hist);
ecc_status_t check_plan(ecc_plan_t plan);

// Event timing around one launch (no-ops unless the plan's timing is on).
struct TimedLaunch {
    ecc_plan_t plan;
    int kind;
    hipEvent_t start = nullptr, stop = nullptr;
    TimedLaunch(ecc_plan_t p, int k);
    ~TimedLaunch();
};
}  // namespace ecc
