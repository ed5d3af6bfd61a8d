// Block-row sweeps over a CSR matrix that consume the assembled vector:
// Jacobi (x_next_i = (b_i - sum_{j != i} a_ij y_j) / a_ii) and the PageRank
// power step (x_next_j = alpha sum_i w_ji y_i + beta), where row i of rank
// block [lo, hi) reads y_j = x_own[j] inside its own block and x_hat[j]
// elsewhere, plus the residual-norm reduction.
//
// Work decomposition (built once per matrix on the host, CSR-Adaptive style
// after Greathouse & Daga, SC'14), in one of four layouts per matrix:
//  - short rows (every row holds at most 8 entries): the entries are copied
//    column-major at set-up; an item is a run of up to 256 rows of one rank,
//    one lane per row, pipelined two items deep;
//  - stream items for other regular matrices: a run of short rows of one
//    rank whose nonzeros fit in LDS -- they are loaded with coalesced
//    accesses and each row is then summed by 1..64 lanes;
//  - sorted stream items for very uneven rows (power-law graphs): the same
//    items over a copy of the matrix, made at set-up, whose rows are ordered
//    by decreasing length within each rank, so that an item holds rows of
//    similar length and its lanes split evenly over them; a map from sorted
//    position to row places each result;
//  - range items for very uneven rows over a vector longer than one column
//    range: every row cut into its entries of each column range (sub-rows),
//    the sub-rows swept range by range as sorted stream items (so that the
//    gathers of a time come from one range of the vector, which stays in
//    L2), each sub-row's sum stored, and every row then finished from its
//    sub-row sums added in range order by a second kernel.
// In the last three, a "vector" item is one long row summed by the whole
// workgroup and a "piece" a fixed-size slice of a very long row whose
// partial sum is recombined, in piece order, at the end.  Items never
// straddle a rank boundary, so [lo, hi) is uniform per item (range items
// excepted: a length class mixes ranks, so each sub-row carries its rank).  Rows summed by
// a single lane accumulate in CSR order with no fused multiply-add, exactly
// like the sequential definition.
//
// Each workgroup writes one partial norm.  Split rows and the reduction of
// the partials (in a fixed order, so results are deterministic run to run)
// belong to a second pass that starts after the sweep has finished: a
// separate one-workgroup launch, or -- in a loop without a tolerance and
// without split rows -- workgroup 0 of the next iteration's launch.  No
// device-wide fence or read-modify-write atomic is used inside a launch: on
// a multi-XCD part an agent-scope release writes back the XCD's L2, which
// would cost more than the launch boundary.
//
// Loop iterations use the same kernel with the staleness decision and the
// assembly fused in: every workgroup evaluates the decision for all ranks
// from the previous versions (read-only in this launch), reads a column of
// another rank from x_own when that rank's block arrives at this step and
// from x_hat otherwise -- exactly the values the assembled vector holds
// after the step's assembly -- and writes its own rows into x_hat when its
// rank arrives.  No entry of x_hat that is written is read in the same
// launch, so the fused step equals assemble-then-sweep bit for bit.
#include <algorithm>
#include <mutex>
#include <vector>

#include <new>

#include "ecc_common.h"

namespace ecc {


// Grids from this size on leave workgroup 0 without items (see item_walk).
constexpr int32_t kReserveMinGrid = 64;

struct SweepArgs {
    const WorkItem *items;
    int32_t n_items;
    const int32_t *row_ptr;
    const int32_t *col;
    const double *val;
    const double *b;
    double alpha, beta;
    const double *x_own;
    double *x_hat;
    double *x_next;
    // what the stream layouts gather: x_own and x_hat, or for a column-value
    // matrix the scaled views c * x_own and c * x_hat
    const double *g_own;
    const double *g_hat;
    // column values, range layout: g_hat at the most gathered columns, which
    // the entries name as -1 - slot (copied to LDS by every workgroup)
    const double *hot;
    int32_t n_hot;
    double *partials;
    double2 *pieces;
    const int32_t *order;    // sorted layout: the row at each sorted position
    const int2 *sinfo;       // range layout: (row, rank) of each sub-row
    double *rpart;           // range layout: [ranges][rn] sums of the sub-rows
    int64_t rn;
    const int32_t *ell_col;  // short layout: column-major copy of the entries
    const double *ell_val;
    const uint8_t *ell_mask;  // short layout, diagonal form: the diagonals of each row
    DiagOffsets dia;          // and their offsets
    int64_t ell_n;
    int32_t interleave;  // items dealt round-robin instead of in XCD ranges
    int32_t reserve0;    // workgroup 0 takes no items (grids of kReserveMinGrid or more)
    // fused loop iteration (step != 0)
    int32_t step;
    int32_t P, S;
    int64_t t;
    const uint8_t *arrived;
    const int32_t *ver_in;
    int32_t *ver_out;
    int32_t *age_state;
    uint8_t *eff_state;
    unsigned long long *forced;
    uint8_t *eff_user;
    int32_t *age_user;
    const int32_t *block_start;
    // workgroup 0: zero partial G; reduce the previous iteration's partials
    int32_t zero_extra;
    const double *prev_partials;
    double *prev_rho;
    int32_t norm;
    const int32_t *done;
    // partial sums per launch (the last one is split rows' share) and, for a
    // queue-scheduled matrix, its ticket counters
    int64_t n_part;
    unsigned *queue;
    int32_t row_part;  // short layout: one partial per row (partials[i] = row i's share)
};

// Rank state staged in LDS by a fused step.
struct StepView {
    const uint8_t *eff;   // [P] this step's decision
    const int32_t *bs;    // [P + 1] block starts
    int32_t P;
};

// Two most recently used rank windows of one lane: [lo, hi) with the rank's
// arrival flag.  Kept across the items of a workgroup (arrivals are fixed
// within a launch); a stencil row's off-block neighbours sit in one or two
// ranks that change only every few items.
struct RankCache {
    int32_t lo0 = 0, hi0 = 0, lo1 = 0, hi1 = 0;
    bool e0 = false, e1 = false, next = false;
};

// Does the assembled vector hold x_own at column c (the rank of c arrives at
// this step)?  Cache hit, else binary search of the LDS-staged block starts.
__device__ __forceinline__ bool col_arrives(const StepView &v, int32_t c, RankCache &rc) {
    if (c >= rc.lo0 && c < rc.hi0) return rc.e0;
    if (c >= rc.lo1 && c < rc.hi1) return rc.e1;
    int32_t a = 0, z = v.P;  // bs[a] <= c < bs[z]
    while (z - a > 1) {
        const int32_t mid = (a + z) >> 1;
        if (v.bs[mid] <= c) a = mid;
        else z = mid;
    }
    const bool e = v.eff[a] != 0;
    if (rc.next) {
        rc.lo1 = v.bs[a];
        rc.hi1 = v.bs[a + 1];
        rc.e1 = e;
    } else {
        rc.lo0 = v.bs[a];
        rc.hi0 = v.bs[a + 1];
        rc.e0 = e;
    }
    rc.next = !rc.next;
    return e;
}

// A gather of the assembled vector.  HOT: a negative column -1 - k names
// slot k of the LDS copy s_hot of the most gathered columns.
template <bool STEP, bool HOT = false>
__device__ __forceinline__ double view_load(int32_t c, int32_t lo, int32_t hi,
                                            const double *__restrict__ x_own,
                                            const double *__restrict__ x_hat,
                                            const StepView &sv, RankCache &rc,
                                            const double *s_hot = nullptr) {
    if constexpr (HOT) {
        if (c < 0) return s_hot[-1 - c];
    }
    bool own = (c >= lo && c < hi);
    if constexpr (STEP) {
        if (!own) own = col_arrives(sv, c, rc);
    }
    return (own ? x_own : x_hat)[c];
}


// Lanes per row of a stream item: rows of at most 16 nonzeros on average are
// summed by one lane in CSR order; longer ones by up to 64 lanes, keeping at
// least 8 nonzeros per lane.
__device__ __forceinline__ int lanes_per_row(int32_t nnz, int32_t nr) {
    int tpr = 1;
    if (nnz > 16 * nr)
        while (tpr < 64 && tpr * 2 * nr <= kSweepThreads && nnz >= 16 * tpr * nr) tpr *= 2;
    return tpr;
}

// Accumulates a lane's entries k0, k0 + stride, ... (< k1) of row i, in that
// order, W at a time: the next W (col, val) loads are in flight while the
// current W gathers of y complete.  With stride 1 this is the row's CSR
// order.  Jacobi skips (and records) the diagonal entry.  CS: the gathers
// come from the scaled views and the entries' values are all 1 (the product
// v * y is then y itself).
template <int KIND, bool STEP, int W, bool CS, bool HOT = false>
__device__ __forceinline__ void seg_accumulate(int32_t i, int32_t k0, int32_t k1, int32_t stride,
                                               const SweepArgs &a, int32_t lo, int32_t hi,
                                               const StepView &sv, RankCache &rc, double &s,
                                               double &dg, const double *s_hot = nullptr) {
    if (k0 >= k1) return;
    int32_t c[W];
    double v[W];
#pragma unroll
    for (int u = 0; u < W; ++u) {
        const int32_t k = k0 + u * stride;
        c[u] = (k < k1) ? a.col[k] : 0;
        v[u] = CS ? 1.0 : (k < k1) ? a.val[k] : 0.0;
    }
    for (int32_t k = k0; k < k1; k += W * stride) {
        double y[W];
#pragma unroll
        for (int u = 0; u < W; ++u)
            y[u] = (k + u * stride < k1)
                       ? view_load<STEP, HOT>(c[u], lo, hi, a.g_own, a.g_hat, sv, rc, s_hot)
                       : 0.0;
        const int32_t kn = k + W * stride;
        int32_t cn[W];
        double vn[W];
#pragma unroll
        for (int u = 0; u < W; ++u) {
            const int32_t kk = kn + u * stride;
            cn[u] = (kk < k1) ? a.col[kk] : 0;
            vn[u] = CS ? 1.0 : (kk < k1) ? a.val[kk] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < W; ++u) {
            if (k + u * stride < k1) {
                if (KIND == ECC_KIND_JACOBI && c[u] == i) dg = v[u];
                else s = s + v[u] * y[u];
            }
        }
#pragma unroll
        for (int u = 0; u < W; ++u) {
            c[u] = cn[u];
            v[u] = vn[u];
        }
    }
}

// Registers that carry the next stream item's data while the current one is
// computed: its nonzeros (eight per thread, coalesced) and the per-row values
// of the row this thread will finish (ri: that row's index, which in the
// sorted layout differs from its position).
struct StreamPrefetch {
    int32_t cv[8];
    double vv[8];
    int32_t rp0, rp1, ri;
    int32_t lo, hi;  // range layout: the row's rank block
    double bi, xo;
};

template <int KIND, int LAY, bool CS>
__device__ __forceinline__ void stream_load(const WorkItem &it, const SweepArgs &a,
                                            StreamPrefetch &pf) {
    const int tid = threadIdx.x;
    const int32_t nnz = it.k1 - it.k0;
    static_assert(kStreamCap == 8 * kSweepThreads, "eight nonzeros per thread");
    if (nnz > 0) {  // reads clamped into [k0, k1) so that all are in flight together
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int32_t kc = min(it.k0 + tid + u * kSweepThreads, it.k1 - 1);
            if constexpr (LAY == kLaySorted || LAY == kLayRanges) {
                // read-once streams that would otherwise evict lines of the
                // gathered vector from L2 (measured on MI355X, PageRank on a
                // scale-22 R-MAT graph: 573 against 600 us per sweep)
                pf.cv[u] = __builtin_nontemporal_load(a.col + kc);
                if constexpr (!CS) pf.vv[u] = __builtin_nontemporal_load(a.val + kc);
            } else {
                pf.cv[u] = a.col[kc];
                if constexpr (!CS) pf.vv[u] = a.val[kc];
            }
        }
    }
    const int tpr = lanes_per_row(nnz, it.nrows);
    const int32_t rr = tid / tpr;
    pf.rp0 = pf.rp1 = pf.ri = pf.lo = pf.hi = 0;
    pf.bi = pf.xo = 0.0;
    if (rr < it.nrows) {
        const int32_t r = it.row0 + rr;
        pf.rp0 = a.row_ptr[r];
        pf.rp1 = a.row_ptr[r + 1];
        if constexpr (LAY == kLayRanges) {
            // a sub-row: its row and that row's rank block; the row's own
            // values are read by the finishing pass
            const int2 si = a.sinfo[r];
            pf.ri = si.x;
            pf.lo = a.block_start[si.y];
            pf.hi = a.block_start[si.y + 1];
        } else {
            const int32_t i = (LAY == kLaySorted) ? a.order[r] : r;
            pf.ri = i;
            pf.xo = a.x_own[i];
            if (KIND == ECC_KIND_JACOBI) pf.bi = a.b[i];
        }
    }
}

template <bool CS>
__device__ __forceinline__ void stream_stage(const WorkItem &it, const StreamPrefetch &pf,
                                             int32_t *s_col, double *s_val) {
    const int32_t nnz = it.k1 - it.k0;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int32_t k = threadIdx.x + u * kSweepThreads;
        if (k < nnz) {
            s_col[k] = pf.cv[u];
            if constexpr (!CS) s_val[k] = pf.vv[u];
        }
    }
}

// The rows of a stream item from the staged nonzeros; returns this thread's
// norm contribution.  i: the index of the row this thread finishes; [lo, hi):
// its rank block.  The range layout stores the sum of a sub-row instead
// (item rank = column range), for the finishing pass.
template <int KIND, bool STEP, int LAY, bool CS>
__device__ __forceinline__ double stream_compute(const WorkItem &it, int32_t rp0, int32_t rp1,
                                                 int32_t i, int32_t lo, int32_t hi, double bi,
                                                 double xo, const SweepArgs &a,
                                                 const int32_t *s_col, const double *s_val,
                                                 const double *s_hot, const StepView &sv,
                                                 RankCache &rc, bool own_arrives) {
    constexpr bool HOT = LAY == kLayRanges && CS;
    const int tid = threadIdx.x;
    const int32_t nnz = it.k1 - it.k0;
    const int tpr = lanes_per_row(nnz, it.nrows);
    const int lane = tid & (tpr - 1);
    const int32_t rr = tid / tpr;
    if (rr >= it.nrows) return 0.0;
    const int32_t rs = rp0 - it.k0, re = rp1 - it.k0;
    double s = 0.0, dg = 0.0;
    if (tpr == 1) {
        // up to eight entries with all gathers in flight, summed in CSR order
        const int32_t len = re - rs;
        int32_t c8[8];
        double v8[8], y8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            // entries past the row's end are read but unused (LDS is padded)
            c8[j] = s_col[rs + j];
            v8[j] = CS ? 1.0 : s_val[rs + j];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j)
            y8[j] = (j < len)
                        ? view_load<STEP, HOT>(c8[j], lo, hi, a.g_own, a.g_hat, sv, rc, s_hot)
                        : 0.0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j < len) {
                if (KIND == ECC_KIND_JACOBI && c8[j] == i) dg = v8[j];
                else s = s + v8[j] * y8[j];
            }
        }
        for (int32_t k = rs + 8; k < re; ++k) {
            const int32_t c = s_col[k];
            const double v = CS ? 1.0 : s_val[k];
            if (KIND == ECC_KIND_JACOBI && c == i) {
                dg = v;
                continue;
            }
            s = s + v * view_load<STEP, HOT>(c, lo, hi, a.g_own, a.g_hat, sv, rc, s_hot);
        }
    } else {
        for (int32_t k = rs + lane; k < re; k += tpr) {
            const int32_t c = s_col[k];
            const double v = CS ? 1.0 : s_val[k];
            if (KIND == ECC_KIND_JACOBI && c == i) {
                dg = v;
                continue;
            }
            s = s + v * view_load<STEP, HOT>(c, lo, hi, a.g_own, a.g_hat, sv, rc, s_hot);
        }
        s = group_sum_dyn(s, tpr);
        if (KIND == ECC_KIND_JACOBI) dg = group_sum_dyn(dg, tpr);
    }
    if (lane != 0) return 0.0;
    if constexpr (LAY == kLayRanges) {
        a.rpart[(int64_t)it.rank * a.rn + i] = s;
        return 0.0;
    } else {
        if (STEP && own_arrives) a.x_hat[i] = xo;
        return row_finish<KIND>(i, s, dg, bi, xo, a.alpha, a.beta, a.x_next);
    }
}

// One long row (or a slice of it) by the whole workgroup; returns the norm
// contribution (in thread 0).
template <int KIND, bool STEP, int LAY, bool CS>
__device__ __forceinline__ double long_compute(const WorkItem &it, const SweepArgs &a,
                                               const StepView &sv, RankCache &rc,
                                               bool own_arrives, double *s_red,
                                               const double *s_hot) {
    constexpr bool HOT = LAY == kLayRanges && CS;
    const int tid = threadIdx.x;
    const int32_t i = it.row0, lo = it.lo, hi = it.hi;
    double s = 0.0, dg = 0.0;
    seg_accumulate<KIND, STEP, 4, CS, HOT>(i, it.k0 + tid, it.k1, kSweepThreads, a, lo, hi, sv,
                                           rc, s, dg, s_hot);
    s = block_sum<kSweepThreads>(s, s_red);
    if (KIND == ECC_KIND_JACOBI) dg = block_sum<kSweepThreads>(dg, s_red);
    if (tid != 0) return 0.0;
    if (it.kind == kItemPiece) {
        a.pieces[it.slot] = make_double2(s, dg);
        return 0.0;
    }
    if constexpr (LAY == kLayRanges) {
        a.rpart[(int64_t)it.rank * a.rn + i] = s;
        return 0.0;
    }
    const double xo = a.x_own[i];
    const double bi = (KIND == ECC_KIND_JACOBI) ? a.b[i] : 0.0;
    if (STEP && own_arrives) a.x_hat[i] = xo;
    return row_finish<KIND>(i, s, dg, bi, xo, a.alpha, a.beta, a.x_next);
}

// Items a workgroup walks: w_first, w_first + w_step, ... below i_end.
// XCD-aware order: workgroups are dispatched round-robin over the 8 XCDs
// (blockIdx mod 8).  The items are split into 8 contiguous ranges, one per
// XCD, and the XCD's workgroups walk its range together, so each XCD's L2
// sees consecutive rows and their neighbours.  Matrices with very uneven
// rows deal items round-robin instead, so that the heavy items (listed
// first) spread over every XCD.  With reserve0, workgroup 0 walks no items:
// in a loop its reduction of the previous partials then overlaps the other
// workgroups' items instead of delaying its own (measured on MI355X, the
// 1024^2 Jacobi loop: 0.3-0.5 us of an 18.5 us launch).  Every launch of a
// matrix walks the same way, so its partial sums, and the norm, do not
// depend on which entry point runs the sweep.
__device__ __forceinline__ void item_walk(const SweepArgs &a, int64_t &i_end, int32_t &w_first,
                                          int32_t &w_step) {
    const int32_t G = gridDim.x;
    const int32_t r = (a.reserve0 && G >= 2) ? 1 : 0;
    i_end = a.n_items;
    w_first = blockIdx.x - r;
    w_step = G - r;
    if (!a.interleave && G % 8 == 0 && G >= 8 * (1 + r)) {
        const int32_t xcd = blockIdx.x % 8;
        const int32_t rx = xcd == 0 ? r : 0;  // XCD 0 walks without workgroup 0
        const int64_t i_begin = (int64_t)a.n_items * xcd / 8;
        i_end = (int64_t)a.n_items * (xcd + 1) / 8;
        w_first = (int32_t)(i_begin + blockIdx.x / 8 - rx);
        w_step = G / 8 - rx;
    }
    if (r && blockIdx.x == 0) w_first = (int32_t)i_end;
}

// Work every workgroup does before its items: a fused step stages this
// step's arrival decision and the block starts in LDS (workgroup 0 also
// records the step's versions, ages and forced arrivals); workgroup 0 zeroes
// partial G and reduces the previous loop iteration's partials.
template <bool STEP>
__device__ __forceinline__ void sweep_prologue(const SweepArgs &a, uint8_t *s_eff, int32_t *s_bs,
                                               double *s_red) {
    const int tid = threadIdx.x;
    if constexpr (STEP) {
        for (int32_t p = tid; p < a.P; p += kSweepThreads)
            s_eff[p] = stale_select(a.ver_in[p], a.arrived[p], a.t, a.S) ? 1 : 0;
        for (int32_t p = tid; p <= a.P; p += kSweepThreads) s_bs[p] = a.block_start[p];
        if (blockIdx.x == 0)
            record_step(a.P, a.S, a.t, a.arrived, a.ver_in, a.ver_out, a.age_state, a.eff_state,
                        a.forced, a.eff_user, a.age_user, nullptr);
    }
    if (blockIdx.x == 0) {
        // no split rows: their norm contribution (the last partial) is zero
        if (a.zero_extra && tid == 0) a.partials[a.n_part - 1] = 0.0;
        // deferred norm of the previous loop iteration, whose partials the
        // kernel boundary has made visible (same order as a separate pass)
        if (a.prev_partials) {
            const double sum = reduce_values(a.prev_partials, a.n_part, false, 0.0, s_red);
            if (tid == 0) *a.prev_rho = (a.norm == ECC_NORM_L2) ? sqrt(sum) : sum;
        }
    }
    if constexpr (STEP) __syncthreads();
}

// LAY selects the layout: stream items over the matrix (kLayStream), over
// its sorted copy (kLaySorted) or over its sub-rows cut by column range
// (kLayRanges); all may contain vector items and pieces.
// The short-row layout has its own body.
template <int KIND, bool STEP, int LAY, bool CS>
__device__ __forceinline__ void sweep_body(const SweepArgs &a) {
    static_assert(LAY == kLayStream || LAY == kLaySorted || LAY == kLayRanges,
                  "stream layouts only");
    // padded by 8 so that a row's first eight entries can be read unclamped
    __shared__ int32_t s_col[kStreamCap + 8];
    __shared__ double s_val[CS ? 1 : kStreamCap + 8];
    __shared__ double s_red[kSweepThreads / 64];
    __shared__ uint8_t s_eff[STEP ? kFusedMaxP : 1];
    __shared__ int32_t s_bs[STEP ? kFusedMaxP + 1 : 1];
    // column values, range layout: the most gathered columns' values.
    // Measured on MI355X (PageRank on a scale-22 R-MAT graph, 64 ranks): 1,024
    // columns (13 % of the gathers) 439 against 453 us per iteration; 2,048
    // the same; 4,096 or 8,192 (25 or 34 %) 539 or 671 us, their LDS leaving
    // fewer workgroups per CU to hide the other gathers.
    constexpr bool HOT = LAY == kLayRanges && CS;
    __shared__ double s_hot[HOT ? kHotCols : 1];
    if (a.done && *a.done) return;
    const int tid = threadIdx.x;
    int64_t i_end;
    int32_t w_first, w_step;
    item_walk(a, i_end, w_first, w_step);
    // the first item's loads go out before the prologue below
    int32_t w = w_first;
    WorkItem cur{}, nxt{};
    StreamPrefetch pf;
    const bool have0 = w < i_end;
    if (have0) {
        cur = a.items[w];
        if (cur.kind == kItemStream) stream_load<KIND, LAY, CS>(cur, a, pf);
    }
    bool have_next = (int64_t)w + w_step < i_end;
    if (have_next) nxt = a.items[w + w_step];

    StepView sv{s_eff, s_bs, a.P};
    sweep_prologue<STEP>(a, s_eff, s_bs, s_red);
    if constexpr (HOT) {
        for (int32_t k = tid; k < a.n_hot; k += kSweepThreads) s_hot[k] = a.hot[k];
        __syncthreads();
    }

    // Software pipeline over this workgroup's items: while an item is computed
    // from LDS, the loads of the next one (and the descriptor of the one
    // after) are in flight.
    double contrib = 0.0;
    RankCache rc;
    bool have = have0;
    while (have) {
        const bool own_arrives = STEP && s_eff[cur.rank] != 0;
        const bool next_stream = have_next && nxt.kind == kItemStream;
        WorkItem nn{};
        const bool have_nn = (int64_t)w + 2 * (int64_t)w_step < i_end;
        if (cur.kind == kItemStream) {
            stream_stage<CS>(cur, pf, s_col, s_val);
            const int32_t rp0 = pf.rp0, rp1 = pf.rp1, ri = pf.ri;
            const int32_t lo = LAY == kLayRanges ? pf.lo : cur.lo;
            const int32_t hi = LAY == kLayRanges ? pf.hi : cur.hi;
            const double bi = pf.bi, xo = pf.xo;
            __syncthreads();
            if (next_stream) stream_load<KIND, LAY, CS>(nxt, a, pf);
            if (have_nn) nn = a.items[w + 2 * w_step];
            contrib += stream_compute<KIND, STEP, LAY, CS>(cur, rp0, rp1, ri, lo, hi, bi, xo, a, s_col,
                                                           s_val, s_hot, sv, rc, own_arrives);
            __syncthreads();  // LDS is reused by the next item
        } else {
            if (have_nn) nn = a.items[w + 2 * w_step];
            contrib += long_compute<KIND, STEP, LAY, CS>(cur, a, sv, rc, own_arrives, s_red, s_hot);
            if (next_stream) stream_load<KIND, LAY, CS>(nxt, a, pf);
        }
        w += w_step;
        have = have_next;
        cur = nxt;
        have_next = have_nn;
        nxt = nn;
    }

    const double total = block_sum<kSweepThreads>(contrib, s_red);
    if (tid == 0) a.partials[blockIdx.x] = total;
}

template <int KIND, bool STEP, int LAY, bool CS = false>
__global__ __launch_bounds__(kSweepThreads) void k_sweep(SweepArgs a) {
    sweep_body<KIND, STEP, LAY, CS>(a);
}

// ---------------------------------------------------------------------------
// Column-value matrices (every entry of column j holds c_j): the sweep adds
// z_j = c_j * y_j, formed here once per element of each view, in place of
// the product w_ij * y_j of each entry.
// ---------------------------------------------------------------------------

// c[col[k]] = val[k] for every entry (any one of a column's values wins).
__global__ void k_col_values(int64_t nnz, const int32_t *__restrict__ col,
                             const double *__restrict__ val, double *__restrict__ c) {
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < nnz;
         k += (int64_t)gridDim.x * blockDim.x)
        c[col[k]] = val[k];
}

// Entries whose value differs, bit for bit, from the value kept for their
// column; *bad = their count.
__global__ void k_col_check(int64_t nnz, const int32_t *__restrict__ col,
                            const double *__restrict__ val, const double *__restrict__ c,
                            unsigned long long *__restrict__ bad) {
    unsigned long long nb = 0;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < nnz;
         k += (int64_t)gridDim.x * blockDim.x)
        nb += __double_as_longlong(val[k]) != __double_as_longlong(c[col[k]]) ? 1 : 0;
    if (nb) atomicAdd(bad, nb);
}

constexpr int kScaleThreads = 256;
constexpr int kScaleElems = 4;  // elements per thread, all loads in flight together

// The scaled views of a plain sweep: z_own = c * x_own, z_hat = c * x_hat;
// and hot[k] = z_hat at column hot_col[k] for the range layout's LDS copy.
__global__ __launch_bounds__(kScaleThreads) void k_col_scale(
    int64_t n, const double *__restrict__ c, const double *__restrict__ x_own,
    const double *__restrict__ x_hat, double *__restrict__ z_own, double *__restrict__ z_hat,
    int32_t n_hot, const int32_t *__restrict__ hot_col, double *__restrict__ hot,
    const int32_t *__restrict__ done) {
    if (done && *done) return;
    const int64_t stride = (int64_t)gridDim.x * kScaleThreads;
    for (int64_t k = (int64_t)blockIdx.x * kScaleThreads + threadIdx.x; k < n_hot; k += stride) {
        const int32_t j = hot_col[k];
        hot[k] = c[j] * x_hat[j];
    }
    for (int64_t j0 = (int64_t)blockIdx.x * kScaleThreads + threadIdx.x; j0 < n;
         j0 += stride * kScaleElems) {
        double cj[kScaleElems], xo[kScaleElems], xh[kScaleElems];
#pragma unroll
        for (int u = 0; u < kScaleElems; ++u) {
            const int64_t j = min(j0 + u * stride, n - 1);
            cj[u] = c[j];
            xo[u] = x_own[j];
            xh[u] = x_hat[j];
        }
#pragma unroll
        for (int u = 0; u < kScaleElems; ++u) {
            const int64_t j = j0 + u * stride;
            if (j < n) {
                z_own[j] = cj[u] * xo[u];
                z_hat[j] = cj[u] * xh[u];
            }
        }
    }
}

// One loop iteration's staleness decision and assembly (as k_assemble, over
// the same tiles) fused with the scaled views: for every element j of a tile
// of rank p, z_own[j] = c_j * x_own[j]; if p's block is taken at this step,
// x_hat[j] = x_own[j] and z_hat[j] = z_own[j] (= c_j * x_hat[j] after the
// copy), else z_hat[j] = c_j * x_hat[j].  Workgroup 0 records the step;
// the workgroups after the n_tiles tiles write the same z_hat at the hot
// columns (kAssembleTile of them each) for the range layout's LDS copy.
__global__ __launch_bounds__(kAssembleThreads) void k_assemble_scaled(
    int32_t P, int32_t S, int64_t t, const uint8_t *__restrict__ arrived,
    const int32_t *__restrict__ ver_in, int32_t *__restrict__ ver_out,
    int32_t *__restrict__ age_state, uint8_t *__restrict__ eff_state,
    unsigned long long *__restrict__ forced, uint8_t *__restrict__ eff_user,
    int32_t *__restrict__ age_user, const Tile *__restrict__ tiles,
    const int64_t *__restrict__ displs, const double *__restrict__ c,
    const double *__restrict__ x_own, double *__restrict__ x_hat, double *__restrict__ z_own,
    double *__restrict__ z_hat, int64_t n_tiles, int32_t n_hot,
    const int32_t *__restrict__ hot_col, const int32_t *__restrict__ hot_rank,
    double *__restrict__ hot, const int32_t *__restrict__ done) {
    if (done && *done) return;
    if (blockIdx.x == 0) {
        record_step(P, S, t, arrived, ver_in, ver_out, age_state, eff_state, forced, eff_user,
                    age_user, nullptr);
        return;
    }
    if ((int64_t)blockIdx.x > n_tiles) {
        // x_hat[j] is read only where j's block is not taken, which no tile
        // of this launch writes
        const int64_t h0 = ((int64_t)blockIdx.x - 1 - n_tiles) * kAssembleTile;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t k = h0 + threadIdx.x + u * kAssembleThreads;
            if (k < n_hot) {
                const int32_t j = hot_col[k], p = hot_rank[k];
                hot[k] = stale_select(ver_in[p], arrived[p], t, S) ? c[j] * x_own[j]
                                                                   : c[j] * x_hat[j];
            }
        }
        return;
    }
    const Tile tile = tiles[blockIdx.x - 1];
    const int32_t p = tile.rank;
    const bool take = stale_select(ver_in[p], arrived[p], t, S);
    const int64_t j0 = displs[p] + tile.off;
    const int32_t len = tile.len;
    static_assert(kAssembleTile / kAssembleThreads == 8, "eight elements per thread");
    if (len <= 0) return;
    const int32_t last = len - 1;
    double cj[8], xo[8], xh[8];
    // clamped reads, all in flight together
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int64_t j = j0 + min((int32_t)threadIdx.x + u * kAssembleThreads, last);
        cj[u] = c[j];
        xo[u] = x_own[j];
        xh[u] = take ? 0.0 : x_hat[j];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int32_t k = threadIdx.x + u * kAssembleThreads;
        if (k < len) {
            const int64_t j = j0 + k;
            const double zo = cj[u] * xo[u];
            z_own[j] = zo;
            if (take) {
                x_hat[j] = xo[u];
                z_hat[j] = zo;
            } else {
                z_hat[j] = cj[u] * xh[u];
            }
        }
    }
}

// Range layout: the sum of a sub-row cut into pieces, its pieces added in
// order (fixup rank = column range).
__global__ void k_range_fix(int32_t n_fix, const Fixup *__restrict__ fix,
                            const double2 *__restrict__ pieces, int64_t rn,
                            double *__restrict__ rpart, const int32_t *done) {
    if (done && *done) return;
    for (int32_t f = blockIdx.x * blockDim.x + threadIdx.x; f < n_fix; f += gridDim.x * blockDim.x) {
        const Fixup x = fix[f];
        double s = 0.0;
        for (int32_t j = 0; j < x.npieces; ++j) s = s + pieces[x.slot0 + j].x;
        rpart[(int64_t)x.rank * rn + x.row] = s;
    }
}

struct RangeFinishArgs {
    int64_t n;
    int32_t n_ranges;
    const uint16_t *rmask;
    const double *rpart;  // [n_ranges][n]
    const double *diag;
    const double *b;
    double alpha, beta;
    const double *x_own;
    double *x_next;
    double *partials;     // [gridDim.x + 1]
    const int32_t *done;
};

// Range layout, second kernel: a row's sum is its sub-rows' sums added in
// range order; then the row is finished as in the other layouts, with one
// norm partial per workgroup (and none for split rows, whose sums are
// already in).  The grid is the sweep's, so workgroups are large and every
// thread takes kFinishRows rows at a time, all their loads in flight.
constexpr int kFinishThreads = 1024;
constexpr int kFinishRows = 4;
template <int KIND>
__global__ __launch_bounds__(kFinishThreads) void k_range_finish(RangeFinishArgs a) {
    __shared__ double s_red[kFinishThreads / 64];
    if (a.done && *a.done) return;
    double contrib = 0.0;
    const int64_t stride = (int64_t)gridDim.x * kFinishThreads;
    for (int64_t i0 = (int64_t)blockIdx.x * kFinishThreads + threadIdx.x; i0 < a.n;
         i0 += stride * kFinishRows) {
        uint32_t mask[kFinishRows];
        double s[kFinishRows], xo[kFinishRows], dg[kFinishRows], bi[kFinishRows];
#pragma unroll
        for (int u = 0; u < kFinishRows; ++u) {
            const int64_t i = i0 + u * stride;
            const bool live = i < a.n;
            mask[u] = live ? a.rmask[i] : 0u;
            xo[u] = live ? a.x_own[i] : 0.0;
            dg[u] = (KIND == ECC_KIND_JACOBI && live) ? a.diag[i] : 0.0;
            bi[u] = (KIND == ECC_KIND_JACOBI && live) ? a.b[i] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < kFinishRows; ++u) {
            const int64_t i = i0 + u * stride;
            s[u] = 0.0;
            for (int x = 0; x < a.n_ranges; ++x)
                if ((mask[u] >> x) & 1u) s[u] = s[u] + a.rpart[(int64_t)x * a.n + i];
        }
#pragma unroll
        for (int u = 0; u < kFinishRows; ++u) {
            const int64_t i = i0 + u * stride;
            if (i < a.n)
                contrib += row_finish<KIND>((int32_t)i, s[u], dg[u], bi[u], xo[u], a.alpha,
                                            a.beta, a.x_next);
        }
    }
    const double total = block_sum<kFinishThreads>(contrib, s_red);
    if (threadIdx.x == 0) {
        a.partials[blockIdx.x] = total;
        if (blockIdx.x == 0) a.partials[gridDim.x] = 0.0;
    }
}

// Entries of one short row in the item-major copy.  Item w's entries start
// at row offset base = w.k0 (a multiple of 32) and are stored entry-major
// over the item's rows padded to a multiple of 32: entry k of the item's
// row l sits at [base * R + k * pad + l], so the lanes of a wave load
// consecutive words and an item's entries are one contiguous run of the
// copy, which is laid out in the order the items are swept.  Padding past a
// row's end has column -1.
// In the diagonal form (DIA) plane k holds the row's entry on diagonal k
// (column row + dia.v[k]), and a byte per row (at [base + l]) says which
// diagonals the row holds: no column indices are stored.  Diagonals are in
// ascending order of offset, so for rows whose entries are sorted by column
// plane order is CSR order.
template <int R>
struct EllEntries {
    int32_t c[R];
    double v[R];
};


template <int R, bool DIA>
__device__ __forceinline__ void ell_entries(const SweepArgs &a, bool live, const WorkItem &w,
                                            int32_t l, EllEntries<R> &e) {
    const int64_t base = (int64_t)w.k0 * R + l;
    const int32_t pad = sell_pad(w.nrows);
    uint32_t mk = 0;
    if constexpr (DIA) mk = live ? a.ell_mask[(int64_t)w.k0 + l] : 0u;
#pragma unroll
    for (int j = 0; j < R; ++j) {
        const int64_t k = base + (int64_t)j * pad;
        if constexpr (DIA) e.c[j] = ((mk >> j) & 1u) ? w.row0 + l + a.dia.v[j] : -1;
        else e.c[j] = live ? a.ell_col[k] : -1;
        e.v[j] = live ? a.ell_val[k] : 0.0;
    }
}

// Short-row layout over the column-major copy, one lane per row, as a
// two-deep pipeline over the workgroup's items: a row's entries depend only
// on the item's descriptor, so while the gathers of item n are in flight
// the entries of item n + 1 are loaded (and the descriptor of item n + 2).
template <int KIND, bool STEP, int R, bool DIA>
__device__ __forceinline__ void short_body(const SweepArgs &a) {
    __shared__ double s_red[kSweepThreads / 64];
    __shared__ uint8_t s_eff[STEP ? kFusedMaxP : 1];
    __shared__ int32_t s_bs[STEP ? kFusedMaxP + 1 : 1];
    if (a.done && *a.done) return;
    const int tid = threadIdx.x;
    int64_t i_end;
    int32_t w, w_step;
    item_walk(a, i_end, w, w_step);
    bool have = w < i_end;
    bool have_next = have && (int64_t)w + w_step < i_end;
    WorkItem cur{}, nxt{};
    EllEntries<R> E;
    if (have) cur = a.items[w];
    ell_entries<R, DIA>(a, have && tid < cur.nrows, cur, tid, E);
    if (have_next) nxt = a.items[w + w_step];
    StepView sv{s_eff, s_bs, a.P};
    sweep_prologue<STEP>(a, s_eff, s_bs, s_red);

    double contrib = 0.0;
    RankCache rc;
    while (have) {
        const bool have_nn = have_next && (int64_t)w + 2 * (int64_t)w_step < i_end;
        WorkItem nn{};
        if (have_nn) nn = a.items[w + 2 * w_step];
        const bool live = tid < cur.nrows;
        const int32_t i = cur.row0 + tid;
        // this item's gathers first, then the next item's entries
        double y[R];
#pragma unroll
        for (int j = 0; j < R; ++j)
            // Jacobi sums the diagonal entry apart: no gather for it
            y[j] = (E.c[j] >= 0 && !(KIND == ECC_KIND_JACOBI && E.c[j] == i))
                       ? view_load<STEP>(E.c[j], cur.lo, cur.hi, a.x_own, a.x_hat, sv, rc)
                       : 0.0;
        double xo = 0.0, bi = 0.0;
        if (live) {
            xo = a.x_own[i];
            if (KIND == ECC_KIND_JACOBI) bi = a.b[i];
        }
        EllEntries<R> En;
        ell_entries<R, DIA>(a, have_next && tid < nxt.nrows, nxt, tid, En);
        if (live) {
            double s = 0.0, dg = 0.0;
#pragma unroll
            for (int j = 0; j < R; ++j) {
                if (E.c[j] >= 0) {
                    if (KIND == ECC_KIND_JACOBI && E.c[j] == i) dg = E.v[j];
                    else s = s + E.v[j] * y[j];
                }
            }
            if (STEP && s_eff[cur.rank] != 0) a.x_hat[i] = xo;
            const double c = row_finish<KIND>(i, s, dg, bi, xo, a.alpha, a.beta, a.x_next);
            if (a.row_part) a.partials[i] = c;
            else contrib += c;
        }
        w += w_step;
        have = have_next;
        have_next = have_nn;
        cur = nxt;
        nxt = nn;
        E = En;
    }
    if (a.row_part) return;  // (uniform across the grid)
    const double total = block_sum<kSweepThreads>(contrib, s_red);
    if (tid == 0) a.partials[blockIdx.x] = total;
}

// Item queue of a short-layout sweep.  With a static walk (item_walk) the
// workgroups of an XCD drift apart: on MI355X, in a 400^3 Jacobi sweep, the
// items an XCD's 160 workgroups start within one round span about 4,400
// items instead of 160, so the rows that neighbour each other one plane
// apart no longer meet in L2.  Here the items are split into kQueueRanges
// contiguous ranges (range r for the workgroups of XCD r), and a workgroup
// claims the next item of its own XCD's range with an agent-scope atomic
// ticket; once that range is exhausted it moves on to the following ranges.
// Every item is claimed exactly once whatever the mapping of workgroups to
// XCDs, and the XCD's active items stay those in flight.  The last workgroup
// to finish zeroes the counters for the next launch.  Each item writes its
// own partial norm (its four waves' sums added in wave order), so the norm
// does not depend on which workgroup took which item.
// Claims item tickets for thread 0: the next item of range r, moving on
// while ranges are exhausted; -1 once every range is.
__device__ __forceinline__ int32_t queue_take(unsigned *q, int64_t n_items, int &r, int &left) {
    while (left > 0) {
        const int64_t b = n_items * r / kQueueRanges, e = n_items * (r + 1) / kQueueRanges;
        const unsigned t = atomicAdd(&q[r * kQueueStride], 1u);
        if ((int64_t)t < e - b) return (int32_t)(b + t);
        r = (r + 1) % kQueueRanges;
        --left;
    }
    return -1;
}

// The hardware id of the XCD running the calling wave (HW_REG_XCC_ID, bits
// 3:0): a read of a hardware register.
__device__ __forceinline__ int xcc_id() {
    return (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15);
}

// Short-row layout with queue-claimed items.  The same two-deep pipeline as
// short_body: tickets are taken three items ahead by thread 0 and handed to
// the workgroup through LDS at the one barrier per item, where the item's
// partial norm is also assembled.
template <int KIND, bool STEP, int R, bool DIA>
__device__ __forceinline__ void short_body_queue(const SweepArgs &a) {
    __shared__ double s_red[kSweepThreads / 64];
    __shared__ double s_ws[2][kSweepThreads / 64];
    __shared__ int32_t s_tk[5];  // [0..1] tickets handed on per item, [2..4] the first three
    __shared__ uint8_t s_eff[STEP ? kFusedMaxP : 1];
    __shared__ int32_t s_bs[STEP ? kFusedMaxP + 1 : 1];
    if (a.done && *a.done) return;
    const int tid = threadIdx.x;
    int r = 0, left = kQueueRanges;
    if (tid == 0) {
        r = xcc_id() % kQueueRanges;
        for (int k = 0; k < 3; ++k) s_tk[2 + k] = queue_take(a.queue, a.n_items, r, left);
    }
    StepView sv{s_eff, s_bs, a.P};
    sweep_prologue<STEP>(a, s_eff, s_bs, s_red);
    __syncthreads();
    int32_t w = s_tk[2], wn = s_tk[3], wnn = s_tk[4];
    WorkItem cur{}, nxt{};
    EllEntries<R> E;
    if (w >= 0) cur = a.items[w];
    ell_entries<R, DIA>(a, w >= 0 && tid < cur.nrows, cur, tid, E);
    if (wn >= 0) nxt = a.items[wn];
    RankCache rc;
    int kk = 0;
    while (w >= 0) {
        int32_t tk = -1;
        if (tid == 0 && wnn >= 0) tk = queue_take(a.queue, a.n_items, r, left);
        WorkItem nn{};
        if (wnn >= 0) nn = a.items[wnn];
        const bool live = tid < cur.nrows;
        const int32_t i = cur.row0 + tid;
        double y[R];
#pragma unroll
        for (int j = 0; j < R; ++j)
            // Jacobi sums the diagonal entry apart: no gather for it
            y[j] = (E.c[j] >= 0 && !(KIND == ECC_KIND_JACOBI && E.c[j] == i))
                       ? view_load<STEP>(E.c[j], cur.lo, cur.hi, a.x_own, a.x_hat, sv, rc)
                       : 0.0;
        double xo = 0.0, bi = 0.0;
        if (live) {
            xo = a.x_own[i];
            if (KIND == ECC_KIND_JACOBI) bi = a.b[i];
        }
        EllEntries<R> En;
        ell_entries<R, DIA>(a, wn >= 0 && tid < nxt.nrows, nxt, tid, En);
        double c = 0.0;
        if (live) {
            double s = 0.0, dg = 0.0;
#pragma unroll
            for (int j = 0; j < R; ++j) {
                if (E.c[j] >= 0) {
                    if (KIND == ECC_KIND_JACOBI && E.c[j] == i) dg = E.v[j];
                    else s = s + E.v[j] * y[j];
                }
            }
            if (STEP && s_eff[cur.rank] != 0) a.x_hat[i] = xo;
            c = row_finish<KIND>(i, s, dg, bi, xo, a.alpha, a.beta, a.x_next);
        }
        c = group_sum<64>(c);
        const int slot = kk & 1;
        if ((tid & 63) == 0) s_ws[slot][tid >> 6] = c;
        if (tid == 0) s_tk[slot] = tk;
        __syncthreads();
        if (tid == 0) {
            double t = s_ws[slot][0];
#pragma unroll
            for (int q = 1; q < kSweepThreads / 64; ++q) t += s_ws[slot][q];
            a.partials[w] = t;
        }
        const int32_t w3 = s_tk[slot];
        ++kk;
        w = wn;
        wn = wnn;
        wnn = w3;
        cur = nxt;
        nxt = nn;
        E = En;
    }
    // the last workgroup out zeroes the counters for the next launch
    if (tid == 0) {
        unsigned *fin = a.queue + kQueueRanges * kQueueStride;
        if (atomicAdd(fin, 1u) == gridDim.x - 1) {
            for (int q = 0; q < kQueueRanges; ++q) atomicExch(a.queue + q * kQueueStride, 0u);
            atomicExch(fin, 0u);
        }
    }
}

// Item-major copy of a matrix whose rows hold at most R entries (layout as
// in ell_entries), one workgroup of kSweepThreads per item: lane l copies
// row row0 + l; lanes of the padding write column -1.
__global__ void k_build_ell(int64_t n_items, int32_t R, const WorkItem *__restrict__ items,
                            const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
                            const double *__restrict__ val, int32_t *__restrict__ ell_col,
                            double *__restrict__ ell_val) {
    for (int64_t w = blockIdx.x; w < n_items; w += gridDim.x) {
        const WorkItem it = items[w];
        const int32_t pad = sell_pad(it.nrows);
        const int32_t l = threadIdx.x;
        if (l >= pad) continue;
        int32_t k0 = 0, len = 0;
        if (l < it.nrows) {
            k0 = row_ptr[it.row0 + l];
            len = row_ptr[it.row0 + l + 1] - k0;
        }
        const int64_t base = (int64_t)it.k0 * R + l;
        for (int32_t j = 0; j < R; ++j) {
            ell_col[base + (int64_t)j * pad] = j < len ? col[k0 + j] : -1;
            ell_val[base + (int64_t)j * pad] = j < len ? val[k0 + j] : 0.0;
        }
    }
}

// The short-row layout holds few values per lane: the register budget is
// capped so that as many waves share each SIMD as the row's registers allow
// without spilling -- 8 for rows of up to 4 entries, 7 for 5, 5 for 7 or 8
// (the fused Jacobi kernel: 61, 69 and 85-93 VGPRs; 8 waves at R = 5 would
// spill).
template <int R>
constexpr int short_waves() {
    return R <= 4 ? 8 : (R == 5 ? 7 : 5);
}
template <int KIND, bool STEP, int R, bool QUEUE, bool DIA>
__global__ __launch_bounds__(kSweepThreads) __attribute__((amdgpu_waves_per_eu(short_waves<R>())))
void k_sweep_short(SweepArgs a) {
    if constexpr (QUEUE) short_body_queue<KIND, STEP, R, DIA>(a);
    else short_body<KIND, STEP, R, DIA>(a);
}

// Diagonal form: the distinct offsets col - row of a short-row matrix's
// entries, at most kDiagMax.  Each workgroup collects them in a set in LDS
// and merges it into the global set; bad[0] counts sets that overflowed,
// bad[1] rows whose entries are not in increasing column order.  A slot
// goes once from kDiagEmpty to an offset and never changes again, so a
// stale read of a slot only costs a failed compare-and-swap.
constexpr int32_t kDiagEmpty = INT32_MIN;

__device__ __forceinline__ bool diag_insert(int32_t *set, int32_t d) {
    for (int k = 0; k < kDiagMax; ++k) {
        const int32_t v = set[k];
        if (v == d) return true;
        if (v == kDiagEmpty) {
            const int32_t old = atomicCAS(&set[k], kDiagEmpty, d);
            if (old == kDiagEmpty || old == d) return true;
        }
    }
    return false;
}

__global__ void k_diag_set(int32_t n_rows, const int32_t *__restrict__ row_ptr,
                           const int32_t *__restrict__ col, int32_t *__restrict__ set,
                           unsigned long long *__restrict__ bad) {
    __shared__ int32_t s_set[kDiagMax];
    __shared__ int s_over;
    if (threadIdx.x < kDiagMax) s_set[threadIdx.x] = kDiagEmpty;
    if (threadIdx.x == 0) s_over = 0;
    __syncthreads();
    unsigned long long unsorted = 0;
    bool over = false;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_rows;
         i += gridDim.x * blockDim.x) {
        const int32_t k0 = row_ptr[i], k1 = row_ptr[i + 1];
        for (int32_t k = k0; k < k1; ++k) {
            const int32_t c = col[k];
            if (k > k0 && c <= col[k - 1]) ++unsorted;
            if (!over && !diag_insert(s_set, c - i)) over = true;
        }
    }
    if (over) s_over = 1;
    if (unsorted) atomicAdd(&bad[1], unsorted);
    __syncthreads();
    if (threadIdx.x == 0) {
        bool gover = s_over != 0;
        for (int k = 0; k < kDiagMax && !gover; ++k)
            if (s_set[k] != kDiagEmpty && !diag_insert(set, s_set[k])) gover = true;
        if (gover) atomicAdd(&bad[0], 1ull);
    }
}

// The diagonal form of the item-major copy (layout as in ell_entries), one
// workgroup per item: lane l writes its row's value planes (0 where the row
// holds no entry on a diagonal) and its diagonal mask.  Columns of rows
// already checked to lie on the D offsets in `off`.
__global__ void k_build_dia(int64_t n_items, int32_t R, int32_t D, DiagOffsets off,
                            const WorkItem *__restrict__ items,
                            const int32_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
                            const double *__restrict__ val, uint8_t *__restrict__ ell_mask,
                            double *__restrict__ ell_val) {
    for (int64_t w = blockIdx.x; w < n_items; w += gridDim.x) {
        const WorkItem it = items[w];
        const int32_t pad = sell_pad(it.nrows);
        const int32_t l = threadIdx.x;
        if (l >= pad) continue;
        const int64_t base = (int64_t)it.k0 * R + l;
        for (int32_t j = 0; j < R; ++j) ell_val[base + (int64_t)j * pad] = 0.0;
        uint32_t mk = 0;
        if (l < it.nrows) {
            const int32_t i = it.row0 + l;
            for (int32_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k) {
                const int32_t d = col[k] - i;
                int32_t j = 0;
                while (j < D - 1 && off.v[j] != d) ++j;
                ell_val[base + (int64_t)j * pad] = val[k];
                mk |= 1u << j;
            }
        }
        ell_mask[(int64_t)it.k0 + l] = (uint8_t)mk;
    }
}

// Second pass of a sweep, one workgroup of kNormThreads.  (1) Rows split into
// pieces are finished: the piece sums are added in piece order, the row
// epilogue runs (and, in a loop iteration, an arrived rank's split row is
// written into x_hat), and their norm contribution becomes partial `G`.
// (2) With norm != 0 the G + 1 partials are reduced in a fixed order to
// sqrt(sum) (L2) or sum (L1) in *rho_out; with a control block, ctrl[1] :=
// t + 1 and ctrl[0] := 1 once the norm is below tol.
struct Pass2Args {
    double *partials;
    int32_t G;
    const Fixup *fixups;
    int32_t n_fixups;
    const double2 *pieces;
    const double *b;
    double alpha, beta;
    const double *x_own;
    double *x_next;
    double *x_hat;
    const uint8_t *eff_state;  // loop iteration: rank arrivals of this step
    int32_t norm;
    double *rho_out;
    double tol;
    int32_t *ctrl;
    int64_t t;
    const int32_t *done;
};

template <int KIND>
__global__ __launch_bounds__(kNormThreads) void k_pass2(Pass2Args a) {
    __shared__ double s_red[kNormThreads / 64];
    __shared__ double s_fx;
    if (a.done && *a.done) return;
    const int tid = threadIdx.x;
    double fx = 0.0;
    for (int32_t f = tid; f < a.n_fixups; f += kNormThreads) {
        const Fixup fu = a.fixups[f];
        double s = 0.0, dg = 0.0;
        for (int32_t j = 0; j < fu.npieces; ++j) {
            const double2 pc = a.pieces[fu.slot0 + j];
            s = s + pc.x;
            dg = dg + pc.y;
        }
        const double xo = a.x_own[fu.row];
        const double bi = (KIND == ECC_KIND_JACOBI) ? a.b[fu.row] : 0.0;
        fx += row_finish<KIND>(fu.row, s, dg, bi, xo, a.alpha, a.beta, a.x_next);
        if (a.eff_state && a.eff_state[fu.rank]) a.x_hat[fu.row] = xo;
    }
    const double fx_total = block_sum<kNormThreads>(fx, s_red);
    if (tid == 0) {
        a.partials[a.G] = fx_total;
        s_fx = fx_total;
    }
    __syncthreads();
    if (a.norm == 0) return;
    const double sum = reduce_values(a.partials, (int64_t)a.G + 1, true, s_fx, s_red);
    if (tid == 0) {
        const double v = (a.norm == ECC_NORM_L2) ? sqrt(sum) : sum;
        if (a.rho_out) *a.rho_out = v;
        if (a.ctrl) {
            a.ctrl[1] = (int32_t)a.t + 1;
            if (a.tol > 0.0 && v < a.tol) a.ctrl[0] = 1;
        }
    }
}

// Standalone second pass: norm of n partial values (same order of operations
// as the last workgroup of a sweep).
__global__ __launch_bounds__(kNormThreads) void k_residual(const double *__restrict__ partials,
                                                          int64_t n, int32_t norm,
                                                          double *__restrict__ out) {
    __shared__ double s_red[kNormThreads / 64];
    const double sum = reduce_values(partials, n, false, 0.0, s_red);
    if (threadIdx.x == 0) *out = (norm == ECC_NORM_L2) ? sqrt(sum) : sum;
}

// Structural check of a matrix for a plan: counts rows whose diagonal entry is
// missing, duplicated or zero (Jacobi only) and entries whose column is out of
// range, and finds the bandwidth max |col - row|.  bad[0] = bad rows,
// bad[1] = bad columns, bad[2] = bandwidth.
// Rows longer than kCheckLong entries are left to k_check_long.
constexpr int32_t kCheckLong = 256;

__global__ void k_check(int32_t n_rows, int32_t n_cols, const int32_t *__restrict__ row_ptr,
                        const int32_t *__restrict__ col, const double *__restrict__ val,
                        int32_t check_diag, unsigned long long *__restrict__ bad) {
    unsigned long long bad_rows = 0, bad_cols = 0, band = 0;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_rows;
         i += gridDim.x * blockDim.x) {
        if (row_ptr[i + 1] - row_ptr[i] > kCheckLong) continue;
        int ndiag = 0;
        bool zero = false;
        for (int32_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k) {
            const int32_t c = col[k];
            if (c < 0 || c >= n_cols) ++bad_cols;
            const int64_t d = (int64_t)c - i;
            band = max(band, (unsigned long long)(d < 0 ? -d : d));
            if (c == i) {
                ++ndiag;
                zero = zero || (val[k] == 0.0);
            }
        }
        if (check_diag && (ndiag != 1 || zero)) ++bad_rows;
    }
    if (bad_rows) atomicAdd(&bad[0], bad_rows);
    if (bad_cols) atomicAdd(&bad[1], bad_cols);
    if (band) atomicMax(&bad[2], band);
}

// The same checks for the rows listed in `rows` (those longer than
// kCheckLong), one workgroup per row.
__global__ void k_check_long(int32_t n_long, const int32_t *__restrict__ rows, int32_t n_cols,
                             const int32_t *__restrict__ row_ptr,
                             const int32_t *__restrict__ col, const double *__restrict__ val,
                             int32_t check_diag, unsigned long long *__restrict__ bad) {
    __shared__ int s_ndiag, s_zero;
    unsigned long long bad_cols = 0, band = 0;
    for (int32_t r = blockIdx.x; r < n_long; r += gridDim.x) {
        const int32_t i = rows[r];
        if (threadIdx.x == 0) {
            s_ndiag = 0;
            s_zero = 0;
        }
        __syncthreads();
        int ndiag = 0;
        bool zero = false;
        for (int32_t k = row_ptr[i] + threadIdx.x; k < row_ptr[i + 1]; k += blockDim.x) {
            const int32_t c = col[k];
            if (c < 0 || c >= n_cols) ++bad_cols;
            const int64_t d = (int64_t)c - i;
            band = max(band, (unsigned long long)(d < 0 ? -d : d));
            if (c == i) {
                ++ndiag;
                zero = zero || (val[k] == 0.0);
            }
        }
        if (ndiag) atomicAdd(&s_ndiag, ndiag);
        if (zero) atomicOr(&s_zero, 1);
        __syncthreads();
        if (threadIdx.x == 0 && check_diag && (s_ndiag != 1 || s_zero))
            atomicAdd(&bad[0], 1ull);
        __syncthreads();
    }
    if (bad_cols) atomicAdd(&bad[1], bad_cols);
    if (band) atomicMax(&bad[2], band);
}

// How the columns of a matrix of bandwidth B sit around each row: the
// distance of an entry from the row is m = min(|d|, ||d| - B|), d = col - row
// (its offset from the row itself or from the rows one plane of B rows
// away).  prof[0] = entries with m > lim, prof[1] = the largest m <= lim.
__global__ void k_band_profile(int32_t n_rows, int64_t B, int64_t lim,
                               const int32_t *__restrict__ row_ptr,
                               const int32_t *__restrict__ col,
                               unsigned long long *__restrict__ prof) {
    unsigned long long far = 0, near = 0;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_rows;
         i += gridDim.x * blockDim.x) {
        for (int32_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k) {
            const int64_t d = (int64_t)col[k] - i;
            const int64_t a = d < 0 ? -d : d;
            const int64_t e = a > B ? a - B : B - a;
            const int64_t m = a < e ? a : e;
            if (m > lim) ++far;
            else near = max(near, (unsigned long long)m);
        }
    }
    if (far) atomicAdd(&prof[0], far);
    if (near) atomicMax(&prof[1], near);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

// Work items of a matrix for a plan's row blocks.  Rows longer than one LDS
// stage become vector items (one workgroup) or pieces of kVectorCap nonzeros
// (recombined in order); they come first.  The other rows form runs of
// consecutive rows (stream items) of up to kStreamRows rows and kStreamCap
// nonzeros.  rp holds the row pointers the items address; with `order` (the
// sorted layout) row position r holds row order[r]: stream items keep
// positions, vector items, pieces and fixups name the row itself.
static bool rows_irregular(const std::vector<int32_t> &rp) {
    const int64_t n = (int64_t)rp.size() - 1;
    if (n <= 0) return false;
    int64_t mx = 0;
    for (int64_t i = 0; i < n; ++i) mx = std::max<int64_t>(mx, (int64_t)rp[i + 1] - rp[i]);
    const double mean = (double)rp[n] / (double)n;
    return mx > 64 && (double)mx > 8.0 * (mean + 1.0);
}

static void build_items(const std::vector<int32_t> &rp, const std::vector<int64_t> &counts,
                        const std::vector<int32_t> *order, std::vector<WorkItem> &items,
                        std::vector<Fixup> &fixups, int64_t &n_pieces) {
    std::vector<WorkItem> big, vec, stream;
    n_pieces = 0;
    int64_t row = 0;
    auto make = [](int64_t r0, int64_t nr, int64_t k0, int64_t k1, int64_t lo, int64_t hi,
                   int kind, int64_t p, int64_t slot) {
        WorkItem w{};
        w.row0 = (int32_t)r0;
        w.nrows = (int32_t)nr;
        w.k0 = (int32_t)k0;
        w.k1 = (int32_t)k1;
        w.lo = (int32_t)lo;
        w.hi = (int32_t)hi;
        w.kind = kind;
        w.rank = (int32_t)p;
        w.slot = (int32_t)slot;
        return w;
    };
    for (size_t p = 0; p < counts.size(); ++p) {
        const int64_t lo = row, hi = row + counts[p];
        int64_t i = lo;
        while (i < hi) {
            const int64_t len = (int64_t)rp[i + 1] - rp[i];
            if (len > kStreamCap) {
                const int64_t ri = order ? (*order)[i] : i;
                if (len <= kVectorCap) {
                    vec.push_back(make(ri, 1, rp[i], rp[i + 1], lo, hi, kItemVector, p, 0));
                } else {
                    const int32_t np = (int32_t)((len + kVectorCap - 1) / kVectorCap);
                    fixups.push_back({(int32_t)ri, (int32_t)n_pieces, np, (int32_t)p});
                    for (int32_t j = 0; j < np; ++j) {
                        const int64_t ka = rp[i] + (int64_t)j * kVectorCap;
                        const int64_t kb = std::min<int64_t>(rp[i + 1], ka + kVectorCap);
                        big.push_back(make(ri, 1, ka, kb, lo, hi, kItemPiece, p, n_pieces + j));
                    }
                    n_pieces += np;
                }
                ++i;
                continue;
            }
            const int64_t start = i;
            int64_t nnz = 0;
            while (i < hi && i - start < kStreamRows) {
                const int64_t l = (int64_t)rp[i + 1] - rp[i];
                if (l > kStreamCap || nnz + l > kStreamCap) break;
                nnz += l;
                ++i;
            }
            stream.push_back(make(start, i - start, rp[start], rp[i], lo, hi, kItemStream, p, 0));
        }
        row = hi;
    }
    items.clear();
    items.insert(items.end(), big.begin(), big.end());
    items.insert(items.end(), vec.begin(), vec.end());
    items.insert(items.end(), stream.begin(), stream.end());
}

// Short-row layout: runs of up to kSweepThreads rows of one rank.  With
// plane tiling (plane B > 0, tile W > 0) the runs are taken segment by
// segment, tile by tile: for tau = 0, W, 2W, ... below B and every plane z,
// the rows [z B + tau, z B + min(tau + W, B)) below n.  Each item's k0 is
// the row offset of its entries in the item-major copy (a multiple of 32);
// returns the copy's padded row count.
static int64_t build_short_items(int64_t n, const std::vector<int64_t> &counts, int64_t plane,
                                 int64_t tile, std::vector<WorkItem> &items) {
    std::vector<int64_t> bs(counts.size() + 1, 0);
    for (size_t p = 0; p < counts.size(); ++p) bs[p + 1] = bs[p] + counts[p];
    items.clear();
    int64_t base = 0;
    auto segment = [&](int64_t a, int64_t b) {
        // the rank holding row a: the last p with bs[p] <= a (after empty ranks)
        int64_t p = (std::upper_bound(bs.begin(), bs.end(), a) - bs.begin()) - 1;
        while (a < b) {
            while (bs[p + 1] <= a) ++p;
            const int64_t e = std::min({b, bs[p + 1], a + (int64_t)kSweepThreads});
            WorkItem w{};
            w.row0 = (int32_t)a;
            w.nrows = (int32_t)(e - a);
            w.k0 = (int32_t)std::min<int64_t>(base, INT32_MAX);
            w.lo = (int32_t)bs[p];
            w.hi = (int32_t)bs[p + 1];
            w.kind = kItemStream;
            w.rank = (int32_t)p;
            items.push_back(w);
            base += (e - a + 31) & ~int64_t(31);
            a = e;
        }
    };
    if (plane > 0 && tile > 0) {
        const int64_t planes = (n + plane - 1) / plane;
        for (int64_t tau = 0; tau < plane; tau += tile)
            for (int64_t z = 0; z < planes; ++z) {
                const int64_t a = z * plane + tau;
                const int64_t b = std::min(n, z * plane + std::min(tau + tile, plane));
                if (a < b) segment(a, b);
            }
    } else if (n > 0) {
        segment(0, n);
    }
    return base;
}

// Sorted layout: the rows of every rank ordered by decreasing length, ties in
// row order.  Returns the row at each position and the row pointers of the
// sorted copy.
static void sort_rows(const std::vector<int32_t> &rp, const std::vector<int64_t> &counts,
                      std::vector<int32_t> &order, std::vector<int32_t> &srp) {
    const int64_t n = (int64_t)rp.size() - 1;
    order.resize(n);
    srp.assign(n + 1, 0);
    int64_t lo = 0;
    for (size_t p = 0; p < counts.size(); ++p) {
        const int64_t hi = lo + counts[p];
        for (int64_t i = lo; i < hi; ++i) order[i] = (int32_t)i;
        std::stable_sort(order.begin() + lo, order.begin() + hi, [&](int32_t x, int32_t y) {
            return rp[x + 1] - rp[x] > rp[y + 1] - rp[y];
        });
        lo = hi;
    }
    for (int64_t r = 0; r < n; ++r) srp[r + 1] = srp[r] + (rp[order[r] + 1] - rp[order[r]]);
}

// Range layout: the number of column ranges for a vector of n doubles,
// about `bytes` of it per range.
static int32_t range_count(int64_t n, int64_t bytes) {
    const int64_t nr = (n * 8 + bytes - 1) / bytes;
    return (int32_t)std::min<int64_t>(kMaxRanges, std::max<int64_t>(1, nr));
}

// The column range of column c: NR ranges of equal width over [0, n).
static inline int32_t range_of(int64_t c, int64_t n, int32_t NR) { return (int32_t)(c * NR / n); }

struct RangeBuild {
    std::vector<int32_t> srp;     // [n_sub + 1] row pointers of the sub-rows
    std::vector<int2> sinfo;      // [n_sub] (row, rank)
    std::vector<int32_t> scol;    // [nnz] entries, sub-row by sub-row
    std::vector<double> sval;
    std::vector<uint16_t> rmask;  // [n] ranges in which a row has entries
    std::vector<double> diag;     // [n] Jacobi diagonal
    std::vector<Fixup> rfix;      // split sub-rows
    std::vector<int32_t> hot_col;   // the most gathered columns, ascending
    std::vector<int32_t> hot_rank;  // the rank whose block holds each
};

// Range layout: every row cut into sub-rows by column range (its entries of
// one range, in CSR order); the sub-rows of a range ordered by decreasing
// length class (octaves) across all ranks, in row order within a class;
// ranges one after another.
// Items: pieces and vector items first, then stream items range by range, so
// that the workgroups, walking the items together, gather from one range of
// the vector at a time.  Item rank = the column range; lo/hi of a vector item
// or piece = its row's rank block (stream items carry theirs per sub-row).
static void build_ranges(const std::vector<int32_t> &rp, const std::vector<int32_t> &col,
                         const std::vector<double> &val, const std::vector<int64_t> &counts,
                         int32_t NR, bool jacobi, int32_t hot_cap, RangeBuild &B,
                         std::vector<WorkItem> &items, int64_t &n_pieces) {
    const int64_t n = (int64_t)rp.size() - 1;
    std::vector<int64_t> bs(counts.size() + 1, 0);
    for (size_t p = 0; p < counts.size(); ++p) bs[p + 1] = bs[p] + counts[p];
    std::vector<int32_t> rank_of(n);
    for (size_t p = 0; p < counts.size(); ++p)
        for (int64_t i = bs[p]; i < bs[p + 1]; ++i) rank_of[i] = (int32_t)p;
    // With hot_cap > 0: the hot_cap columns gathered most often from outside
    // their own rank block (at least twice, ties to the lower column), whose
    // entries outside the row's block then name slot k as -1 - k; the sweep
    // reads them from a copy in LDS (the same values: the sums do not change).
    std::vector<int32_t> hot_slot;
    if (hot_cap > 0 && n > 0) {
        std::vector<int64_t> g(n, 0);
        for (int64_t i = 0; i < n; ++i) {
            const int64_t lo = bs[rank_of[i]], hi = bs[rank_of[i] + 1];
            for (int32_t k = rp[i]; k < rp[i + 1]; ++k)
                if (col[k] < lo || col[k] >= hi) ++g[col[k]];
        }
        std::vector<int32_t> cand;
        for (int64_t c = 0; c < n; ++c)
            if (g[c] >= 2) cand.push_back((int32_t)c);
        if ((int64_t)cand.size() > hot_cap) {
            std::nth_element(cand.begin(), cand.begin() + hot_cap, cand.end(),
                             [&](int32_t u, int32_t v) { return g[u] > g[v] || (g[u] == g[v] && u < v); });
            cand.resize(hot_cap);
        }
        std::sort(cand.begin(), cand.end());
        hot_slot.assign(n, -1);
        B.hot_col = cand;
        B.hot_rank.resize(cand.size());
        for (size_t k = 0; k < cand.size(); ++k) {
            hot_slot[cand[k]] = (int32_t)k;
            B.hot_rank[k] = rank_of[cand[k]];
        }
    }
    // sub-rows of each range in row order: (row, length)
    std::vector<std::vector<int32_t>> srow(NR), slen(NR);
    std::vector<int32_t> cnt(NR);
    B.rmask.assign(n, 0);
    B.diag.assign(jacobi ? n : 0, 0.0);
    for (int64_t i = 0; i < n; ++i) {
        std::fill(cnt.begin(), cnt.end(), 0);
        for (int32_t k = rp[i]; k < rp[i + 1]; ++k) {
            ++cnt[range_of(col[k], n, NR)];
            if (jacobi && col[k] == i) B.diag[i] = val[k];
        }
        for (int32_t x = 0; x < NR; ++x)
            if (cnt[x] > 0) {
                srow[x].push_back((int32_t)i);
                slen[x].push_back(cnt[x]);
                B.rmask[i] |= (uint16_t)(1u << x);
            }
    }
    // sorted position of the j-th sub-row (row order) of range x: base[x] + inv[x][j]
    std::vector<int64_t> base(NR + 1, 0);
    std::vector<std::vector<int32_t>> inv(NR);
    for (int32_t x = 0; x < NR; ++x) base[x + 1] = base[x] + (int64_t)srow[x].size();
    const int64_t n_sub = base[NR];
    B.srp.assign(n_sub + 1, 0);
    B.sinfo.resize(n_sub);
    for (int32_t x = 0; x < NR; ++x) {
        const int64_t m = (int64_t)srow[x].size();
        std::vector<int32_t> perm(m);
        for (int64_t j = 0; j < m; ++j) perm[j] = (int32_t)j;
        // decreasing length class (octaves), rows in row order within a class:
        // neighbouring sub-rows then write their sums close together
        auto octave = [&](int32_t u) { return 31 - __builtin_clz((uint32_t)slen[x][u]); };
        std::stable_sort(perm.begin(), perm.end(),
                         [&](int32_t u, int32_t v) { return octave(u) > octave(v); });
        inv[x].resize(m);
        for (int64_t q = 0; q < m; ++q) {
            const int32_t j = perm[q];
            inv[x][j] = (int32_t)q;
            const int64_t r = base[x] + q;
            B.srp[r + 1] = slen[x][j];
            B.sinfo[r] = make_int2(srow[x][j], rank_of[srow[x][j]]);
        }
    }
    for (int64_t r = 0; r < n_sub; ++r) B.srp[r + 1] += B.srp[r];
    // entries: each row's entries of range x to its sub-row, in CSR order
    B.scol.resize(col.size());
    B.sval.resize(val.size());
    std::vector<int32_t> seen(NR, 0);
    std::vector<int64_t> cur(NR);
    for (int64_t i = 0; i < n; ++i) {
        for (int32_t x = 0; x < NR; ++x)
            if ((B.rmask[i] >> x) & 1u) cur[x] = B.srp[base[x] + inv[x][seen[x]++]];
        const int64_t lo = bs[rank_of[i]], hi = bs[rank_of[i] + 1];
        for (int32_t k = rp[i]; k < rp[i + 1]; ++k) {
            const int32_t c = col[k];
            const int64_t d = cur[range_of(c, n, NR)]++;
            const bool hot = !hot_slot.empty() && hot_slot[c] >= 0 && (c < lo || c >= hi);
            B.scol[d] = hot ? -1 - hot_slot[c] : c;
            B.sval[d] = val[k];
        }
    }
    // items
    auto make = [](int64_t r0, int64_t nr, int64_t k0, int64_t k1, int64_t lo, int64_t hi,
                   int kind, int64_t x, int64_t slot) {
        WorkItem w{};
        w.row0 = (int32_t)r0;
        w.nrows = (int32_t)nr;
        w.k0 = (int32_t)k0;
        w.k1 = (int32_t)k1;
        w.lo = (int32_t)lo;
        w.hi = (int32_t)hi;
        w.kind = kind;
        w.rank = (int32_t)x;
        w.slot = (int32_t)slot;
        return w;
    };
    std::vector<WorkItem> big, vec, stream;
    n_pieces = 0;
    for (int32_t x = 0; x < NR; ++x) {
        int64_t r = base[x];
        const int64_t end = base[x + 1];
        while (r < end) {
            const int64_t len = (int64_t)B.srp[r + 1] - B.srp[r];
            if (len > kStreamCap) {
                const int32_t i = B.sinfo[r].x, p = B.sinfo[r].y;
                if (len <= kVectorCap) {
                    vec.push_back(make(i, 1, B.srp[r], B.srp[r + 1], bs[p], bs[p + 1], kItemVector,
                                       x, 0));
                } else {
                    const int32_t np = (int32_t)((len + kVectorCap - 1) / kVectorCap);
                    B.rfix.push_back({i, (int32_t)n_pieces, np, x});
                    for (int32_t j = 0; j < np; ++j) {
                        const int64_t ka = B.srp[r] + (int64_t)j * kVectorCap;
                        const int64_t kb = std::min<int64_t>(B.srp[r + 1], ka + kVectorCap);
                        big.push_back(make(i, 1, ka, kb, bs[p], bs[p + 1], kItemPiece, x,
                                           n_pieces + j));
                    }
                    n_pieces += np;
                }
                ++r;
                continue;
            }
            const int64_t start = r;
            int64_t nnz = 0;
            while (r < end && r - start < kStreamRows) {
                const int64_t l = (int64_t)B.srp[r + 1] - B.srp[r];
                if (l > kStreamCap || nnz + l > kStreamCap) break;
                nnz += l;
                ++r;
            }
            stream.push_back(make(start, r - start, B.srp[start], B.srp[r], 0, 0, kItemStream, x, 0));
        }
    }
    items.clear();
    items.insert(items.end(), big.begin(), big.end());
    items.insert(items.end(), vec.begin(), vec.end());
    items.insert(items.end(), stream.begin(), stream.end());
}

// Copies row order[r] of the matrix to position r of the sorted copy, one
// wave per row.
__global__ void k_sort_rows(int32_t n, const int32_t *__restrict__ order,
                            const int32_t *__restrict__ row_ptr,
                            const int32_t *__restrict__ srow_ptr, const int32_t *__restrict__ col,
                            const double *__restrict__ val, int32_t *__restrict__ scol,
                            double *__restrict__ sval) {
    const int lane = threadIdx.x & 63;
    const int64_t per_block = blockDim.x / 64;
    const int64_t waves = (int64_t)gridDim.x * per_block;
    for (int64_t r = (int64_t)blockIdx.x * per_block + threadIdx.x / 64; r < n; r += waves) {
        const int32_t i = order[r];
        const int32_t src = row_ptr[i], len = row_ptr[i + 1] - src, dst = srow_ptr[r];
        for (int32_t k = lane; k < len; k += 64) {
            scol[dst + k] = col[src + k];
            if (sval) sval[dst + k] = val[src + k];
        }
    }
}

// Workgroups of a sweep: as many as the device holds at once (each then
// walks several items through the load/compute pipeline), at most one per
// item, rounded down to a multiple of the 8 XCDs.
// Occupancy of the kernel a loop iteration launches: the fused one, except
// for the sorted and range layouts, which are never fused.
template <int LAY>
static hipError_t sweep_occupancy(int *per_cu, int kind, bool colscale) {
    constexpr bool S = LAY != kLaySorted && LAY != kLayRanges;
    if constexpr (!S) {
        if (colscale)
            return hipOccupancyMaxActiveBlocksPerMultiprocessor(
                per_cu, k_sweep<ECC_KIND_POWER, false, LAY, true>, kSweepThreads, 0);
    }
    return kind == ECC_KIND_JACOBI
               ? hipOccupancyMaxActiveBlocksPerMultiprocessor(
                     per_cu, k_sweep<ECC_KIND_JACOBI, S, LAY>, kSweepThreads, 0)
               : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                     per_cu, k_sweep<ECC_KIND_POWER, S, LAY>, kSweepThreads, 0);
}

template <int R, bool DIA>
static hipError_t short_occupancy_r(int *per_cu, int kind) {
    return kind == ECC_KIND_JACOBI
               ? hipOccupancyMaxActiveBlocksPerMultiprocessor(
                     per_cu, k_sweep_short<ECC_KIND_JACOBI, true, R, false, DIA>, kSweepThreads, 0)
               : hipOccupancyMaxActiveBlocksPerMultiprocessor(
                     per_cu, k_sweep_short<ECC_KIND_POWER, true, R, false, DIA>, kSweepThreads, 0);
}

// Entries per row of the short-layout kernel that serves rows of at most
// `max_row` entries (the launch below uses the same classes).
static int short_class(int32_t max_row) {
    return max_row <= 3 ? 3 : max_row == 4 ? 4 : max_row == 5 ? 5 : max_row <= 7 ? 7 : 8;
}

template <bool DIA>
static hipError_t short_occupancy(int *per_cu, int kind, int32_t short_r) {
    switch (short_class(short_r)) {
        case 3: return short_occupancy_r<3, DIA>(per_cu, kind);
        case 4: return short_occupancy_r<4, DIA>(per_cu, kind);
        case 5: return short_occupancy_r<5, DIA>(per_cu, kind);
        case 7: return short_occupancy_r<7, DIA>(per_cu, kind);
        default: return short_occupancy_r<8, DIA>(per_cu, kind);
    }
}

static int32_t sweep_grid(int64_t n_items, int kind, int layout, int32_t short_r,
                          bool colscale, bool dia) {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        cus = 256;
    const hipError_t e =
        layout == kLaySorted   ? sweep_occupancy<kLaySorted>(&per_cu, kind, colscale)
        : layout == kLayRanges ? sweep_occupancy<kLayRanges>(&per_cu, kind, colscale)
        : layout == kLayShort  ? (dia ? short_occupancy<true>(&per_cu, kind, short_r)
                                      : short_occupancy<false>(&per_cu, kind, short_r))
                               : sweep_occupancy<kLayStream>(&per_cu, kind, false);
    if (e != hipSuccess || per_cu < 1) per_cu = 4;
    const int64_t resident = (int64_t)std::max(cus, 1) * per_cu;
    int64_t g = std::max<int64_t>(1, std::min<int64_t>({n_items, resident, (int64_t)kMaxSweepBlocks}));
    if (g >= 8) g -= g % 8;
    return (int32_t)g;
}

// The short-row kernel of a matrix's row class.
template <int K, bool S, bool Q, bool D>
static void launch_short(ecc_matrix_t M, dim3 grid, dim3 block, hipStream_t st,
                         const SweepArgs &a) {
    switch (short_class(M->short_r)) {
        case 3: hipLaunchKernelGGL((k_sweep_short<K, S, 3, Q, D>), grid, block, 0, st, a); break;
        case 4: hipLaunchKernelGGL((k_sweep_short<K, S, 4, Q, D>), grid, block, 0, st, a); break;
        case 5: hipLaunchKernelGGL((k_sweep_short<K, S, 5, Q, D>), grid, block, 0, st, a); break;
        case 7: hipLaunchKernelGGL((k_sweep_short<K, S, 7, Q, D>), grid, block, 0, st, a); break;
        default: hipLaunchKernelGGL((k_sweep_short<K, S, 8, Q, D>), grid, block, 0, st, a); break;
    }
}

// The kernel of a matrix's layout.  Matrices with very uneven rows are only
// swept after a separate assembly (see ecc_solve), so their fused kernel is
// never built.
template <int K, bool S>
static void launch_layout(ecc_matrix_t M, dim3 grid, dim3 block, hipStream_t st,
                          const SweepArgs &a) {
    if (K == ECC_KIND_POWER && !S && M->colscale) {
        if (M->layout == kLaySorted)
            hipLaunchKernelGGL((k_sweep<ECC_KIND_POWER, false, kLaySorted, true>), grid, block, 0,
                               st, a);
        else
            hipLaunchKernelGGL((k_sweep<ECC_KIND_POWER, false, kLayRanges, true>), grid, block, 0,
                               st, a);
    } else if (M->layout == kLaySorted) {
        if constexpr (!S) hipLaunchKernelGGL((k_sweep<K, S, kLaySorted>), grid, block, 0, st, a);
    } else if (M->layout == kLayRanges) {
        if constexpr (!S) hipLaunchKernelGGL((k_sweep<K, S, kLayRanges>), grid, block, 0, st, a);
    } else if (M->layout == kLayShort) {
        if (M->queue) {
            if (M->dia) launch_short<K, S, true, true>(M, grid, block, st, a);
            else launch_short<K, S, true, false>(M, grid, block, st, a);
        } else {
            if (M->dia) launch_short<K, S, false, true>(M, grid, block, st, a);
            else launch_short<K, S, false, false>(M, grid, block, st, a);
        }
    } else {
        hipLaunchKernelGGL((k_sweep<K, S, kLayStream>), grid, block, 0, st, a);
    }
}

ecc_status_t launch_sweep(ecc_matrix_t M, const SweepLaunch &L) {
    ecc_plan_t pl = M->plan;
    SweepArgs a{};
    a.items = M->d_items;
    a.n_items = (int32_t)M->n_items;
    const bool sorted = M->layout == kLaySorted || M->layout == kLayRanges;
    a.row_ptr = sorted ? M->d_srow_ptr : M->A.d_row_ptr;
    a.col = sorted ? M->d_scol : M->A.d_col;
    a.val = sorted ? M->d_sval : M->A.d_val;
    a.b = L.b;
    a.alpha = L.alpha;
    a.beta = L.beta;
    a.x_own = L.x_own;
    a.x_hat = L.x_hat;
    a.x_next = L.x_next;
    a.g_own = M->colscale ? M->d_zown : L.x_own;
    a.g_hat = M->colscale ? M->d_zhat : L.x_hat;
    a.hot = M->d_hot;
    a.n_hot = M->n_hot;
    a.partials = L.partials;
    a.pieces = M->d_pieces;
    a.order = M->d_order;
    a.sinfo = M->d_sinfo;
    a.rpart = M->d_rpart;
    a.rn = M->A.n_rows;
    a.block_start = pl->d_block_start;
    a.ell_col = M->d_ell_col;
    a.ell_val = M->d_ell_val;
    a.ell_mask = M->d_ell_mask;
    a.dia = M->dia_off;
    a.ell_n = M->A.n_rows;
    a.interleave = M->irregular ? 1 : 0;
    // a queue-scheduled sweep needs no reserved workgroup: workgroup 0 takes
    // items once its reduction of the previous partials is done
    a.reserve0 = (M->grid >= kReserveMinGrid && !M->queue) ? 1 : 0;
    a.n_part = M->n_part;
    a.queue = M->queue ? M->d_queue : nullptr;
    a.row_part = M->tiny ? 1 : 0;
    a.zero_extra = M->n_fixups == 0 ? 1 : 0;
    a.prev_partials = L.prev_partials;
    a.prev_rho = L.prev_rho;
    a.norm = L.norm;
    a.done = L.done;
    const bool step = L.arrived != nullptr;
    if (step) {
        const int64_t t = pl->clock;
        if (pl->P > kFusedMaxP || !pl->d_block_start || M->layout == kLaySorted ||
            M->layout == kLayRanges) {
            set_error("internal: fused step does not fit the plan or the matrix");
            return ECC_ERR_STATE;
        }
        a.step = 1;
        a.P = pl->P;
        a.S = pl->S;
        a.t = t;
        a.arrived = L.arrived;
        a.ver_in = pl->d_version + (t & 1) * pl->P;
        a.ver_out = pl->d_version + ((t + 1) & 1) * pl->P;
        a.age_state = pl->d_age;
        a.eff_state = pl->d_eff;
        a.forced = pl->d_forced;
        a.eff_user = L.eff_user;
        a.age_user = L.age_user;
        a.block_start = pl->d_block_start;
    }
    TimedLaunch timed(pl, ECC_TIMING_SWEEP);
    const dim3 grid(M->grid), block(kSweepThreads);
    hipStream_t st = pl->stream;
    if (M->colscale && !L.scaled && M->A.n_rows > 0) {
        // the views this sweep gathers, scaled by the column values
        const int64_t n = M->A.n_rows;
        const int64_t per = (int64_t)kScaleThreads * kScaleElems;
        const int sg = (int)std::min<int64_t>(8192, (n + per - 1) / per);
        hipLaunchKernelGGL(k_col_scale, dim3(sg), dim3(kScaleThreads), 0, st, n, M->d_cscale,
                           L.x_own, L.x_hat, M->d_zown, M->d_zhat, M->n_hot, M->d_hot_col,
                           M->d_hot, L.done);
        ECC_LAUNCH_CHECK();
    }
    if (M->kind == ECC_KIND_JACOBI) {
        if (step) launch_layout<ECC_KIND_JACOBI, true>(M, grid, block, st, a);
        else launch_layout<ECC_KIND_JACOBI, false>(M, grid, block, st, a);
    } else {
        if (step) launch_layout<ECC_KIND_POWER, true>(M, grid, block, st, a);
        else launch_layout<ECC_KIND_POWER, false>(M, grid, block, st, a);
    }
    ECC_LAUNCH_CHECK();
    if (M->layout == kLayRanges) {
        // the split sub-rows' sums, then every row from its sub-rows' sums
        if (M->n_rfix > 0) {
            const int fb = (int)std::min<int64_t>(1024, (M->n_rfix + 255) / 256);
            hipLaunchKernelGGL(k_range_fix, dim3(fb), dim3(256), 0, st, (int32_t)M->n_rfix,
                               M->d_rfix, M->d_pieces, (int64_t)M->A.n_rows, M->d_rpart, L.done);
            ECC_LAUNCH_CHECK();
        }
        RangeFinishArgs f{};
        f.n = M->A.n_rows;
        f.n_ranges = M->n_ranges;
        f.rmask = M->d_rmask;
        f.rpart = M->d_rpart;
        f.diag = M->d_diag;
        f.b = L.b;
        f.alpha = L.alpha;
        f.beta = L.beta;
        f.x_own = L.x_own;
        f.x_next = L.x_next;
        f.partials = L.partials;
        f.done = L.done;
        const dim3 fblock(kFinishThreads);
        if (M->kind == ECC_KIND_JACOBI)
            hipLaunchKernelGGL(k_range_finish<ECC_KIND_JACOBI>, grid, fblock, 0, st, f);
        else
            hipLaunchKernelGGL(k_range_finish<ECC_KIND_POWER>, grid, fblock, 0, st, f);
        ECC_LAUNCH_CHECK();
    }
    if (step) pl->clock += 1;
    return ECC_OK;
}

ecc_status_t launch_assemble_scaled(ecc_matrix_t M, const double *x_own, double *x_hat,
                                    const uint8_t *d_arrived, uint8_t *d_eff_out,
                                    int32_t *d_age_out, const int32_t *d_done) {
    ecc_plan_t plan = M->plan;
    if (!M->colscale) {
        set_error("internal: scaled assembly for a matrix without column values");
        return ECC_ERR_STATE;
    }
    const int64_t t = plan->clock;
    const int32_t *ver_in = plan->d_version + (t & 1) * plan->P;
    int32_t *ver_out = plan->d_version + ((t + 1) & 1) * plan->P;
    // the tiles, then the hot columns' copy (kAssembleTile per workgroup)
    const int64_t grid = 1 + plan->n_tiles + (M->n_hot + kAssembleTile - 1) / kAssembleTile;
    if (grid > 0x7fffffff) {
        set_error("too many assembly tiles");
        return ECC_ERR_RANGE;
    }
    TimedLaunch timed(plan, ECC_TIMING_ASSEMBLE);
    hipLaunchKernelGGL(k_assemble_scaled, dim3((unsigned)grid), dim3(kAssembleThreads), 0,
                       plan->stream, plan->P, plan->S, t, d_arrived, ver_in, ver_out, plan->d_age,
                       plan->d_eff, plan->d_forced, d_eff_out, d_age_out, plan->d_tiles,
                       plan->d_displs, M->d_cscale, x_own, x_hat, M->d_zown, M->d_zhat,
                       plan->n_tiles, M->n_hot, M->d_hot_col, M->d_hot_rank, M->d_hot, d_done);
    ECC_LAUNCH_CHECK();
    plan->clock = t + 1;
    return ECC_OK;
}

ecc_status_t launch_pass2(ecc_matrix_t M, const Pass2Launch &L) {
    ecc_plan_t pl = M->plan;
    Pass2Args a{};
    a.partials = L.partials;
    a.G = (int32_t)(M->n_part - 1);
    a.fixups = M->d_fixups;
    a.n_fixups = (int32_t)M->n_fixups;
    a.pieces = M->d_pieces;
    a.b = L.b;
    a.alpha = L.alpha;
    a.beta = L.beta;
    a.x_own = L.x_own;
    a.x_next = L.x_next;
    a.x_hat = L.x_hat;
    a.eff_state = L.step ? pl->d_eff : nullptr;
    a.norm = L.norm;
    a.rho_out = L.rho_out;
    a.tol = L.tol;
    a.ctrl = L.ctrl;
    a.t = L.t;
    a.done = L.done;
    TimedLaunch timed(pl, ECC_TIMING_NORM);
    if (M->kind == ECC_KIND_JACOBI)
        hipLaunchKernelGGL(k_pass2<ECC_KIND_JACOBI>, dim3(1), dim3(kNormThreads), 0, pl->stream, a);
    else
        hipLaunchKernelGGL(k_pass2<ECC_KIND_POWER>, dim3(1), dim3(kNormThreads), 0, pl->stream, a);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

}  // namespace ecc

using namespace ecc;

extern "C" {

static ecc_status_t ecc_matrix_create_impl(ecc_plan_t plan, const ecc_csr_t *A, int32_t kind,
                                           const ecc_matrix_opts_t *opts_in, ecc_matrix_t *out) {
    clear_error();
    ECC_ARG(out != nullptr, "out is NULL");
    *out = nullptr;
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(A != nullptr, "A is NULL");
    const ecc_matrix_opts_t opts = opts_in ? *opts_in : ecc_matrix_opts_t{0, 0, 0, 0};
    ECC_ARG(opts.range_bytes >= 0, "range_bytes is negative");
    ECC_ARG(opts.schedule == ECC_SCHEDULE_AUTO || opts.schedule == ECC_SCHEDULE_STATIC ||
                opts.schedule == ECC_SCHEDULE_QUEUE || opts.schedule == ECC_SCHEDULE_SINGLE,
            "unknown schedule %d", opts.schedule);
    ECC_ARG(opts.compact == ECC_COMPACT_AUTO || opts.compact == ECC_COMPACT_NONE,
            "unknown compact choice %d", opts.compact);
    ECC_ARG(kind == ECC_KIND_JACOBI || kind == ECC_KIND_POWER, "unknown kind %d", kind);
    ECC_ARG(A->n_rows >= 0 && A->n_cols >= 0 && A->nnz >= 0, "negative matrix size");
    if (A->nnz >= (int64_t(1) << 31) || A->n_rows >= (int64_t(1) << 31) ||
        A->n_cols >= (int64_t(1) << 31)) {
        set_error("matrix too large for int32 indices");
        return ECC_ERR_RANGE;
    }
    if (!plan->has_layout || !plan->tiles_rows || !plan->d_block_start) {
        set_error("iterations need a plan whose blocks tile [0, n) in rank order");
        return ECC_ERR_STATE;
    }
    if (A->n_rows != A->n_cols || A->n_rows != plan->extent) {
        set_error("matrix must be square with n_rows = %lld (the plan's extent)",
                  (long long)plan->extent);
        return ECC_ERR_STATE;
    }
    ECC_ARG(A->d_row_ptr != nullptr, "row_ptr is NULL");
    ECC_ARG(A->nnz == 0 || (A->d_col && A->d_val), "col/val are NULL");

    const int64_t n = A->n_rows;
    std::vector<int32_t> rp(n + 1);
    ECC_HIP(hipStreamSynchronize(plan->stream));
    ECC_HIP(hipMemcpy(rp.data(), A->d_row_ptr, sizeof(int32_t) * (n + 1), hipMemcpyDeviceToHost));
    ECC_ARG(rp[0] == 0, "row_ptr[0] must be 0");
    for (int64_t i = 0; i < n; ++i)
        ECC_ARG(rp[i + 1] >= rp[i], "row_ptr must be non-decreasing (row %lld)", (long long)i);
    ECC_ARG(rp[n] == A->nnz, "row_ptr[n] = %d differs from nnz = %lld", rp[n], (long long)A->nnz);

    // structural check on the device: short rows one per lane, long rows
    // (listed here) one per workgroup
    int64_t bandwidth = 0;
    if (n > 0) {
        std::vector<int32_t> long_rows;
        for (int64_t i = 0; i < n; ++i)
            if (rp[i + 1] - rp[i] > kCheckLong) long_rows.push_back((int32_t)i);
        unsigned long long *d_bad = nullptr;
        int32_t *d_long = nullptr;
        unsigned long long h_bad[3] = {0, 0, 0};
        hipError_t e = hipMalloc((void **)&d_bad, 3 * sizeof(unsigned long long));
        if (e == hipSuccess && !long_rows.empty())
            e = hipMalloc((void **)&d_long, sizeof(int32_t) * long_rows.size());
        if (e == hipSuccess && d_long)
            e = hipMemcpy(d_long, long_rows.data(), sizeof(int32_t) * long_rows.size(),
                          hipMemcpyHostToDevice);
        if (e == hipSuccess) e = hipMemcpy(d_bad, h_bad, sizeof(h_bad), hipMemcpyHostToDevice);
        if (e == hipSuccess) {
            const int blocks = (int)std::min<int64_t>(4096, (n + 255) / 256);
            hipLaunchKernelGGL(k_check, dim3(blocks), dim3(256), 0, plan->stream, (int32_t)n,
                               (int32_t)A->n_cols, A->d_row_ptr, A->d_col, A->d_val,
                               kind == ECC_KIND_JACOBI ? 1 : 0, d_bad);
            if (d_long) {
                const int lb = (int)std::min<size_t>(4096, long_rows.size());
                hipLaunchKernelGGL(k_check_long, dim3(lb), dim3(256), 0, plan->stream,
                                   (int32_t)long_rows.size(), d_long, (int32_t)A->n_cols,
                                   A->d_row_ptr, A->d_col, A->d_val,
                                   kind == ECC_KIND_JACOBI ? 1 : 0, d_bad);
            }
            e = hipGetLastError();
            if (e == hipSuccess) e = hipStreamSynchronize(plan->stream);
            if (e == hipSuccess) e = hipMemcpy(h_bad, d_bad, sizeof(h_bad), hipMemcpyDeviceToHost);
        }
        (void)hipFree(d_bad);
        (void)hipFree(d_long);
        if (e != hipSuccess) {
            set_error("matrix check failed: %s", hipGetErrorString(e));
            return ECC_ERR_DEVICE;
        }
        ECC_ARG(h_bad[1] == 0, "%llu column indices are out of range", h_bad[1]);
        ECC_ARG(h_bad[0] == 0, "%llu rows lack a single non-zero diagonal entry", h_bad[0]);
        bandwidth = (int64_t)h_bad[2];
    }

    std::vector<WorkItem> items;
    std::vector<Fixup> fixups;
    int64_t n_pieces = 0;
    // Sorted layout for matrices whose row lengths vary widely (power-law
    // graphs): in row order, neighbouring rows differ so much in length that
    // no split of an item's lanes suits them all.  Measured on MI355X
    // (PageRank on a scale-22 R-MAT graph, 64 ranks): 544 against 644 us per
    // sweep for rows binned into length classes read in place, whose
    // scattered row reads kept the texture address units busier than the
    // gathers of x do.
    const bool irregular = rows_irregular(rp);
    // Short-row layout, over a column-major copy of the entries, for
    // matrices whose rows all hold at most kShortRow entries.  Measured on
    // MI355X (Jacobi on 2-D 5-point and 3-D 7-point Laplacians, 4K-64M rows)
    // it beats the LDS-staged stream layout at every size: 3-D 400^3, 1,715
    // against 1,842 us per sweep.
    int32_t max_row = 0;
    for (int64_t i = 0; i < n; ++i) max_row = std::max(max_row, rp[i + 1] - rp[i]);
    const bool short_rows = max_row <= kShortRow;
    // Column values: a power matrix with very uneven rows whose every column
    // holds one value (the PageRank matrix) is swept from c and the scaled
    // views, without the entries' values.  Measured on MI355X (PageRank on a
    // scale-22 R-MAT graph, 64 ranks, ecc_solve): 472 against 533 us per
    // iteration at 8 MiB ranges.
    double *d_cscale = nullptr;
    bool colscale = false;
    if (kind == ECC_KIND_POWER && irregular && opts.compact == ECC_COMPACT_AUTO && n > 0 &&
        A->nnz > 0) {
        unsigned long long *d_bad = nullptr;
        unsigned long long h_bad = 1;
        hipError_t e = hipMalloc((void **)&d_cscale, sizeof(double) * n);
        if (e == hipSuccess) e = hipMalloc((void **)&d_bad, sizeof(unsigned long long));
        if (e == hipSuccess) e = hipMemsetAsync(d_cscale, 0, sizeof(double) * n, plan->stream);
        if (e == hipSuccess) e = hipMemsetAsync(d_bad, 0, sizeof(unsigned long long), plan->stream);
        if (e == hipSuccess) {
            const int blocks = (int)std::min<int64_t>(8192, (A->nnz + 255) / 256);
            hipLaunchKernelGGL(k_col_values, dim3(blocks), dim3(256), 0, plan->stream, A->nnz,
                               A->d_col, A->d_val, d_cscale);
            hipLaunchKernelGGL(k_col_check, dim3(blocks), dim3(256), 0, plan->stream, A->nnz,
                               A->d_col, A->d_val, d_cscale, d_bad);
            e = hipGetLastError();
            if (e == hipSuccess) e = hipStreamSynchronize(plan->stream);
            if (e == hipSuccess)
                e = hipMemcpy(&h_bad, d_bad, sizeof(h_bad), hipMemcpyDeviceToHost);
        }
        (void)hipFree(d_bad);
        if (e != hipSuccess) {
            (void)hipFree(d_cscale);
            set_error("column value check failed: %s", hipGetErrorString(e));
            return e == hipErrorOutOfMemory ? ECC_ERR_ALLOC : ECC_ERR_DEVICE;
        }
        colscale = h_bad == 0;
        if (!colscale) {
            (void)hipFree(d_cscale);
            d_cscale = nullptr;
        }
    }
    // owned by the handle from here on (freed by fail() below or by destroy)
    struct CscaleGuard {
        double **p;
        ~CscaleGuard() {
            if (*p) (void)hipFree(*p);
        }
    } cscale_guard{&d_cscale};
    // Very uneven rows over a vector of more than one range: the range layout
    // (each range of the vector, about kRangeBytes, is gathered by all
    // workgroups at once, so that the gathers of a time hit one window of
    // the vector).  Without a value stream
    // the sub-rows' own costs weigh more, and wider ranges pay: measured on
    // MI355X (the same PageRank), 452 us per iteration at 16 MiB against 472
    // at 8 MiB and 512 unsplit; the general form takes 533 at 8 MiB and 539
    // at 16 MiB.
    const int64_t range_bytes = opts.range_bytes > 0 ? opts.range_bytes
                                : colscale            ? kRangeBytesColumns
                                                      : kRangeBytes;
    const int32_t n_ranges = irregular ? range_count(n, range_bytes) : 1;
    const int layout = irregular ? (n_ranges >= 2 ? kLayRanges : kLaySorted)
                                 : (short_rows ? kLayShort : kLayStream);
    std::vector<int32_t> order, srp;
    RangeBuild RB;
    int64_t tile_plane = 0, tile_rows = 0, short_rows_total = 0;
    bool dia = false;  // short layout in diagonal form
    int32_t n_dia = 0;
    DiagOffsets dia_off{};
    if (layout == kLayRanges) {
        std::vector<int32_t> hcol(A->nnz);
        std::vector<double> hval(A->nnz);
        ECC_HIP(hipMemcpy(hcol.data(), A->d_col, sizeof(int32_t) * A->nnz, hipMemcpyDeviceToHost));
        ECC_HIP(hipMemcpy(hval.data(), A->d_val, sizeof(double) * A->nnz, hipMemcpyDeviceToHost));
        build_ranges(rp, hcol, hval, plan->counts, n_ranges, kind == ECC_KIND_JACOBI,
                     colscale ? kHotCols : 0, RB, items,
                     n_pieces);
    } else if (irregular) {
        sort_rows(rp, plan->counts, order, srp);
        build_items(srp, plan->counts, &order, items, fixups, n_pieces);
    } else if (layout == kLayShort) {
        // Plane tiling for a matrix whose columns sit near the row or near
        // the rows one bandwidth B away (a 3-D grid stencil, B = one plane),
        // when B rows stream more than an XCD's L2 holds: in row order the
        // neighbours one plane ahead are read B rows before their own rows
        // are swept, and have left L2 by then.
        // A caller's tile size applies whenever the columns qualify.
        const int64_t row_bytes = 12 * (int64_t)short_class(std::max(1, max_row)) + 24;
        const bool big = bandwidth >= 1024 && bandwidth * row_bytes > kTileMinBytes;
        if (opts.tile_rows >= 0 && bandwidth >= 16 && n >= 3 * bandwidth &&
            (big || opts.tile_rows > 0)) {
            unsigned long long h_prof[2] = {0, 0};
            unsigned long long *d_prof = nullptr;
            ECC_HIP(hipMalloc((void **)&d_prof, sizeof(h_prof)));
            hipError_t e = hipMemcpy(d_prof, h_prof, sizeof(h_prof), hipMemcpyHostToDevice);
            if (e == hipSuccess) {
                const int blocks = (int)std::min<int64_t>(4096, (n + 255) / 256);
                hipLaunchKernelGGL(k_band_profile, dim3(blocks), dim3(256), 0, plan->stream,
                                   (int32_t)n, bandwidth, bandwidth / 16, A->d_row_ptr, A->d_col,
                                   d_prof);
                e = hipGetLastError();
                if (e == hipSuccess) e = hipStreamSynchronize(plan->stream);
                if (e == hipSuccess)
                    e = hipMemcpy(h_prof, d_prof, sizeof(h_prof), hipMemcpyDeviceToHost);
            }
            (void)hipFree(d_prof);
            if (e != hipSuccess) {
                set_error("band profile failed: %s", hipGetErrorString(e));
                return ECC_ERR_DEVICE;
            }
            if (h_prof[0] == 0) {
                // tiles wide against the in-plane offsets (the edge rows of a
                // tile re-read their neighbours in the next tile)
                int64_t w = opts.tile_rows > 0 ? opts.tile_rows
                                               : std::max<int64_t>(kTileMinRows,
                                                                   kTileNearFactor * (int64_t)h_prof[1]);
                w = (w + kSweepThreads - 1) / kSweepThreads * kSweepThreads;
                if (w < bandwidth) {
                    tile_plane = bandwidth;
                    tile_rows = w;
                }
            }
        }
        short_rows_total = build_short_items(n, plan->counts, tile_plane, tile_rows, items);
        if (short_rows_total >= (int64_t(1) << 31)) {
            set_error("the short-row copy needs more than 2^31 padded rows");
            return ECC_ERR_RANGE;
        }
        // Diagonal form: entries on at most as many offsets col - row as the
        // row class holds, every row in increasing column order.  Measured
        // on MI355X (Jacobi on the 400^3 7-point stencil): see the sweep
        // profiles.
        if (opts.compact == ECC_COMPACT_AUTO && A->nnz > 0) {
            int32_t h_set[kDiagMax];
            unsigned long long h_bad[2] = {1, 1};
            int32_t *d_set = nullptr;
            unsigned long long *d_bad = nullptr;
            for (int k = 0; k < kDiagMax; ++k) h_set[k] = kDiagEmpty;
            hipError_t e = hipMalloc((void **)&d_set, sizeof(h_set));
            if (e == hipSuccess) e = hipMalloc((void **)&d_bad, sizeof(h_bad));
            const unsigned long long zero2[2] = {0, 0};
            if (e == hipSuccess) e = hipMemcpy(d_set, h_set, sizeof(h_set), hipMemcpyHostToDevice);
            if (e == hipSuccess) e = hipMemcpy(d_bad, zero2, sizeof(zero2), hipMemcpyHostToDevice);
            if (e == hipSuccess) {
                const int blocks = (int)std::min<int64_t>(4096, (n + 255) / 256);
                hipLaunchKernelGGL(k_diag_set, dim3(blocks), dim3(256), 0, plan->stream,
                                   (int32_t)n, A->d_row_ptr, A->d_col, d_set, d_bad);
                e = hipGetLastError();
                if (e == hipSuccess) e = hipStreamSynchronize(plan->stream);
                if (e == hipSuccess) e = hipMemcpy(h_set, d_set, sizeof(h_set), hipMemcpyDeviceToHost);
                if (e == hipSuccess) e = hipMemcpy(h_bad, d_bad, sizeof(h_bad), hipMemcpyDeviceToHost);
            }
            (void)hipFree(d_set);
            (void)hipFree(d_bad);
            if (e != hipSuccess) {
                set_error("diagonal check failed: %s", hipGetErrorString(e));
                return ECC_ERR_DEVICE;
            }
            std::vector<int32_t> offs;
            for (int k = 0; k < kDiagMax; ++k)
                if (h_set[k] != kDiagEmpty) offs.push_back(h_set[k]);
            std::sort(offs.begin(), offs.end());
            const int32_t cls = short_class(std::max(1, max_row));
            if (h_bad[0] == 0 && h_bad[1] == 0 && !offs.empty() &&
                short_class((int32_t)offs.size()) == cls) {
                dia = true;
                n_dia = (int32_t)offs.size();
                for (int k = 0; k < kDiagMax; ++k) dia_off.v[k] = k < n_dia ? offs[k] : 0;
            }
        }
    } else {
        build_items(rp, plan->counts, nullptr, items, fixups, n_pieces);
    }
    if ((int64_t)items.size() >= (int64_t(1) << 31)) {
        set_error("too many work items");
        return ECC_ERR_RANGE;
    }

    ecc_matrix_s *M = new (std::nothrow) ecc_matrix_s();
    if (!M) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
    M->plan = plan;
    M->A = *A;
    M->kind = kind;
    M->n_items = (int64_t)items.size();
    M->n_fixups = (int64_t)fixups.size();
    M->n_pieces = n_pieces;
    M->irregular = irregular;
    M->layout = layout;
    M->short_r = std::max(1, max_row);
    M->bandwidth = bandwidth;
    M->tile_plane = tile_plane;
    M->tile_rows = tile_rows;
    M->grid = sweep_grid(M->n_items, kind, layout, M->short_r, colscale, dia);
    M->dia = dia;
    M->n_dia = n_dia;
    M->dia_off = dia_off;
    M->colscale = colscale;
    M->d_cscale = d_cscale;
    d_cscale = nullptr;
    // Queue-claimed items for a short-layout matrix that gives each workgroup
    // many items (the static walk's drift grows with them): measured on
    // MI355X, Jacobi on the 400^3 7-point stencil, 1.55 against 1.66 ms per
    // sweep.
    M->queue = layout == kLayShort && (opts.schedule == ECC_SCHEDULE_QUEUE ||
                                       (opts.schedule == ECC_SCHEDULE_AUTO &&
                                        M->n_items >= kQueueMinItems * (int64_t)M->grid));
    // A small short-row problem is solved by one launch (tiny.hip), whose
    // norm reduces one partial per row: its sweeps write per-row partials
    // too, so that every entry point gives the same norm.
    M->tiny = layout == kLayShort && tiny_fits(n, M->short_r, M->n_items, plan->P) &&
              (opts.schedule == ECC_SCHEDULE_AUTO || opts.schedule == ECC_SCHEDULE_SINGLE);
    if (M->tiny) M->queue = false;
    M->n_part = M->tiny ? n + 1 : M->queue ? M->n_items + 1 : (int64_t)M->grid + 1;
    auto fail = [&](const char *what) {
        set_error("%s", what);
        ecc_matrix_destroy(M);
        return ECC_ERR_ALLOC;
    };
    if (!items.empty()) {
        if (hipMalloc((void **)&M->d_items, sizeof(WorkItem) * items.size()) != hipSuccess)
            return fail("hipMalloc of work items failed");
        if (hipMemcpy(M->d_items, items.data(), sizeof(WorkItem) * items.size(),
                      hipMemcpyHostToDevice) != hipSuccess)
            return fail("copy of work items failed");
    }
    if (!fixups.empty()) {
        if (hipMalloc((void **)&M->d_fixups, sizeof(Fixup) * fixups.size()) != hipSuccess)
            return fail("hipMalloc of fixups failed");
        if (hipMemcpy(M->d_fixups, fixups.data(), sizeof(Fixup) * fixups.size(),
                      hipMemcpyHostToDevice) != hipSuccess)
            return fail("copy of fixups failed");
    }
    if (n_pieces > 0 && hipMalloc((void **)&M->d_pieces, sizeof(double2) * n_pieces) != hipSuccess)
        return fail("hipMalloc of piece sums failed");
    if (layout == kLaySorted && n > 0) {
        if (hipMalloc((void **)&M->d_order, sizeof(int32_t) * n) != hipSuccess ||
            hipMalloc((void **)&M->d_srow_ptr, sizeof(int32_t) * (n + 1)) != hipSuccess ||
            hipMalloc((void **)&M->d_scol, sizeof(int32_t) * std::max<int64_t>(1, A->nnz)) !=
                hipSuccess ||
            (!colscale &&
             hipMalloc((void **)&M->d_sval, sizeof(double) * std::max<int64_t>(1, A->nnz)) !=
                 hipSuccess))
            return fail("hipMalloc of the sorted copy failed");
        if (hipMemcpy(M->d_order, order.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice) !=
                hipSuccess ||
            hipMemcpy(M->d_srow_ptr, srp.data(), sizeof(int32_t) * (n + 1),
                      hipMemcpyHostToDevice) != hipSuccess)
            return fail("copy of the row order failed");
        const int blocks = (int)std::min<int64_t>(65536, (n + 3) / 4);
        hipLaunchKernelGGL(k_sort_rows, dim3(blocks), dim3(256), 0, plan->stream, (int32_t)n,
                           M->d_order, A->d_row_ptr, M->d_srow_ptr, A->d_col, A->d_val, M->d_scol,
                           M->d_sval);
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(plan->stream) != hipSuccess)
            return fail("building the sorted copy failed");
    }
    if (layout == kLayRanges) {
        M->n_ranges = n_ranges;
        M->n_sub = (int64_t)RB.sinfo.size();
        M->n_rfix = (int64_t)RB.rfix.size();
        auto up = [&](void **dst, const void *src, size_t bytes) {
            if (hipMalloc(dst, std::max<size_t>(bytes, 8)) != hipSuccess) return false;
            return bytes == 0 || hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice) == hipSuccess;
        };
        if (!up((void **)&M->d_srow_ptr, RB.srp.data(), sizeof(int32_t) * RB.srp.size()) ||
            !up((void **)&M->d_sinfo, RB.sinfo.data(), sizeof(int2) * RB.sinfo.size()) ||
            !up((void **)&M->d_scol, RB.scol.data(), sizeof(int32_t) * RB.scol.size()) ||
            (!colscale &&
             !up((void **)&M->d_sval, RB.sval.data(), sizeof(double) * RB.sval.size())) ||
            !up((void **)&M->d_rmask, RB.rmask.data(), sizeof(uint16_t) * RB.rmask.size()) ||
            !up((void **)&M->d_diag, RB.diag.data(), sizeof(double) * RB.diag.size()) ||
            !up((void **)&M->d_rfix, RB.rfix.data(), sizeof(Fixup) * RB.rfix.size()))
            return fail("building the range layout failed");
        M->n_hot = (int32_t)RB.hot_col.size();
        if (M->n_hot > 0 &&
            (!up((void **)&M->d_hot_col, RB.hot_col.data(), sizeof(int32_t) * RB.hot_col.size()) ||
             !up((void **)&M->d_hot_rank, RB.hot_rank.data(),
                 sizeof(int32_t) * RB.hot_rank.size()) ||
             hipMalloc((void **)&M->d_hot, sizeof(double) * RB.hot_col.size()) != hipSuccess))
            return fail("building the hot-column copy failed");
        if (hipMalloc((void **)&M->d_rpart, sizeof(double) * (size_t)n_ranges * (size_t)n) !=
            hipSuccess)
            return fail("hipMalloc of the range sums failed");
    }
    if (layout == kLayShort && n > 0) {
        const int64_t R = short_class(M->short_r);
        if ((dia ? hipMalloc((void **)&M->d_ell_mask, short_rows_total)
                 : hipMalloc((void **)&M->d_ell_col, sizeof(int32_t) * R * short_rows_total)) !=
                hipSuccess ||
            hipMalloc((void **)&M->d_ell_val, sizeof(double) * R * short_rows_total) != hipSuccess)
            return fail("hipMalloc of the item-major entries failed");
        const int blocks = (int)std::min<int64_t>(65536, M->n_items);
        if (dia)
            hipLaunchKernelGGL(k_build_dia, dim3(blocks), dim3(kSweepThreads), 0, plan->stream,
                               M->n_items, (int32_t)R, n_dia, dia_off, M->d_items, A->d_row_ptr,
                               A->d_col, A->d_val, M->d_ell_mask, M->d_ell_val);
        else
            hipLaunchKernelGGL(k_build_ell, dim3(blocks), dim3(kSweepThreads), 0, plan->stream,
                               M->n_items, (int32_t)R, M->d_items, A->d_row_ptr, A->d_col,
                               A->d_val, M->d_ell_col, M->d_ell_val);
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(plan->stream) != hipSuccess)
            return fail("building the item-major entries failed");
    }
    if (colscale && (hipMalloc((void **)&M->d_zown, sizeof(double) * n) != hipSuccess ||
                     hipMalloc((void **)&M->d_zhat, sizeof(double) * n) != hipSuccess))
        return fail("hipMalloc of the scaled views failed");
    // two buffers of G + 1 partials: a loop iteration writes one while the
    // next launch reduces the other
    if (hipMalloc((void **)&M->d_partials, sizeof(double) * 2 * M->n_part) != hipSuccess)
        return fail("hipMalloc of partials failed");
    if (M->queue) {
        const size_t qb = sizeof(unsigned) * (kQueueRanges + 1) * kQueueStride;
        if (hipMalloc((void **)&M->d_queue, qb) != hipSuccess ||
            hipMemsetAsync(M->d_queue, 0, qb, plan->stream) != hipSuccess ||
            hipStreamSynchronize(plan->stream) != hipSuccess)
            return fail("allocating the item queue failed");
    }
    *out = M;
    return ECC_OK;
}

// Host allocations of the set-up throw std::bad_alloc when memory runs
// out: the C ABI reports ECC_ERR_ALLOC instead of letting it escape.
ecc_status_t ecc_matrix_create(ecc_plan_t plan, const ecc_csr_t *A, int32_t kind,
                               ecc_matrix_t *out) {
    return ecc_matrix_create_ex(plan, A, kind, nullptr, out);
}

ecc_status_t ecc_matrix_create_ex(ecc_plan_t plan, const ecc_csr_t *A, int32_t kind,
                                  const ecc_matrix_opts_t *opts, ecc_matrix_t *out) {
    try {
        return ecc_matrix_create_impl(plan, A, kind, opts, out);
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
}

ecc_status_t ecc_matrix_destroy(ecc_matrix_t M) {
    if (!M) return ECC_OK;
    if (M->plan) (void)hipStreamSynchronize(M->plan->stream);
    (void)hipFree(M->d_items);
    (void)hipFree(M->d_fixups);
    (void)hipFree(M->d_pieces);
    (void)hipFree(M->d_partials);
    (void)hipFree(M->d_order);
    (void)hipFree(M->d_srow_ptr);
    (void)hipFree(M->d_scol);
    (void)hipFree(M->d_sval);
    (void)hipFree(M->d_sinfo);
    (void)hipFree(M->d_rpart);
    (void)hipFree(M->d_rmask);
    (void)hipFree(M->d_diag);
    (void)hipFree(M->d_rfix);
    (void)hipFree(M->d_ell_col);
    (void)hipFree(M->d_ell_mask);
    (void)hipFree(M->d_ell_val);
    (void)hipFree(M->d_queue);
    (void)hipFree(M->d_cscale);
    (void)hipFree(M->d_zown);
    (void)hipFree(M->d_zhat);
    (void)hipFree(M->d_hot_col);
    (void)hipFree(M->d_hot_rank);
    (void)hipFree(M->d_hot);
    delete M;
    return ECC_OK;
}

ecc_status_t ecc_matrix_layout(ecc_matrix_t M, int32_t *layout, int32_t *row_slots) {
    clear_error();
    ECC_ARG(M != nullptr, "matrix is NULL");
    ECC_ARG(layout != nullptr && row_slots != nullptr, "NULL output");
    *layout = M->layout == kLayShort ? ECC_LAYOUT_SHORT
              : M->layout == kLaySorted ? ECC_LAYOUT_SORTED
              : M->layout == kLayRanges ? ECC_LAYOUT_RANGES
                                      : ECC_LAYOUT_STREAM;
    *row_slots = M->layout == kLayShort    ? short_class(M->short_r)
                 : M->layout == kLayRanges ? M->n_ranges
                                           : 0;
    return ECC_OK;
}

ecc_status_t ecc_matrix_tiling(ecc_matrix_t M, int64_t *plane_rows, int64_t *tile_rows) {
    clear_error();
    ECC_ARG(M != nullptr, "matrix is NULL");
    ECC_ARG(plane_rows != nullptr && tile_rows != nullptr, "NULL output");
    *plane_rows = M->tile_plane;
    *tile_rows = M->tile_rows;
    return ECC_OK;
}

ecc_status_t ecc_matrix_form(ecc_matrix_t M, int32_t *form, int32_t *n_diagonals,
                             int32_t *offsets) {
    clear_error();
    ECC_ARG(M != nullptr, "matrix is NULL");
    ECC_ARG(form != nullptr, "NULL output");
    *form = M->colscale ? ECC_FORM_COLUMN_VALUES : M->dia ? ECC_FORM_DIAGONALS : ECC_FORM_GENERAL;
    if (n_diagonals) *n_diagonals = M->dia ? M->n_dia : 0;
    if (offsets)
        for (int k = 0; k < ECC_MAX_DIAGONALS; ++k)
            offsets[k] = (M->dia && k < M->n_dia) ? M->dia_off.v[k] : 0;
    return ECC_OK;
}

ecc_status_t ecc_matrix_schedule(ecc_matrix_t M, int32_t *schedule) {
    clear_error();
    ECC_ARG(M != nullptr, "matrix is NULL");
    ECC_ARG(schedule != nullptr, "NULL output");
    *schedule = M->tiny ? ECC_SCHEDULE_SINGLE : M->queue ? ECC_SCHEDULE_QUEUE : ECC_SCHEDULE_STATIC;
    return ECC_OK;
}

int64_t ecc_partials_size(ecc_matrix_t M) {
    if (!M) return 0;
    return M->n_part;
}

static ecc_status_t iterate(ecc_plan_t plan, ecc_matrix_t M, int32_t kind, const double *d_b,
                            double alpha, double beta, const double *d_x_own,
                            const double *d_x_hat, double *d_x_next, double *d_partials) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(M != nullptr, "matrix is NULL");
    if (M->plan != plan || M->kind != kind) {
        set_error("matrix was created for another plan or kind");
        return ECC_ERR_STATE;
    }
    const int64_t n = M->A.n_rows;
    ECC_ARG(d_partials != nullptr, "d_partials is NULL");
    ECC_ARG(n == 0 || (d_x_own && d_x_hat && d_x_next), "NULL vector argument");
    ECC_ARG(kind != ECC_KIND_JACOBI || n == 0 || d_b, "d_b is NULL");
    ECC_ARG(n == 0 || (d_x_next != d_x_own && d_x_next != d_x_hat && d_x_next != d_b),
            "d_x_next must not alias an input");
    // x_hat is only read by a plain sweep
    SweepLaunch L;
    L.b = d_b;
    L.alpha = alpha;
    L.beta = beta;
    L.x_own = d_x_own;
    L.x_hat = const_cast<double *>(d_x_hat);
    L.x_next = d_x_next;
    L.partials = d_partials;
    st = launch_sweep(M, L);
    if (st != ECC_OK || M->n_fixups == 0) return st;
    // finish the rows split into pieces (their norm contribution -> partial G)
    Pass2Launch F;
    F.partials = d_partials;
    F.b = d_b;
    F.alpha = alpha;
    F.beta = beta;
    F.x_own = d_x_own;
    F.x_next = d_x_next;
    return launch_pass2(M, F);
}

ecc_status_t ecc_iterate_jacobi(ecc_plan_t plan, ecc_matrix_t A, const double *d_b,
                                const double *d_x_own, const double *d_x_hat, double *d_x_next,
                                double *d_partials) {
    return iterate(plan, A, ECC_KIND_JACOBI, d_b, 0.0, 0.0, d_x_own, d_x_hat, d_x_next,
                   d_partials);
}

ecc_status_t ecc_iterate_spmv(ecc_plan_t plan, ecc_matrix_t W, double alpha, double beta,
                              const double *d_x_own, const double *d_x_hat, double *d_x_next,
                              double *d_partials) {
    return iterate(plan, W, ECC_KIND_POWER, nullptr, alpha, beta, d_x_own, d_x_hat, d_x_next,
                   d_partials);
}

// ---------------------------------------------------------------------------
// The sweep's partial sums without a caller workspace: a static device array
// of ECC_SCRATCH_DOUBLES doubles, one copy on every GPU the library runs on.
// Host code never passes the array's name to a kernel (in host code it is a
// stand-in, not a device address): its device address is looked up once per
// device with hipGetSymbolAddress, with that device current, and kept here.
// ---------------------------------------------------------------------------
namespace {

static __device__ __align__(256) double scratch[ECC_SCRATCH_DOUBLES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double *g_scratch_ptr[kMaxDevices] = {};

// The address of the array on the device that runs `stream`.
ecc_status_t scratch_on(hipStream_t stream, double **out) {
    int dev = 0;
    if (stream) {
        hipDevice_t d = 0;
        ECC_HIP(hipStreamGetDevice(stream, &d));
        dev = (int)d;
    } else {
        ECC_HIP(hipGetDevice(&dev));
    }
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("device %d beyond the %d devices the scratch table holds", dev, kMaxDevices);
        return ECC_ERR_RANGE;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        int cur = 0;
        ECC_HIP(hipGetDevice(&cur));
        if (cur != dev) ECC_HIP(hipSetDevice(dev));
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) ECC_HIP(hipSetDevice(cur));
        if (e != hipSuccess || !p) {
            set_error("hipGetSymbolAddress of the scratch array failed: %s", hipGetErrorString(e));
            return ECC_ERR_DEVICE;
        }
        g_scratch_ptr[dev] = static_cast<double *>(p);
    }
    *out = g_scratch_ptr[dev];
    return ECC_OK;
}

}  // namespace

ecc_status_t ecc_iterate_jacobi_noalloc(ecc_plan_t plan, ecc_matrix_t A, const double *d_b,
                                        const double *d_x_own, const double *d_x_hat,
                                        double *d_x_next, double *d_rho) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(A != nullptr, "matrix is NULL");
    ECC_ARG(d_rho != nullptr, "d_rho is NULL");
    if (A->n_part > ECC_SCRATCH_DOUBLES) {
        set_error("the sweep writes %lld partial sums; the scratch array holds %d",
                  (long long)A->n_part, ECC_SCRATCH_DOUBLES);
        return ECC_ERR_RANGE;
    }
    double *part = nullptr;
    st = scratch_on(plan->stream, &part);
    if (st != ECC_OK) return st;
    // the same kernels as ecc_iterate_jacobi + ecc_residual: every partial
    // is written by the sweep (and its split-row pass), so nothing in the
    // array needs clearing
    st = iterate(plan, A, ECC_KIND_JACOBI, d_b, 0.0, 0.0, d_x_own, d_x_hat, d_x_next, part);
    if (st != ECC_OK) return st;
    TimedLaunch timed(plan, ECC_TIMING_NORM);
    hipLaunchKernelGGL(k_residual, dim3(1), dim3(kNormThreads), 0, plan->stream, part,
                       A->n_part, ECC_NORM_L2, d_rho);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

ecc_status_t ecc_residual(ecc_plan_t plan, const double *d_partials, int64_t n_partials,
                          int32_t norm, double *h_out, double *d_out) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(norm == ECC_NORM_L1 || norm == ECC_NORM_L2, "norm must be 1 or 2");
    ECC_ARG(n_partials >= 1 && d_partials, "need at least one partial");
    ECC_ARG(h_out || d_out, "h_out and d_out are both NULL");
    double *dst = d_out ? d_out : plan->d_scalar;
    {
        TimedLaunch timed(plan, ECC_TIMING_NORM);
        hipLaunchKernelGGL(k_residual, dim3(1), dim3(kNormThreads), 0, plan->stream, d_partials,
                           n_partials, norm, dst);
        ECC_LAUNCH_CHECK();
    }
    if (h_out) {
        ECC_HIP(hipMemcpyAsync(h_out, dst, sizeof(double), hipMemcpyDeviceToHost, plan->stream));
        ECC_HIP(hipStreamSynchronize(plan->stream));
    }
    return ECC_OK;
}

}  // extern "C"
