// Single-launch solve of a small block-row problem: the loop control of
// ecc_solve (staleness decision + assembly -> sweep -> norm -> swap, T times
// or until the norm is below the tolerance) run by one workgroup of
// kTinyThreads, with the iterate, the next iterate and the assembled vector
// held in LDS.  For a short-row matrix of at most kTinyMaxRows rows a loop of
// launches is bound by launch latency (on MI355X, the tridiagonal n = 4,096
// Jacobi loop: about 6 us per launch for 0.3 MB of data); here an iteration
// costs a few barriers.
//
// The arithmetic is that of the launch-per-iteration path bit for bit:
//  - the staleness decision and bookkeeping as record_step;
//  - every row is summed by one thread in CSR order (its entries read once
//    from the item-major copy and kept in registers);
//  - the norm reduces the rows' shares (r_i^2 or |dx_i|) as reduce_values
//    does,
// so iterates, norms, eff/age histories and the plan state equal those of
// ecc_iterate_* + ecc_residual over the same matrix (whose sweeps write one
// partial per row).
#include "ecc_common.h"

namespace ecc {

// Workgroup barrier for data exchanged through LDS only: waits for this
// wave's LDS operations, not for its global loads and stores (which
// __syncthreads' fence would drain at every barrier: the arrival flags
// prefetched for the next iteration, the norms and histories written).  The
// memory clobber keeps the compiler from moving accesses across it.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

struct TinyArgs {
    const WorkItem *items;
    int32_t n_items;
    int32_t n;
    const int32_t *ell_col;
    const double *ell_val;
    const double *b;
    double alpha, beta;
    double *x;      // in: x^0; out: the last iterate
    double *x_hat;  // out: the assembled vector after the last iteration
    const uint8_t *mask;
    int32_t T;
    double tol;
    double *rho;
    uint8_t *eff_hist;
    int32_t *age_hist;
    int32_t P, S;
    int64_t t0;
    int32_t *version;  // the plan's [2][P] versions (read half t0 & 1)
    int32_t *age_state;
    uint8_t *eff_state;
    unsigned long long *forced;
    int32_t *ctrl;     // ctrl[0] := 1 when stopped by the tolerance, ctrl[1] := iterations
    int32_t norm;
};

// RPT rows per thread: thread tid sweeps rows tid, tid + kTinyThreads, ...,
// with their entries in registers (4 rows of 3 entries, or 2 of up to 8,
// fit the 128 VGPRs of a 1,024-thread workgroup without spilling).

template <int KIND, int R, int RPT>
__global__ __launch_bounds__(kTinyThreads) void k_solve_tiny(TinyArgs a) {
    static_assert(RPT * kTinyThreads <= kTinyMaxRows, "rows of a thread beyond the LDS arrays");
    // [0], [1]: the iterate and the next one (in turn); [2]: the assembled vector
    __shared__ double s_v[3][kTinyMaxRows];
    __shared__ double s_c[kTinyMaxRows];        // each row's norm contribution
    __shared__ uint8_t s_item[kTinyMaxRows];    // the work item of each row
    __shared__ int32_t s_ver[2][kTinyMaxP];     // versions before / after a step
    __shared__ double s_red[kNormThreads / 64];
    __shared__ unsigned s_forced;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int32_t n = a.n, P = a.P, NI = a.n_items;
    for (int32_t i = tid; i < n; i += kTinyThreads) s_v[0][i] = a.x[i];
    const int32_t *ver_in = a.version + (a.t0 & 1) * P;
    for (int32_t p = tid; p < P; p += kTinyThreads) s_ver[0][p] = ver_in[p];
    for (int32_t q = tid; q < NI * kSweepThreads; q += kTinyThreads) {
        const int32_t w = q / kSweepThreads, l = q % kSweepThreads;
        const WorkItem it = a.items[w];
        if (l < it.nrows) s_item[it.row0 + l] = (uint8_t)w;
    }
    if (tid == 0) s_forced = 0;
    __syncthreads();
    // this thread's rows: entries, right-hand side, rank block, held in
    // registers for the whole solve (the item-major copy, read once)
    int32_t col[RPT][R];
    double val[RPT][R];
    double bi[RPT];
    int32_t blk[RPT], rk[RPT];  // rank block [lo, hi) packed as lo | hi << 16 (n <= 4096)
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
        const int32_t i = tid + k * kTinyThreads;
        blk[k] = rk[k] = 0;
        bi[k] = 0.0;
#pragma unroll
        for (int j = 0; j < R; ++j) {
            col[k][j] = -1;
            val[k][j] = 0.0;
        }
        if (i < n) {
            const WorkItem it = a.items[s_item[i]];
            const int32_t l = i - it.row0;
            const int64_t base = (int64_t)it.k0 * R + l;
            const int32_t pad = sell_pad(it.nrows);
#pragma unroll
            for (int j = 0; j < R; ++j) {
                col[k][j] = a.ell_col[base + (int64_t)j * pad];
                val[k][j] = a.ell_val[base + (int64_t)j * pad];
            }
            blk[k] = it.lo | (it.hi << 16);
            rk[k] = it.rank;
            if (KIND == ECC_KIND_JACOBI) bi[k] = a.b[i];
        }
    }
    int cur = 0, iters = 0, stopped = 0;
    unsigned forced = 0;
    // arrival flags, loaded one iteration ahead: of rank tid (its official
    // decision) and of this thread's rows' ranks (their assembly)
    uint8_t ar_p = (tid < P && a.T > 0) ? a.mask[tid] : 0;
    uint8_t ar_r[RPT];
#pragma unroll
    for (int k = 0; k < RPT; ++k) ar_r[k] = a.T > 0 ? a.mask[rk[k]] : 0;
    for (int32_t t = 0; t < a.T; ++t) {
        const int64_t tt = a.t0 + t;
        const int vb = t & 1;
        const uint8_t arp = ar_p;
        uint8_t arr[RPT];
#pragma unroll
        for (int k = 0; k < RPT; ++k) arr[k] = ar_r[k];
        if (t + 1 < a.T) {
            const uint8_t *mn = a.mask + (int64_t)(t + 1) * P;
            if (tid < P) ar_p = mn[tid];
#pragma unroll
            for (int k = 0; k < RPT; ++k) ar_r[k] = mn[rk[k]];
        }
        // staleness decision of rank tid (P <= kTinyThreads): the plan's
        // bookkeeping; every thread also decides its own rows' ranks from the
        // same versions (the same result) and assembles those rows
        if (tid < P) {
            const int32_t v = s_ver[vb][tid];
            const bool e = stale_select(v, arp, tt, a.S);
            if (e && arp == 0 && v >= 0) ++forced;
            const int32_t nv = e ? (int32_t)tt : v;
            s_ver[vb ^ 1][tid] = nv;
            if (a.eff_hist) a.eff_hist[(int64_t)t * P + tid] = e ? 1 : 0;
            if (a.age_hist) a.age_hist[(int64_t)t * P + tid] = (int32_t)(tt - nv);
        }
        const double *xo = s_v[cur];
        double *xn = s_v[cur ^ 1];
        double *xh = s_v[2];
#pragma unroll
        for (int k = 0; k < RPT; ++k) {
            const int32_t i = tid + k * kTinyThreads;
            if (i < n && stale_select(s_ver[vb][rk[k]], arr[k], tt, a.S)) xh[i] = xo[i];
        }
        lds_barrier();
        // sweep: one thread per row, entries in CSR order, without branches
        // (padding gathers entry 0 and is not added); every row's gathers
        // first, so that the rows' arithmetic chains overlap
        double y[RPT][R], xoi[RPT];
#pragma unroll
        for (int k = 0; k < RPT; ++k) {
            const int32_t i = tid + k * kTinyThreads;
#pragma unroll
            for (int j = 0; j < R; ++j) {
                const int32_t cj = col[k][j];
                const int32_t c = cj >= 0 ? cj : 0;
                const bool own = cj >= (blk[k] & 0xffff) && cj < (blk[k] >> 16);
                y[k][j] = s_v[own ? cur : 2][c];  // one load: the view's source by index
            }
            xoi[k] = xo[i];
        }
#pragma unroll
        for (int k = 0; k < RPT; ++k) {
            const int32_t i = tid + k * kTinyThreads;
            double s = 0.0, dg = 0.0;
#pragma unroll
            for (int j = 0; j < R; ++j) {
                const int32_t cj = col[k][j];
                const bool diag = KIND == ECC_KIND_JACOBI && cj == i;
                if (diag) dg = val[k][j];
                const double sn = s + val[k][j] * y[k][j];
                s = (cj >= 0 && !diag) ? sn : s;
            }
            // rows past n (up to RPT x kTinyThreads <= kTinyMaxRows) compute
            // into the unread tail of the LDS arrays: no branch per row
            s_c[i] = row_finish<KIND>(i, s, dg, bi[k], xoi[k], a.alpha, a.beta, xn);
        }
        lds_barrier();
        // the norm: the rows' shares and a last, zero, partial reduced in
        // reduce_values' order (thread j takes rows j, j + 256, ..., groups of
        // eight as pairwise trees, then the waves' sums in order)
        if (tid < kNormThreads) {
            double acc = 0.0;
            int32_t k = tid;
            for (; k + 7 * kNormThreads <= n; k += 8 * kNormThreads) {
                double t8[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int32_t q = k + j * kNormThreads;
                    t8[j] = q < n ? s_c[q] : 0.0;
                }
                acc += tree8(t8);
            }
            for (; k <= n; k += kNormThreads) acc += k < n ? s_c[k] : 0.0;
            acc = wave_sum_lane63(acc);
            if (lane == 63) s_red[wave] = acc;
        }
        lds_barrier();
        double sum = s_red[0];
        for (int w = 1; w < kNormThreads / 64; ++w) sum += s_red[w];
        const double v = (a.norm == ECC_NORM_L2) ? sqrt(sum) : sum;
        if (tid == 0) a.rho[t] = v;
        cur ^= 1;
        ++iters;
        if (a.tol > 0.0 && v < a.tol) {
            stopped = 1;
            break;
        }
    }
    // state after the last iteration: the iterate, the assembled vector, the
    // plan's versions (half (t0 + iters) & 1), ages, decisions, forced count
    if (forced) atomicAdd(&s_forced, forced);
    __syncthreads();
    for (int32_t i = tid; i < n; i += kTinyThreads) {
        a.x[i] = s_v[cur][i];
        a.x_hat[i] = s_v[2][i];
    }
    if (iters > 0) {
        int32_t *ver_out = a.version + ((a.t0 + iters) & 1) * P;
        const int64_t tl = a.t0 + iters - 1;
        const int vb = iters & 1;
        for (int32_t p = tid; p < P; p += kTinyThreads) {
            const int32_t nv = s_ver[vb][p];
            ver_out[p] = nv;
            a.age_state[p] = (int32_t)(tl - nv);
            a.eff_state[p] = nv == (int32_t)tl ? 1 : 0;
        }
    }
    if (tid == 0) {
        *a.forced = *a.forced + s_forced;
        a.ctrl[0] = stopped;
        a.ctrl[1] = iters;
    }
}

ecc_status_t launch_solve_tiny(ecc_matrix_t M, const double *d_b, double alpha, double beta,
                               double *d_x, double *d_x_hat, const uint8_t *d_mask, int32_t T,
                               double tol, double *d_rho, uint8_t *d_eff_hist,
                               int32_t *d_age_hist) {
    ecc_plan_t pl = M->plan;
    TinyArgs a{};
    a.items = M->d_items;
    a.n_items = (int32_t)M->n_items;
    a.n = (int32_t)M->A.n_rows;
    a.ell_col = M->d_ell_col;
    a.ell_val = M->d_ell_val;
    a.b = d_b;
    a.alpha = alpha;
    a.beta = beta;
    a.x = d_x;
    a.x_hat = d_x_hat;
    a.mask = d_mask;
    a.T = T;
    a.tol = tol;
    a.rho = d_rho;
    a.eff_hist = d_eff_hist;
    a.age_hist = d_age_hist;
    a.P = pl->P;
    a.S = pl->S;
    a.t0 = pl->clock;
    a.version = pl->d_version;
    a.age_state = pl->d_age;
    a.eff_state = pl->d_eff;
    a.forced = pl->d_forced;
    a.ctrl = pl->d_ctrl;
    a.norm = M->kind == ECC_KIND_JACOBI ? ECC_NORM_L2 : ECC_NORM_L1;
    if (!tiny_fits(a.n, M->short_r, M->n_items, a.P) || M->layout != kLayShort) {
        set_error("internal: the single-launch solve does not fit the matrix");
        return ECC_ERR_STATE;
    }
    TimedLaunch timed(pl, ECC_TIMING_SWEEP);
    const dim3 grid(1), block(kTinyThreads);
    hipStream_t st = pl->stream;
#define ECC_TINY(K, RR, RP) hipLaunchKernelGGL((k_solve_tiny<K, RR, RP>), grid, block, 0, st, a)
#define ECC_TINY_KIND(K)                                  \
    if (a.n > 2 * kTinyThreads) {                         \
        ECC_TINY(K, 3, 4);                                \
    } else {                                              \
        switch (R) {                                      \
            case 3: ECC_TINY(K, 3, 2); break;             \
            case 4: ECC_TINY(K, 4, 2); break;             \
            case 5: ECC_TINY(K, 5, 2); break;             \
            case 7: ECC_TINY(K, 7, 2); break;             \
            default: ECC_TINY(K, 8, 2); break;            \
        }                                                 \
    }
    const int32_t R = M->short_r <= 3 ? 3 : M->short_r == 4 ? 4 : M->short_r == 5 ? 5
                      : M->short_r <= 7 ? 7 : 8;
    if (M->kind == ECC_KIND_JACOBI) {
        ECC_TINY_KIND(ECC_KIND_JACOBI)
    } else {
        ECC_TINY_KIND(ECC_KIND_POWER)
    }
#undef ECC_TINY_KIND
#undef ECC_TINY
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

}  // namespace ecc
