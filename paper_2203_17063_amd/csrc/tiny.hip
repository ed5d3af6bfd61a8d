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
    const uint8_t *ell_mask;  // diagonal form: the diagonals of each row (no ell_col)
    DiagOffsets dia;
    const double *b;
    double alpha, beta;
    double *x;      // in: x^0; out: the last iterate
    double *x_hat;  // in: the assembled vector of the plan's last clock; out: after the last iteration
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
    int32_t *ctrl_host;  // the same two values in pinned host memory
    int32_t norm;
};

// Rows of a thread: with j = tid mod 256 and q = tid / 256, rows
// j + 256 (RPT q + m), m = 0 .. RPT-1.  The norm adds the rows' shares as
// reduce_values does with 256 threads: thread j adds rows j, j + 256, ...
// eight at a time as a pairwise tree; the RPT rows of one thread here are
// one subtree of such a group of eight (a pair, or a half), which the thread
// sums in registers, so only those subtree sums pass through LDS.  Rows in a
// group of eight that is not complete (the last rows before n) are added one
// by one, through LDS, as reduce_values adds them.
// The entries of a thread's rows (the diagonal entry held apart for Jacobi;
// padding turned into a zero value that gathers a zero), the LDS offsets
// their gathers read, its right-hand sides and its rows' current iterate
// stay in registers.  The iterate has one copy in LDS: the sweep keeps the
// new values in registers, and each thread writes its rows' values over
// the old ones only once every gather of the sweep is done (a barrier).
// The staleness decisions depend only on the arrival flags and the versions
// (Algorithm 1's acceptance test), not on the iterate: thread p decides rank
// p's steps for a chunk of iterations at once, into LDS, and the
// iterations then only read them.  The loop thus issues no global load: no
// wait on the memory counter (which also counts the history stores) stalls
// an iteration.  Two barriers per iteration: between the assembly and the
// gathers, and between the gathers and the new iterate; the norm's waves
// sums are kept per step and finished once per chunk, so only a tolerance
// needs a third barrier (every thread then compares the norm).
constexpr int kTinyMaskBytes = 1024;  // arrival flags staged per chunk
constexpr int kTinyChunkMax = 256;    // iterations per chunk at most

template <int KIND, int R, int RPT>
__global__ __launch_bounds__(kTinyThreads) void k_solve_tiny(TinyArgs a) {
    static_assert(RPT == 2 || RPT == 4, "a thread's rows form a subtree of a group of eight");
    static_assert(RPT * kTinyThreads <= kTinyMaxRows, "rows of a thread beyond the LDS arrays");
    static_assert(kTinyThreads == 4 * kNormThreads, "four row sets per norm thread");
    constexpr int N = kTinyMaxRows;
    constexpr int RO = KIND == ECC_KIND_JACOBI ? R - 1 : R;  // entries summed per row
    static_assert(RPT * RO <= 32, "one bit per entry in a 32-bit mask");
    // [0, N): the iterate; [N, 2N): the assembled vector; [2N]: zero,
    // gathered by padding entries
    __shared__ double s_v[2 * N + 2];
    __shared__ double s_c[N];                    // shares of rows outside complete groups
    __shared__ double s_h[4][kNormThreads];      // subtree sums of complete groups, [q][j]
    __shared__ uint8_t s_item[N];                // the work item of each row
    __shared__ uint8_t s_mask[kTinyMaskBytes];   // arrival flags of a chunk, [u][p]
    __shared__ uint8_t s_eff[kTinyMaskBytes];    // its decisions: bit 0 taken, bit 1 forced
    __shared__ int32_t s_nv[kTinyMaskBytes];     // the versions after each of its steps
    __shared__ double s_sum[kTinyChunkMax][kNormThreads / 64];  // waves' norm sums per step
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int jn = tid & (kNormThreads - 1), qn = tid / kNormThreads;
    const int32_t n = a.n, P = a.P, NI = a.n_items;
    for (int32_t i = tid; i < n; i += kTinyThreads) {
        s_v[i] = a.x[i];
        s_v[N + i] = a.x_hat[i];  // the assembled vector of the plan's last clock
    }
    if (tid == 0) s_v[2 * N] = 0.0;
    for (int32_t q = tid; q < NI * kSweepThreads; q += kTinyThreads) {
        const int32_t w = q / kSweepThreads, l = q % kSweepThreads;
        const WorkItem it = a.items[w];
        if (l < it.nrows) s_item[it.row0 + l] = (uint8_t)w;
    }
    // rank tid's version (its state between the decisions of two chunks)
    int32_t ver = tid < P ? a.version[(a.t0 & 1) * P + tid] : 0;
    __syncthreads();
    // row m of this thread is row0 + 256 m; rank of row m in bits 16 (m & 1)
    // of rkp[m / 2] (ranks < 1024)
    const int32_t row0 = jn + kNormThreads * RPT * qn;
    uint32_t rkp[RPT / 2] = {};
    int32_t ad[RPT][RO];  // byte offset in s_v of each gather
    double val[RPT][RO];
    double dg[RPT], bi[RPT], xr[RPT];
#pragma unroll
    for (int m = 0; m < RPT; ++m) {
        const int32_t i = row0 + kNormThreads * m;
        dg[m] = bi[m] = xr[m] = 0.0;
        int32_t c8[R];
        double v8[R];
        int32_t lo = 0, hi = 0;
#pragma unroll
        for (int e = 0; e < R; ++e) {
            c8[e] = -1;
            v8[e] = 0.0;
        }
        if (i < n) {
            const WorkItem it = a.items[s_item[i]];
            const int32_t l = i - it.row0;
            const int64_t base = (int64_t)it.k0 * R + l;
            const int32_t pad = sell_pad(it.nrows);
            const uint32_t mk = a.ell_mask ? a.ell_mask[(int64_t)it.k0 + l] : 0u;
#pragma unroll
            for (int e = 0; e < R; ++e) {
                c8[e] = a.ell_mask ? (((mk >> e) & 1u) ? i + a.dia.v[e] : -1)
                                   : a.ell_col[base + (int64_t)e * pad];
                v8[e] = a.ell_val[base + (int64_t)e * pad];
            }
            lo = it.lo;
            hi = it.hi;
            rkp[m / 2] |= (uint32_t)it.rank << (16 * (m & 1));
            if (KIND == ECC_KIND_JACOBI) bi[m] = a.b[i];
            xr[m] = s_v[i];
        }
        int dpos = R;  // Jacobi: the diagonal entry, summed apart
        if constexpr (KIND == ECC_KIND_JACOBI) {
#pragma unroll
            for (int e = R - 1; e >= 0; --e)
                if (c8[e] == i) dpos = e;
#pragma unroll
            for (int e = 0; e < R; ++e)
                if (e == dpos) dg[m] = v8[e];
        }
#pragma unroll
        for (int o = 0; o < RO; ++o) {
            // the others in CSR order (selects with fixed indices keep the
            // arrays in registers)
            const int32_t c = (KIND == ECC_KIND_JACOBI && o >= dpos) ? c8[o + 1] : c8[o];
            const double v = (KIND == ECC_KIND_JACOBI && o >= dpos) ? v8[o + 1] : v8[o];
            const bool in_own = c >= lo && c < hi;
            // padding: value 0 times the zero slot adds +0 to a sum that
            // is never -0 (it starts at +0, and only -0 + -0 gives -0), so
            // it leaves the sum unchanged, as if the entry were skipped
            val[m][o] = c >= 0 ? v : 0.0;
            ad[m][o] = 8 * (c < 0 ? 2 * N : in_own ? c : N + c);
        }
    }
    // the group of eight of this thread's rows, and whether it is complete
    // (its eight values, the zero partial at index n included, all exist)
    const int32_t grp = (RPT * qn) / 8;
    const bool complete = jn + 8 * kNormThreads * grp + 7 * kNormThreads <= n;
    const char *sb = reinterpret_cast<const char *>(s_v);
    int32_t iters = 0, stopped = 0;
    unsigned forced = 0;
    const int32_t chunk = min(kTinyChunkMax, max(1, kTinyMaskBytes / max(P, 1)));

    // The norm of step u of the chunk from its waves' sums.
    auto norm_of = [&](int32_t u) -> double {
        double sum = s_sum[u][0];
        for (int w = 1; w < kNormThreads / 64; ++w) sum += s_sum[u][w];
        return (a.norm == ECC_NORM_L2) ? sqrt(sum) : sum;
    };

    // One iteration: the assembly of the taken ranks' rows, the sweep, the
    // new iterate over the old one, the norm.  Returns whether the tolerance
    // stops the loop.
    auto iteration = [&](int32_t u) -> bool {
        const uint8_t *ef = s_eff + u * P;
#pragma unroll
        for (int m = 0; m < RPT; ++m) {
            const int32_t i = row0 + kNormThreads * m;
            const uint32_t r = (rkp[m / 2] >> (16 * (m & 1))) & 0xffffu;
            if (i < n && (ef[r] & 1)) s_v[N + i] = xr[m];
        }
        lds_barrier();
        // every row's gathers first, so that the rows' arithmetic chains
        // overlap
        double y[RPT][RO];
#pragma unroll
        for (int m = 0; m < RPT; ++m)
#pragma unroll
            for (int o = 0; o < RO; ++o)
                y[m][o] = *reinterpret_cast<const double *>(sb + ad[m][o]);
        double sh[RPT];
#pragma unroll
        for (int m = 0; m < RPT; ++m) {
            double sum = 0.0;
#pragma unroll
            for (int o = 0; o < RO; ++o) sum = sum + val[m][o] * y[m][o];
            double xnew, share;
            if constexpr (KIND == ECC_KIND_JACOBI) {
                const double bs = bi[m] - sum;
                xnew = bs / dg[m];
                const double r = bs - dg[m] * xr[m];
                share = r * r;
            } else {
                xnew = a.alpha * sum + a.beta;
                share = fabs(xnew - xr[m]);
            }
            xr[m] = xnew;
            sh[m] = row0 + kNormThreads * m < n ? share : 0.0;  // index n: the zero partial
        }
        if (complete) {
            double h;
            if constexpr (RPT == 4) h = (sh[0] + sh[1]) + (sh[2] + sh[3]);
            else h = sh[0] + sh[1];
            s_h[qn][jn] = h;
        } else {
#pragma unroll
            for (int m = 0; m < RPT; ++m)
                if (row0 + kNormThreads * m < n) s_c[row0 + kNormThreads * m] = sh[m];
        }
        lds_barrier();
        // every gather of the sweep is done: the new iterate replaces the old
        // (rows past n write into the unread tail of the array)
#pragma unroll
        for (int m = 0; m < RPT; ++m) s_v[row0 + kNormThreads * m] = xr[m];
        // the norm in reduce_values' order: each complete group of eight as
        // its tree, then the remaining values one by one
        if (tid < kNormThreads) {
            double acc = 0.0;
            int32_t k = tid;
            for (int g = 0; g < RPT / 2 && k + 7 * kNormThreads <= n;
                 ++g, k += 8 * kNormThreads) {
                if constexpr (RPT == 4) acc += s_h[2 * g][tid] + s_h[2 * g + 1][tid];
                else acc += (s_h[0][tid] + s_h[1][tid]) + (s_h[2][tid] + s_h[3][tid]);
            }
            for (; k <= n; k += kNormThreads) acc += k < n ? s_c[k] : 0.0;
            acc = wave_sum_lane63(acc);
            if (lane == 63) s_sum[u][wave] = acc;
        }
        // Without a tolerance nothing here needs the norm: the next step's
        // first barrier orders these reads of s_h and s_c before their next
        // writes, and the norms of the chunk are finished after it.
        if (a.tol > 0.0) {
            lds_barrier();
            return norm_of(u) < a.tol;
        }
        return false;
    };

    for (int32_t tc = 0; tc < a.T && !stopped; tc += chunk) {
        const int32_t cn = min(chunk, a.T - tc);
        __syncthreads();  // the previous chunk's decisions are no longer read
        for (int32_t q = tid; q < cn * P; q += kTinyThreads)
            s_mask[q] = a.mask[(int64_t)tc * P + q];
        __syncthreads();
        if (tid < P) {
            // rank tid's decisions at the chunk's steps, in order: taken if
            // fresh, never taken, or too stale (as record_step)
            for (int32_t u0 = 0; u0 < cn; u0 += 8) {
                uint8_t ar[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) ar[k] = u0 + k < cn ? s_mask[(u0 + k) * P + tid] : 0;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    if (u0 + k < cn) {
                        const int64_t tt = a.t0 + tc + u0 + k;
                        const bool e = stale_select(ver, ar[k], tt, a.S);
                        const bool f = e && ar[k] == 0 && ver >= 0;
                        ver = e ? (int32_t)tt : ver;
                        s_eff[(u0 + k) * P + tid] = (uint8_t)((e ? 1 : 0) | (f ? 2 : 0));
                        s_nv[(u0 + k) * P + tid] = ver;
                    }
                }
            }
        }
        __syncthreads();
        int32_t u = 0;
        bool stop = false;
        while (!stop && u < cn) {
            stop = iteration(u);
            ++u;
        }
        __syncthreads();  // the chunk's norm sums are in
        for (int32_t k = tid; k < u; k += kTinyThreads) a.rho[tc + k] = norm_of(k);
        // the histories and forced arrivals of the iterations run
        if (tid < P) {
            for (int32_t k = 0; k < u; ++k) {
                const uint8_t e = s_eff[k * P + tid];
                const int64_t tt = a.t0 + tc + k;
                if (a.eff_hist) a.eff_hist[(int64_t)(tc + k) * P + tid] = e & 1;
                if (a.age_hist) a.age_hist[(int64_t)(tc + k) * P + tid] =
                    (int32_t)(tt - s_nv[k * P + tid]);
                forced += (e >> 1) & 1;
            }
            if (u < cn) ver = s_nv[(u - 1) * P + tid];  // stopped: the last step run
        }
        iters += u;
        if (stop) stopped = 1;
    }
    // state after the last iteration: the iterate, the assembled vector, the
    // plan's versions (half (t0 + iters) & 1), ages, decisions, forced count
    __syncthreads();
#pragma unroll
    for (int m = 0; m < RPT; ++m)
        if (row0 + kNormThreads * m < n) a.x[row0 + kNormThreads * m] = xr[m];
    for (int32_t i = tid; i < n; i += kTinyThreads) a.x_hat[i] = s_v[N + i];
    if (iters > 0 && tid < P) {
        const int64_t tl = a.t0 + iters - 1;
        a.version[((a.t0 + iters) & 1) * P + tid] = ver;
        a.age_state[tid] = (int32_t)(tl - ver);
        a.eff_state[tid] = ver == (int32_t)tl ? 1 : 0;
    }
    // the forced arrivals, added in rank order (one thread: P <= kTinyMaxP)
    __shared__ unsigned s_forced[kTinyMaxP];
    if (tid < P) s_forced[tid] = forced;
    __syncthreads();
    if (tid == 0) {
        unsigned long long total = 0;
        for (int32_t p = 0; p < P; ++p) total += s_forced[p];
        *a.forced = *a.forced + total;
        a.ctrl[0] = stopped;
        a.ctrl[1] = iters;
        a.ctrl_host[0] = stopped;
        a.ctrl_host[1] = iters;
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
    a.ell_mask = M->dia ? M->d_ell_mask : nullptr;
    a.dia = M->dia_off;
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
    a.ctrl_host = pl->h_ctrl;
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
