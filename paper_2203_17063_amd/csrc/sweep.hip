// Block-row sweeps over a CSR matrix that consume the assembled vector:
// Jacobi (x_next_i = (b_i - sum_{j != i} a_ij y_j) / a_ii) and the PageRank
// power step (x_next_j = alpha sum_i w_ji y_i + beta), where row i of rank
// block [lo, hi) reads y_j = x_own[j] inside its own block and x_hat[j]
// elsewhere, plus the residual-norm reduction.
//
// Work decomposition (built once per matrix on the host, CSR-Adaptive style
// after Greathouse & Daga, SC'14): a "stream" item is a run of short rows of
// one rank whose nonzeros fit in LDS -- they are loaded with coalesced
// accesses and each row is then summed by 1..64 lanes; a "vector" item is one
// long row summed by the whole workgroup; a "piece" is a fixed-size slice of
// a very long row whose partial sum is recombined, in piece order, by the
// second pass.  Items never straddle a rank boundary, so [lo, hi) is uniform
// per item.  Rows summed by a single lane accumulate in CSR order with no
// fused multiply-add, exactly like the sequential definition.
#include <algorithm>
#include <vector>

#include "ecc_common.h"

namespace ecc {

constexpr int kMaxSweepBlocks = 8192;

// Row epilogue; returns the row's contribution to the norm (r_i^2 for Jacobi,
// |x_next_j - x_own_j| for the power step).
template <int KIND>
__device__ __forceinline__ double row_finish(int32_t i, double s, double dg,
                                             const double *__restrict__ b, double alpha,
                                             double beta, const double *__restrict__ x_own,
                                             double *__restrict__ x_next) {
    if constexpr (KIND == ECC_KIND_JACOBI) {
        const double bs = b[i] - s;
        const double xn = bs / dg;
        x_next[i] = xn;
        const double r = bs - dg * x_own[i];
        return r * r;
    } else {
        const double xn = alpha * s + beta;
        x_next[i] = xn;
        return fabs(xn - x_own[i]);
    }
}

// Accumulate entries [k_begin, k_end) of row i with stride `step` starting at
// `first`, reading (col, val) through the given accessors.
template <int KIND>
__device__ __forceinline__ void row_accumulate_global(
    int32_t i, int32_t first, int32_t k_end, int32_t step, const int32_t *__restrict__ col,
    const double *__restrict__ val, int32_t lo, int32_t hi, const double *__restrict__ x_own,
    const double *__restrict__ x_hat, double &s, double &dg) {
    int32_t k = first;
    // four independent loads in flight per lane
    for (; k + 3 * step < k_end; k += 4 * step) {
        int32_t c[4];
        double v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            c[u] = col[k + u * step];
            v[u] = val[k + u * step];
        }
        double y[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const double *src = (c[u] >= lo && c[u] < hi) ? x_own : x_hat;
            y[u] = src[c[u]];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (KIND == ECC_KIND_JACOBI && c[u] == i) {
                dg = v[u];
            } else {
                s = s + v[u] * y[u];
            }
        }
    }
    for (; k < k_end; k += step) {
        const int32_t c = col[k];
        const double v = val[k];
        if (KIND == ECC_KIND_JACOBI && c == i) {
            dg = v;
            continue;
        }
        const double *src = (c >= lo && c < hi) ? x_own : x_hat;
        s = s + v * src[c];
    }
}

template <int KIND>
__global__ __launch_bounds__(kSweepThreads) void k_sweep(
    const WorkItem *__restrict__ items, int32_t n_items, const int32_t *__restrict__ row_ptr,
    const int32_t *__restrict__ col, const double *__restrict__ val,
    const int32_t *__restrict__ block_start, const double *__restrict__ b, double alpha,
    double beta, const double *__restrict__ x_own, const double *__restrict__ x_hat,
    double *__restrict__ x_next, double *__restrict__ partials, double2 *__restrict__ pieces,
    int32_t zero_extra, const int32_t *__restrict__ done) {
    __shared__ int32_t s_col[kStreamCap];
    __shared__ double s_val[kStreamCap];
    __shared__ double s_red[kSweepThreads / 64];
    if (done && *done) return;
    const int tid = threadIdx.x;
    double contrib = 0.0;

    for (int32_t w = blockIdx.x; w < n_items; w += gridDim.x) {
        const WorkItem it = items[w];
        const int kind = it.kind_rank >> 24;
        const int32_t p = it.kind_rank & 0xffffff;
        const int32_t lo = block_start[p], hi = block_start[p + 1];

        if (kind == kItemStream) {
            const int32_t r0 = it.row0, nr = it.a;
            const int32_t k0 = row_ptr[r0], k1 = row_ptr[r0 + nr];
            for (int32_t k = k0 + tid; k < k1; k += kSweepThreads) {
                s_col[k - k0] = col[k];
                s_val[k - k0] = val[k];
            }
            __syncthreads();
            // lanes per row: short rows (<= 16 nonzeros on average) are summed by
            // one lane in CSR order; longer ones by up to 64 lanes, keeping at
            // least 4 nonzeros per lane
            const int32_t nnz_item = k1 - k0;
            int tpr = 1;
            if (nnz_item > 16 * nr)
                while (tpr < 64 && tpr * 2 * nr <= kSweepThreads && nnz_item >= 8 * tpr * nr)
                    tpr *= 2;
            const int lane = tid & (tpr - 1);
            const int32_t rr = tid / tpr;
            if (rr < nr) {
                const int32_t i = r0 + rr;
                const int32_t rs = row_ptr[i] - k0, re = row_ptr[i + 1] - k0;
                double s = 0.0, dg = 0.0;
                for (int32_t k = rs + lane; k < re; k += tpr) {
                    const int32_t c = s_col[k];
                    const double v = s_val[k];
                    if (KIND == ECC_KIND_JACOBI && c == i) {
                        dg = v;
                        continue;
                    }
                    const double *src = (c >= lo && c < hi) ? x_own : x_hat;
                    s = s + v * src[c];
                }
                if (tpr > 1) {
                    s = group_sum_dyn(s, tpr);
                    if (KIND == ECC_KIND_JACOBI) dg = group_sum_dyn(dg, tpr);
                }
                if (lane == 0) contrib += row_finish<KIND>(i, s, dg, b, alpha, beta, x_own, x_next);
            }
            __syncthreads();  // LDS is reused by the next item
        } else {
            const int32_t i = it.row0;
            int32_t ks = row_ptr[i], ke = row_ptr[i + 1];
            if (kind == kItemPiece) {
                ks = ks + it.a * kVectorCap;
                ke = min(ke, ks + kVectorCap);
            }
            double s = 0.0, dg = 0.0;
            row_accumulate_global<KIND>(i, ks + tid, ke, kSweepThreads, col, val, lo, hi, x_own,
                                        x_hat, s, dg);
            s = block_sum<kSweepThreads>(s, s_red);
            if (KIND == ECC_KIND_JACOBI) dg = block_sum<kSweepThreads>(dg, s_red);
            if (tid == 0) {
                if (kind == kItemPiece)
                    pieces[it.b] = make_double2(s, dg);
                else
                    contrib += row_finish<KIND>(i, s, dg, b, alpha, beta, x_own, x_next);
            }
        }
    }
    const double total = block_sum<kSweepThreads>(contrib, s_red);
    if (tid == 0) partials[blockIdx.x] = total;
    // no split rows: the extra partial (split-row contributions) is zero
    if (zero_extra && blockIdx.x == 0 && tid == 0) partials[gridDim.x] = 0.0;
}

// Second pass, one workgroup.  (1) Rows split into pieces are finished: their
// piece sums are added in piece order, the row epilogue runs, and the
// contributions go to partials[n_main].  (2) If `norm` is non-zero, the
// n_main + 1 partials are reduced in a fixed order to sqrt(sum) (L2) or sum
// (L1), written to *out; with a control block, ctrl[1] := t + 1 and
// ctrl[0] := 1 once the norm is below tol.
template <int KIND>
__global__ __launch_bounds__(kPass2Threads) void k_pass2(
    double *__restrict__ partials, int64_t n_main, int32_t do_fixups,
    const Fixup *__restrict__ fixups, int32_t n_fixups, const double2 *__restrict__ pieces,
    const double *__restrict__ b,
    double alpha, double beta, const double *__restrict__ x_own, double *__restrict__ x_next,
    int32_t norm, double *__restrict__ out, double tol, int32_t *__restrict__ ctrl, int32_t t,
    const int32_t *__restrict__ done) {
    __shared__ double s_red[kPass2Threads / 64];
    if (done && *done) return;
    const int tid = threadIdx.x;
    if (do_fixups) {
        double acc = 0.0;
        for (int32_t f = tid; f < n_fixups; f += kPass2Threads) {
            const Fixup fx = fixups[f];
            double s = 0.0, dg = 0.0;
            for (int32_t j = 0; j < fx.npieces; ++j) {
                const double2 pc = pieces[fx.slot0 + j];
                s = s + pc.x;
                dg = dg + pc.y;
            }
            acc += row_finish<KIND>(fx.row, s, dg, b, alpha, beta, x_own, x_next);
        }
        const double tot = block_sum<kPass2Threads>(acc, s_red);
        if (tid == 0) partials[n_main] = tot;
        __syncthreads();
        __threadfence_block();
    }
    if (norm == 0) return;
    const int64_t n = n_main + 1;
    double acc = 0.0;
    for (int64_t k = tid; k < n; k += kPass2Threads) acc += partials[k];
    const double tot = block_sum<kPass2Threads>(acc, s_red);
    if (tid == 0) {
        const double v = (norm == ECC_NORM_L2) ? sqrt(tot) : tot;
        if (out) *out = v;
        if (ctrl) {
            ctrl[1] = t + 1;
            if (tol > 0.0 && v < tol) ctrl[0] = 1;
        }
    }
}

// Structural check of a matrix for a plan: counts rows whose diagonal entry is
// missing, duplicated or zero (Jacobi only) and entries whose column is out of
// range.  bad[0] = bad rows, bad[1] = bad columns.
__global__ void k_check(int32_t n_rows, int32_t n_cols, const int32_t *__restrict__ row_ptr,
                        const int32_t *__restrict__ col, const double *__restrict__ val,
                        int32_t check_diag, unsigned long long *__restrict__ bad) {
    unsigned long long bad_rows = 0, bad_cols = 0;
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n_rows;
         i += gridDim.x * blockDim.x) {
        int ndiag = 0;
        bool zero = false;
        for (int32_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k) {
            const int32_t c = col[k];
            if (c < 0 || c >= n_cols) ++bad_cols;
            if (c == i) {
                ++ndiag;
                zero = zero || (val[k] == 0.0);
            }
        }
        if (check_diag && (ndiag != 1 || zero)) ++bad_rows;
    }
    if (bad_rows) atomicAdd(&bad[0], bad_rows);
    if (bad_cols) atomicAdd(&bad[1], bad_cols);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

static void build_items(const std::vector<int32_t> &rp, const std::vector<int64_t> &counts,
                        std::vector<WorkItem> &items, std::vector<Fixup> &fixups,
                        int64_t &n_pieces) {
    std::vector<WorkItem> big, vec, stream;
    n_pieces = 0;
    int64_t row = 0;
    for (size_t p = 0; p < counts.size(); ++p) {
        const int64_t hi = row + counts[p];
        int64_t i = row;
        while (i < hi) {
            const int64_t len = (int64_t)rp[i + 1] - rp[i];
            if (len > kStreamCap) {
                if (len <= kVectorCap) {
                    vec.push_back({(int32_t)i, 1, 0, (int32_t)((kItemVector << 24) | (int32_t)p)});
                } else {
                    const int32_t np = (int32_t)((len + kVectorCap - 1) / kVectorCap);
                    fixups.push_back({(int32_t)i, (int32_t)n_pieces, np, (int32_t)p});
                    for (int32_t j = 0; j < np; ++j)
                        big.push_back({(int32_t)i, j, (int32_t)(n_pieces + j),
                                       (int32_t)((kItemPiece << 24) | (int32_t)p)});
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
            stream.push_back({(int32_t)start, (int32_t)(i - start), 0,
                              (int32_t)((kItemStream << 24) | (int32_t)p)});
        }
        row = hi;
    }
    items.clear();
    items.insert(items.end(), big.begin(), big.end());
    items.insert(items.end(), vec.begin(), vec.end());
    items.insert(items.end(), stream.begin(), stream.end());
}

ecc_status_t launch_sweep(ecc_matrix_t M, const double *d_b, double alpha, double beta,
                          const double *d_x_own, const double *d_x_hat, double *d_x_next,
                          double *d_partials, int32_t zero_extra, const int32_t *d_done) {
    ecc_plan_t pl = M->plan;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(M->n_items, kMaxSweepBlocks));
    if (M->kind == ECC_KIND_JACOBI)
        hipLaunchKernelGGL(k_sweep<ECC_KIND_JACOBI>, dim3(grid), dim3(kSweepThreads), 0,
                           pl->stream, M->d_items, (int32_t)M->n_items, M->A.d_row_ptr, M->A.d_col,
                           M->A.d_val, pl->d_block_start, d_b, alpha, beta, d_x_own, d_x_hat,
                           d_x_next, d_partials, M->d_pieces, zero_extra, d_done);
    else
        hipLaunchKernelGGL(k_sweep<ECC_KIND_POWER>, dim3(grid), dim3(kSweepThreads), 0,
                           pl->stream, M->d_items, (int32_t)M->n_items, M->A.d_row_ptr, M->A.d_col,
                           M->A.d_val, pl->d_block_start, d_b, alpha, beta, d_x_own, d_x_hat,
                           d_x_next, d_partials, M->d_pieces, zero_extra, d_done);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

static int64_t n_main_partials(ecc_matrix_t M) {
    return std::max<int64_t>(1, std::min<int64_t>(M->n_items, kMaxSweepBlocks));
}

static ecc_status_t launch_pass2_impl(ecc_plan_t pl, ecc_matrix_t M, double *d_partials,
                                      int64_t n_main, bool do_fixups, int32_t norm,
                                      const double *d_b, double alpha, double beta,
                                      const double *d_x_own, double *d_x_next, double *d_out,
                                      double tol, int32_t *d_ctrl, int32_t t,
                                      const int32_t *d_done) {
    const Fixup *fx = (M && M->n_fixups > 0) ? M->d_fixups : nullptr;
    const int32_t nf = fx ? (int32_t)M->n_fixups : 0;
    const double2 *pc = M ? M->d_pieces : nullptr;
    const int kind = M ? M->kind : ECC_KIND_POWER;
    const int32_t fix = do_fixups ? 1 : 0;
    if (kind == ECC_KIND_JACOBI)
        hipLaunchKernelGGL(k_pass2<ECC_KIND_JACOBI>, dim3(1), dim3(kPass2Threads), 0, pl->stream,
                           d_partials, n_main, fix, fx, nf, pc, d_b, alpha, beta, d_x_own,
                           d_x_next, norm, d_out, tol, d_ctrl, t, d_done);
    else
        hipLaunchKernelGGL(k_pass2<ECC_KIND_POWER>, dim3(1), dim3(kPass2Threads), 0, pl->stream,
                           d_partials, n_main, fix, fx, nf, pc, d_b, alpha, beta, d_x_own,
                           d_x_next, norm, d_out, tol, d_ctrl, t, d_done);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

}  // namespace ecc

using namespace ecc;

extern "C" {

ecc_status_t ecc_matrix_create(ecc_plan_t plan, const ecc_csr_t *A, int32_t kind,
                               ecc_matrix_t *out) {
    clear_error();
    ECC_ARG(out != nullptr, "out is NULL");
    *out = nullptr;
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(A != nullptr, "A is NULL");
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

    // structural check on the device
    if (n > 0) {
        unsigned long long *d_bad = nullptr;
        ECC_HIP(hipMalloc((void **)&d_bad, 2 * sizeof(unsigned long long)));
        unsigned long long h_bad[2] = {0, 0};
        hipError_t e = hipMemcpy(d_bad, h_bad, sizeof(h_bad), hipMemcpyHostToDevice);
        if (e == hipSuccess) {
            const int blocks = (int)std::min<int64_t>(4096, (n + 255) / 256);
            hipLaunchKernelGGL(k_check, dim3(blocks), dim3(256), 0, plan->stream, (int32_t)n,
                               (int32_t)A->n_cols, A->d_row_ptr, A->d_col, A->d_val,
                               kind == ECC_KIND_JACOBI ? 1 : 0, d_bad);
            e = hipGetLastError();
            if (e == hipSuccess) e = hipStreamSynchronize(plan->stream);
            if (e == hipSuccess) e = hipMemcpy(h_bad, d_bad, sizeof(h_bad), hipMemcpyDeviceToHost);
        }
        (void)hipFree(d_bad);
        if (e != hipSuccess) {
            set_error("matrix check failed: %s", hipGetErrorString(e));
            return ECC_ERR_DEVICE;
        }
        ECC_ARG(h_bad[1] == 0, "%llu column indices are out of range", h_bad[1]);
        ECC_ARG(h_bad[0] == 0, "%llu rows lack a single non-zero diagonal entry", h_bad[0]);
    }

    std::vector<WorkItem> items;
    std::vector<Fixup> fixups;
    int64_t n_pieces = 0;
    build_items(rp, plan->counts, items, fixups, n_pieces);

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
    if (hipMalloc((void **)&M->d_partials, sizeof(double) * (n_main_partials(M) + 1)) != hipSuccess)
        return fail("hipMalloc of partials failed");
    *out = M;
    return ECC_OK;
}

ecc_status_t ecc_matrix_destroy(ecc_matrix_t M) {
    if (!M) return ECC_OK;
    if (M->plan) (void)hipStreamSynchronize(M->plan->stream);
    (void)hipFree(M->d_items);
    (void)hipFree(M->d_fixups);
    (void)hipFree(M->d_pieces);
    (void)hipFree(M->d_partials);
    delete M;
    return ECC_OK;
}

int64_t ecc_partials_size(ecc_matrix_t M) {
    if (!M) return 0;
    return n_main_partials(M) + 1;
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
    ECC_ARG(n == 0 || (d_x_own && d_x_hat && d_x_next && d_partials), "NULL vector argument");
    ECC_ARG(kind != ECC_KIND_JACOBI || n == 0 || d_b, "d_b is NULL");
    ECC_ARG(n == 0 || (d_x_next != d_x_own && d_x_next != d_x_hat && d_x_next != d_b),
            "d_x_next must not alias an input");
    const bool split = M->n_fixups > 0;
    st = launch_sweep(M, d_b, alpha, beta, d_x_own, d_x_hat, d_x_next, d_partials,
                      split ? 0 : 1, nullptr);
    if (st != ECC_OK || !split) return st;
    // finish the rows that were split into pieces
    return launch_pass2_impl(plan, M, d_partials, n_main_partials(M), true, 0, d_b, alpha, beta,
                             d_x_own, d_x_next, nullptr, 0.0, nullptr, 0, nullptr);
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

ecc_status_t ecc_residual(ecc_plan_t plan, const double *d_partials, int64_t n_partials,
                          int32_t norm, double *h_out, double *d_out) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(norm == ECC_NORM_L1 || norm == ECC_NORM_L2, "norm must be 1 or 2");
    ECC_ARG(n_partials >= 1 && d_partials, "need at least one partial");
    ECC_ARG(h_out || d_out, "h_out and d_out are both NULL");
    double *dst = d_out ? d_out : plan->d_scalar;
    st = launch_pass2_impl(plan, nullptr, const_cast<double *>(d_partials), n_partials - 1, false,
                           norm, nullptr, 0.0, 0.0, nullptr, nullptr, dst, 0.0, nullptr, 0,
                           nullptr);
    if (st != ECC_OK) return st;
    if (h_out) {
        ECC_HIP(hipMemcpyAsync(h_out, dst, sizeof(double), hipMemcpyDeviceToHost, plan->stream));
        ECC_HIP(hipStreamSynchronize(plan->stream));
    }
    return ECC_OK;
}

}  // extern "C"

namespace ecc {
ecc_status_t solve_pass2(ecc_matrix_t M, int32_t norm, const double *d_b, double alpha,
                         double beta, const double *d_x_own, double *d_x_next, double *d_out,
                         double tol, int32_t *d_ctrl, int32_t t, const int32_t *d_done) {
    return launch_pass2_impl(M->plan, M, M->d_partials, n_main_partials(M), true, norm, d_b,
                             alpha, beta, d_x_own, d_x_next, d_out, tol, d_ctrl, t, d_done);
}
}  // namespace ecc
