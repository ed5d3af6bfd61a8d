// Data-parallel matrix factorisation by gradient steps over the eventually
// consistent partial allreduce: the workload of the paper's allreduce_SSP
// experiment (Section IV), P workers each holding a shard of the ratings
// and a replica of the model W = [U; V] (rows of `rank` doubles).
//
// One iteration, enqueued on the plan's stream:
//  (1) k_mf_err: e_k = r_k - U[u_k] . V[i_k] for every rating (products
//      added for j = 0 .. rank-1 in order), and per-workgroup sums of e_k^2;
//  (2) k_mf_grad: every worker's gradient of its shard's squared error --
//      row (p, entity) accumulates (-2 e_k) times the other factor's row
//      over the worker's ratings of that entity, in shard order; `rank`
//      lanes per row, one per column; rows without ratings are written 0;
//  (3) the partial allreduce of the workers' gradients (ecc_allreduce_partial:
//      staleness decision, stale gradients substituted from the slots);
//  (4) k_mf_step: W := W - eta * (G * c_row + 2 lam W), c_row = 1 / (number
//      of ratings of the row, at least 1);
//  (5) k_mf_rmse: sqrt(sum e_k^2 / N) from the workgroup sums in a fixed
//      order.
// The per-worker row index (ratings of each (worker, entity) row in shard
// order) is built once, on the host, by counting sorts.
#include <algorithm>
#include <vector>

#include "ecc_common.h"

namespace ecc {

constexpr int kMfThreads = 256;
constexpr int kMfMaxRank = 64;

struct MfView {
    int32_t n_users, n_items;
    int64_t N;
    const int32_t *users, *items;
    const double *ratings;
    const double *W;  // [U; V]
};

template <int R>
__global__ __launch_bounds__(kMfThreads) void k_mf_err(MfView v, double *__restrict__ err,
                                                       double *__restrict__ partials) {
    __shared__ double s_red[kMfThreads / 64];
    const double *U = v.W, *V = v.W + (int64_t)v.n_users * R;
    double sq = 0.0;
    const int64_t stride = (int64_t)gridDim.x * kMfThreads;
    for (int64_t k = (int64_t)blockIdx.x * kMfThreads + threadIdx.x; k < v.N; k += stride) {
        const double *ur = U + (int64_t)v.users[k] * R;
        const double *vr = V + (int64_t)v.items[k] * R;
        double acc = 0.0;
#pragma unroll
        for (int j = 0; j < R; ++j) acc = acc + ur[j] * vr[j];
        const double e = v.ratings[k] - acc;
        err[k] = e;
        sq = sq + e * e;
    }
    const double tot = block_sum<kMfThreads>(sq, s_red);
    if (threadIdx.x == 0) partials[blockIdx.x] = tot;
}

// Row r of the gradient index: worker p = r / E, entity e = r % E (E =
// n_users + n_items; users first).  Its ratings are perm[rp[r] .. rp[r+1]),
// and oidx holds, in the same order, the index of the other factor's row.
template <int R>
__global__ __launch_bounds__(kMfThreads) void k_mf_grad(MfView v, const double *__restrict__ err,
                                                        const int32_t *__restrict__ perm,
                                                        const int32_t *__restrict__ oidx,
                                                        const int32_t *__restrict__ rp,
                                                        int64_t n_rows,
                                                        double *const *__restrict__ grads) {
    constexpr int ROWS = kMfThreads / R;  // rows per workgroup and pass
    const int lane = threadIdx.x % R;
    const int64_t E = (int64_t)v.n_users + v.n_items;
    const double *U = v.W, *V = v.W + (int64_t)v.n_users * R;
    for (int64_t row = (int64_t)blockIdx.x * ROWS + threadIdx.x / R; row < n_rows;
         row += (int64_t)gridDim.x * ROWS) {
        const int32_t p = (int32_t)(row / E);
        const int64_t e = row - (int64_t)p * E;
        const bool user = e < v.n_users;
        const double *other = user ? V : U;
        const int32_t a = rp[row], b = rp[row + 1];
        double acc = 0.0;
        int32_t x = a;
        // four ratings' loads in flight, added in order
        for (; x + 4 <= b; x += 4) {
            int32_t k[4];
            double t[4], o[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) k[u] = perm[x + u];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                t[u] = -2.0 * err[k[u]];
                o[u] = other[(int64_t)oidx[x + u] * R + lane];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) acc = acc + t[u] * o[u];
        }
        for (; x < b; ++x) {
            const int32_t k = perm[x];
            acc = acc + (-2.0 * err[k]) * other[(int64_t)oidx[x] * R + lane];
        }
        grads[p][e * R + lane] = acc;
    }
}

__global__ __launch_bounds__(kMfThreads) void k_mf_step(int64_t m, int log2r, double eta,
                                                        double lam2,
                                                        const double *__restrict__ G,
                                                        const double *__restrict__ row_scale,
                                                        double *__restrict__ W) {
    const int64_t stride = (int64_t)gridDim.x * kMfThreads;
    for (int64_t x = (int64_t)blockIdx.x * kMfThreads + threadIdx.x; x < m; x += stride) {
        const double w = W[x];
        W[x] = w - eta * (G[x] * row_scale[x >> log2r] + lam2 * w);
    }
}

__global__ __launch_bounds__(kNormThreads) void k_mf_rmse(const double *__restrict__ partials,
                                                          int64_t n, int64_t N,
                                                          double *__restrict__ out) {
    __shared__ double s_red[kNormThreads / 64];
    const double sum = reduce_values(partials, n, false, 0.0, s_red);
    if (threadIdx.x == 0) *out = sqrt(sum / (double)N);
}

int32_t mf_grid(int64_t work, int per_cu) {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        cus = 256;
    return (int32_t)std::max<int64_t>(1, std::min<int64_t>(work, (int64_t)cus * per_cu));
}

}  // namespace ecc

using namespace ecc;

struct ecc_mf_s {
    int32_t n_users = 0, n_items = 0, rank = 0, P = 0;
    int64_t N = 0;
    const int32_t *d_users = nullptr, *d_items = nullptr;
    const double *d_ratings = nullptr;
    double *d_err = nullptr;        // [N]
    int32_t *d_perm = nullptr;      // [2N]
    int32_t *d_oidx = nullptr;      // [2N] other factor's row of perm[x]
    int32_t *d_rp = nullptr;        // [P * (n_users + n_items) + 1]
    double *d_scale = nullptr;      // [n_users + n_items]
    double *d_partials = nullptr;   // [err_grid]
    int32_t err_grid = 1, grad_grid = 1, step_grid = 1;
};

extern "C" {

ecc_status_t ecc_mf_destroy(ecc_mf_t h) {
    if (!h) return ECC_OK;
    (void)hipDeviceSynchronize();
    (void)hipFree(h->d_err);
    (void)hipFree(h->d_perm);
    (void)hipFree(h->d_oidx);
    (void)hipFree(h->d_rp);
    (void)hipFree(h->d_scale);
    (void)hipFree(h->d_partials);
    delete h;
    return ECC_OK;
}

ecc_status_t ecc_mf_create(int32_t n_users, int32_t n_items, int32_t rank, int32_t P, int64_t N,
                           const int32_t *d_users, const int32_t *d_items,
                           const double *d_ratings, ecc_mf_t *out) {
    clear_error();
    ECC_ARG(out != nullptr, "out is NULL");
    *out = nullptr;
    ECC_ARG(n_users >= 1 && n_items >= 1, "need at least one user and one item");
    ECC_ARG(rank >= 1 && rank <= kMfMaxRank && (rank & (rank - 1)) == 0,
            "rank = %d must be a power of two in [1, 64]", rank);
    ECC_ARG(P >= 1, "P must be >= 1");
    ECC_ARG(N >= 1 && 2 * N < (int64_t(1) << 31), "N must lie in [1, 2^30)");
    ECC_ARG(d_users && d_items && d_ratings, "NULL rating arrays");
    const int64_t E = (int64_t)n_users + n_items;
    const int64_t n_rows = (int64_t)P * E;
    if (n_rows + 1 >= (int64_t(1) << 31)) {
        set_error("P * (n_users + n_items) too large");
        return ECC_ERR_RANGE;
    }
    std::vector<int32_t> users(N), items(N);
    ECC_HIP(hipMemcpy(users.data(), d_users, sizeof(int32_t) * N, hipMemcpyDeviceToHost));
    ECC_HIP(hipMemcpy(items.data(), d_items, sizeof(int32_t) * N, hipMemcpyDeviceToHost));
    std::vector<int64_t> cnt(E, 0);
    for (int64_t k = 0; k < N; ++k) {
        ECC_ARG(users[k] >= 0 && users[k] < n_users, "users[%lld] out of range", (long long)k);
        ECC_ARG(items[k] >= 0 && items[k] < n_items, "items[%lld] out of range", (long long)k);
        ++cnt[users[k]];
        ++cnt[(int64_t)n_users + items[k]];
    }
    // rows (p, entity): users then items of worker p; their ratings in shard
    // order, user rows' in perm[2 a_p ...] and item rows' after them
    std::vector<int32_t> rp(n_rows + 1, 0), perm(2 * N);
    std::vector<int32_t> fill(E);
    int64_t pos = 0;
    for (int32_t p = 0; p < P; ++p) {
        const int64_t a = N * p / P, b = N * (p + 1) / P;
        std::fill(fill.begin(), fill.end(), 0);
        for (int64_t k = a; k < b; ++k) {
            ++fill[users[k]];
            ++fill[(int64_t)n_users + items[k]];
        }
        const int64_t base = (int64_t)p * E;
        for (int64_t e = 0; e < E; ++e) {
            rp[base + e] = (int32_t)pos;
            pos += fill[e];
            fill[e] = rp[base + e];
        }
        for (int64_t k = a; k < b; ++k) {
            perm[fill[users[k]]++] = (int32_t)k;
            perm[fill[(int64_t)n_users + items[k]]++] = (int32_t)k;
        }
    }
    rp[n_rows] = (int32_t)pos;
    std::vector<int32_t> oidx(2 * N);
    for (int32_t p = 0; p < P; ++p) {
        const int64_t base = (int64_t)p * E;
        for (int64_t e = 0; e < E; ++e)
            for (int32_t x = rp[base + e]; x < rp[base + e + 1]; ++x)
                oidx[x] = e < n_users ? items[perm[x]] : users[perm[x]];
    }
    std::vector<double> scale(E);
    for (int64_t e = 0; e < E; ++e) scale[e] = 1.0 / (double)std::max<int64_t>(1, cnt[e]);

    ecc_mf_s *h = new (std::nothrow) ecc_mf_s();
    if (!h) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
    h->n_users = n_users;
    h->n_items = n_items;
    h->rank = rank;
    h->P = P;
    h->N = N;
    h->d_users = d_users;
    h->d_items = d_items;
    h->d_ratings = d_ratings;
    h->err_grid = mf_grid((N + kMfThreads - 1) / kMfThreads, 8);
    h->grad_grid = mf_grid((n_rows + kMfThreads / rank - 1) / (kMfThreads / rank), 8);
    h->step_grid = mf_grid((E * rank + kMfThreads - 1) / kMfThreads, 8);
    auto fail = [&](const char *what) {
        set_error("%s", what);
        ecc_mf_destroy(h);
        return ECC_ERR_ALLOC;
    };
    if (hipMalloc((void **)&h->d_err, sizeof(double) * N) != hipSuccess ||
        hipMalloc((void **)&h->d_perm, sizeof(int32_t) * 2 * N) != hipSuccess ||
        hipMalloc((void **)&h->d_oidx, sizeof(int32_t) * 2 * N) != hipSuccess ||
        hipMalloc((void **)&h->d_rp, sizeof(int32_t) * (n_rows + 1)) != hipSuccess ||
        hipMalloc((void **)&h->d_scale, sizeof(double) * E) != hipSuccess ||
        hipMalloc((void **)&h->d_partials, sizeof(double) * h->err_grid) != hipSuccess)
        return fail("hipMalloc of the factorisation state failed");
    if (hipMemcpy(h->d_perm, perm.data(), sizeof(int32_t) * 2 * N, hipMemcpyHostToDevice) !=
            hipSuccess ||
        hipMemcpy(h->d_oidx, oidx.data(), sizeof(int32_t) * 2 * N, hipMemcpyHostToDevice) !=
            hipSuccess ||
        hipMemcpy(h->d_rp, rp.data(), sizeof(int32_t) * (n_rows + 1), hipMemcpyHostToDevice) !=
            hipSuccess ||
        hipMemcpy(h->d_scale, scale.data(), sizeof(double) * E, hipMemcpyHostToDevice) !=
            hipSuccess)
        return fail("upload of the factorisation state failed");
    *out = h;
    return ECC_OK;
}

ecc_status_t ecc_mf_iterate(ecc_mf_t h, ecc_plan_t plan, double eta, double lam, double *d_W,
                            double *const *d_grads, double *const *d_slots, double *d_G,
                            const uint8_t *d_arrived, double *d_rmse, uint8_t *d_eff_out) {
    clear_error();
    ECC_ARG(h != nullptr, "factorisation state is NULL");
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    if (plan->P != h->P) {
        set_error("plan has %d ranks, the factorisation %d workers", plan->P, h->P);
        return ECC_ERR_STATE;
    }
    ECC_ARG(d_W && d_grads && d_slots && d_G && d_arrived && d_rmse, "NULL argument");
    hipStream_t s = plan->stream;
    MfView v{h->n_users, h->n_items, h->N, h->d_users, h->d_items, h->d_ratings, d_W};
    const int64_t E = (int64_t)h->n_users + h->n_items;
    const int64_t n_rows = (int64_t)h->P * E;
    const int64_t m = E * h->rank;
    int log2r = 0;
    while ((1 << log2r) < h->rank) ++log2r;
#define ECC_MF_RANKS(X) X(1) X(2) X(4) X(8) X(16) X(32) X(64)
#define ECC_MF_LAUNCH(R)                                                                      \
    case R: {                                                                                 \
        {                                                                                     \
            TimedLaunch timed(plan, ECC_TIMING_MF_ERROR);                                     \
            hipLaunchKernelGGL(k_mf_err<R>, dim3(h->err_grid), dim3(kMfThreads), 0, s, v,     \
                               h->d_err, h->d_partials);                                      \
        }                                                                                     \
        TimedLaunch timed(plan, ECC_TIMING_MF_GRAD);                                          \
        hipLaunchKernelGGL(k_mf_grad<R>, dim3(h->grad_grid), dim3(kMfThreads), 0, s, v,       \
                           h->d_err, h->d_perm, h->d_oidx, h->d_rp, n_rows, d_grads);         \
        break;                                                                                \
    }
    switch (h->rank) {
        ECC_MF_RANKS(ECC_MF_LAUNCH)
        default:
            set_error("internal: rank %d", h->rank);
            return ECC_ERR_STATE;
    }
#undef ECC_MF_LAUNCH
#undef ECC_MF_RANKS
    ECC_LAUNCH_CHECK();
    st = ecc_allreduce_partial(plan, m, d_grads, d_slots, d_G, d_arrived, d_eff_out, nullptr);
    if (st != ECC_OK) return st;
    {
        TimedLaunch timed(plan, ECC_TIMING_MF_STEP);
        hipLaunchKernelGGL(k_mf_rmse, dim3(1), dim3(kNormThreads), 0, s, h->d_partials,
                           (int64_t)h->err_grid, h->N, d_rmse);
        hipLaunchKernelGGL(k_mf_step, dim3(h->step_grid), dim3(kMfThreads), 0, s, m, log2r, eta,
                           2.0 * lam, d_G, h->d_scale, d_W);
    }
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

}  // extern "C"
