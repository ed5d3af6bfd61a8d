// Data-parallel matrix factorisation by minibatch stochastic gradient
// descent over the eventually consistent partial allreduce: the workload of
// the paper's allreduce_SSP experiment (Section IV), P workers each holding
// a shard of the ratings, cut into K minibatches of consecutive ratings, and
// a replica of the model W = [U; V] (rows of `rank` doubles).
//
// One iteration, enqueued on the plan's stream, worker p using minibatch
// batch[p] (a device array, so that a schedule can be replayed without the
// host):
//  (1) k_mf_grad: every row (p, entity) of every worker's gradient of its
//      minibatch's squared error.  For the minibatch's ratings of that
//      entity, in storage order, the rating's error e_k = r_k - U[u_k] .
//      V[i_k] (products added for j = 0 .. rank-1 in order) and then
//      row += (-2 e_k) times the other factor's row; rows without ratings in
//      the minibatch are 0.  The errors met in user rows (every rating lies in
//      exactly one) also feed per-workgroup sums of e_k^2.  A worker taken
//      at this clock writes its gradient into its slot, one not taken into
//      its gradient buffer (its slot keeps its last taken gradient);
//  (2) the partial allreduce of the workers' gradients (ecc_allreduce_partial:
//      staleness decision, every gradient read from the slots in place);
//  (3) k_mf_step: W := W - eta * (G * c_row + 2 lam W), c_row = K / (number
//      of ratings of the row, at least 1); its workgroup 0 also reduces the
//      minibatch error sqrt(sum e_k^2 / ratings used) from the gradient
//      kernel's workgroup sums, in a fixed order.
// ecc_mf_error evaluates sqrt(sum e_k^2 / N) over all ratings at a model.
//
// The gradient index is built once, on the host, for every (worker,
// minibatch): the ratings of each row in storage order (other factor's row
// index and rating value, stored in that order), and every entity's row in
// order of its number of ratings, longest first.  The gradient kernel's
// grid holds g workgroups per worker, which walk the rows of its
// minibatch's list; with a multiple of 8 workers every worker's workgroups
// run on one XCD (workgroups are dealt to the 8 XCDs round-robin), so that
// the factor rows its list gathers most stay in that XCD's L2.
//  - A row of more than kMfHeavy ratings takes a whole workgroup: chunks of
//    its ratings are spread over the workgroup, whose lane groups compute
//    the errors and products into LDS, and then `rank` lanes add the
//    products in storage order.  The longest rows (hundreds of ratings for
//    the most popular items) thus wait on a few memory latencies per chunk
//    instead of a serial chain of loads per rating.
//  - Other rows take a group of rank / 4 lanes (4 columns each; one lane
//    for rank < 4), so a wave of rank 16 carries 16 rows of similar
//    length (rows sorted by length); kMfBatch ratings' loads
//    are in flight and the next batch's indices are loaded while one is
//    summed; the next item's row descriptors are loaded one item ahead.
//  - Rows without ratings in the minibatch (about half of each list at the
//    benchmark's shape) end the list; every workgroup of the worker first
//    writes zeros over a contiguous share of them, with the entity indices
//    of several passes loaded together.
// A rating's dot product is the running sum of the group's lanes in column
// order, handed from lane to lane by shuffles, so errors and gradients are
// the sequential definition's, bit for bit.
#include <algorithm>
#include <vector>

#include <new>

#include "ecc_common.h"

namespace ecc {

constexpr int kMfThreads = 256;
constexpr int kMfMaxRank = 64;
constexpr int kMfHeavy = 128;   // rows with more ratings take a whole workgroup
constexpr int kMfStage = 2048;  // doubles of LDS for one chunk of a heavy row
constexpr int kMfBatch = 4;     // ratings of a light row in flight together
constexpr int kMfZeroPasses = 8;  // passes of rows without ratings with loads in flight together

// Rows without ratings: R / V lanes per row, V doubles per lane.
template <int R>
struct MfZero {
    static constexpr int V = R >= 2 ? 2 : 1;
    static constexpr int LPR = R / V;
    static constexpr int ROWS = kMfThreads / LPR;  // rows of one pass of the workgroup
};

template <int R>
struct MfShape {
    static constexpr int C = R < 4 ? R : 4;               // columns per lane
    static constexpr int LPR = R / C;                     // lanes per row
    static constexpr int GROUPS = kMfThreads / LPR;       // rows of a light item
    static constexpr int CHUNK = kMfStage / R;            // ratings of a heavy chunk
    static constexpr int J = CHUNK / GROUPS > 0 ? CHUNK / GROUPS : 1;  // per group and chunk
};

struct MfGradArgs {
    int32_t n_users;
    int64_t E;                    // n_users + n_items
    int32_t K;                    // minibatches per worker
    const double *W;              // [U; V]
    const int32_t *oidx;          // [2N] other factor's row, ratings of each row in storage order
    const double *rv;             // [2N] rating values, same order
    const int32_t *row_of;        // [P K E] entity of each row of each (worker, minibatch)
                                  // list, longest first
    const int32_t *start_of;      // same order: first rating of that row in oidx / rv
    const int32_t *len_of;        // same order: its number of ratings
    const int32_t *n_heavy;       // [P K] rows of more than kMfHeavy ratings, per list
    const int32_t *n_rated;       // [P K] rows with ratings, per list (the rows without follow)
    const int32_t *batch;         // [P] this iteration's minibatch of each worker
    double *const *grads;         // [P] -> m doubles: gradients of workers not taken
    double *const *slots;         // [P] -> m doubles: gradients of workers taken
    const int32_t *ver_in;        // [P] versions at this clock (the plan's)
    const uint8_t *arrived;       // [P] arrivals of this clock
    int64_t t;                    // the plan's clock
    int32_t S;                    // its slack
    double *partials;             // [P][g] sums of e^2 over user rows
    int32_t g;                    // workgroups per worker
    int32_t pin;                  // P a multiple of 8: a worker's workgroups on one XCD
};

// own . other over a lane group: lane l holds columns l*C .. l*C + C-1 of
// both rows; lane s continues the running sum of lane s - 1 (received by a
// shuffle), so the products are added for j = 0 .. R-1 in order from +0.0.
template <int R>
__device__ __forceinline__ double mf_dot(const double (&ow)[MfShape<R>::C],
                                         const double (&o)[MfShape<R>::C]) {
    constexpr int LPR = MfShape<R>::LPR, C = MfShape<R>::C;
    double d = 0.0;
#pragma unroll
    for (int s = 0; s < LPR; ++s) {
        double v = d;
#pragma unroll
        for (int c = 0; c < C; ++c) v = v + ow[c] * o[c];
        d = (LPR == 1) ? v : __shfl(v, s, LPR);
    }
    return d;
}

// One light row on the lane group (lane = column block); returns the lane's
// sum of e^2 (user rows, lane 0 only).
template <int R>
__device__ __forceinline__ double mf_light_row(const MfGradArgs &a, double *gd, int32_t ent,
                                               int32_t x0, int32_t len, int lane) {
    constexpr int C = MfShape<R>::C, K = kMfBatch;
    const int64_t e = ent;
    const bool user = e < a.n_users;
    const double *own = a.W + e * R + lane * C;
    const double *other = (user ? a.W + (int64_t)a.n_users * R : a.W) + lane * C;
    const int32_t x1 = x0 + len;
    double acc[C], ow[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        acc[c] = 0.0;
        ow[c] = len > 0 ? own[c] : 0.0;
    }
    int32_t ki[K];
    double kr[K];
#pragma unroll
    for (int u = 0; u < K; ++u) {
        ki[u] = (x0 + u < x1) ? a.oidx[x0 + u] : 0;
        kr[u] = (x0 + u < x1) ? a.rv[x0 + u] : 0.0;
    }
    double sq = 0.0;
    for (int32_t x = x0; x < x1; x += K) {
        double o[K][C], r[K];
#pragma unroll
        for (int u = 0; u < K; ++u) {
            r[u] = kr[u];
#pragma unroll
            for (int c = 0; c < C; ++c)
                o[u][c] = (x + u < x1) ? other[(int64_t)ki[u] * R + c] : 0.0;
        }
        const int32_t xn = x + K;
#pragma unroll
        for (int u = 0; u < K; ++u) {
            ki[u] = (xn + u < x1) ? a.oidx[xn + u] : 0;
            kr[u] = (xn + u < x1) ? a.rv[xn + u] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < K; ++u) {
            if (x + u < x1) {
                const double err = r[u] - mf_dot<R>(ow, o[u]);
                const double t = -2.0 * err;
#pragma unroll
                for (int c = 0; c < C; ++c) acc[c] = acc[c] + t * o[u][c];
                if (user) sq = sq + err * err;
            }
        }
    }
    double *g = gd + e * R + lane * C;
#pragma unroll
    for (int c = 0; c < C; ++c) g[c] = acc[c];
    return lane == 0 ? sq : 0.0;
}

// One heavy row on the whole workgroup; returns the thread's sum of e^2.
template <int R>
__device__ __forceinline__ double mf_heavy_row(const MfGradArgs &a, double *gd, int32_t ent,
                                               int32_t x0, int32_t len, double *s_prod) {
    constexpr int LPR = MfShape<R>::LPR, C = MfShape<R>::C, NG = MfShape<R>::GROUPS;
    constexpr int CH = MfShape<R>::CHUNK, J = MfShape<R>::J;
    const int tid = threadIdx.x, lane = tid % LPR, grp = tid / LPR;
    const int64_t e = ent;
    const bool user = e < a.n_users;
    const double *own = a.W + e * R + lane * C;
    const double *other = (user ? a.W + (int64_t)a.n_users * R : a.W) + lane * C;
    double ow[C];
#pragma unroll
    for (int c = 0; c < C; ++c) ow[c] = own[c];
    double acc = 0.0, sq = 0.0;
    for (int32_t xb = 0; xb < len; xb += CH) {
        const int32_t n = min(CH, len - xb);
        // ratings grp, grp + NG, ... of the chunk: loads first, then products
        int32_t ki[J];
        double kr[J], o[J][C];
#pragma unroll
        for (int q = 0; q < J; ++q) {
            const int32_t j = grp + q * NG;
            ki[q] = j < n ? a.oidx[x0 + xb + j] : 0;
            kr[q] = j < n ? a.rv[x0 + xb + j] : 0.0;
        }
#pragma unroll
        for (int q = 0; q < J; ++q) {
            const int32_t j = grp + q * NG;
#pragma unroll
            for (int c = 0; c < C; ++c)
                o[q][c] = j < n ? other[(int64_t)ki[q] * R + c] : 0.0;
        }
#pragma unroll
        for (int q = 0; q < J; ++q) {
            const int32_t j = grp + q * NG;
            if (j < n) {
                const double err = kr[q] - mf_dot<R>(ow, o[q]);
                const double t = -2.0 * err;
#pragma unroll
                for (int c = 0; c < C; ++c) s_prod[j * R + lane * C + c] = t * o[q][c];
                if (user && lane == 0) sq = sq + err * err;
            }
        }
        __syncthreads();
        if (tid < R)
            for (int32_t j = 0; j < n; ++j) acc = acc + s_prod[j * R + tid];
        __syncthreads();
    }
    if (tid < R) gd[e * R + tid] = acc;
    return sq;
}

template <int R>
__global__ __launch_bounds__(kMfThreads) void k_mf_grad(MfGradArgs a) {
    __shared__ double s_prod[kMfStage];
    __shared__ double s_red[kMfThreads / 64];
    constexpr int LPR = MfShape<R>::LPR, G = MfShape<R>::GROUPS;
    using Z = MfZero<R>;
    static_assert(MfShape<R>::CHUNK * R == kMfStage, "a heavy chunk fills the stage");
    const int lane = threadIdx.x % LPR, grp = threadIdx.x / LPR;
    // worker p's list for its minibatch of this iteration
    // this workgroup's worker p and its index wgx among the worker's g:
    // workgroup b runs on XCD b mod 8, and with pinning the workers
    // x, x + 8, ... take XCD x's workgroups in turn (measured on MI355X, 25M
    // ratings, 32 workers: 742 against 774 us per iteration, bitwise the same)
    const int64_t g = a.g;
    int32_t p;
    int64_t wgx;
    if (a.pin) {
        const int64_t xb = blockIdx.x & 7, kb = blockIdx.x >> 3;
        p = (int32_t)(xb + 8 * (kb / g));
        wgx = kb % g;
    } else {
        p = (int32_t)(blockIdx.x / g);
        wgx = blockIdx.x % g;
    }
    const int32_t bp = min(max(a.batch[p], 0), a.K - 1);  // (values outside [0, K) clamped)
    // a worker whose contribution the allreduce takes at this clock writes
    // its gradient straight into its slot, which the allreduce then reads in
    // place (the decision is the allreduce's own, from the same versions);
    // measured on MI355X, 25M ratings, rank 16, 32 workers: the allreduce
    // 197 against 326 us, the iteration 620 against 744 us
    double *const gd = stale_select(a.ver_in[p], a.arrived[p], a.t, a.S) ? a.slots[p] : a.grads[p];
    const int64_t list = (int64_t)p * a.K + bp;
    const int32_t *row_of = a.row_of + list * a.E;
    const int32_t *start_of = a.start_of + list * a.E;
    const int32_t *len_of = a.len_of + list * a.E;
    const int64_t n_rows = a.E, n_heavy = a.n_heavy[list], n_rated = a.n_rated[list];
    const int64_t n_work = n_heavy + (n_rated - n_heavy + G - 1) / G;
    double sq = 0.0;
    // Rows without ratings (list positions n_rated .. E-1, in entity order):
    // this workgroup's contiguous share is written as zeros first,
    // kMfZeroPasses passes at a time with all their entity loads in flight
    // (measured on MI355X, 25M ratings, rank 16, 32 workers: 806 against
    // 863 us per iteration when they were light rows of length 0 at the end
    // of the list; writing them last, or first in every other workgroup,
    // 815 and 810 us).
    const int64_t n_zero = n_rows - n_rated;
    const int64_t z_lo = n_rated + n_zero * wgx / g;
    const int64_t z_hi = n_rated + n_zero * (wgx + 1) / g;
    {
        double *const grad = gd;
        const int zl = threadIdx.x % Z::LPR, zr = threadIdx.x / Z::LPR;
        for (int64_t zq = z_lo; zq < z_hi; zq += (int64_t)kMfZeroPasses * Z::ROWS) {
            int32_t ent[kMfZeroPasses];
#pragma unroll
            for (int s = 0; s < kMfZeroPasses; ++s) {
                const int64_t q = zq + (int64_t)s * Z::ROWS + zr;
                ent[s] = q < z_hi ? row_of[q] : -1;
            }
#pragma unroll
            for (int s = 0; s < kMfZeroPasses; ++s) {
                if (ent[s] >= 0) {
                    double *gz = grad + (int64_t)ent[s] * R + zl * Z::V;
#pragma unroll
                    for (int c = 0; c < Z::V; ++c) gz[c] = 0.0;
                }
            }
        }
    }
    // this lane group's row in a light item w (descriptors one item ahead)
    auto light_q = [&](int64_t w) { return n_heavy + (w - n_heavy) * G + grp; };
    int32_t nrow = 0, nx0 = 0, nlen = -1;
    int64_t w = wgx;
    if (w < n_work && w >= n_heavy && light_q(w) < n_rated) {
        const int64_t q = light_q(w);
        nrow = row_of[q];
        nx0 = start_of[q];
        nlen = len_of[q];
    }
    for (; w < n_work; w += g) {
        if (w < n_heavy) {
            sq += mf_heavy_row<R>(a, gd, row_of[w], start_of[w], len_of[w], s_prod);
            const int64_t wn = w + g;
            nlen = -1;
            if (wn < n_work && wn >= n_heavy && light_q(wn) < n_rated) {
                const int64_t q = light_q(wn);
                nrow = row_of[q];
                nx0 = start_of[q];
                nlen = len_of[q];
            }
            continue;
        }
        const int32_t row = nrow, x0 = nx0, len = nlen;
        const int64_t wn = w + g;
        nlen = -1;
        if (wn < n_work && light_q(wn) < n_rated) {
            const int64_t q = light_q(wn);
            nrow = row_of[q];
            nx0 = start_of[q];
            nlen = len_of[q];
        }
        if (len >= 0) sq += mf_light_row<R>(a, gd, row, x0, len, lane);
    }
    const double tot = block_sum<kMfThreads>(sq, s_red);
    if (threadIdx.x == 0) a.partials[(int64_t)p * g + wgx] = tot;
}

// The minibatch error of an iteration: sqrt(sum / count) of the gradient
// kernel's per-workgroup sums of e^2, reduced in a fixed order (see
// k_mf_rmse).
struct MfRmseArgs {
    const double *partials;
    int64_t n, N;
    int32_t P, K;
    const int32_t *batch;
    const int64_t *sizes;
    double *out;
};

__device__ __forceinline__ void mf_rmse_body(const MfRmseArgs &r, double *s_red) {
    static_assert(kMfThreads == kNormThreads, "the reduction's thread count");
    const double sum = reduce_values(r.partials, r.n, false, 0.0, s_red);
    if (threadIdx.x == 0) {
        int64_t cnt = r.N;
        if (r.batch) {
            cnt = 0;
            for (int32_t p = 0; p < r.P; ++p)
                cnt += r.sizes[(int64_t)p * r.K + min(max(r.batch[p], 0), r.K - 1)];
        }
        *r.out = cnt > 0 ? sqrt(sum / (double)cnt) : 0.0;
    }
}

// The step, one element per thread and one workgroup per kMfThreads
// elements; workgroup 0 first reduces the iteration's minibatch error, which
// then overlaps the other workgroups' elements (measured on MI355X, 25M
// ratings, rank 16, 32 workers: 21 us for both against 17 + 18 us as a
// grid-stride step over the resident workgroups and a separate reduction).
__global__ __launch_bounds__(kMfThreads) void k_mf_step(int64_t m, int log2r, double eta,
                                                        double lam2,
                                                        const double *__restrict__ G,
                                                        const double *__restrict__ row_scale,
                                                        double *__restrict__ W, MfRmseArgs r) {
    __shared__ double s_red[kNormThreads / 64];
    if (blockIdx.x == 0) mf_rmse_body(r, s_red);
    const int64_t x = (int64_t)blockIdx.x * kMfThreads + threadIdx.x;
    if (x < m) {
        const double w = W[x];
        W[x] = w - eta * (G[x] * row_scale[x >> log2r] + lam2 * w);
    }
}

// sqrt(sum / count): the n partial sums of e^2 reduced in a fixed order,
// over the ratings of the minibatches used (sizes[p K + batch[p]] for each
// worker), or over N ratings when batch is NULL.
__global__ __launch_bounds__(kNormThreads) void k_mf_rmse(const double *__restrict__ partials,
                                                          int64_t n, int64_t N, int32_t P,
                                                          int32_t K,
                                                          const int32_t *__restrict__ batch,
                                                          const int64_t *__restrict__ sizes,
                                                          double *__restrict__ out) {
    __shared__ double s_red[kNormThreads / 64];
    mf_rmse_body(MfRmseArgs{partials, n, N, P, K, batch, sizes, out}, s_red);
}

// Errors of every rating at W, one lane group per rating (products in
// column order as in the gradient kernel): per-workgroup sums of e^2.
template <int R>
__global__ __launch_bounds__(kMfThreads) void k_mf_error(int64_t N, int32_t n_users,
                                                         const int32_t *__restrict__ users,
                                                         const int32_t *__restrict__ items,
                                                         const double *__restrict__ ratings,
                                                         const double *__restrict__ W,
                                                         double *__restrict__ partials) {
    __shared__ double s_red[kMfThreads / 64];
    constexpr int LPR = MfShape<R>::LPR, C = MfShape<R>::C, G = MfShape<R>::GROUPS;
    const int lane = threadIdx.x % LPR, grp = threadIdx.x / LPR;
    double sq = 0.0;
    for (int64_t k0 = (int64_t)blockIdx.x * G; k0 < N; k0 += (int64_t)gridDim.x * G) {
        const int64_t k = k0 + grp;
        const bool live = k < N;
        double ow[C], o[C];
        const int64_t u = live ? users[k] : 0, i = live ? items[k] : 0;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            ow[c] = live ? W[u * R + lane * C + c] : 0.0;
            o[c] = live ? W[((int64_t)n_users + i) * R + lane * C + c] : 0.0;
        }
        const double d = mf_dot<R>(ow, o);
        if (live && lane == 0) {
            const double err = ratings[k] - d;
            sq = sq + err * err;
        }
    }
    const double tot = block_sum<kMfThreads>(sq, s_red);
    if (threadIdx.x == 0) partials[blockIdx.x] = tot;
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
    int32_t n_users = 0, n_items = 0, rank = 0, P = 0, K = 1;
    int64_t N = 0;
    int32_t *d_oidx = nullptr;      // [2N] other factor's row, ratings of each row in storage order
    double *d_rv = nullptr;         // [2N] rating values, same order
    int32_t *d_row_of = nullptr;    // [P K E] entity of each row of each list, longest first
    int32_t *d_start_of = nullptr;  // same order: first rating in d_oidx / d_rv
    int32_t *d_len_of = nullptr;    // same order: number of ratings
    int32_t *d_n_heavy = nullptr;   // [P K] rows of more than kMfHeavy ratings, per list
    int32_t *d_n_rated = nullptr;   // [P K] rows with ratings, per list
    int64_t *d_sizes = nullptr;     // [P K] ratings of each minibatch
    int32_t *d_users = nullptr;     // [N] copies of the ratings, for ecc_mf_error
    int32_t *d_items = nullptr;
    double *d_ratings = nullptr;
    double *d_scale = nullptr;      // [n_users + n_items]: K / ratings of the row
    double *d_partials = nullptr;   // [max(grad_grid * P, err_grid)]
    int32_t grad_grid = 1, err_grid = 1;
};

extern "C" {

ecc_status_t ecc_mf_destroy(ecc_mf_t h) {
    if (!h) return ECC_OK;
    (void)hipDeviceSynchronize();
    (void)hipFree(h->d_oidx);
    (void)hipFree(h->d_rv);
    (void)hipFree(h->d_row_of);
    (void)hipFree(h->d_start_of);
    (void)hipFree(h->d_len_of);
    (void)hipFree(h->d_n_heavy);
    (void)hipFree(h->d_n_rated);
    (void)hipFree(h->d_sizes);
    (void)hipFree(h->d_users);
    (void)hipFree(h->d_items);
    (void)hipFree(h->d_ratings);
    (void)hipFree(h->d_scale);
    (void)hipFree(h->d_partials);
    delete h;
    return ECC_OK;
}

static ecc_status_t ecc_mf_create_impl(int32_t n_users, int32_t n_items, int32_t rank, int32_t P,
                                       int32_t K, int64_t N, const int32_t *d_users,
                                       const int32_t *d_items, const double *d_ratings,
                                       ecc_mf_t *out) {
    clear_error();
    ECC_ARG(out != nullptr, "out is NULL");
    *out = nullptr;
    ECC_ARG(n_users >= 1 && n_items >= 1, "need at least one user and one item");
    ECC_ARG(rank >= 1 && rank <= kMfMaxRank && (rank & (rank - 1)) == 0,
            "rank = %d must be a power of two in [1, 64]", rank);
    ECC_ARG(P >= 1, "P must be >= 1");
    ECC_ARG(K >= 1, "K must be >= 1");
    ECC_ARG(N >= 1 && 2 * N < (int64_t(1) << 31), "N must lie in [1, 2^30)");
    ECC_ARG(d_users && d_items && d_ratings, "NULL rating arrays");
    const int64_t E = (int64_t)n_users + n_items;
    const int64_t n_lists = (int64_t)P * K;
    if (n_lists * E >= (int64_t(1) << 40) || P > 65535) {
        set_error("P * K * (n_users + n_items) too large");
        return ECC_ERR_RANGE;
    }
    std::vector<int32_t> users(N), items(N);
    std::vector<double> ratings(N);
    ECC_HIP(hipMemcpy(users.data(), d_users, sizeof(int32_t) * N, hipMemcpyDeviceToHost));
    ECC_HIP(hipMemcpy(items.data(), d_items, sizeof(int32_t) * N, hipMemcpyDeviceToHost));
    ECC_HIP(hipMemcpy(ratings.data(), d_ratings, sizeof(double) * N, hipMemcpyDeviceToHost));
    std::vector<int64_t> cnt(E, 0);
    for (int64_t k = 0; k < N; ++k) {
        ECC_ARG(users[k] >= 0 && users[k] < n_users, "users[%lld] out of range", (long long)k);
        ECC_ARG(items[k] >= 0 && items[k] < n_items, "items[%lld] out of range", (long long)k);
        ++cnt[users[k]];
        ++cnt[(int64_t)n_users + items[k]];
    }
    // For every (worker p, minibatch b): the rows of all E entities, their
    // ratings of the minibatch in storage order (counting sort), stored as
    // the other factor's row and the value; then the rows by number of
    // ratings, longest first (rows of equal length in entity order): heavy
    // rows by a sort, the rest by a counting sort.
    std::vector<int32_t> oidx(2 * N), row_of(n_lists * E), start_of(n_lists * E),
        len_of(n_lists * E), n_heavy(n_lists), n_rated(n_lists);
    std::vector<int64_t> sizes(n_lists);
    std::vector<double> rv(2 * N);
    std::vector<int32_t> rp(E + 1), fill(E), heavy, by_len(kMfHeavy + 2);
    std::vector<int64_t> slot(kMfHeavy + 1);
    int64_t pos = 0;
    for (int32_t p = 0; p < P; ++p) {
        const int64_t a = N * p / P, c = N * (p + 1) / P, L = c - a;
        for (int32_t b = 0; b < K; ++b) {
            const int64_t lo = a + L * b / K, hi = a + L * (b + 1) / K;
            const int64_t list = (int64_t)p * K + b;
            sizes[list] = hi - lo;
            std::fill(fill.begin(), fill.end(), 0);
            for (int64_t k = lo; k < hi; ++k) {
                ++fill[users[k]];
                ++fill[(int64_t)n_users + items[k]];
            }
            for (int64_t e = 0; e < E; ++e) {
                rp[e] = (int32_t)pos;
                pos += fill[e];
                fill[e] = rp[e];
            }
            rp[E] = (int32_t)pos;
            for (int64_t k = lo; k < hi; ++k) {
                const int32_t xu = fill[users[k]]++;
                const int32_t xi = fill[(int64_t)n_users + items[k]]++;
                oidx[xu] = items[k];
                rv[xu] = ratings[k];
                oidx[xi] = users[k];
                rv[xi] = ratings[k];
            }
            heavy.clear();
            std::fill(by_len.begin(), by_len.end(), 0);
            for (int64_t e = 0; e < E; ++e) {
                const int32_t len = rp[e + 1] - rp[e];
                if (len > kMfHeavy) heavy.push_back((int32_t)e);
                else ++by_len[len];
            }
            std::stable_sort(heavy.begin(), heavy.end(), [&](int32_t x, int32_t y) {
                return rp[x + 1] - rp[x] > rp[y + 1] - rp[y];
            });
            int32_t *ro = row_of.data() + list * E;
            int64_t next = (int64_t)heavy.size();
            for (int32_t len = kMfHeavy; len >= 0; --len) {
                slot[len] = next;
                next += by_len[len];
            }
            for (size_t j = 0; j < heavy.size(); ++j) ro[j] = heavy[j];
            for (int64_t e = 0; e < E; ++e) {
                const int32_t len = rp[e + 1] - rp[e];
                if (len <= kMfHeavy) ro[slot[len]++] = (int32_t)e;
            }
            for (int64_t q = 0; q < E; ++q) {
                start_of[list * E + q] = rp[ro[q]];
                len_of[list * E + q] = rp[ro[q] + 1] - rp[ro[q]];
            }
            n_heavy[list] = (int32_t)heavy.size();
            n_rated[list] = (int32_t)(E - by_len[0]);
        }
    }
    std::vector<double> scale(E);
    for (int64_t e = 0; e < E; ++e) scale[e] = (double)K / (double)std::max<int64_t>(1, cnt[e]);

    ecc_mf_s *h = new (std::nothrow) ecc_mf_s();
    if (!h) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
    h->n_users = n_users;
    h->n_items = n_items;
    h->rank = rank;
    h->P = P;
    h->K = K;
    h->N = N;
    // a worker's workgroups: its share of 16 per CU (four times what the
    // device holds at once), at most one per light item of a whole list, at
    // least 1.  Measured on MI355X (25M ratings, rank 16, 32 workers: 107
    // workgroups per worker): 763 us per iteration, against 798 us with 8
    // per CU and 783-785 us with 160-512 per worker.
    const int64_t groups = kMfThreads / (rank < 4 ? 1 : rank / 4);
    h->grad_grid = std::max<int32_t>(1, mf_grid((E + groups - 1) / groups, 16) / P);
    h->err_grid = mf_grid((N + groups - 1) / groups, 8);
    const int64_t n_part = std::max<int64_t>((int64_t)h->grad_grid * P, h->err_grid);
    auto fail = [&](const char *what) {
        set_error("%s", what);
        ecc_mf_destroy(h);
        return ECC_ERR_ALLOC;
    };
    auto up = [&](void **dst, const void *src, size_t bytes) {
        if (hipMalloc(dst, std::max<size_t>(bytes, 8)) != hipSuccess) return false;
        return hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice) == hipSuccess;
    };
    if (!up((void **)&h->d_oidx, oidx.data(), sizeof(int32_t) * 2 * N) ||
        !up((void **)&h->d_rv, rv.data(), sizeof(double) * 2 * N) ||
        !up((void **)&h->d_row_of, row_of.data(), sizeof(int32_t) * n_lists * E) ||
        !up((void **)&h->d_start_of, start_of.data(), sizeof(int32_t) * n_lists * E) ||
        !up((void **)&h->d_len_of, len_of.data(), sizeof(int32_t) * n_lists * E) ||
        !up((void **)&h->d_n_heavy, n_heavy.data(), sizeof(int32_t) * n_lists) ||
        !up((void **)&h->d_n_rated, n_rated.data(), sizeof(int32_t) * n_lists) ||
        !up((void **)&h->d_sizes, sizes.data(), sizeof(int64_t) * n_lists) ||
        !up((void **)&h->d_users, users.data(), sizeof(int32_t) * N) ||
        !up((void **)&h->d_items, items.data(), sizeof(int32_t) * N) ||
        !up((void **)&h->d_ratings, ratings.data(), sizeof(double) * N) ||
        !up((void **)&h->d_scale, scale.data(), sizeof(double) * E))
        return fail("allocating or uploading the factorisation state failed");
    if (hipMalloc((void **)&h->d_partials, sizeof(double) * n_part) != hipSuccess)
        return fail("hipMalloc of the partial sums failed");
    *out = h;
    return ECC_OK;
}

// Host allocations of the set-up throw std::bad_alloc when memory runs
// out: the C ABI reports ECC_ERR_ALLOC instead of letting it escape.
ecc_status_t ecc_mf_create(int32_t n_users, int32_t n_items, int32_t rank, int32_t P, int32_t K,
                           int64_t N, const int32_t *d_users, const int32_t *d_items,
                           const double *d_ratings, ecc_mf_t *out) {
    try {
        return ecc_mf_create_impl(n_users, n_items, rank, P, K, N, d_users, d_items, d_ratings,
                                  out);
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
}

#define ECC_MF_RANKS(KERNEL, GRID, ...)                                              \
    switch (h->rank) {                                                               \
        case 1: hipLaunchKernelGGL(KERNEL<1>, GRID, dim3(kMfThreads), 0, s, __VA_ARGS__); break;   \
        case 2: hipLaunchKernelGGL(KERNEL<2>, GRID, dim3(kMfThreads), 0, s, __VA_ARGS__); break;   \
        case 4: hipLaunchKernelGGL(KERNEL<4>, GRID, dim3(kMfThreads), 0, s, __VA_ARGS__); break;   \
        case 8: hipLaunchKernelGGL(KERNEL<8>, GRID, dim3(kMfThreads), 0, s, __VA_ARGS__); break;   \
        case 16: hipLaunchKernelGGL(KERNEL<16>, GRID, dim3(kMfThreads), 0, s, __VA_ARGS__); break; \
        case 32: hipLaunchKernelGGL(KERNEL<32>, GRID, dim3(kMfThreads), 0, s, __VA_ARGS__); break; \
        case 64: hipLaunchKernelGGL(KERNEL<64>, GRID, dim3(kMfThreads), 0, s, __VA_ARGS__); break; \
        default: set_error("internal: rank %d", h->rank); return ECC_ERR_STATE;      \
    }

ecc_status_t ecc_mf_iterate(ecc_mf_t h, ecc_plan_t plan, double eta, double lam, double *d_W,
                            double *const *d_grads, double *const *d_slots, double *d_G,
                            const uint8_t *d_arrived, const int32_t *d_batch, double *d_rmse,
                            uint8_t *d_eff_out) {
    clear_error();
    ECC_ARG(h != nullptr, "factorisation state is NULL");
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    if (plan->P != h->P) {
        set_error("plan has %d ranks, the factorisation %d workers", plan->P, h->P);
        return ECC_ERR_STATE;
    }
    ECC_ARG(d_W && d_grads && d_slots && d_G && d_arrived && d_batch && d_rmse, "NULL argument");
    hipStream_t s = plan->stream;
    const int64_t E = (int64_t)h->n_users + h->n_items;
    const int64_t m = E * h->rank;
    int log2r = 0;
    while ((1 << log2r) < h->rank) ++log2r;
    MfGradArgs ga{};
    ga.n_users = h->n_users;
    ga.E = E;
    ga.K = h->K;
    ga.W = d_W;
    ga.oidx = h->d_oidx;
    ga.rv = h->d_rv;
    ga.row_of = h->d_row_of;
    ga.start_of = h->d_start_of;
    ga.len_of = h->d_len_of;
    ga.n_heavy = h->d_n_heavy;
    ga.n_rated = h->d_n_rated;
    ga.batch = d_batch;
    ga.grads = d_grads;
    ga.slots = d_slots;
    ga.ver_in = plan->d_version + (plan->clock & 1) * plan->P;
    ga.arrived = d_arrived;
    ga.t = plan->clock;
    ga.S = plan->S;
    ga.partials = h->d_partials;
    {
        TimedLaunch timed(plan, ECC_TIMING_MF_GRAD);
        ga.g = h->grad_grid;
        ga.pin = (h->P % 8) == 0;
        const dim3 grid((unsigned)((int64_t)h->grad_grid * h->P));
        ECC_MF_RANKS(k_mf_grad, grid, ga)
        ECC_LAUNCH_CHECK();
    }
    // every contribution is read from its slot: the taken ones were written
    // there by the gradient kernel
    st = ecc_allreduce_partial(plan, m, d_slots, d_slots, d_G, d_arrived, d_eff_out, nullptr);
    if (st != ECC_OK) return st;
    {
        TimedLaunch timed(plan, ECC_TIMING_MF_STEP);
        const MfRmseArgs r{h->d_partials, (int64_t)h->grad_grid * h->P, h->N, h->P, h->K,
                           d_batch, h->d_sizes, d_rmse};
        const int64_t sg = std::max<int64_t>(1, (m + kMfThreads - 1) / kMfThreads);
        if (sg > 0x7fffffff) {
            set_error("model too large for one step launch");
            return ECC_ERR_RANGE;
        }
        hipLaunchKernelGGL(k_mf_step, dim3((unsigned)sg), dim3(kMfThreads), 0, s, m, log2r, eta,
                           2.0 * lam, d_G, h->d_scale, d_W, r);
    }
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

ecc_status_t ecc_mf_error(ecc_mf_t h, const double *d_W, double *d_rmse, void *hip_stream) {
    clear_error();
    ECC_ARG(h != nullptr, "factorisation state is NULL");
    ECC_ARG(d_W && d_rmse, "NULL argument");
    hipStream_t s = (hipStream_t)hip_stream;
    ECC_MF_RANKS(k_mf_error, dim3(h->err_grid), h->N, h->n_users, h->d_users, h->d_items,
                 h->d_ratings, d_W, h->d_partials)
    ECC_LAUNCH_CHECK();
    hipLaunchKernelGGL(k_mf_rmse, dim3(1), dim3(kNormThreads), 0, s, h->d_partials,
                       (int64_t)h->err_grid, h->N, h->P, h->K, nullptr, nullptr, d_rmse);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

}  // extern "C"
