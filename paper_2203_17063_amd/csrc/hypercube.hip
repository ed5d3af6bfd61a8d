// SSP hypercube allreduce with one view per receiver (Section III-A,
// Algorithm 1): P = 2^d virtual processes on one GPU, each with d dedicated
// receive slots (data and clock of the last message that landed there).
//
// One call is one iteration of every process, as one kernel launch:
//  (1) every workgroup replays the scalar part of the call in LDS -- which
//      slot of which process takes this call's message from its partner
//      (process XOR 2^k) and which reuses its last message -- from the slot
//      clocks of the previous call (read-only in this launch; workgroup 0
//      writes the new ones into the other half of a double buffer);
//  (2) the data part is elementwise: element j of every result depends only
//      on element j of the contributions and slots, so one thread (or a few
//      lanes) carries element j of all P partial reductions through the d
//      steps, storing each arriving message into its slot and reading each
//      reused slot, and no workgroup waits for another.
// A partial reduction is updated as partial + received, in that order, in
// fp64 without contraction: the same operations as the sequential
// definition, so results are bitwise reproducible.
#include <algorithm>

#include <new>

#include "ecc_common.h"

namespace ecc {

// Contributions, slots and results are each touched once per call and the
// slots of all processes (P d m doubles) far exceed the caches: non-temporal
// accesses (measured on MI355X, 32 processes x 16 MB: 973 us against 1,019
// us with ordinary ones).
__device__ __forceinline__ void hc_st(double *p, double v) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ double hc_ld(const double *p) { return __builtin_nontemporal_load(p); }

constexpr int kHcThreads = 256;
constexpr int kHcMaxDims = 5;  // P <= 32: one launch, one lane per process in the scalar phase
constexpr int kHcMaxDimsBig = 12;  // P <= 4096: decisions, sub-cubes, then step by step
constexpr int kHcCubeDims = 5;     // sub-cubes of 32 processes in the P > 32 path
constexpr int kHcDecideThreads = 1024;
constexpr int32_t kHcNever = INT32_MIN;  // clock of a slot that was never written

struct HcArgs {
    int32_t P, D, slack;
    int32_t t;
    int64_t m;
    const double *contrib;      // [P][m]
    const uint8_t *delivered;   // [P][D]: the partner's message of this call has landed
    double *slots;              // [P][D][m]
    const int32_t *clk_in;      // [P][D] slot clocks before the call
    int32_t *clk_out;           // [P][D] after the call (workgroup 0)
    unsigned long long *waits;  // [P][D] cumulative waits (workgroup 0)
    double *result;             // [P][m] (may alias contrib)
    int32_t *result_clock;      // [P] or null (workgroup 0)
    uint8_t *outcome;           // [P][D] or null (workgroup 0)
};

// Scalar phase on wave 0, lane r = process r.  Returns nothing; leaves in
// s_fresh[k] the set of processes whose slot k takes this call's message.
__device__ __forceinline__ void hc_decide(const HcArgs &a, unsigned long long *s_fresh) {
    const int lane = threadIdx.x;
    if (lane >= 64) return;
    const bool live = lane < a.P;
    // slack is at most INT32_MAX; ECC_UNBOUNDED accepts every received message
    const int64_t min_accepted =
        a.slack == ECC_UNBOUNDED ? INT64_MIN : (int64_t)a.t - (int64_t)a.slack;
    int32_t pc = a.t;  // clock of this process's partial reduction
    for (int k = 0; k < a.D; ++k) {
        const int partner = lane ^ (1 << k);
        const int32_t sent_clock = __shfl(pc, partner, 64);
        int32_t sc = live ? a.clk_in[lane * a.D + k] : 0;
        const bool arrived = live && a.delivered[lane * a.D + k] != 0;
        uint8_t how;
        if (arrived) how = 1;                                   // delivered
        else if (sc == kHcNever) how = 3;                       // first receipt: wait
        else if ((int64_t)sc < min_accepted) how = 2;           // too old: wait
        else how = 0;                                           // reuse the slot
        const bool fresh = live && how != 0;
        if (fresh) sc = sent_clock;
        const unsigned long long mask = __ballot(fresh);
        if (lane == 0) s_fresh[k] = mask;
        if (live) pc = min(pc, sc);
        if (blockIdx.x == 0 && live) {
            a.clk_out[lane * a.D + k] = sc;
            if (how == 2) a.waits[lane * a.D + k] += 1;
            if (a.outcome) a.outcome[lane * a.D + k] = how;
        }
    }
    if (blockIdx.x == 0 && live && a.result_clock) a.result_clock[lane] = pc;
}

__device__ __forceinline__ unsigned long long uniform64(unsigned long long v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((unsigned long long)hi << 32) | lo;
}

// Column layout: a thread carries element j of all P = 2^D partial
// reductions in registers (P <= 32), so every load and store of a wave
// covers contiguous bytes of one row.  At step k the two processes of each
// pair (r, r XOR 2^k) sit in the same thread and are updated together from
// their old partials.  A scheduling barrier between steps keeps the loads of
// a step from being hoisted above the stores of the previous one (register
// pressure).  The grid has one thread per element and no loop: a loop over
// elements kept every row address live across it, and the 224 addresses of
// P = 32 then spilled 620 SGPRs (942 against 933 us per call).  Measured on
// MI355X (slack 2, 80 % delivery): P = 32 x 16 MB, 166 VGPRs, 4.03 TB/s.
// Sixty-four processes take the multi-launch path below: 1,202 us per call
// of 8 MB vectors, against 1,530 us with all 64 partials of an element in
// one thread (255 VGPRs, one wave per SIMD), and slower still with two lanes
// per element, whose per-lane delivery bits make every slot access divergent.
template <int D>
__global__ __launch_bounds__(kHcThreads) void k_allreduce_ssp(HcArgs a) {
    constexpr int Pt = 1 << D;
    __shared__ unsigned long long s_fresh[kHcMaxDims];
    hc_decide(a, s_fresh);
    __syncthreads();
    unsigned long long fresh[D > 0 ? D : 1];
#pragma unroll
    for (int k = 0; k < D; ++k) fresh[k] = uniform64(s_fresh[k]);
    const int64_t m = a.m;
    const int64_t j = (int64_t)blockIdx.x * kHcThreads + threadIdx.x;
    if (j < m) {
        double part[Pt];
#pragma unroll
        for (int i = 0; i < Pt; ++i) part[i] = hc_ld(a.contrib + i * m + j);
#pragma unroll
        for (int k = 0; k < D; ++k) {
            double *srow = a.slots + (int64_t)k * m + j;  // + r * D * m
            const int bit = 1 << k;
#pragma unroll
            for (int i = 0; i < Pt; ++i) {
                if (i & bit) continue;
                const int q = i | bit;
                const bool fr = (fresh[k] >> i) & 1ull, fq = (fresh[k] >> q) & 1ull;
                double *sr = srow + (int64_t)i * D * m, *sq = srow + (int64_t)q * D * m;
                const double gr = fr ? part[q] : hc_ld(sr);
                const double gq = fq ? part[i] : hc_ld(sq);
                if (fr) hc_st(sr, gr);
                if (fq) hc_st(sq, gq);
                part[i] = part[i] + gr;
                part[q] = part[q] + gq;
            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int i = 0; i < Pt; ++i) hc_st(a.result + i * m + j, part[i]);
    }
}

// More than 32 processes.  One call is then three kinds of launch:
//  (1) k_hc_decide_big, one workgroup: process r's thread replays its d
//      steps in order (its partner's partial clock read from LDS after every
//      step), writes the (process, step) fresh flags for the data kernels
//      and the same bookkeeping as hc_decide;
//  (2) k_hc_cube: the first five steps inside every sub-cube of 32
//      processes (partners r XOR 2^k, k < 5, share the sub-cube), a thread
//      carrying element j of the sub-cube's 32 partials in registers as
//      k_allreduce_ssp<5> does, the partials then stored in the result;
//  (3) k_hc_pair_step for every further step k: a thread takes element j of
//      one pair (r, r XOR 2^k) of partials from the result, receives for
//      each from the partner's partial or its slot, and stores both
//      partial + received.
// The additions are those of the one-launch kernel, in the same order.
__global__ __launch_bounds__(kHcDecideThreads) void k_hc_decide_big(HcArgs a,
                                                                    uint8_t *__restrict__ fresh) {
    __shared__ int32_t s_pc[2][1 << kHcMaxDimsBig];
    const int64_t min_accepted =
        a.slack == ECC_UNBOUNDED ? INT64_MIN : (int64_t)a.t - (int64_t)a.slack;
    for (int32_t r = threadIdx.x; r < a.P; r += kHcDecideThreads) s_pc[0][r] = a.t;
    __syncthreads();
    for (int k = 0; k < a.D; ++k) {
        const int cur = k & 1;
        for (int32_t r = threadIdx.x; r < a.P; r += kHcDecideThreads) {
            const int32_t sent_clock = s_pc[cur][r ^ (1 << k)];
            const int64_t sk = (int64_t)r * a.D + k;
            int32_t sc = a.clk_in[sk];
            const bool arrived = a.delivered[sk] != 0;
            uint8_t how;
            if (arrived) how = 1;                              // delivered
            else if (sc == kHcNever) how = 3;                  // first receipt: wait
            else if ((int64_t)sc < min_accepted) how = 2;      // too old: wait
            else how = 0;                                      // reuse the slot
            if (how != 0) sc = sent_clock;
            fresh[sk] = how != 0 ? 1 : 0;
            s_pc[cur ^ 1][r] = min(s_pc[cur][r], sc);
            a.clk_out[sk] = sc;
            if (how == 2) a.waits[sk] += 1;
            if (a.outcome) a.outcome[sk] = how;
        }
        __syncthreads();
    }
    if (a.result_clock)
        for (int32_t r = threadIdx.x; r < a.P; r += kHcDecideThreads)
            a.result_clock[r] = s_pc[a.D & 1][r];
}

// Steps 0 .. kHcCubeDims-1 of sub-cube blockIdx.y (processes 32 y .. 32 y +
// 31); element blockIdx.x * kHcThreads + threadIdx.x.
__global__ __launch_bounds__(kHcThreads) void k_hc_cube(HcArgs a,
                                                        const uint8_t *__restrict__ fresh_in) {
    constexpr int DL = kHcCubeDims, Pt = 1 << DL;
    __shared__ unsigned long long s_fresh[DL];
    const int32_t p0 = (int32_t)blockIdx.y * Pt;
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        for (int k = 0; k < DL; ++k) {
            const bool f = lane < Pt && fresh_in[(int64_t)(p0 + lane) * a.D + k] != 0;
            const unsigned long long mask = __ballot(f);
            if (lane == 0) s_fresh[k] = mask;
        }
    }
    __syncthreads();
    unsigned long long fresh[DL];
#pragma unroll
    for (int k = 0; k < DL; ++k) fresh[k] = uniform64(s_fresh[k]);
    const int64_t m = a.m;
    const int64_t j = (int64_t)blockIdx.x * kHcThreads + threadIdx.x;
    if (j >= m) return;
    double part[Pt];
#pragma unroll
    for (int i = 0; i < Pt; ++i) part[i] = hc_ld(a.contrib + (int64_t)(p0 + i) * m + j);
#pragma unroll
    for (int k = 0; k < DL; ++k) {
        double *srow = a.slots + ((int64_t)p0 * a.D + k) * m + j;  // + i * D * m
        const int bit = 1 << k;
#pragma unroll
        for (int i = 0; i < Pt; ++i) {
            if (i & bit) continue;
            const int q = i | bit;
            const bool fr = (fresh[k] >> i) & 1ull, fq = (fresh[k] >> q) & 1ull;
            double *sr = srow + (int64_t)i * a.D * m, *sq = srow + (int64_t)q * a.D * m;
            const double gr = fr ? part[q] : hc_ld(sr);
            const double gq = fq ? part[i] : hc_ld(sq);
            if (fr) hc_st(sr, gr);
            if (fq) hc_st(sq, gq);
            part[i] = part[i] + gr;
            part[q] = part[q] + gq;
        }
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < Pt; ++i) hc_st(a.result + (int64_t)(p0 + i) * m + j, part[i]);
}

// Step k >= kHcCubeDims for pair blockIdx.y of the partials in the result.
__global__ __launch_bounds__(kHcThreads) void k_hc_pair_step(HcArgs a,
                                                             const uint8_t *__restrict__ fresh_in,
                                                             int32_t k) {
    const int64_t pi = blockIdx.y;
    const int32_t bit = 1 << k;
    const int32_t r = (int32_t)(((pi >> k) << (k + 1)) | (pi & (bit - 1)));
    const int32_t q = r | bit;
    const bool fr = fresh_in[(int64_t)r * a.D + k] != 0, fq = fresh_in[(int64_t)q * a.D + k] != 0;
    const int64_t m = a.m;
    const int64_t j = (int64_t)blockIdx.x * kHcThreads + threadIdx.x;
    if (j >= m) return;
    double *pr = a.result + (int64_t)r * m + j, *pq = a.result + (int64_t)q * m + j;
    double *sr = a.slots + ((int64_t)r * a.D + k) * m + j;
    double *sq = a.slots + ((int64_t)q * a.D + k) * m + j;
    const double xr = hc_ld(pr), xq = hc_ld(pq);
    const double gr = fr ? xq : hc_ld(sr);
    const double gq = fq ? xr : hc_ld(sq);
    if (fr) hc_st(sr, gr);
    if (fq) hc_st(sq, gq);
    hc_st(pr, xr + gr);
    hc_st(pq, xq + gq);
}

}  // namespace ecc

using namespace ecc;

struct ecc_hypercube_s {
    int32_t P = 0, D = 0, slack = 0;
    int64_t m = 0;
    int64_t clock = 0;
    hipStream_t stream = nullptr;
    int32_t grid = 1;
    double *d_slots = nullptr;               // [P][D][m]
    int32_t *d_clk = nullptr;                // [2][P][D]
    unsigned long long *d_waits = nullptr;   // [P][D]
    uint8_t *d_fresh = nullptr;              // P > 64: [P][D] this call's fresh slots
};

namespace {

__global__ void k_hc_reset(int32_t n, int32_t *clk, unsigned long long *waits) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        clk[i] = kHcNever;
        clk[n + i] = kHcNever;
        waits[i] = 0;
    }
}

ecc_status_t hc_reset(ecc_hypercube_t h) {
    const int32_t n = h->P * h->D;
    if (n > 0) {
        hipLaunchKernelGGL(k_hc_reset, dim3(1), dim3(256), 0, h->stream, n, h->d_clk, h->d_waits);
        ECC_LAUNCH_CHECK();
    }
    h->clock = 0;
    return ECC_OK;
}

template <int D>
void hc_launch(dim3 grid, hipStream_t st, const HcArgs &a) {
    hipLaunchKernelGGL((k_allreduce_ssp<D>), grid, dim3(kHcThreads), 0, st, a);
}

}  // namespace

extern "C" {

ecc_status_t ecc_hypercube_create(int32_t P, int64_t m, int32_t slack, void *hip_stream,
                                  ecc_hypercube_t *out) {
    clear_error();
    ECC_ARG(out != nullptr, "out is NULL");
    *out = nullptr;
    ECC_ARG(P >= 1 && P <= (1 << kHcMaxDimsBig) && (P & (P - 1)) == 0,
            "P = %d must be a power of two in [1, %d]", P, 1 << kHcMaxDimsBig);
    ECC_ARG(m >= 0, "m must be >= 0");
    ECC_ARG(slack >= 0, "slack must be >= 0 (ECC_UNBOUNDED for no limit)");
    int D = 0;
    while ((1 << D) < P) ++D;
    const int64_t slot_elems = (int64_t)P * D * m;
    if (m > (int64_t(1) << 40) / std::max(1, P * std::max(D, 1))) {
        set_error("P * d * m too large");
        return ECC_ERR_RANGE;
    }
    // one thread per element: the grid's x extent holds at most 2^31 - 1 workgroups
    if (m > (int64_t)0x7fffffff * kHcThreads) {
        set_error("m too large");
        return ECC_ERR_RANGE;
    }
    ecc_hypercube_s *h = new (std::nothrow) ecc_hypercube_s();
    if (!h) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
    h->P = P;
    h->D = D;
    h->m = m;
    h->slack = slack;
    h->stream = (hipStream_t)hip_stream;
    auto fail = [&](const char *what) {
        set_error("%s", what);
        ecc_hypercube_destroy(h);
        return ECC_ERR_ALLOC;
    };
    if (slot_elems > 0 && hipMalloc((void **)&h->d_slots, sizeof(double) * slot_elems) != hipSuccess)
        return fail("hipMalloc of the receive slots failed");
    const int32_t n = P * D;
    if (n > 0) {
        if (hipMalloc((void **)&h->d_clk, sizeof(int32_t) * 2 * n) != hipSuccess)
            return fail("hipMalloc of the slot clocks failed");
        if (hipMalloc((void **)&h->d_waits, sizeof(unsigned long long) * n) != hipSuccess)
            return fail("hipMalloc of the wait counters failed");
        if (D > kHcMaxDims && hipMalloc((void **)&h->d_fresh, n) != hipSuccess)
            return fail("hipMalloc of the fresh flags failed");
    }
    // grid: one workgroup per pass over its elements (measured on MI355X,
    // 32 processes x 16 MB: 945 us, against 974 us with the resident
    // workgroups walking the vector)
    const int64_t per_wg = kHcThreads;  // elements of one workgroup
    h->grid = (int32_t)std::max<int64_t>(1, (m + per_wg - 1) / per_wg);
    ecc_status_t st = hc_reset(h);
    if (st != ECC_OK) {
        ecc_hypercube_destroy(h);
        return st;
    }
    *out = h;
    return ECC_OK;
}

ecc_status_t ecc_hypercube_destroy(ecc_hypercube_t h) {
    if (!h) return ECC_OK;
    (void)hipStreamSynchronize(h->stream);
    (void)hipFree(h->d_slots);
    (void)hipFree(h->d_clk);
    (void)hipFree(h->d_waits);
    (void)hipFree(h->d_fresh);
    delete h;
    return ECC_OK;
}

ecc_status_t ecc_hypercube_reset(ecc_hypercube_t h) {
    clear_error();
    ECC_ARG(h != nullptr, "hypercube is NULL");
    return hc_reset(h);
}

ecc_status_t ecc_allreduce_ssp(ecc_hypercube_t h, const double *d_contrib,
                               const uint8_t *d_delivered, double *d_result,
                               int32_t *d_result_clock, uint8_t *d_outcome) {
    clear_error();
    ECC_ARG(h != nullptr, "hypercube is NULL");
    ECC_ARG(h->m == 0 || (d_contrib && d_result), "NULL contribution or result");
    ECC_ARG(h->D == 0 || d_delivered, "d_delivered is NULL");
    if (h->clock >= INT32_MAX - 1) {
        set_error("clock overflow");
        return ECC_ERR_RANGE;
    }
    if (h->m > 0 && d_result != d_contrib) {
        const uintptr_t a0 = (uintptr_t)d_contrib, a1 = a0 + 8 * (uintptr_t)h->P * h->m;
        const uintptr_t b0 = (uintptr_t)d_result, b1 = b0 + 8 * (uintptr_t)h->P * h->m;
        ECC_ARG(a1 <= b0 || b1 <= a0, "result overlaps the contributions without being them");
    }
    HcArgs a{};
    a.P = h->P;
    a.D = h->D;
    a.slack = h->slack;
    a.t = (int32_t)h->clock;
    a.m = h->m;
    a.contrib = d_contrib;
    a.delivered = d_delivered;
    a.slots = h->d_slots;
    const int32_t n = h->P * h->D;
    a.clk_in = h->d_clk ? h->d_clk + (h->clock & 1) * n : nullptr;
    a.clk_out = h->d_clk ? h->d_clk + ((h->clock + 1) & 1) * n : nullptr;
    a.waits = h->d_waits;
    a.result = d_result;
    a.result_clock = d_result_clock;
    a.outcome = d_outcome;
    const dim3 grid(h->grid);
    if (h->D > kHcMaxDims) {
        // decisions, the sub-cubes' steps, then one launch per further step
        hipLaunchKernelGGL(k_hc_decide_big, dim3(1), dim3(kHcDecideThreads), 0, h->stream, a,
                           h->d_fresh);
        ECC_LAUNCH_CHECK();
        hipLaunchKernelGGL(k_hc_cube, dim3(h->grid, h->P >> kHcCubeDims), dim3(kHcThreads), 0,
                           h->stream, a, h->d_fresh);
        ECC_LAUNCH_CHECK();
        for (int32_t k = kHcCubeDims; k < h->D; ++k) {
            hipLaunchKernelGGL(k_hc_pair_step, dim3(h->grid, h->P / 2), dim3(kHcThreads), 0,
                               h->stream, a, h->d_fresh, k);
            ECC_LAUNCH_CHECK();
        }
        h->clock += 1;
        return ECC_OK;
    }
    switch (h->D) {
        case 0: hc_launch<0>(grid, h->stream, a); break;
        case 1: hc_launch<1>(grid, h->stream, a); break;
        case 2: hc_launch<2>(grid, h->stream, a); break;
        case 3: hc_launch<3>(grid, h->stream, a); break;
        case 4: hc_launch<4>(grid, h->stream, a); break;
        default: hc_launch<5>(grid, h->stream, a); break;
    }
    ECC_LAUNCH_CHECK();
    h->clock += 1;
    return ECC_OK;
}

static ecc_status_t ecc_hypercube_stats_impl(ecc_hypercube_t h, int64_t *clock, uint64_t *waits_total,
                                 int32_t *h_slot_clock, uint64_t *h_waits) {
    clear_error();
    ECC_ARG(h != nullptr, "hypercube is NULL");
    const int32_t n = h->P * h->D;
    std::vector<int32_t> clk(n);
    std::vector<unsigned long long> w(n);
    if (n > 0) {
        ECC_HIP(hipStreamSynchronize(h->stream));
        ECC_HIP(hipMemcpy(clk.data(), h->d_clk + (h->clock & 1) * n, sizeof(int32_t) * n,
                          hipMemcpyDeviceToHost));
        ECC_HIP(hipMemcpy(w.data(), h->d_waits, sizeof(unsigned long long) * n,
                          hipMemcpyDeviceToHost));
    }
    if (clock) *clock = h->clock;
    uint64_t tot = 0;
    for (int32_t i = 0; i < n; ++i) tot += w[i];
    if (waits_total) *waits_total = tot;
    if (h_slot_clock)
        for (int32_t i = 0; i < n; ++i) h_slot_clock[i] = clk[i];
    if (h_waits)
        for (int32_t i = 0; i < n; ++i) h_waits[i] = w[i];
    return ECC_OK;
}

// Host allocations of the set-up throw std::bad_alloc when memory runs
// out: the C ABI reports ECC_ERR_ALLOC instead of letting it escape.
ecc_status_t ecc_hypercube_stats(ecc_hypercube_t h, int64_t *clock, uint64_t *waits_total,
                                 int32_t *h_slot_clock, uint64_t *h_waits) {
    try {
        return ecc_hypercube_stats_impl(h, clock, waits_total, h_slot_clock, h_waits);
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
}

}  // extern "C"
