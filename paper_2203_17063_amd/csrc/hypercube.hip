// SSP hypercube allreduce with one view per receiver (Section III-A,
// Algorithm 1): P = 2^d virtual processes on one GPU, each with d dedicated
// receive slots (data and clock of the last message that landed there).
//
// One call is one iteration of every process, as one kernel launch (up to
// 32 processes; beyond, see k_hc_decide_big):
//  (1) every workgroup replays the scalar part of the call in LDS -- which
//      slot of which process takes this call's message from its partner
//      (process XOR 2^k) and which reuses its last message -- from the slot
//      clocks of the previous call (read-only in this launch; workgroup 0
//      writes the new ones into the other half of a double buffer);
//  (2) the data part is elementwise: element j of every result depends only
//      on element j of the contributions and slots, so one thread (up to 4
//      processes) or one lane of each of four waves (8 to 32) carries element
//      j of all P partial reductions through the d steps, storing each
//      arriving message into its slot and reading each reused slot, and no
//      workgroup waits for another.
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

// Column layout, for up to 4 processes: a thread carries element j of all
// P = 2^D partial reductions in registers, so every load and store of a wave
// covers contiguous bytes of one row.  At step k the two processes of each
// pair (r, r XOR 2^k) sit in the same thread and are updated together from
// their old partials.  A scheduling barrier between steps keeps the loads of
// a step from being hoisted above the stores of the previous one (register
// pressure).  The grid has one thread per element and no loop (a loop over
// elements kept every row address live across it).
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

// Split layout, for 8 to 32 processes and for the 32-process sub-cubes of
// larger calls: the 2^D partials of element j are held by the W = 2^LW
// waves of a workgroup, 2^D / W each (wave w holds processes w 2^D / W + i),
// so that every decision stays uniform in a wave and a thread holds few
// partials.  Steps 0 .. D-LW-1 pair processes within a wave; each of the
// last LW steps pairs process w 2^D / W + i with the same i of wave
// w XOR 2^(k-D+LW), whose old partials the waves exchange through LDS.  The
// additions are those of k_allreduce_ssp, in the same order.  With CUBE,
// blockIdx.y selects the sub-cube of processes 2^D y .. 2^D (y + 1) - 1,
// whose fresh flags for steps 0 .. D-1 come from fresh_in, and the partials
// go to the result for the remaining steps.  Measured on MI355X (32
// processes x 16 MB, slack 2, 80 % delivery): 789 us per call with four
// waves (50 VGPRs, 8 waves per SIMD), 885 us with two (90 VGPRs), 827 us
// with eight, against 937 us with the 32 partials in one thread.
template <int D, int LW, bool CUBE>
__global__ __launch_bounds__(64 << LW) void k_allreduce_ssp_split(HcArgs a,
                                                                  const uint8_t *__restrict__ fresh_in) {
    constexpr int Pt = 1 << D, W = 1 << LW, H = Pt / W;
    static_assert(LW >= 1 && LW < D && D <= kHcMaxDims, "a split of at most 32 processes");
    __shared__ unsigned long long s_fresh[kHcMaxDims];
    __shared__ double s_x[W][H][64];
    const int32_t pc = CUBE ? (int32_t)blockIdx.y * Pt : 0;  // the sub-cube's first process
    if constexpr (CUBE) {
        if (threadIdx.x < 64) {
            const int lane = threadIdx.x;
            for (int k = 0; k < D; ++k) {
                const bool f = lane < Pt && fresh_in[(int64_t)(pc + lane) * a.D + k] != 0;
                const unsigned long long mask = __ballot(f);
                if (lane == 0) s_fresh[k] = mask;
            }
        }
    } else {
        hc_decide(a, s_fresh);
    }
    __syncthreads();
    unsigned long long fresh[D];
#pragma unroll
    for (int k = 0; k < D; ++k) fresh[k] = uniform64(s_fresh[k]);
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t m = a.m;
    const int64_t sd = CUBE ? (int64_t)a.D : D;  // slots per process
    const int64_t j = (int64_t)blockIdx.x * 64 + lane;
    const bool live = j < m;
    const int p0 = wv * H;  // this wave's first process in the (sub-)cube
    auto slot = [&](int i, int k) { return a.slots + ((int64_t)(pc + p0 + i) * sd + k) * m + j; };
    double part[H];
#pragma unroll
    for (int i = 0; i < H; ++i)
        part[i] = live ? hc_ld(a.contrib + (int64_t)(pc + p0 + i) * m + j) : 0.0;
#pragma unroll
    for (int k = 0; k < D - LW; ++k) {
        const int bit = 1 << k;
#pragma unroll
        for (int i = 0; i < H; ++i) {
            if (i & bit) continue;
            const int q = i | bit;
            const bool fr = (fresh[k] >> (p0 + i)) & 1ull, fq = (fresh[k] >> (p0 + q)) & 1ull;
            double *sr = slot(i, k), *sq = slot(q, k);
            const double gr = fr ? part[q] : (live ? hc_ld(sr) : 0.0);
            const double gq = fq ? part[i] : (live ? hc_ld(sq) : 0.0);
            if (fr && live) hc_st(sr, gr);
            if (fq && live) hc_st(sq, gq);
            part[i] = part[i] + gr;
            part[q] = part[q] + gq;
        }
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int k = D - LW; k < D; ++k) {
        const int pw = wv ^ (1 << (k - (D - LW)));  // the partner wave
#pragma unroll
        for (int i = 0; i < H; ++i) s_x[wv][i][lane] = part[i];
        __syncthreads();
#pragma unroll
        for (int i = 0; i < H; ++i) {
            const bool fr = (fresh[k] >> (p0 + i)) & 1ull;
            double *sr = slot(i, k);
            const double gr = fr ? s_x[pw][i][lane] : (live ? hc_ld(sr) : 0.0);
            if (fr && live) hc_st(sr, gr);
            part[i] = part[i] + gr;
        }
        if (k + 1 < D) __syncthreads();  // every partner read before the next writes
    }
    if (live) {
#pragma unroll
        for (int i = 0; i < H; ++i) hc_st(a.result + (int64_t)(pc + p0 + i) * m + j, part[i]);
    }
}

// More than 32 processes.  One call is then three kinds of launch:
//  (1) k_hc_decide_big, one workgroup: process r's thread replays its d
//      steps in order (its partner's partial clock read from LDS after every
//      step), writes the (process, step) fresh flags for the data kernels
//      and the same bookkeeping as hc_decide;
//  (2) k_allreduce_ssp_split<5, 2, true>: the first five steps inside every
//      sub-cube of 32 processes (partners r XOR 2^k, k < 5, share the
//      sub-cube) in the split layout, the partials then stored in the result;
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
    uint8_t *d_fresh = nullptr;              // P > 32: [P][D] this call's fresh slots
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

constexpr int kHcSplitLW = 2;  // four waves per 64 elements

template <int D>
void hc_launch_split(int64_t m, hipStream_t st, const HcArgs &a) {
    const int64_t g = std::max<int64_t>(1, (m + 63) / 64);
    hipLaunchKernelGGL((k_allreduce_ssp_split<D, kHcSplitLW, false>), dim3((unsigned)g),
                       dim3(64 << kHcSplitLW), 0, st, a, nullptr);
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
    // one thread per element and at most 64 elements per workgroup: the
    // grid's x extent holds at most 2^31 - 1 workgroups
    if (m > (int64_t)0x7fffffff * 64) {
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
        const int64_t g = std::max<int64_t>(1, (h->m + 63) / 64);
        hipLaunchKernelGGL((k_allreduce_ssp_split<kHcCubeDims, kHcSplitLW, true>),
                           dim3((unsigned)g, h->P >> kHcCubeDims), dim3(64 << kHcSplitLW), 0,
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
        case 3: hc_launch_split<3>(h->m, h->stream, a); break;
        case 4: hc_launch_split<4>(h->m, h->stream, a); break;
        default: hc_launch_split<5>(h->m, h->stream, a); break;
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
