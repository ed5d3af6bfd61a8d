// Collectives of one clock step on P virtual ranks in HBM:
//   - the staleness decision of Algorithm 1 (fused into both kernels below),
//   - allgatherv-style assembly into the last-received vector,
//   - the partial allreduce with stale substitution and the min-clock rule.
//
// Both kernels read the versions of the previous step from one half of a
// double buffer and write the new versions to the other half, so the
// workgroups that copy or reduce data (which all evaluate the decision for
// the ranks they touch) never race with the workgroup that records it.
#include <algorithm>

#include "ecc_common.h"

namespace ecc {

// Assembly: workgroup 0 records the step; workgroup 1 + k copies tile k if
// its rank's block is taken at this step.  Copies use 16-byte accesses when
// source and destination have the same alignment modulo 16 bytes.
__global__ __launch_bounds__(kAssembleThreads) void k_assemble(
    int32_t P, int32_t S, int64_t t, const uint8_t *__restrict__ arrived,
    const int32_t *__restrict__ ver_in, int32_t *__restrict__ ver_out,
    int32_t *__restrict__ age_state, uint8_t *__restrict__ eff_state,
    unsigned long long *__restrict__ forced, uint8_t *__restrict__ eff_user,
    int32_t *__restrict__ age_user, const Tile *__restrict__ tiles,
    const int64_t *__restrict__ displs, const double *const *__restrict__ send_ptrs,
    const double *__restrict__ send_base, double *__restrict__ recv,
    const int32_t *__restrict__ done) {
    if (done && *done) return;
    if (blockIdx.x == 0) {
        record_step(P, S, t, arrived, ver_in, ver_out, age_state, eff_state, forced, eff_user,
                    age_user, nullptr);
        return;
    }
    const Tile tile = tiles[blockIdx.x - 1];
    const int32_t p = tile.rank;
    if (!stale_select(ver_in[p], arrived[p], t, S)) return;
    const int64_t d0 = displs[p];
    const double *src = (send_ptrs ? send_ptrs[p] : send_base + d0) + tile.off;
    double *dst = recv + d0 + tile.off;
    const int32_t len = tile.len;
    const int tid = threadIdx.x;
    if ((((uintptr_t)src ^ (uintptr_t)dst) & 15) == 0) {
        const int32_t h = (((uintptr_t)dst & 15) != 0 && len > 0) ? 1 : 0;
        if (tid == 0 && h) dst[0] = src[0];
        const int32_t body = len - h;
        const int32_t npair = body >> 1;
        const double2 *s2 = reinterpret_cast<const double2 *>(src + h);
        double2 *d2 = reinterpret_cast<double2 *>(dst + h);
        static_assert(kAssembleTile / 2 / kAssembleThreads == 4, "four pairs per thread");
        // reads are clamped into range so that all four are in flight together
        if (npair > 0) {
            const int32_t last = npair - 1;
            const int32_t k0 = tid, k1 = tid + kAssembleThreads, k2 = tid + 2 * kAssembleThreads,
                          k3 = tid + 3 * kAssembleThreads;
            const double2 v0 = s2[min(k0, last)], v1 = s2[min(k1, last)],
                          v2 = s2[min(k2, last)], v3 = s2[min(k3, last)];
            if (k0 < npair) d2[k0] = v0;
            if (k1 < npair) d2[k1] = v1;
            if (k2 < npair) d2[k2] = v2;
            if (k3 < npair) d2[k3] = v3;
        }
        if (tid == 0 && (body & 1)) dst[len - 1] = src[len - 1];
    } else {
        static_assert(kAssembleTile / kAssembleThreads == 8, "eight elements per thread");
        if (len > 0) {
            const int32_t last = len - 1;
            double v[8];
            // fully unrolled with clamped reads: the array lives in registers
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = src[min(tid + u * kAssembleThreads, last)];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int32_t k = tid + u * kAssembleThreads;
                if (k < len) dst[k] = v[u];
            }
        }
    }
}

// Partial allreduce: workgroup 0 records the step; every other workgroup owns
// kReduceThreads * kReduceElems consecutive elements and, for p = 0..P-1 in
// order, takes the fresh contribution of eff ranks (writing it to the rank's
// slot) or the slot of the others, summing in rank order.  A contribution
// that its producer wrote into the slot itself (fresh[p] == slots[p]) is
// read there and not written back.
__global__ __launch_bounds__(kReduceThreads) void k_allreduce(
    int32_t P, int32_t S, int64_t t, const uint8_t *__restrict__ arrived,
    const int32_t *__restrict__ ver_in, int32_t *__restrict__ ver_out,
    int32_t *__restrict__ age_state, uint8_t *__restrict__ eff_state,
    unsigned long long *__restrict__ forced, uint8_t *__restrict__ eff_user,
    int32_t *__restrict__ result_clock, int64_t m, const double *const *__restrict__ fresh,
    double *const *__restrict__ slots, double *__restrict__ result) {
    if (blockIdx.x == 0) {
        record_step(P, S, t, arrived, ver_in, ver_out, age_state, eff_state, forced, eff_user,
                    nullptr, result_clock);
        return;
    }
    const int tid = threadIdx.x;
    // 16-byte path only if every pointer involved is 16-byte aligned.
    int ok = (((uintptr_t)result & 15) == 0) && ((m & 1) == 0);
    for (int32_t p = tid; p < P; p += kReduceThreads)
        ok = ok && ((((uintptr_t)fresh[p] | (uintptr_t)slots[p]) & 15) == 0);
    const int vec = __syncthreads_and(ok);

    const int64_t base = (int64_t)(blockIdx.x - 1) * (kReduceThreads * kReduceElems);
    constexpr int U = kReduceU;
    constexpr int VP = kReduceElems / 2;  // 16-byte pairs per thread
    static_assert(kReduceElems % 2 == 0, "pairs of elements");
    if (vec) {
        // element pairs q[j] = chunk pair offset + tid + j * kReduceThreads
        int64_t q[VP];
        bool in[VP];
        double2 acc[VP];
#pragma unroll
        for (int j = 0; j < VP; ++j) {
            q[j] = base / 2 + tid + (int64_t)j * kReduceThreads;
            in[j] = 2 * q[j] < m;
            acc[j] = make_double2(0.0, 0.0);
        }
        for (int32_t p0 = 0; p0 < P; p0 += U) {
            double2 v[U][VP];
            bool e[U], wr[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t p = p0 + u;
                if (p < P) {
                    e[u] = stale_select(ver_in[p], arrived[p], t, S);
                    const double *fp = fresh[p], *sp = slots[p];
                    wr[u] = e[u] && fp != sp;
                    const double2 *src = reinterpret_cast<const double2 *>(e[u] ? fp : sp);
#pragma unroll
                    for (int j = 0; j < VP; ++j)
                        if (in[j]) v[u][j] = src[q[j]];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t p = p0 + u;
                if (p < P) {
                    if (wr[u]) {
                        double2 *dst = reinterpret_cast<double2 *>(slots[p]);
#pragma unroll
                        for (int j = 0; j < VP; ++j) {
                            if (in[j]) dst[q[j]] = v[u][j];
                        }
                    }
#pragma unroll
                    for (int j = 0; j < VP; ++j) {
                        if (p == 0) {
                            acc[j] = v[u][j];
                        } else {
                            acc[j].x = acc[j].x + v[u][j].x;
                            acc[j].y = acc[j].y + v[u][j].y;
                        }
                    }
                }
            }
        }
        double2 *r2 = reinterpret_cast<double2 *>(result);
#pragma unroll
        for (int j = 0; j < VP; ++j)
            if (in[j]) r2[q[j]] = acc[j];
    } else {
        int64_t idx[kReduceElems];
        double acc[kReduceElems];
#pragma unroll
        for (int j = 0; j < kReduceElems; ++j) {
            idx[j] = base + tid + (int64_t)j * kReduceThreads;
            acc[j] = 0.0;
        }
        for (int32_t p = 0; p < P; ++p) {
            const bool e = stale_select(ver_in[p], arrived[p], t, S);
            const double *fp = fresh[p];
            double *sp = slots[p];
            const bool wr = e && fp != sp;
            const double *src = e ? fp : sp;
            double v[kReduceElems];
#pragma unroll
            for (int j = 0; j < kReduceElems; ++j)
                if (idx[j] < m) v[j] = src[idx[j]];
#pragma unroll
            for (int j = 0; j < kReduceElems; ++j) {
                if (idx[j] < m) {
                    if (wr) sp[idx[j]] = v[j];
                    acc[j] = (p == 0) ? v[j] : acc[j] + v[j];
                }
            }
        }
#pragma unroll
        for (int j = 0; j < kReduceElems; ++j)
            if (idx[j] < m) result[idx[j]] = acc[j];
    }
}

ecc_status_t launch_assemble(ecc_plan_t plan, const double *const *d_send,
                             const double *d_send_base, double *d_recv,
                             const uint8_t *d_arrived, uint8_t *d_eff_out, int32_t *d_age_out,
                             const int32_t *d_done) {
    const int64_t t = plan->clock;
    const int32_t *ver_in = plan->d_version + (t & 1) * plan->P;
    int32_t *ver_out = plan->d_version + ((t + 1) & 1) * plan->P;
    const int64_t grid = 1 + plan->n_tiles;
    if (grid > 0x7fffffff) {
        set_error("too many assembly tiles");
        return ECC_ERR_RANGE;
    }
    TimedLaunch timed(plan, ECC_TIMING_ASSEMBLE);
    hipLaunchKernelGGL(k_assemble, dim3((unsigned)grid), dim3(kAssembleThreads), 0, plan->stream,
                       plan->P, plan->S, t, d_arrived, ver_in, ver_out, plan->d_age, plan->d_eff,
                       plan->d_forced, d_eff_out, d_age_out, plan->d_tiles, plan->d_displs,
                       d_send, d_send_base, d_recv, d_done);
    ECC_LAUNCH_CHECK();
    plan->clock = t + 1;
    return ECC_OK;
}

}  // namespace ecc

using namespace ecc;

extern "C" {

ecc_status_t ecc_allgatherv_assemble(ecc_plan_t plan, const double *const *d_send,
                                     double *d_recv, const uint8_t *d_arrived,
                                     uint8_t *d_eff_out, int32_t *d_age_out) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    if (!plan->has_layout) {
        set_error("plan was created without counts/displs");
        return ECC_ERR_STATE;
    }
    ECC_ARG(d_send != nullptr, "d_send is NULL");
    ECC_ARG(d_arrived != nullptr, "d_arrived is NULL");
    ECC_ARG(d_recv != nullptr || plan->extent == 0, "d_recv is NULL");
    return launch_assemble(plan, d_send, nullptr, d_recv, d_arrived, d_eff_out, d_age_out,
                           nullptr);
}

ecc_status_t ecc_allgatherv_assemble_packed(ecc_plan_t plan, const double *d_send_base,
                                            double *d_recv, const uint8_t *d_arrived,
                                            uint8_t *d_eff_out, int32_t *d_age_out) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    if (!plan->has_layout) {
        set_error("plan was created without counts/displs");
        return ECC_ERR_STATE;
    }
    ECC_ARG(d_send_base != nullptr || plan->extent == 0, "d_send_base is NULL");
    ECC_ARG(d_arrived != nullptr, "d_arrived is NULL");
    ECC_ARG(d_recv != nullptr || plan->extent == 0, "d_recv is NULL");
    ECC_ARG(d_send_base != d_recv || plan->extent == 0, "d_send_base must not alias d_recv");
    return launch_assemble(plan, nullptr, d_send_base, d_recv, d_arrived, d_eff_out, d_age_out,
                           nullptr);
}

ecc_status_t ecc_allreduce_partial(ecc_plan_t plan, int64_t m, const double *const *d_fresh,
                                   double *const *d_slots, double *d_result,
                                   const uint8_t *d_arrived, uint8_t *d_eff_out,
                                   int32_t *d_result_clock) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(m >= 0, "m must be >= 0");
    ECC_ARG(d_fresh && d_slots, "d_fresh and d_slots must be device arrays of P pointers");
    ECC_ARG(d_arrived != nullptr, "d_arrived is NULL");
    ECC_ARG(d_result != nullptr || m == 0, "d_result is NULL");
    const int64_t chunk = (int64_t)kReduceThreads * kReduceElems;
    const int64_t grid = 1 + (m + chunk - 1) / chunk;
    if (grid > 0x7fffffff) {
        set_error("m too large");
        return ECC_ERR_RANGE;
    }
    const int64_t t = plan->clock;
    const int32_t *ver_in = plan->d_version + (t & 1) * plan->P;
    int32_t *ver_out = plan->d_version + ((t + 1) & 1) * plan->P;
    TimedLaunch timed(plan, ECC_TIMING_ALLREDUCE);
    hipLaunchKernelGGL(k_allreduce, dim3((unsigned)grid), dim3(kReduceThreads), 0, plan->stream,
                       plan->P, plan->S, t, d_arrived, ver_in, ver_out, plan->d_age, plan->d_eff,
                       plan->d_forced, d_eff_out, d_result_clock, m, d_fresh, d_slots, d_result);
    ECC_LAUNCH_CHECK();
    plan->clock = t + 1;
    return ECC_OK;
}

}  // extern "C"
