// Plan lifecycle: the set-up / shut-down phases of the collective (resources
// are allocated and the layout is exchanged once, then reused every clock),
// host-side validation, error reporting and state read-back.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>

#include <new>

#include "ecc_common.h"

namespace ecc {

static thread_local char g_err[1024] = "";

void set_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
}

void clear_error() { g_err[0] = '\0'; }

ecc_status_t check_plan(ecc_plan_t plan) {
    if (!plan) {
        set_error("plan is NULL");
        return ECC_ERR_ARG;
    }
    return ECC_OK;
}

// Reset of the per-rank state: versions := -1, age := 0, forced := 0.  A
// kernel rather than a memset so that it can be recorded in a graph.
__global__ void k_plan_reset(int32_t P, int32_t *version, int32_t *age, uint8_t *eff,
                             unsigned long long *forced, int32_t *ctrl) {
    for (int32_t p = blockIdx.x * blockDim.x + threadIdx.x; p < P;
         p += gridDim.x * blockDim.x) {
        version[p] = -1;
        version[P + p] = -1;
        age[p] = 0;
        eff[p] = 0;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *forced = 0ull;
        ctrl[0] = 0;
        ctrl[1] = 0;
    }
}

// Assembly tiles for a layout: every non-empty block is cut into pieces of at
// most kAssembleTile elements; ranks are visited in order of displacement.
static std::vector<Tile> make_tiles(const std::vector<int64_t> &counts,
                                    const std::vector<int64_t> &displs) {
    const int32_t P = (int32_t)counts.size();
    std::vector<int32_t> order(P);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int32_t a, int32_t b) { return displs[a] < displs[b]; });
    std::vector<Tile> tiles;
    for (int32_t p : order) {
        for (int64_t off = 0; off < counts[p]; off += kAssembleTile) {
            Tile t;
            t.off = off;
            t.rank = p;
            t.len = (int32_t)std::min<int64_t>(kAssembleTile, counts[p] - off);
            tiles.push_back(t);
        }
    }
    return tiles;
}

static hipEvent_t take_event(ecc_plan_t plan) {
    if (!plan->event_pool.empty()) {
        hipEvent_t e = plan->event_pool.back();
        plan->event_pool.pop_back();
        return e;
    }
    // no system-scope fence: the events only order work on this device
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

TimedLaunch::TimedLaunch(ecc_plan_t p, int k) : plan(p), kind(k) {
    if (!plan || !plan->timing) return;
    start = take_event(plan);
    stop = take_event(plan);
    if (start && stop && hipEventRecord(start, plan->stream) == hipSuccess) return;
    start = stop = nullptr;
}

TimedLaunch::~TimedLaunch() {
    if (!start || !stop) return;
    if (hipEventRecord(stop, plan->stream) == hipSuccess)
        plan->pending[kind].push_back({start, stop});
}

}  // namespace ecc

using namespace ecc;

extern "C" {

int32_t ecc_abi_version(void) { return 3; }

const char *ecc_last_error(void) { return g_err; }

const char *ecc_status_string(ecc_status_t s) {
    switch (s) {
    case ECC_OK: return "ECC_OK";
    case ECC_ERR_ARG: return "ECC_ERR_ARG";
    case ECC_ERR_OVERLAP: return "ECC_ERR_OVERLAP";
    case ECC_ERR_RANGE: return "ECC_ERR_RANGE";
    case ECC_ERR_ALLOC: return "ECC_ERR_ALLOC";
    case ECC_ERR_DEVICE: return "ECC_ERR_DEVICE";
    case ECC_ERR_STATE: return "ECC_ERR_STATE";
    }
    return "ECC_ERR_UNKNOWN";
}

static ecc_status_t ecc_plan_validate_impl(int32_t P, const int64_t *h_counts, const int64_t *h_displs,
                               int32_t max_staleness) {
    clear_error();
    ECC_ARG(P >= 1, "P must be >= 1 (got %d)", P);
    ECC_ARG(P < (1 << 24), "P must be < 2^24 (got %d)", P);
    ECC_ARG(max_staleness >= 0, "max_staleness must be >= 0 (got %d)", max_staleness);
    if (!h_counts && !h_displs) return ECC_OK;
    ECC_ARG(h_counts && h_displs, "counts and displs must both be given or both be NULL");
    std::vector<std::pair<int64_t, int64_t>> seg;
    for (int32_t p = 0; p < P; ++p) {
        ECC_ARG(h_counts[p] >= 0, "counts[%d] = %lld is negative", p, (long long)h_counts[p]);
        ECC_ARG(h_displs[p] >= 0, "displs[%d] = %lld is negative", p, (long long)h_displs[p]);
        if (h_displs[p] + h_counts[p] >= (int64_t(1) << 40) || h_counts[p] >= (int64_t(1) << 40)) {
            set_error("block of rank %d ends beyond 2^40 elements", p);
            return ECC_ERR_RANGE;
        }
        if (h_counts[p] > 0) seg.push_back({h_displs[p], h_displs[p] + h_counts[p]});
    }
    std::sort(seg.begin(), seg.end());
    for (size_t i = 1; i < seg.size(); ++i) {
        if (seg[i].first < seg[i - 1].second) {
            set_error("blocks [%lld,%lld) and [%lld,%lld) overlap",
                      (long long)seg[i - 1].first, (long long)seg[i - 1].second,
                      (long long)seg[i].first, (long long)seg[i].second);
            return ECC_ERR_OVERLAP;
        }
    }
    return ECC_OK;
}

// Host allocations of the set-up throw std::bad_alloc when memory runs
// out: the C ABI reports ECC_ERR_ALLOC instead of letting it escape.
ecc_status_t ecc_plan_validate(int32_t P, const int64_t *h_counts, const int64_t *h_displs,
                               int32_t max_staleness) {
    try {
        return ecc_plan_validate_impl(P, h_counts, h_displs, max_staleness);
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
}

static ecc_status_t ecc_plan_create_impl(int32_t P, const int64_t *h_counts, const int64_t *h_displs,
                             int32_t max_staleness, void *hip_stream, ecc_plan_t *out) {
    ECC_ARG(out != nullptr, "out is NULL");
    *out = nullptr;
    ecc_status_t st = ecc_plan_validate(P, h_counts, h_displs, max_staleness);
    if (st != ECC_OK) return st;

    ecc_plan_s *pl = new (std::nothrow) ecc_plan_s();
    if (!pl) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
    pl->P = P;
    pl->S = max_staleness;
    pl->stream = (hipStream_t)hip_stream;
    auto fail = [&](ecc_status_t s) {
        ecc_plan_destroy(pl);
        return s;
    };
    if (hipGetDevice(&pl->device) != hipSuccess) {
        set_error("hipGetDevice failed");
        delete pl;
        return ECC_ERR_DEVICE;
    }
    if (h_counts) {
        pl->has_layout = true;
        pl->counts.assign(h_counts, h_counts + P);
        pl->displs.assign(h_displs, h_displs + P);
        int64_t acc = 0;
        bool tiles = true;
        for (int32_t p = 0; p < P; ++p) {
            if (pl->displs[p] != acc) tiles = false;
            acc += pl->counts[p];
            pl->extent = std::max(pl->extent, pl->displs[p] + pl->counts[p]);
        }
        pl->tiles_rows = tiles;
    }

#define ALLOC(ptr, bytes)                                                        \
    do {                                                                         \
        if (hipMalloc((void **)&(ptr), (bytes)) != hipSuccess) {                 \
            set_error("hipMalloc of %zu bytes failed", (size_t)(bytes));         \
            return fail(ECC_ERR_ALLOC);                                          \
        }                                                                        \
    } while (0)

    ALLOC(pl->d_version, sizeof(int32_t) * 2 * P);
    ALLOC(pl->d_age, sizeof(int32_t) * P);
    ALLOC(pl->d_eff, sizeof(uint8_t) * P);
    ALLOC(pl->d_forced, sizeof(unsigned long long));
    ALLOC(pl->d_ctrl, sizeof(int32_t) * 4);
    if (hipHostMalloc((void **)&pl->h_ctrl, sizeof(int32_t) * 2, hipHostMallocDefault) !=
        hipSuccess) {
        pl->h_ctrl = nullptr;
        set_error("hipHostMalloc of the loop control failed");
        return fail(ECC_ERR_ALLOC);
    }
    ALLOC(pl->d_scalar, sizeof(double) * 2);
    if (pl->has_layout) {
        ALLOC(pl->d_displs, sizeof(int64_t) * P);
        if (hipMemcpy(pl->d_displs, pl->displs.data(), sizeof(int64_t) * P,
                      hipMemcpyHostToDevice) != hipSuccess) {
            set_error("copy of displs failed");
            return fail(ECC_ERR_DEVICE);
        }
        std::vector<Tile> tiles = make_tiles(pl->counts, pl->displs);
        pl->n_tiles = (int64_t)tiles.size();
        if (!tiles.empty()) {
            ALLOC(pl->d_tiles, sizeof(Tile) * tiles.size());
            if (hipMemcpy(pl->d_tiles, tiles.data(), sizeof(Tile) * tiles.size(),
                          hipMemcpyHostToDevice) != hipSuccess) {
                set_error("copy of tiles failed");
                return fail(ECC_ERR_DEVICE);
            }
        }
        if (pl->tiles_rows && pl->extent < (int64_t(1) << 31)) {
            std::vector<int32_t> bs(P + 1);
            bs[0] = 0;
            for (int32_t p = 0; p < P; ++p) bs[p + 1] = (int32_t)(bs[p] + pl->counts[p]);
            ALLOC(pl->d_block_start, sizeof(int32_t) * (P + 1));
            if (hipMemcpy(pl->d_block_start, bs.data(), sizeof(int32_t) * (P + 1),
                          hipMemcpyHostToDevice) != hipSuccess) {
                set_error("copy of block starts failed");
                return fail(ECC_ERR_DEVICE);
            }
        }
    }
#undef ALLOC
    st = ecc_plan_reset(pl);
    if (st != ECC_OK) return fail(st);
    if (hipStreamSynchronize(pl->stream) != hipSuccess) {
        set_error("stream synchronise after plan reset failed");
        return fail(ECC_ERR_DEVICE);
    }
    *out = pl;
    return ECC_OK;
}

// Host allocations of the set-up throw std::bad_alloc when memory runs
// out: the C ABI reports ECC_ERR_ALLOC instead of letting it escape.
ecc_status_t ecc_plan_create(int32_t P, const int64_t *h_counts, const int64_t *h_displs,
                             int32_t max_staleness, void *hip_stream, ecc_plan_t *out) {
    try {
        return ecc_plan_create_impl(P, h_counts, h_displs, max_staleness, hip_stream, out);
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return ECC_ERR_ALLOC;
    }
}

ecc_status_t ecc_plan_destroy(ecc_plan_t plan) {
    if (!plan) return ECC_OK;
    (void)hipStreamSynchronize(plan->stream);
    (void)hipFree(plan->d_version);
    (void)hipFree(plan->d_age);
    (void)hipFree(plan->d_eff);
    (void)hipFree(plan->d_forced);
    (void)hipFree(plan->d_ctrl);
    if (plan->h_ctrl) (void)hipHostFree(plan->h_ctrl);
    (void)hipFree(plan->d_scalar);
    (void)hipFree(plan->d_displs);
    (void)hipFree(plan->d_tiles);
    (void)hipFree(plan->d_block_start);
    for (auto &v : plan->pending)
        for (auto &pr : v) {
            (void)hipEventDestroy(pr.first);
            (void)hipEventDestroy(pr.second);
        }
    for (hipEvent_t e : plan->event_pool) (void)hipEventDestroy(e);
    delete plan;
    return ECC_OK;
}

ecc_status_t ecc_plan_set_timing(ecc_plan_t plan, int32_t enable) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    plan->timing = enable != 0;
    return ECC_OK;
}

ecc_status_t ecc_plan_timing(ecc_plan_t plan, int32_t kernel, double *total_ms,
                             int64_t *launches, int32_t reset) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(kernel >= 0 && kernel < ECC_TIMING_KINDS, "unknown kernel %d", kernel);
    ECC_HIP(hipStreamSynchronize(plan->stream));
    for (int k = 0; k < ECC_TIMING_KINDS; ++k) {
        for (auto &pr : plan->pending[k]) {
            float ms = 0.f;
            ECC_HIP(hipEventElapsedTime(&ms, pr.first, pr.second));
            plan->timed_ms[k] += ms;
            plan->timed_launches[k] += 1;
            plan->event_pool.push_back(pr.first);
            plan->event_pool.push_back(pr.second);
        }
        plan->pending[k].clear();
    }
    if (total_ms) *total_ms = plan->timed_ms[kernel];
    if (launches) *launches = plan->timed_launches[kernel];
    if (reset) {
        plan->timed_ms[kernel] = 0.0;
        plan->timed_launches[kernel] = 0;
    }
    return ECC_OK;
}

ecc_status_t ecc_plan_reset(ecc_plan_t plan) {
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    const int threads = 256;
    const int blocks = (int)std::min<int64_t>(64, (plan->P + threads - 1) / threads);
    hipLaunchKernelGGL(k_plan_reset, dim3(blocks), dim3(threads), 0, plan->stream, plan->P,
                       plan->d_version, plan->d_age, plan->d_eff, plan->d_forced, plan->d_ctrl);
    ECC_LAUNCH_CHECK();
    plan->clock = 0;
    return ECC_OK;
}

ecc_status_t ecc_plan_set_stream(ecc_plan_t plan, void *hip_stream) {
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    plan->stream = (hipStream_t)hip_stream;
    return ECC_OK;
}

ecc_status_t ecc_plan_stats(ecc_plan_t plan, int64_t *clock, int64_t *forced_total,
                            int32_t *h_version, int32_t *h_age) {
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_HIP(hipStreamSynchronize(plan->stream));
    if (clock) *clock = plan->clock;
    if (forced_total) {
        unsigned long long f = 0;
        ECC_HIP(hipMemcpy(&f, plan->d_forced, sizeof(f), hipMemcpyDeviceToHost));
        *forced_total = (int64_t)f;
    }
    if (h_version) {
        const int32_t *cur = plan->d_version + (plan->clock & 1) * plan->P;
        ECC_HIP(hipMemcpy(h_version, cur, sizeof(int32_t) * plan->P, hipMemcpyDeviceToHost));
    }
    if (h_age)
        ECC_HIP(hipMemcpy(h_age, plan->d_age, sizeof(int32_t) * plan->P, hipMemcpyDeviceToHost));
    return ECC_OK;
}

}  // extern "C"
