// Plain streaming copy (16-byte accesses, one per thread): the
// reference kernel for the measured copy ceiling and for calibrating the
// HBM byte counters against a kernel of known traffic.  And a gather probe:
// the rate of gathers of one vector over an index stream.
#include <algorithm>

#include "ecc_common.h"

namespace ecc {

constexpr int kCopyThreads = 256;
// One 16-byte pair per thread and one workgroup per 256 pairs (measured on
// MI355X, 4 GiB + 4 GiB: 6.26 TB/s, against 5.76 and 5.63 TB/s with two and
// four pairs per thread).
constexpr int kCopyPairs = 1;

// Copies npair 16-byte pairs; an odd trailing element (tail != 0) is copied
// by thread 0 of block 0.
__global__ __launch_bounds__(kCopyThreads) void k_stream_copy(double2 *__restrict__ dst,
                                                              const double2 *__restrict__ src,
                                                              int64_t npair, int tail) {
    if (tail && blockIdx.x == 0 && threadIdx.x == 0)
        reinterpret_cast<double *>(dst)[2 * npair] =
            reinterpret_cast<const double *>(src)[2 * npair];
    if (npair == 0) return;
    const int64_t base = (int64_t)blockIdx.x * (kCopyThreads * kCopyPairs) + threadIdx.x;
    double2 v[kCopyPairs];
#pragma unroll
    for (int u = 0; u < kCopyPairs; ++u) {
        const int64_t k = base + (int64_t)u * kCopyThreads;
        v[u] = src[k < npair ? k : npair - 1];
    }
#pragma unroll
    for (int u = 0; u < kCopyPairs; ++u) {
        const int64_t k = base + (int64_t)u * kCopyThreads;
        if (k < npair) dst[k] = v[u];
    }
}

// Copy of 8-byte elements for buffers that are not 16-byte aligned.
__global__ __launch_bounds__(kCopyThreads) void k_copy_f64(double *__restrict__ dst,
                                                           const double *__restrict__ src,
                                                           int64_t n) {
    const int64_t k = (int64_t)blockIdx.x * kCopyThreads + threadIdx.x;
    if (k < n) dst[k] = src[k];
}

// Gather probe: workgroup w sums d_x at indices [w C, (w + 1) C) (C =
// kGatherChunk), eight per thread with every load in flight, and writes the
// workgroup's sum.
constexpr int kGatherThreads = 256;
constexpr int kGatherPer = ECC_GATHER_CHUNK / kGatherThreads;
static_assert(kGatherPer == 8, "eight indices per thread");

__global__ __launch_bounds__(kGatherThreads) void k_gather_probe(const int32_t *__restrict__ idx,
                                                                 int64_t n,
                                                                 const double *__restrict__ x,
                                                                 int64_t n_x,
                                                                 double *__restrict__ out) {
    __shared__ double s_red[kGatherThreads / 64];
    const int64_t base = (int64_t)blockIdx.x * ECC_GATHER_CHUNK + threadIdx.x;
    int32_t c[kGatherPer];
#pragma unroll
    for (int u = 0; u < kGatherPer; ++u) {
        const int64_t k = base + (int64_t)u * kGatherThreads;
        c[u] = k < n ? __builtin_nontemporal_load(idx + k) : -1;
    }
    double y[kGatherPer];
#pragma unroll
    for (int u = 0; u < kGatherPer; ++u)
        y[u] = (c[u] >= 0 && (int64_t)c[u] < n_x) ? x[c[u]] : 0.0;
    double s = 0.0;
#pragma unroll
    for (int u = 0; u < kGatherPer; ++u) s = s + y[u];
    const double total = block_sum<kGatherThreads>(s, s_red);
    if (threadIdx.x == 0) out[blockIdx.x] = total;
}

}  // namespace ecc

using namespace ecc;

extern "C" ecc_status_t ecc_gather_probe(const int32_t *d_idx, int64_t n, const double *d_x,
                                         int64_t n_x, double *d_out, int64_t n_out,
                                         void *hip_stream) {
    clear_error();
    ECC_ARG(n >= 0 && n_x >= 0, "negative size");
    if (n == 0) return ECC_OK;
    ECC_ARG(d_idx && d_x && d_out, "NULL pointer");
    const int64_t grid = (n + ECC_GATHER_CHUNK - 1) / ECC_GATHER_CHUNK;
    ECC_ARG(n_out >= grid, "d_out holds %lld doubles; %lld needed", (long long)n_out,
            (long long)grid);
    ECC_ARG(grid < 0x7fffffff, "n too large");
    hipLaunchKernelGGL(k_gather_probe, dim3((unsigned)grid), dim3(kGatherThreads), 0,
                       (hipStream_t)hip_stream, d_idx, n, d_x, n_x, d_out);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

extern "C" ecc_status_t ecc_stream_copy(double *d_dst, const double *d_src, int64_t n,
                                        void *hip_stream) {
    clear_error();
    ECC_ARG(n >= 0, "n must be >= 0");
    if (n == 0) return ECC_OK;
    ECC_ARG(d_dst && d_src, "NULL pointer");
    ECC_ARG((((uintptr_t)d_dst | (uintptr_t)d_src) & 7) == 0, "buffers must be 8-byte aligned");
    const uintptr_t lo = (uintptr_t)d_dst, hi = lo + 8 * (uintptr_t)n;
    const uintptr_t slo = (uintptr_t)d_src, shi = slo + 8 * (uintptr_t)n;
    ECC_ARG(hi <= slo || shi <= lo, "source and destination overlap");
    if ((((uintptr_t)d_dst | (uintptr_t)d_src) & 15) != 0) {
        const int64_t grid = (n + kCopyThreads - 1) / kCopyThreads;
        ECC_ARG(grid < 0x7fffffff, "n too large");
        hipLaunchKernelGGL(k_copy_f64, dim3((unsigned)grid), dim3(kCopyThreads), 0,
                           (hipStream_t)hip_stream, d_dst, d_src, n);
        ECC_LAUNCH_CHECK();
        return ECC_OK;
    }
    const int64_t npair = n / 2;
    const int64_t grid =
        std::max<int64_t>(1, (npair + kCopyThreads * kCopyPairs - 1) / (kCopyThreads * kCopyPairs));
    ECC_ARG(grid < 0x7fffffff, "n too large");
    hipLaunchKernelGGL(k_stream_copy, dim3((unsigned)grid), dim3(kCopyThreads), 0,
                       (hipStream_t)hip_stream, reinterpret_cast<double2 *>(d_dst),
                       reinterpret_cast<const double2 *>(d_src), npair, (int)(n & 1));
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}
