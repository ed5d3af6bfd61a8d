// Plain streaming copy (16-byte accesses, four per thread in flight): the
// reference kernel for the measured copy ceiling and for calibrating the
// HBM byte counters against a kernel of known traffic.
#include "ecc_common.h"

namespace ecc {

constexpr int kCopyThreads = 256;
constexpr int kCopyPairs = 4;  // 16-byte pairs per thread

__global__ __launch_bounds__(kCopyThreads) void k_stream_copy(double2 *__restrict__ dst,
                                                              const double2 *__restrict__ src,
                                                              int64_t npair) {
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

}  // namespace ecc

using namespace ecc;

extern "C" ecc_status_t ecc_stream_copy(double *d_dst, const double *d_src, int64_t n,
                                        void *hip_stream) {
    clear_error();
    ECC_ARG(n >= 0, "n must be >= 0");
    if (n == 0) return ECC_OK;
    ECC_ARG(d_dst && d_src, "NULL pointer");
    ECC_ARG((((uintptr_t)d_dst | (uintptr_t)d_src) & 15) == 0 && (n & 1) == 0,
            "the copy needs 16-byte aligned buffers and an even element count");
    const int64_t npair = n / 2;
    const int64_t grid = (npair + kCopyThreads * kCopyPairs - 1) / (kCopyThreads * kCopyPairs);
    ECC_ARG(grid < 0x7fffffff, "n too large");
    hipLaunchKernelGGL(k_stream_copy, dim3((unsigned)grid), dim3(kCopyThreads), 0,
                       (hipStream_t)hip_stream, reinterpret_cast<double2 *>(d_dst),
                       reinterpret_cast<const double2 *>(d_src), npair);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}
