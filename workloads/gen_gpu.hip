/*
 * Device-side counterpart of gen.c's uniform generator, for inputs too large
 * to produce on the host for every repetition of a test (for example, the
 * contributions of 256 ranks x 2^22 elements at each of 1,000 repetitions).
 *
 * Like gen.c it holds no arithmetic of the method: it only writes the same
 * counter-based SplitMix64 uniforms (Steele, Lea, Flood, OOPSLA 2014) that
 * gen_uniform_range produces on the host, bit for bit -- integer mixing,
 * the top 53 bits scaled by 2^-53 (exact), then lo + (hi - lo) * u, built
 * without floating-point contraction.
 */
#include <hip/hip_runtime.h>
#include <stdint.h>

#define GOLDEN 0x9e3779b97f4a7c15ULL

__host__ __device__ static inline uint64_t sm64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

__host__ __device__ static inline uint64_t sm64_nth(uint64_t state, uint64_t k) {
    return sm64_mix(state + k * GOLDEN);
}

/* out[i] = lo + w * U[0,1)(key, ctr0 + i), i < n; key = the stream's key. */
__global__ void k_uniform_range(uint64_t key, uint64_t ctr0, int64_t n, double lo, double w,
                                double *__restrict__ out) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const double u = (double)(sm64_nth(key, ctr0 + (uint64_t)i + 1) >> 11) * 0x1.0p-53;
        out[i] = lo + w * u;
    }
}

/* d_out[i] = lo + (hi - lo) * U[0,1)(seed, stream, ctr0 + i) for 0 <= i < n,
 * as gen_uniform_range, enqueued on hip_stream.  Returns 0, or the HIP error. */
extern "C" int gen_uniform_range_device(uint64_t seed, uint64_t stream, uint64_t ctr0, int64_t n,
                                        double lo, double hi, double *d_out, void *hip_stream) {
    if (n <= 0) return 0;
    const uint64_t key = sm64_nth(seed, stream + 1);
    const int64_t blocks = (n + 255) / 256;
    const unsigned grid = (unsigned)(blocks < 65536 ? blocks : 65536);
    hipLaunchKernelGGL(k_uniform_range, dim3(grid), dim3(256), 0, (hipStream_t)hip_stream, key,
                       ctr0, n, lo, hi - lo, d_out);
    return (int)hipGetLastError();
}
