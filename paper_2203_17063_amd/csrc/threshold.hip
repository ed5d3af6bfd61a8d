// Eventually consistent Broadcast and Reduce with a threshold (Section III-B,
// with the threshold/status parameters of Section III), and the partial
// allreduce that drops the contributions that did not arrive.
//
// Binomial spanning tree (BST) over P processes numbered relative to the
// root: the children of q are q + 2^i for every i above q's highest set bit
// with q + 2^i < P, so stage s involves min(2^s, P) processes.
//  - Broadcast delivers the first ceil(theta * m) elements of the root's
//    vector to every other process: on one GPU the tree's forwarding
//    reduces to prefix copies (every receiver gets the root's data); each
//    tile of the prefix is read once and written P - 1 times.
//  - Reduce sums either the first ceil(theta * m) elements of every process
//    or the full vectors of the processes of the first stages of the tree
//    (at least ceil(theta * P) of them).  The order is the tree's: a parent
//    adds its children's partial sums leaves first, which is, stage by stage
//    from the last one, q += partial(q + 2^s) for every q < 2^s.  A thread
//    carries one element of every involved process in registers; beyond 32
//    processes it sums them in the same tree as a pairwise sum (below).
//  - The dropping allreduce sums, in rank order from +0.0, the contributions
//    of the ranks that arrived in this step.
// All sums are fp64 without contraction, in the order stated, so results
// are bitwise reproducible.
#include <algorithm>
#include <cmath>

#include "ecc_common.h"

namespace ecc {

constexpr int kThrThreads = 256;
constexpr int kThrMaxStages = 5;  // Reduce: at most 32 processes in registers
constexpr int kThrMaxStagesBig = 12;  // Reduce beyond 32 processes: up to 4096
constexpr int kBcastTile = 4096;  // elements one workgroup copies

// One workgroup per tile of kBcastTile elements of the prefix: the tile is
// loaded from the root's vector once, into registers (kBcastPairs pairs per
// thread), and stored into every other process's buffer -- 16-byte stores
// where the destination row allows, else 8-byte.
constexpr int kBcastPairs = kBcastTile / (2 * kThrThreads);

__global__ __launch_bounds__(kThrThreads) void k_bcast_prefix(int32_t P, int32_t root, int64_t k,
                                                              const double *__restrict__ src,
                                                              double *const *__restrict__ dst) {
    const int64_t t0 = (int64_t)blockIdx.x * kBcastTile;
    const bool src16 = ((uintptr_t)src & 15) == 0;
    double2 v[kBcastPairs];
#pragma unroll
    for (int u = 0; u < kBcastPairs; ++u) {
        const int64_t e = t0 + 2 * ((int64_t)threadIdx.x + (int64_t)u * kThrThreads);
        if (e + 1 < k) {
            if (src16) v[u] = *reinterpret_cast<const double2 *>(src + e);
            else v[u] = make_double2(src[e], src[e + 1]);
        } else {
            v[u] = make_double2(e < k ? src[e] : 0.0, 0.0);
        }
    }
    for (int32_t p = 0; p < P; ++p) {
        if (p == root) continue;
        double *__restrict__ d = dst[p];
        const bool d16 = ((uintptr_t)d & 15) == 0;
#pragma unroll
        for (int u = 0; u < kBcastPairs; ++u) {
            const int64_t e = t0 + 2 * ((int64_t)threadIdx.x + (int64_t)u * kThrThreads);
            if (e + 1 < k) {
                if (d16) *reinterpret_cast<double2 *>(d + e) = v[u];
                else {
                    d[e] = v[u].x;
                    d[e + 1] = v[u].y;
                }
            } else if (e < k) {
                d[e] = v[u].x;
            }
        }
    }
}

// Reduce over relative ranks 0 .. n-1 (n <= 2^S) of the first k elements.
// Every contribution is read once: non-temporal loads (measured on MI355X,
// 32 processes x 4.2M elements: 190 us against 261 us with ordinary loads
// and a grid capped at 8 workgroups per CU), and one workgroup per 256
// elements.
template <int S>
__global__ __launch_bounds__(kThrThreads) void k_reduce_bst(int32_t P, int32_t root, int32_t n,
                                                            int64_t k,
                                                            const double *const *__restrict__ src,
                                                            double *__restrict__ result) {
    static_assert(S >= 0 && S <= kThrMaxStages, "the register fold holds at most 32 processes");
    constexpr int N = 1 << S;
    const int64_t stride = (int64_t)gridDim.x * kThrThreads;
    for (int64_t j = (int64_t)blockIdx.x * kThrThreads + threadIdx.x; j < k; j += stride) {
        double part[N];
#pragma unroll
        for (int q = 0; q < N; ++q) {
            if (q < n) {
                const int32_t p = (q + root) % P;
                part[q] = __builtin_nontemporal_load(src[p] + j);
            }
        }
#pragma unroll
        for (int s = S - 1; s >= 0; --s) {
#pragma unroll
            for (int q = 0; q < (1 << s); ++q)
                if (q + (1 << s) < n) part[q] = part[q] + part[q + (1 << s)];
        }
        result[j] = part[0];
    }
}

// More than 32 processes (measured on MI355X, 64 x 32 MB: 362 against 369
// us with all 64 in registers, 169 VGPRs; 32 x 64 MB: 377 against 360 us,
// so the register fold stays up to 32).  Stage by stage from the last,
// q += partial(q + 2^s) builds a binary tree whose leaves, read left to
// right, are the relative ranks in the bit-reversed order of D =
// ceil(log2 n) bits: the two children of a node combined at stage s are
// its halves, the lower rank on the left and added first.  A rank at or beyond n is absent; as
// absence grows with the rank, a node whose left child is absent has an
// absent right child too, and a node with an absent right child is its
// left child.  So the reduction is a pairwise sum over that order, and a
// thread computes it for its element with a stack of one node per level:
// the 8 leaves of each group of 8 consecutive positions are loaded
// together and added into one node, which is merged into the stack as a
// binary counter over the group index.
constexpr int kBrev3[8] = {0, 4, 2, 6, 1, 5, 3, 7};

template <int D>
__global__ __launch_bounds__(kThrThreads) void k_reduce_bst_big(
    int32_t P, int32_t root, int32_t n, int64_t k, const double *const *__restrict__ src,
    double *__restrict__ result) {
    constexpr int H = D - 3;  // levels above a group of 8 leaves
    static_assert(H >= 1 && D <= kThrMaxStagesBig, "between 9 and 4,096 processes");
    const int64_t stride = (int64_t)gridDim.x * kThrThreads;
    for (int64_t j = (int64_t)blockIdx.x * kThrThreads + threadIdx.x; j < k; j += stride) {
        double st[H];
        bool sv[H];
#pragma unroll
        for (int l = 0; l < H; ++l) {
            st[l] = 0.0;
            sv[l] = false;
        }
        double node = 0.0;
        for (int32_t b = 0; b < (1 << H); ++b) {
            // leaf u of group b sits at position 8 b + u: relative rank
            // bitrev3(u) 2^H + bitrev_H(b)
            const int32_t hb = (int32_t)(__brev((uint32_t)b) >> (32 - H));
            double v[8];
            bool e[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int32_t q = (kBrev3[u] << H) | hb;
                e[u] = q < n;
                int32_t p = (e[u] ? q : 0) + root;  // (an absent leaf names no process)
                if (p >= P) p -= P;
                v[u] = e[u] ? __builtin_nontemporal_load(src[p] + j) : 0.0;
            }
            // the group's node: pairs, then quads, then the eight
#pragma unroll
            for (int w = 1; w < 8; w *= 2) {
#pragma unroll
                for (int u = 0; u < 8; u += 2 * w)
                    if (e[u + w]) v[u] = v[u] + v[u + w];
            }
            node = v[0];
            bool nv = e[0];
            // merge as a binary counter: level l holds the left sibling while
            // bit l of b is 1
            bool carry = true;
#pragma unroll
            for (int l = 0; l < H; ++l) {
                if (carry) {
                    if ((b >> l) & 1) {
                        if (sv[l] && nv) node = st[l] + node;
                        else if (sv[l]) node = st[l];
                        nv = sv[l];
                    } else {
                        st[l] = node;
                        sv[l] = nv;
                        carry = false;
                    }
                }
            }
        }
        // the last group (b = 2^H - 1) carried through every level: the root
        result[j] = node;
    }
}

// Dropping partial allreduce: eight ranks' loads in flight, summed in rank
// order; only arrived ranks are added.
constexpr int kDropU = 8;

__global__ __launch_bounds__(kThrThreads) void k_allreduce_drop(int32_t P, int64_t m,
                                                                const double *const *__restrict__ fresh,
                                                                const uint8_t *__restrict__ arrived,
                                                                double *__restrict__ result,
                                                                int32_t *__restrict__ count) {
    if (count && blockIdx.x == 0 && threadIdx.x == 0) {
        int32_t c = 0;
        for (int32_t p = 0; p < P; ++p) c += arrived[p] != 0;
        *count = c;
    }
    const int64_t stride = (int64_t)gridDim.x * kThrThreads;
    for (int64_t j = (int64_t)blockIdx.x * kThrThreads + threadIdx.x; j < m; j += stride) {
        double acc = 0.0;
        for (int32_t p0 = 0; p0 < P; p0 += kDropU) {
            bool on[kDropU];
            double v[kDropU];
#pragma unroll
            for (int u = 0; u < kDropU; ++u) {
                const int32_t p = p0 + u;
                on[u] = p < P && arrived[p] != 0;
                v[u] = on[u] ? fresh[p][j] : 0.0;
            }
#pragma unroll
            for (int u = 0; u < kDropU; ++u)
                if (on[u]) acc = acc + v[u];
        }
        result[j] = acc;
    }
}

int64_t thr_prefix(double theta, int64_t m) {
    const double x = std::ceil(theta * (double)m);
    return std::min<int64_t>(m, (int64_t)x);
}

int32_t thr_involved(double theta, int32_t P) {
    const int64_t need = std::max<int64_t>(1, (int64_t)std::ceil(theta * (double)P));
    int64_t n = 1;
    while (n < need) n *= 2;
    return (int32_t)std::min<int64_t>(n, P);
}

int32_t thr_grid(int64_t elems) {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        cus = 256;
    const int64_t need = std::max<int64_t>(1, (elems + kThrThreads - 1) / kThrThreads);
    return (int32_t)std::min<int64_t>(need, (int64_t)cus * 8);
}

int32_t thr_grid_once(int64_t elems) {
    const int64_t need = std::max<int64_t>(1, (elems + kThrThreads - 1) / kThrThreads);
    return (int32_t)std::min<int64_t>(need, 0x7fffffff);
}

}  // namespace ecc

using namespace ecc;

extern "C" {

ecc_status_t ecc_bcast_threshold(int32_t P, int32_t root, int64_t m, double theta,
                                 const double *d_src, double *const *d_dst, int64_t *h_count,
                                 void *hip_stream) {
    clear_error();
    ECC_ARG(P >= 1, "P must be >= 1");
    ECC_ARG(root >= 0 && root < P, "root %d outside [0, P)", root);
    ECC_ARG(m >= 0, "m must be >= 0");
    ECC_ARG(theta >= 0.0 && theta <= 1.0, "theta must lie in [0, 1]");
    const int64_t k = thr_prefix(theta, m);
    if (h_count) *h_count = k;
    if (k == 0 || P == 1) return ECC_OK;
    ECC_ARG(d_src != nullptr && d_dst != nullptr, "NULL source or destination array");
    const int64_t tiles = (k + kBcastTile - 1) / kBcastTile;
    ECC_ARG(tiles < 0x7fffffff, "too many tiles");
    hipLaunchKernelGGL(k_bcast_prefix, dim3((unsigned)tiles), dim3(kThrThreads), 0,
                       (hipStream_t)hip_stream, P, root, k, d_src, d_dst);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

ecc_status_t ecc_reduce_threshold(int32_t P, int32_t root, int64_t m, double theta, int32_t mode,
                                  const double *const *d_src, double *d_result,
                                  int64_t *h_elements, int32_t *h_processes, void *hip_stream) {
    clear_error();
    ECC_ARG(P >= 1 && P <= (1 << kThrMaxStagesBig), "P = %d must lie in [1, %d]", P,
            1 << kThrMaxStagesBig);
    ECC_ARG(root >= 0 && root < P, "root %d outside [0, P)", root);
    ECC_ARG(m >= 0, "m must be >= 0");
    ECC_ARG(mode == ECC_THRESHOLD_DATA || mode == ECC_THRESHOLD_PROCS, "unknown mode %d", mode);
    int64_t k;
    int32_t n;
    if (mode == ECC_THRESHOLD_DATA) {
        ECC_ARG(theta >= 0.0 && theta <= 1.0, "theta must lie in [0, 1]");
        k = thr_prefix(theta, m);
        n = P;
    } else {
        ECC_ARG(theta > 0.0 && theta <= 1.0, "theta must lie in (0, 1]");
        k = m;
        n = thr_involved(theta, P);
    }
    if (h_elements) *h_elements = k;
    if (h_processes) *h_processes = n;
    if (k == 0) return ECC_OK;
    ECC_ARG(d_src != nullptr && d_result != nullptr, "NULL source array or result");
    int S = 0;
    while ((1 << S) < n) ++S;
    const dim3 grid(thr_grid_once(k)), block(kThrThreads);
    hipStream_t st = (hipStream_t)hip_stream;
    switch (S) {
        case 0: hipLaunchKernelGGL(k_reduce_bst<0>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 1: hipLaunchKernelGGL(k_reduce_bst<1>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 2: hipLaunchKernelGGL(k_reduce_bst<2>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 3: hipLaunchKernelGGL(k_reduce_bst<3>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 4: hipLaunchKernelGGL(k_reduce_bst<4>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 5: hipLaunchKernelGGL(k_reduce_bst<5>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 6: hipLaunchKernelGGL(k_reduce_bst_big<6>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 7: hipLaunchKernelGGL(k_reduce_bst_big<7>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 8: hipLaunchKernelGGL(k_reduce_bst_big<8>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 9: hipLaunchKernelGGL(k_reduce_bst_big<9>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 10: hipLaunchKernelGGL(k_reduce_bst_big<10>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        case 11: hipLaunchKernelGGL(k_reduce_bst_big<11>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
        default: hipLaunchKernelGGL(k_reduce_bst_big<12>, grid, block, 0, st, P, root, n, k, d_src, d_result); break;
    }
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

ecc_status_t ecc_allreduce_drop(int32_t P, int64_t m, const double *const *d_fresh,
                                const uint8_t *d_arrived, double *d_result, int32_t *d_count,
                                void *hip_stream) {
    clear_error();
    ECC_ARG(P >= 1, "P must be >= 1");
    ECC_ARG(m >= 0, "m must be >= 0");
    ECC_ARG(d_arrived != nullptr, "d_arrived is NULL");
    ECC_ARG(m == 0 || (d_fresh && d_result), "NULL contribution array or result");
    if (m == 0 && !d_count) return ECC_OK;
    hipLaunchKernelGGL(k_allreduce_drop, dim3(thr_grid(m)), dim3(kThrThreads), 0,
                       (hipStream_t)hip_stream, P, m, d_fresh, d_arrived, d_result, d_count);
    ECC_LAUNCH_CHECK();
    return ECC_OK;
}

}  // extern "C"
