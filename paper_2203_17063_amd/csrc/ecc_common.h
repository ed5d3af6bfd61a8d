// Internal definitions shared by the libecc translation units (HIP, gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "libecc.h"

namespace ecc {

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

#define ECC_HIP(expr)                                                                   \
    do {                                                                                \
        hipError_t e_ = (expr);                                                         \
        if (e_ != hipSuccess) {                                                         \
            ::ecc::set_error("%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_),     \
                             __FILE__, __LINE__);                                       \
            return ECC_ERR_DEVICE;                                                      \
        }                                                                               \
    } while (0)

#define ECC_LAUNCH_CHECK()                                                              \
    do {                                                                                \
        hipError_t e_ = hipGetLastError();                                              \
        if (e_ != hipSuccess) {                                                         \
            ::ecc::set_error("kernel launch failed: %s (%s:%d)", hipGetErrorString(e_), \
                             __FILE__, __LINE__);                                       \
            return ECC_ERR_DEVICE;                                                      \
        }                                                                               \
    } while (0)

#define ECC_ARG(cond, ...)                                                              \
    do {                                                                                \
        if (!(cond)) {                                                                  \
            ::ecc::set_error(__VA_ARGS__);                                              \
            return ECC_ERR_ARG;                                                         \
        }                                                                               \
    } while (0)

// ---------------------------------------------------------------------------
// layouts shared by host and device
// ---------------------------------------------------------------------------
constexpr int kAssembleThreads = 256;
constexpr int kAssembleTile = 2048;      // elements copied by one workgroup
constexpr int kReduceThreads = 256;
constexpr int kReduceElems = 4;          // elements per thread per rank (2 x 16 B)
constexpr int kSweepThreads = 256;
constexpr int kStreamCap = 2048;         // nonzeros staged in LDS by a stream item
constexpr int kStreamRows = 256;         // rows of one stream item at most
constexpr int kVectorCap = 16384;        // nonzeros of one vector item / piece
constexpr int kPass2Threads = 1024;

// One assembly tile: `len` elements of rank `rank` starting `off` elements
// into its block.
struct Tile {
    int64_t off;
    int32_t rank;
    int32_t len;
};

// One sweep work item.  kind: 0 stream (rows [row0, row0 + a)), 1 vector (row
// row0 by the whole workgroup), 2 piece a of row row0 (nonzeros
// [row_ptr[row0] + a*kVectorCap, ...), result to piece slot b).
enum { kItemStream = 0, kItemVector = 1, kItemPiece = 2 };
struct WorkItem {
    int32_t row0;
    int32_t a;
    int32_t b;
    int32_t kind_rank;  // kind << 24 | rank
};

// A row split into pieces, recombined by the second pass in piece order.
struct Fixup {
    int32_t row;
    int32_t slot0;
    int32_t npieces;
    int32_t rank;
};

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

// Staleness decision of Algorithm 1 for one rank at clock step t: the data
// last received (version) is used unless it is older than S steps, in which
// case the caller waits for an update (a forced arrival); never-received
// blocks arrive with the initial exchange.
__device__ __forceinline__ bool stale_select(int32_t version, uint8_t arrived, int64_t t,
                                             int32_t S) {
    return version < 0 || arrived != 0 || (t - (int64_t)version) > (int64_t)S;
}

// 64-bit lane exchange through two 32-bit DPP moves.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), CTRL, 0xf, 0xf, false);
    return __hiloint2double(hi, lo);
}

constexpr int kDppQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

// Sum over aligned groups of G lanes (G a power of two <= 64); every lane of
// the group receives the group's sum.  The pairing is fixed, so the result is
// deterministic.  All lanes of a group must be active.
template <int G>
__device__ __forceinline__ double group_sum(double v) {
    if constexpr (G >= 2) v += dpp_f64<kDppQuadXor1>(v);
    if constexpr (G >= 4) v += dpp_f64<kDppQuadXor2>(v);
    if constexpr (G >= 8) v += dpp_f64<kDppRowHalfMirror>(v);
    if constexpr (G >= 16) v += dpp_f64<kDppRowMirror>(v);
    if constexpr (G >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (G >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// Runtime group size version (g in {1,2,4,...,64}).
__device__ __forceinline__ double group_sum_dyn(double v, int g) {
    if (g >= 2) v += dpp_f64<kDppQuadXor1>(v);
    if (g >= 4) v += dpp_f64<kDppQuadXor2>(v);
    if (g >= 8) v += dpp_f64<kDppRowHalfMirror>(v);
    if (g >= 16) v += dpp_f64<kDppRowMirror>(v);
    if (g >= 32) v += __shfl_xor(v, 16, 64);
    if (g >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

// Deterministic workgroup sum (NT threads, a multiple of 64).  Returns the
// total in thread 0.  `scratch` holds NT/64 doubles of LDS.
template <int NT>
__device__ __forceinline__ double block_sum(double v, double *scratch) {
    v = group_sum<64>(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) scratch[wave] = v;
    __syncthreads();
    double total = 0.0;
    if (threadIdx.x == 0) {
        total = scratch[0];
        for (int w = 1; w < NT / 64; ++w) total += scratch[w];
    }
    __syncthreads();
    return total;
}

}  // namespace ecc

// ---------------------------------------------------------------------------
// opaque handles
// ---------------------------------------------------------------------------
struct ecc_plan_s {
    int32_t P = 0;
    int32_t S = 0;
    int device = 0;
    hipStream_t stream = nullptr;
    int64_t clock = 0;

    bool has_layout = false;
    bool tiles_rows = false;  // displs = exclusive scan of counts
    std::vector<int64_t> counts, displs;
    int64_t extent = 0;       // max(displs + counts)

    // device state (owned)
    int32_t *d_version = nullptr;   // [2][P], buffer (clock & 1) holds the current versions
    int32_t *d_age = nullptr;       // [P]
    uint8_t *d_eff = nullptr;       // [P] eff of the last call
    unsigned long long *d_forced = nullptr;  // total forced arrivals
    int64_t *d_displs = nullptr;    // [P]
    int32_t *d_block_start = nullptr;  // [P+1] when tiles_rows and extent < 2^31
    ecc::Tile *d_tiles = nullptr;   // assembly tiles (packed layout)
    int64_t n_tiles = 0;
    int32_t *d_ctrl = nullptr;      // [0] done flag, [1] iterations run (loop control)
    double *d_scalar = nullptr;     // scratch result of ecc_residual
};

struct ecc_matrix_s {
    ecc_plan_t plan = nullptr;
    ecc_csr_t A{};
    int32_t kind = 0;
    ecc::WorkItem *d_items = nullptr;
    int64_t n_items = 0;
    ecc::Fixup *d_fixups = nullptr;
    int64_t n_fixups = 0;
    double2 *d_pieces = nullptr;    // (partial sum, diagonal) per piece
    int64_t n_pieces = 0;
    double *d_partials = nullptr;   // internal partials used by ecc_solve
};

namespace ecc {
// kernels and launchers implemented in the .hip files
ecc_status_t launch_assemble(ecc_plan_t plan, const double *const *d_send,
                             const double *d_send_base, double *d_recv,
                             const uint8_t *d_arrived, uint8_t *d_eff_out, int32_t *d_age_out,
                             const int32_t *d_done);
ecc_status_t launch_sweep(ecc_matrix_t M, const double *d_b, double alpha, double beta,
                          const double *d_x_own, const double *d_x_hat, double *d_x_next,
                          double *d_partials, int32_t zero_extra, const int32_t *d_done);
// Split-row fix-up plus norm of one loop iteration (internal partials).
ecc_status_t solve_pass2(ecc_matrix_t M, int32_t norm, const double *d_b, double alpha,
                         double beta, const double *d_x_own, double *d_x_next, double *d_out,
                         double tol, int32_t *d_ctrl, int32_t t, const int32_t *d_done);
ecc_status_t check_plan(ecc_plan_t plan);
}  // namespace ecc
