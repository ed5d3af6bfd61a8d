// Loop control of the data path: T iterations of
//   staleness decision + assembly  ->  block-row sweep  ->  norm  ->  swap,
// each on the plan's next clock, enqueued without host round trips.  Each
// iteration is one fused kernel launch (see sweep.hip) unless the plan has
// more ranks than a workgroup stages in LDS, or the matrix has very uneven
// rows; then the assembly is its own launch.  A tolerance is checked on the
// device: the norm pass raises a flag that makes every later kernel of the
// loop return at entry, so the state (versions, ages, iterate) is exactly
// that after the first iteration below tolerance.
#include <algorithm>

#include "ecc_common.h"

namespace ecc {

__global__ void k_ctrl_reset(int32_t *ctrl) {
    if (threadIdx.x == 0) {
        ctrl[0] = 0;
        ctrl[1] = 0;
    }
}

}  // namespace ecc

using namespace ecc;

extern "C" ecc_status_t ecc_solve(ecc_plan_t plan, ecc_matrix_t A, const double *d_b,
                                  double alpha, double beta, double *d_x, double *d_x_tmp,
                                  double *d_x_hat, const uint8_t *d_mask, int32_t T, double tol,
                                  double *d_rho, uint8_t *d_eff_hist, int32_t *d_age_hist,
                                  int32_t *h_iters) {
    clear_error();
    ecc_status_t st = check_plan(plan);
    if (st != ECC_OK) return st;
    ECC_ARG(A != nullptr, "matrix is NULL");
    if (A->plan != plan) {
        set_error("matrix was created for another plan");
        return ECC_ERR_STATE;
    }
    ECC_ARG(T >= 0, "T must be >= 0");
    ECC_ARG(h_iters != nullptr, "h_iters is NULL");
    const int64_t n = A->A.n_rows;
    ECC_ARG(n == 0 || (d_x && d_x_tmp && d_x_hat), "NULL vector argument");
    ECC_ARG(d_x != d_x_tmp && d_x != d_x_hat && d_x_tmp != d_x_hat, "vectors must be distinct");
    ECC_ARG(T == 0 || (d_mask && d_rho), "d_mask and d_rho are required");
    ECC_ARG(A->kind != ECC_KIND_JACOBI || n == 0 || d_b, "d_b is NULL");
    const int32_t norm = (A->kind == ECC_KIND_JACOBI) ? ECC_NORM_L2 : ECC_NORM_L1;
    ECC_ARG(n == 0 || plan->d_block_start, "plan blocks do not tile the rows");
    const int64_t clock0 = plan->clock;
    const int32_t P = plan->P;

    if (A->tiny && T > 0 && n > 0) {
        // the whole loop in one launch; the last iterate lands in d_x, and the
        // kernel writes the loop control (which it sets whole) to the device
        // and to pinned host memory (every earlier solve of the plan has
        // synchronised, so no kernel still writes it)
        plan->h_ctrl[0] = 0;
        plan->h_ctrl[1] = -1;
        st = launch_solve_tiny(A, d_b, alpha, beta, d_x, d_x_hat, d_mask, T, tol, d_rho,
                               d_eff_hist, d_age_hist);
        if (st != ECC_OK) return st;
        ECC_HIP(hipStreamSynchronize(plan->stream));
        const int32_t iters = plan->h_ctrl[1];
        if (iters < 0 || iters > T) {
            set_error("the single-launch solve reported %d iterations", iters);
            return ECC_ERR_DEVICE;
        }
        plan->clock = clock0 + iters;
        *h_iters = iters;
        return ECC_OK;
    }
    hipLaunchKernelGGL(k_ctrl_reset, dim3(1), dim3(64), 0, plan->stream, plan->d_ctrl);
    ECC_LAUNCH_CHECK();
    const int32_t *done = plan->d_ctrl;
    const int64_t G1 = A->n_part;
    // Without a tolerance and without split rows, every iteration is a single
    // launch: workgroup 0 of launch t reduces launch t-1's partials (double
    // buffer), and one last pass reduces those of the final iteration.
    // Otherwise a one-workgroup pass follows each sweep (split rows, norm and
    // the convergence flag).  The assembly is fused into the sweep while the
    // rank state fits in LDS.
    // For matrices with very uneven rows (power-law graphs), whose columns are
    // spread at random, the fused kernel's rank lookup of every off-block
    // gather costs more than assembling first: assemble, then a sweep that
    // reads every other rank from the assembled vector (measured on MI355X,
    // PageRank on a scale-22 R-MAT graph: 67.2 against 70.0 ms per solve).
    const bool fused = P <= kFusedMaxP && A->layout != kLaySorted && A->layout != kLayRanges;
    const bool deferred = fused && tol <= 0.0 && A->n_fixups == 0;
    double *cur = d_x, *nxt = d_x_tmp;
    for (int32_t t = 0; t < T; ++t) {
        const int64_t tt = plan->clock;
        const uint8_t *mask_t = d_mask + (int64_t)t * P;
        uint8_t *eff_t = d_eff_hist ? d_eff_hist + (int64_t)t * P : nullptr;
        int32_t *age_t = d_age_hist ? d_age_hist + (int64_t)t * P : nullptr;
        double *part = A->d_partials + (deferred ? (t & 1) * G1 : 0);
        if (!fused) {
            // a column-value matrix's assembly also forms the scaled views
            st = A->colscale
                     ? launch_assemble_scaled(A, cur, d_x_hat, mask_t, eff_t, age_t, done)
                     : launch_assemble(plan, nullptr, cur, d_x_hat, mask_t, eff_t, age_t, done);
            if (st != ECC_OK) return st;
        }
        SweepLaunch L;
        L.b = d_b;
        L.alpha = alpha;
        L.beta = beta;
        L.x_own = cur;
        L.x_hat = d_x_hat;
        L.x_next = nxt;
        L.partials = part;
        L.norm = norm;
        L.done = done;
        L.scaled = !fused && A->colscale;
        if (fused) {
            L.arrived = mask_t;
            L.eff_user = eff_t;
            L.age_user = age_t;
        }
        if (deferred && t > 0) {
            L.prev_partials = A->d_partials + ((t - 1) & 1) * G1;
            L.prev_rho = d_rho + (t - 1);
        }
        st = launch_sweep(A, L);
        if (st != ECC_OK) return st;
        if (!deferred || t == T - 1) {
            Pass2Launch F;
            F.partials = part;
            F.b = d_b;
            F.alpha = alpha;
            F.beta = beta;
            F.x_own = cur;
            F.x_next = nxt;
            F.x_hat = d_x_hat;
            F.step = fused;
            F.norm = norm;
            F.rho_out = d_rho + t;
            F.tol = tol;
            F.ctrl = plan->d_ctrl;
            F.t = tt - clock0;
            F.done = done;
            st = launch_pass2(A, F);
            if (st != ECC_OK) return st;
        }
        std::swap(cur, nxt);
    }
    int32_t ctrl[2] = {0, 0};
    ECC_HIP(hipMemcpyAsync(ctrl, plan->d_ctrl, sizeof(ctrl), hipMemcpyDeviceToHost, plan->stream));
    ECC_HIP(hipStreamSynchronize(plan->stream));
    const int32_t iters = ctrl[1];
    plan->clock = clock0 + iters;
    *h_iters = iters;
    // iterate x^iters sits in d_x for an even count, in d_x_tmp for an odd one
    if ((iters & 1) && n > 0) {
        ECC_HIP(hipMemcpyAsync(d_x, d_x_tmp, sizeof(double) * n, hipMemcpyDeviceToDevice,
                               plan->stream));
        ECC_HIP(hipStreamSynchronize(plan->stream));
    }
    return ECC_OK;
}
