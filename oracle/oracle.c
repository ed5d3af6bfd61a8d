/*
 * ORACLE -- test infrastructure only.
 *
 * A plain, slow, sequential CPU statement of what the eventually consistent
 * collective data path computes.  Only the tests, the smoke check and the
 * CPU-baseline leg of the benchmark may load it; the product path never
 * does.  It shares no code, header or table with the GPU library.
 *
 * Built with gcc -O2 -ffp-contract=off: every a*b+c below is a rounded
 * product followed by a rounded sum, exactly in the order written.  Row
 * loops may run on several OpenMP threads; each row is computed by one
 * thread in the same order, so the results do not depend on the thread
 * count.  Sums over many elements are done afterwards, sequentially.
 *
 * Notation (paper: Iakymchuk et al., "Efficient and Eventually Consistent
 * Collective Operations", Section III-A and Algorithm 1):
 *   P ranks own blocks [displs[p], displs[p] + counts[p]);
 *   t   = iteration index = the paper's clock minus one (the clock is
 *         incremented on entry to the collective);
 *   S   = the paper's slack, the maximum accepted staleness;
 *   version[p] = iteration at which block p last arrived (-1: never).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ------------------------------------------------------------------------
 * Staleness decision.  Algorithm 1 accepts the last received contribution
 * when its clock is at least clock - slack (age <= S) and otherwise waits
 * for an update.  In a step-by-step emulation the only newer data is the
 * current iterate, so a wait delivers version t ("forced" arrival).  A
 * block never received before (version -1) is delivered by the initial
 * exchange and is not counted as forced.
 *   eff[p]     = version[p] < 0  or  arrived[p]  or  t - version[p] > S
 *   version[p] = t where eff[p]
 *   age[p]     = t - version[p]       (always 0 <= age <= S afterwards)
 * Returns the number of forced arrivals in this step.
 * ---------------------------------------------------------------------- */
int64_t orc_select(int32_t P, int64_t S, int64_t t, const uint8_t *arrived,
                   int32_t *version, uint8_t *eff, int32_t *age) {
    int64_t forced = 0;
    for (int32_t p = 0; p < P; ++p) {
        const int never = version[p] < 0;
        const int too_stale = !never && (t - (int64_t)version[p] > S);
        const int e = never || arrived[p] || too_stale;
        if (e && !arrived[p] && !never) forced += 1;
        eff[p] = (uint8_t)e;
        if (e) version[p] = (int32_t)t;
        age[p] = (int32_t)(t - (int64_t)version[p]);
    }
    return forced;
}

/* ------------------------------------------------------------------------
 * allgatherv assembly with last-received semantics.  Every rank's block has
 * dedicated receive memory that a new contribution overwrites and that is
 * re-read when no new contribution arrives (the paper's rcv_data_vec).
 * For each p with eff[p]:  recv[displs[p] + j] = send[p][j],  0 <= j < counts[p].
 * Blocks without eff, and gaps between blocks, are left untouched.
 * ---------------------------------------------------------------------- */
void orc_allgatherv(int32_t P, const int64_t *counts, const int64_t *displs,
                    const uint8_t *eff, const double *const *send, double *recv) {
    for (int32_t p = 0; p < P; ++p) {
        if (!eff[p]) continue;
        for (int64_t j = 0; j < counts[p]; ++j) recv[displs[p] + j] = send[p][j];
    }
}

/* ------------------------------------------------------------------------
 * Partial allreduce (sum).  Algorithm 1 starts from the rank's own new
 * contribution and reduces it with the last received data, so the result
 * combines, per rank, the newest contribution it holds: the fresh one where
 * eff[p], else the one kept in the rank's slot (stale contributions are
 * substituted).
 *   for eff p:  slot[p] = fresh[p]
 *   result[i] = ((slot[0][i] + slot[1][i]) + slot[2][i]) + ...   (rank order)
 * ---------------------------------------------------------------------- */
void orc_allreduce(int32_t P, int64_t m, const uint8_t *eff, const double *const *fresh,
                   double *const *slots, double *result) {
    for (int32_t p = 0; p < P; ++p)
        if (eff[p])
            for (int64_t i = 0; i < m; ++i) slots[p][i] = fresh[p][i];
    for (int64_t i = 0; i < m; ++i) {
        double acc = slots[0][i];
        for (int32_t p = 1; p < P; ++p) acc = acc + slots[p][i];
        result[i] = acc;
    }
}

/* Clock of a reduced result: the minimum of the clocks reduced into it. */
int64_t orc_result_clock(int32_t P, const int32_t *version) {
    int64_t c = version[0];
    for (int32_t p = 1; p < P; ++p)
        if (version[p] < c) c = version[p];
    return c;
}

/* ------------------------------------------------------------------------
 * Block-row Jacobi sweep (textbook Jacobi, e.g. Saad, "Iterative Methods
 * for Sparse Linear Systems", Sec. 4.1) on the view rank p has of x:
 * its own block from x_own (always current), every other block from the
 * assembled vector x_hat.  For row i of block p = [lo, hi):
 *   y_j      = x_own[j] if lo <= j < hi, else x_hat[j]
 *   s        = sum over the row's off-diagonal entries, in CSR order, of a_ij*y_j
 *   x_next_i = (b_i - s) / a_ii
 *   r_i      = (b_i - s) - a_ii * x_own[i]
 * ---------------------------------------------------------------------- */
void orc_jacobi_sweep(int32_t P, const int64_t *block_start, const int32_t *row_ptr,
                      const int32_t *col, const double *val, const double *b,
                      const double *x_own, const double *x_hat, double *x_next,
                      double *r, int nthreads) {
    for (int32_t p = 0; p < P; ++p) {
        const int64_t lo = block_start[p], hi = block_start[p + 1];
#pragma omp parallel for schedule(static) num_threads(nthreads)
        for (int64_t i = lo; i < hi; ++i) {
            double s = 0.0, aii = 0.0;
            for (int64_t k = row_ptr[i]; k < row_ptr[i + 1]; ++k) {
                const int64_t j = col[k];
                if (j == i) {
                    aii = val[k];
                    continue;
                }
                const double y = (j >= lo && j < hi) ? x_own[j] : x_hat[j];
                s = s + val[k] * y;
            }
            x_next[i] = (b[i] - s) / aii;
            r[i] = (b[i] - s) - aii * x_own[i];
        }
    }
}

/* ------------------------------------------------------------------------
 * Block-row power-iteration step for PageRank (Page, Brin, Motwani,
 * Winograd 1999) with W = A^T D^-1 stored row by row (row j lists the
 * sources i of the edges i -> j):
 *   s        = sum over row j, in CSR order, of w_ji * y_i  (y as for Jacobi)
 *   x_next_j = alpha * s + beta
 *   d_j      = |x_next_j - x_own[j]|
 * ---------------------------------------------------------------------- */
void orc_power_sweep(int32_t P, const int64_t *block_start, const int32_t *row_ptr,
                     const int32_t *col, const double *val, double alpha, double beta,
                     const double *x_own, const double *x_hat, double *x_next, double *d,
                     int nthreads) {
    for (int32_t p = 0; p < P; ++p) {
        const int64_t lo = block_start[p], hi = block_start[p + 1];
#pragma omp parallel for schedule(dynamic, 4096) num_threads(nthreads)
        for (int64_t j = lo; j < hi; ++j) {
            double s = 0.0;
            for (int64_t k = row_ptr[j]; k < row_ptr[j + 1]; ++k) {
                const int64_t i = col[k];
                const double y = (i >= lo && i < hi) ? x_own[i] : x_hat[i];
                s = s + val[k] * y;
            }
            x_next[j] = alpha * s + beta;
            d[j] = fabs(x_next[j] - x_own[j]);
        }
    }
}

/* ------------------------------------------------------------------------
 * Norms.  Neumaier's compensated summation (Neumaier 1974; Higham,
 * "Accuracy and Stability of Numerical Algorithms", ch. 4), sequential
 * over i, so the oracle's norms are accurate to a few units in the last
 * place independently of n.
 *   L2: sqrt(sum_i v_i*v_i)        L1: sum_i |v_i|
 * ---------------------------------------------------------------------- */
double orc_norm(int64_t n, const double *v, int32_t which) {
    double s = 0.0, c = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double x = (which == 2) ? v[i] * v[i] : fabs(v[i]);
        const double t = s + x;
        if (fabs(s) >= fabs(x)) c = c + ((s - t) + x);
        else c = c + ((x - t) + s);
        s = t;
    }
    return (which == 2) ? sqrt(s + c) : s + c;
}
