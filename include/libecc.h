/*
 * libecc -- eventually consistent collectives and the iterations they feed,
 * on one AMD Instinct MI355X (gfx950).
 *
 * Method: Iakymchuk et al., "Efficient and Eventually Consistent Collective
 * Operations" (arXiv 2203.17063).  Section III-A and Algorithm 1 define the
 * stale-synchronous (SSP) collective: each call advances a logical clock,
 * a contribution is used if its clock is at least clock - slack, and only
 * data that is too stale makes the caller wait for an update; the last data
 * received for each source is kept in dedicated receive memory and re-read
 * when nothing newer has arrived; a reduced result carries the minimum
 * clock of its inputs.  Section III also names the two extra collective
 * parameters this library exposes as outputs ("status": which blocks were
 * used, their age, the clock of the result).  Table I and Section II give
 * the resource model: resources are allocated and metadata exchanged once
 * at set-up and released at shut-down.
 *
 * Here P "virtual ranks" live on one GPU: rank p's contribution is a block
 * of a vector in HBM, a delivery is a copy plus a version update, and the
 * arrival of each block at each clock comes from a caller-supplied mask.
 *
 * Conventions for every call:
 *   - Pointers prefixed d_ are device (HBM) pointers, h_ are host pointers.
 *     The caller owns every vector, mask, slot and matrix array; the library
 *     never frees caller memory.  A plan owns only its small metadata.
 *   - Calls are asynchronous on the plan's HIP stream unless stated.  Buffers
 *     passed to a call must stay valid until the stream reaches that work.
 *   - Every call returns an ecc_status_t.  Argument errors are detected on the
 *     host before anything is enqueued and leave the plan unchanged; the text
 *     of the last error of the calling thread is ecc_last_error().
 *   - A plan is not thread-safe.  Calls that share a plan, or that write the
 *     same buffers, must not overlap.
 *   - Indices of CSR matrices are int32 (nnz < 2^31); values are fp64.
 */
#ifndef LIBECC_H
#define LIBECC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ecc_plan_s *ecc_plan_t;
typedef struct ecc_matrix_s *ecc_matrix_t;
typedef struct ecc_hypercube_s *ecc_hypercube_t;
typedef struct ecc_mf_s *ecc_mf_t;

typedef enum {
    ECC_OK = 0,
    ECC_ERR_ARG = 1,      /* a bad argument (null pointer, negative size, ...) */
    ECC_ERR_OVERLAP = 2,  /* two ranks' blocks overlap in the receive vector   */
    ECC_ERR_RANGE = 3,    /* a size exceeds what the layout supports           */
    ECC_ERR_ALLOC = 4,    /* a device or host allocation failed                */
    ECC_ERR_DEVICE = 5,   /* a HIP call or kernel launch failed                */
    ECC_ERR_STATE = 6     /* the call does not fit the plan or matrix          */
} ecc_status_t;

/* max_staleness value meaning "no bound": after the initial exchange a block
 * is taken only when it arrives, never forced. */
#define ECC_UNBOUNDED 0x7fffffff

#define ECC_NORM_L1 1
#define ECC_NORM_L2 2

#define ECC_KIND_JACOBI 0  /* x_next_i = (b_i - sum_{j!=i} a_ij y_j) / a_ii       */
#define ECC_KIND_POWER 1   /* x_next_j = alpha * sum_i w_ji y_i + beta           */

typedef struct {
    int64_t n_rows, n_cols, nnz;
    const int32_t *d_row_ptr; /* [n_rows + 1], row_ptr[0] = 0, non-decreasing */
    const int32_t *d_col;     /* [nnz], each in [0, n_cols)                   */
    const double *d_val;      /* [nnz]                                        */
} ecc_csr_t;

/* ---------------------------------------------------------------------------
 * Host-only helpers (no GPU needed).
 * ------------------------------------------------------------------------- */

/* Version of this interface (incremented on incompatible changes). */
int32_t ecc_abi_version(void);

/* Text of the last error on the calling thread ("" if none). */
const char *ecc_last_error(void);

/* Name of a status code. */
const char *ecc_status_string(ecc_status_t s);

/* Check a block layout without creating anything.  Same rules as
 * ecc_plan_create: P >= 1; max_staleness >= 0; if h_counts is non-NULL then
 * h_displs must be too, every count and displacement is >= 0, and no two
 * non-empty blocks [displs[p], displs[p] + counts[p]) overlap
 * (ECC_ERR_OVERLAP); the extent max(displs + counts) must be < 2^40
 * (ECC_ERR_RANGE).  Unsorted displacements and gaps are allowed. */
ecc_status_t ecc_plan_validate(int32_t P, const int64_t *h_counts, const int64_t *h_displs,
                               int32_t max_staleness);

/* ---------------------------------------------------------------------------
 * Plan: the set-up phase of Table I.  A plan holds the rank layout, the
 * slack S (max_staleness), the logical clock and, per rank, the version
 * (clock at which its data last arrived; -1 before the first call) and age.
 * ------------------------------------------------------------------------- */

/* Create a plan for P ranks.  h_counts/h_displs (host, P entries each,
 * copied) describe where rank p's block lives in the assembled vector; both
 * may be NULL for a plan used only with ecc_allreduce_partial.  hip_stream is
 * a hipStream_t (NULL: the default stream).  Allocates a few KB of device
 * memory on the current device.  Validation as ecc_plan_validate. */
ecc_status_t ecc_plan_create(int32_t P, const int64_t *h_counts, const int64_t *h_displs,
                             int32_t max_staleness, void *hip_stream, ecc_plan_t *out);

/* Release the plan's device metadata (waits for its stream first). */
ecc_status_t ecc_plan_destroy(ecc_plan_t plan);

/* Clock := 0, every version := -1, forced counter := 0 (asynchronous). */
ecc_status_t ecc_plan_reset(ecc_plan_t plan);

/* Change the stream later calls are enqueued on. */
ecc_status_t ecc_plan_set_stream(ecc_plan_t plan, void *hip_stream);

/* Synchronising read of the plan state: clock (= number of collective calls
 * since create/reset), total forced arrivals, and optionally the per-rank
 * version and age after the last call (host arrays of P int32, nullable). */
ecc_status_t ecc_plan_stats(ecc_plan_t plan, int64_t *clock, int64_t *forced_total,
                            int32_t *h_version, int32_t *h_age);

/* Optional per-kernel timing on the plan's stream (diagnostics).  While
 * enabled, each launch of the libecc kernels below is bracketed by two HIP
 * events recorded on the plan's stream; ecc_plan_timing synchronises, adds
 * up the elapsed times of the launches recorded so far for one kernel, and
 * optionally clears them.  Disabled by default; enabling it adds two event
 * records per launch. */
#define ECC_TIMING_ASSEMBLE 0   /* staleness decision + assembly */
#define ECC_TIMING_ALLREDUCE 1  /* partial allreduce             */
#define ECC_TIMING_SWEEP 2      /* Jacobi / power-iteration sweep */
#define ECC_TIMING_NORM 3       /* split-row fix-up + norm pass  */
#define ECC_TIMING_MF_GRAD 4    /* factorisation: errors + worker gradients */
#define ECC_TIMING_MF_STEP 5    /* factorisation: model step + RMSE */
#define ECC_TIMING_KINDS 6
ecc_status_t ecc_plan_set_timing(ecc_plan_t plan, int32_t enable);
ecc_status_t ecc_plan_timing(ecc_plan_t plan, int32_t kernel, double *total_ms,
                             int64_t *launches, int32_t reset);

/* ---------------------------------------------------------------------------
 * Collectives.  Each call is one clock step t = current clock (Algorithm 1
 * increments the clock on entry; t is that value minus one) and advances the
 * clock by one.  The staleness decision for every rank p is
 *     eff[p] = version[p] < 0  ||  arrived[p]  ||  t - version[p] > S
 * (the caller waits only for data older than the slack: a block older than S
 * clocks is delivered now, a *forced* arrival); then version[p] := t where
 * eff[p] and age[p] := t - version[p], so 0 <= age <= S.
 * ------------------------------------------------------------------------- */

/* allgatherv-style assembly with last-received semantics (the per-source
 * receive memory of Section III-A, rcv_data_vec).  For every rank with
 * eff[p]:  d_recv[displs[p] + j] = d_send[p][j] for 0 <= j < counts[p].
 * Blocks without eff, and gaps between blocks, keep their previous contents.
 *   d_send     device array of P device pointers (rank p's block); entries of
 *              ranks with count 0 are not read.  The blocks must not overlap
 *              d_recv's written ranges.
 *   d_recv     device vector of at least max(displs + counts) doubles.
 *   d_arrived  device array of P bytes (non-zero: arrived at this clock).
 *   d_eff_out  optional device array of P bytes: eff of this call.
 *   d_age_out  optional device array of P int32: age after this call.
 * Requires a plan created with counts/displs (else ECC_ERR_STATE). */
ecc_status_t ecc_allgatherv_assemble(ecc_plan_t plan, const double *const *d_send,
                                     double *d_recv, const uint8_t *d_arrived,
                                     uint8_t *d_eff_out, int32_t *d_age_out);

/* Same, with every rank's block at the same offset in one packed send
 * vector: rank p's block starts at d_send_base + displs[p]. */
ecc_status_t ecc_allgatherv_assemble_packed(ecc_plan_t plan, const double *d_send_base,
                                            double *d_recv, const uint8_t *d_arrived,
                                            uint8_t *d_eff_out, int32_t *d_age_out);

/* Partial allreduce (sum) with stale substitution: the reduction of
 * Algorithm 1 over the newest contribution held for each rank.  This is the
 * stale mode of the partial allreduce; the mode that drops contributions
 * that did not arrive is the separate call ecc_allreduce_drop (it keeps no
 * slots, versions or clock, so it takes no plan) instead of a mode argument
 * here.
 *   for every p with eff[p]:  d_slots[p][i] = d_fresh[p][i]
 *   d_result[i] = ((slot_0[i] + slot_1[i]) + slot_2[i]) + ...   (rank order,
 *                 so the result is bitwise reproducible)
 *   *d_result_clock = min_p version[p]  (the minimum-clock rule; nullable)
 *   m          elements per rank (>= 0).
 *   d_fresh    device array of P device pointers to this clock's
 *              contributions (read only where eff[p]).
 *   d_slots    device array of P device pointers to the caller-owned receive
 *              memory of each rank (m doubles each); read every call, written
 *              where eff[p].  At the plan's first call every rank is eff, so
 *              the slots need no initialisation.  d_fresh[p] may equal
 *              d_slots[p]: the contribution was then written into the slot
 *              by its producer, which must do so only where eff[p] (the
 *              slot keeps the newest taken contribution), and the slot is
 *              read without being written.
 *   d_result   device vector of m doubles; must not alias any slot or fresh.
 *   d_arrived, d_eff_out as for the assembly. */
ecc_status_t ecc_allreduce_partial(ecc_plan_t plan, int64_t m, const double *const *d_fresh,
                                   double *const *d_slots, double *d_result,
                                   const uint8_t *d_arrived, uint8_t *d_eff_out,
                                   int32_t *d_result_clock);

/* ---------------------------------------------------------------------------
 * Block-row iterations consuming the assembled vector.  Rank p owns rows
 * [displs[p], displs[p] + counts[p]); the plan's blocks must tile
 * [0, n_rows) in rank order (displs = exclusive prefix sum of counts) and
 * the matrix must be square, else ECC_ERR_STATE.  Row i of block
 * p = [lo, hi) reads the view
 *     y_j = x_own[j] if lo <= j < hi  (a rank's own block is always current)
 *     y_j = x_hat[j] otherwise        (the assembled, possibly stale, vector)
 * ------------------------------------------------------------------------- */

/* Analyse a CSR matrix once for a plan (set-up, synchronising): builds the
 * row-block work list (blocks never straddle a rank boundary; rows longer
 * than one work item are split and recombined in a fixed order), and for
 * ECC_KIND_JACOBI checks that every row has exactly one diagonal entry and
 * that it is non-zero (else ECC_ERR_ARG).  It chooses the sweep layout:
 *   ECC_LAYOUT_SHORT   every row holds at most 8 entries: work items are
 *                      runs of up to 256 rows of one rank, one lane per row,
 *                      and the entries are copied item by item in the order
 *                      the items are swept, each item's entries stored
 *                      entry-major (entry k of all its rows together) and
 *                      padded to the longest row's class R in {3, 4, 5, 7, 8}
 *                      (about 12 bytes x R x n_rows of device memory).  When
 *                      the columns of every row lie near the row itself or
 *                      near the rows one "plane" away (the bandwidth B: a
 *                      3-D grid stencil), and B rows are too many for the
 *                      rows one plane apart to meet in L2, the items are
 *                      swept in plane tiles: rows [z B + tau W, z B + (tau
 *                      + 1) W) for every plane z, tile after tile, so that
 *                      a row's neighbours one plane away were read a few
 *                      items earlier (ecc_matrix_tiling reports B and W);
 *   ECC_LAYOUT_SORTED  very uneven rows (longest > 64 and > 8 x (mean + 1))
 *                      over a vector of at most one column range (below):
 *                      the rows of every rank are copied in order of
 *                      decreasing length (12 bytes x nnz + 8 bytes x n_rows
 *                      of device memory) and swept in runs staged in LDS;
 *   ECC_LAYOUT_RANGES  very uneven rows over a longer vector: the columns are
 *                      cut into R = ceil(8 x n_rows / 8 MiB) ranges of equal
 *                      width (16 MiB in the column-value form below;
 *                      2 <= R <= 16; ecc_matrix_opts_t.range_bytes
 *                      replaces the 8 MiB), every row into its entries of
 *                      each range, and these
 *                      sub-rows are copied range by range in order of
 *                      decreasing length class (12 bytes x nnz, 12 bytes per
 *                      sub-row, 8 x R + 2 bytes x n_rows of device memory,
 *                      plus 8 bytes x n_rows for Jacobi; the host copies the
 *                      entries once here).  A sweep sums every sub-row,
 *                      then adds a row's sub-row sums in range order: the
 *                      result differs from the CSR-order sum by rounding;
 *   ECC_LAYOUT_STREAM  otherwise: runs of rows staged in LDS.
 * ECC_LAYOUT_STREAM reads the matrix arrays at every sweep: they must then
 * outlive the handle and stay unchanged.  The other layouts sweep the copy
 * made here.  Two compact forms of the copy, reported by ecc_matrix_form,
 * leave the results bit for bit as the general form gives them:
 * Diagonals (ECC_LAYOUT_SHORT): when every row's entries are in increasing
 * column order and lie on at most as many offsets col - row as the row class
 * R holds (a grid stencil: 3 offsets in 1-D, 5 in 2-D, 7 in 3-D), the copy
 * keeps each row's values by diagonal and one byte per row naming the
 * diagonals it holds, in place of the column indices (8 bytes x R per row
 * instead of 12 bytes x R); diagonals are summed in increasing offset order,
 * which is the rows' CSR order.
 * Column values (ECC_KIND_POWER in ECC_LAYOUT_SORTED or ECC_LAYOUT_RANGES):
 * when all entries of every column j hold one value c_j, bit for bit -- the
 * PageRank matrix W = A^T D^-1 of Section IV holds 1 / outdeg(j) throughout
 * column j -- the copy keeps c (8 bytes x n_rows) in place of the entries'
 * values (8 bytes x nnz).  Every sweep then first forms z_own = c * x_own
 * and z_hat = c * x_hat elementwise (in 16 bytes x n_rows the handle owns)
 * and adds z_j where the general form adds w_ij * y_j: the same IEEE
 * product of the same two operands, so the iterates are bit for bit those
 * of the general form (the residual norm agrees to rounding: the kernel
 * stages no values, more of its workgroups fit on the device, and the
 * per-workgroup partial sums group the rows differently).  In
 * ECC_LAYOUT_RANGES the 1,024 columns gathered most often from outside
 * their own rank block also get a copy of their z_hat values (16 bytes per
 * column in the handle, 8 bytes more formed with the views) that every
 * sweep workgroup reads into LDS; the values gathered are the same. */
#define ECC_LAYOUT_STREAM 0
#define ECC_LAYOUT_SORTED 1
#define ECC_LAYOUT_SHORT 2
#define ECC_LAYOUT_RANGES 3
ecc_status_t ecc_matrix_create(ecc_plan_t plan, const ecc_csr_t *A, int32_t kind,
                               ecc_matrix_t *out);
ecc_status_t ecc_matrix_destroy(ecc_matrix_t A);

/* Set-up choices of ecc_matrix_create_ex; all zero gives ecc_matrix_create's
 * defaults.  They change how a sweep is laid out and ordered, never what it
 * computes, except that range_bytes changes the ECC_LAYOUT_RANGES rounding
 * (the number of sub-row sums added per row).
 *   range_bytes  ECC_LAYOUT_RANGES: bytes of the vector per column range
 *                (0: 8 MiB, 16 MiB in the column-value form).
 *   tile_rows    ECC_LAYOUT_SHORT plane tiles: 0 chosen from the matrix, > 0
 *                that many rows per tile (rounded up to a multiple of 256;
 *                applied only to a matrix that qualifies for tiling), < 0
 *                items in row order.
 *   schedule     ECC_LAYOUT_SHORT: how a sweep's workgroups share the items.
 *                ECC_SCHEDULE_STATIC: each walks a fixed set (items cut into
 *                eight ranges, one per XCD).  ECC_SCHEDULE_QUEUE: each claims
 *                the next item of its XCD's range with an atomic ticket (and
 *                of the other ranges once its own is exhausted); each item
 *                then writes its own partial norm, so ecc_partials_size is
 *                the item count + 1.  ECC_SCHEDULE_SINGLE: ecc_solve runs
 *                the whole loop as one launch of one 1,024-thread workgroup
 *                holding the vectors in LDS, for at most 2,048 rows (4,096
 *                rows of at most 3 entries), 64 items and 1,024 ranks (else
 *                as ECC_SCHEDULE_AUTO); the other calls use the queue's
 *                per-item partials.
 *                ECC_SCHEDULE_AUTO (0): the single launch when the problem
 *                fits it, else the queue when a workgroup would walk at
 *                least 16 items, else the static walk.
 *   compact      ECC_COMPACT_AUTO (0): a compact form of the copy (above)
 *                whenever the matrix qualifies; ECC_COMPACT_NONE: the
 *                general form always.
 * opts may be NULL (the defaults).  ECC_ERR_ARG for a negative range_bytes,
 * an unknown schedule or an unknown compact choice. */
#define ECC_SCHEDULE_AUTO 0
#define ECC_SCHEDULE_STATIC 1
#define ECC_SCHEDULE_QUEUE 2
#define ECC_SCHEDULE_SINGLE 3
#define ECC_COMPACT_AUTO 0
#define ECC_COMPACT_NONE 1
typedef struct {
    int64_t range_bytes;
    int64_t tile_rows;
    int32_t schedule;
    int32_t compact;
} ecc_matrix_opts_t;
ecc_status_t ecc_matrix_create_ex(ecc_plan_t plan, const ecc_csr_t *A, int32_t kind,
                                  const ecc_matrix_opts_t *opts, ecc_matrix_t *out);

/* ECC_LAYOUT_SHORT plane tiling chosen at set-up (host only): *plane_rows =
 * the bandwidth B taken as the plane size and *tile_rows = W, both 0 when
 * the items are swept in row order. */
ecc_status_t ecc_matrix_tiling(ecc_matrix_t A, int64_t *plane_rows, int64_t *tile_rows);

/* The form of the copy ecc_matrix_create made (host only):
 * ECC_FORM_GENERAL, ECC_FORM_DIAGONALS or ECC_FORM_COLUMN_VALUES.  For the
 * diagonal form *n_diagonals = their number and offsets[0 ..
 * ECC_MAX_DIAGONALS - 1] their offsets col - row in increasing order (0
 * past the last); otherwise 0 and zeros.  n_diagonals and offsets may be
 * NULL. */
#define ECC_FORM_GENERAL 0
#define ECC_FORM_COLUMN_VALUES 1
#define ECC_FORM_DIAGONALS 2
#define ECC_MAX_DIAGONALS 8
ecc_status_t ecc_matrix_form(ecc_matrix_t A, int32_t *form, int32_t *n_diagonals,
                             int32_t *offsets);

/* Schedule chosen at set-up (host only): ECC_SCHEDULE_STATIC,
 * ECC_SCHEDULE_QUEUE or ECC_SCHEDULE_SINGLE. */
ecc_status_t ecc_matrix_schedule(ecc_matrix_t A, int32_t *schedule);

/* The layout ecc_matrix_create chose (ECC_LAYOUT_*) and, for
 * ECC_LAYOUT_SHORT, the entries held per row R, for ECC_LAYOUT_RANGES the
 * number of column ranges (0 otherwise).  Host only. */
ecc_status_t ecc_matrix_layout(ecc_matrix_t A, int32_t *layout, int32_t *row_slots);

/* Number of doubles a d_partials buffer for this matrix must hold. */
int64_t ecc_partials_size(ecc_matrix_t A);

/* One Jacobi sweep (textbook Jacobi on the block-row view above):
 *   s_i = sum over the row's off-diagonal entries of a_ij * y_j (CSR order)
 *   d_x_next[i] = (b_i - s_i) / a_ii
 *   r_i = (b_i - s_i) - a_ii * x_own[i]
 * and writes ecc_partials_size(A) partial sums of r_i^2 to d_partials, whose
 * total ecc_residual(..., ECC_NORM_L2, ...) turns into ||r||_2.  d_x_next
 * must not alias d_x_own, d_x_hat or d_b.  Does not advance the clock. */
ecc_status_t ecc_iterate_jacobi(ecc_plan_t plan, ecc_matrix_t A, const double *d_b,
                                const double *d_x_own, const double *d_x_hat,
                                double *d_x_next, double *d_partials);

/* One power-iteration step (PageRank with W = A^T D^-1 stored by rows):
 *   d_x_next[j] = alpha * (sum_i w_ji * y_i) + beta
 * with partial sums of |x_next_j - x_own_j| in d_partials (ECC_NORM_L1). */
ecc_status_t ecc_iterate_spmv(ecc_plan_t plan, ecc_matrix_t W, double alpha, double beta,
                              const double *d_x_own, const double *d_x_hat, double *d_x_next,
                              double *d_partials);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): one
 * ecc_iterate_jacobi sweep followed by its ecc_residual(..., ECC_NORM_L2,
 * ...), without the caller's d_partials workspace.  The partial sums are
 * kept in a static device array of the library, ECC_SCRATCH_DOUBLES doubles
 * (8 MiB) on each GPU it runs on, held until the process ends; *d_rho
 * (device, asynchronous) receives ||r||_2.  Results are bitwise those of
 * ecc_iterate_jacobi + ecc_residual (the same kernels and order).  Calls no
 * allocation routine.  ECC_ERR_RANGE when ecc_partials_size(A) exceeds
 * ECC_SCRATCH_DOUBLES; other errors as ecc_iterate_jacobi.  Every call on a
 * GPU uses that GPU's one array: calls that overlap on one GPU (from other
 * streams or threads) race. */
#define ECC_SCRATCH_DOUBLES (1 << 20)
ecc_status_t ecc_iterate_jacobi_noalloc(ecc_plan_t plan, ecc_matrix_t A, const double *d_b,
                                        const double *d_x_own, const double *d_x_hat,
                                        double *d_x_next, double *d_rho);

/* Second pass of the norm: reduces n_partials values in a fixed order
 * (deterministic) to sqrt(sum) (ECC_NORM_L2) or sum (ECC_NORM_L1).  Writes
 * *d_out (device, asynchronous) and/or *h_out (host: synchronises); at least
 * one must be non-NULL. */
ecc_status_t ecc_residual(ecc_plan_t plan, const double *d_partials, int64_t n_partials,
                          int32_t norm, double *h_out, double *d_out);

/* ---------------------------------------------------------------------------
 * Loop control: T iterations of  assemble -> sweep -> norm -> swap, each on
 * the plan's next clock.  ECC_KIND_JACOBI uses d_b and the L2 residual;
 * ECC_KIND_POWER uses alpha, beta and the L1 norm of the update.  If tol > 0
 * the loop stops after the first iteration whose norm is below tol (checked
 * on the device: no host round trip per iteration).
 *   d_x       in: x^0; out: the last iterate.  n_rows doubles.
 *   d_x_tmp   workspace, n_rows doubles.
 *   d_x_hat   the assembled vector, n_rows doubles.  in: as the plan's last
 *             clock left it (blocks that do not arrive at the first iteration
 *             keep these values; unused at the plan's first clock, when every
 *             block arrives); out: as the last iteration leaves it.
 *   d_mask    device [T][P] bytes; row t is the arrival mask of iteration t.
 *   d_rho     device [T] doubles: the norm of every iteration run.
 *   d_eff_hist, d_age_hist  optional device [T][P] histories.
 *   h_iters   out: iterations run.
 * Synchronises at the end. */
ecc_status_t ecc_solve(ecc_plan_t plan, ecc_matrix_t A, const double *d_b, double alpha,
                       double beta, double *d_x, double *d_x_tmp, double *d_x_hat,
                       const uint8_t *d_mask, int32_t T, double tol, double *d_rho,
                       uint8_t *d_eff_hist, int32_t *d_age_hist, int32_t *h_iters);

/* ---------------------------------------------------------------------------
 * SSP hypercube allreduce with one view per receiver: Algorithm 1
 * (allreduce_SSP, Section III-A) for P = 2^d processes emulated on one GPU.
 *
 * Every process owns d receive slots, one per hypercube step (the paper's
 * rcv_data_vec): m doubles plus the clock of the message that last landed
 * there.  One ecc_allreduce_ssp call is one call of every process, with
 * clock t = number of earlier calls since create/reset:
 *   - the partial reduction starts as the process's contribution (clock t);
 *   - at step k = 0 .. d-1 process r sends its partial reduction and clock to
 *     process r XOR 2^k, whose slot k it overwrites -- if that message has
 *     landed before r' reads its slot (d_delivered[r'][k] != 0); otherwise r'
 *     reuses the slot's last message when its clock >= t - slack, and waits
 *     for this call's message when it is older (or when the slot was never
 *     written: a first receipt);
 *   - partial := partial + received (fp64, in that order); its clock becomes
 *     the smaller of the two (the minimum-clock rule of Section III-A).
 * All processes take the steps of one call in lock step: the message of step
 * k of call t is the sender's partial reduction at step k of call t.
 * --------------------------------------------------------------------------- */

/* Create the hypercube state for P processes (a power of two, 1..4096) with
 * vectors of m doubles and the given slack (ECC_UNBOUNDED: never wait for a
 * slot that holds a message).  Allocates P * d * m doubles of receive slots
 * (d = log2 P) and their clocks on the current device; work is enqueued on
 * hip_stream.  Up to 32 processes a call is one kernel launch; beyond, it is
 * d - 3 launches (the decisions, the first five steps in sub-cubes of 32
 * processes, then one launch per further step, partials kept in the result),
 * with the same results bit for bit.  ECC_ERR_ARG for a bad P, m or slack; ECC_ERR_RANGE when the
 * slots would exceed 2^40 elements or m exceeds 64 (2^31 - 1) (one thread
 * per element, 64 elements per workgroup); ECC_ERR_ALLOC when allocation
 * fails. */
ecc_status_t ecc_hypercube_create(int32_t P, int64_t m, int32_t slack, void *hip_stream,
                                  ecc_hypercube_t *out);
ecc_status_t ecc_hypercube_destroy(ecc_hypercube_t h);
/* Clock back to 0, every slot "never written", wait counters to 0. */
ecc_status_t ecc_hypercube_reset(ecc_hypercube_t h);

/* One call of every process (enqueued; asynchronous).
 *   d_contrib     [P][m] doubles, row r = process r's new contribution.
 *   d_delivered   [P][d] bytes (device): != 0 when the message process
 *                 r XOR 2^k sends at step k of this call lands in slot k of
 *                 process r before r reads it.  Ignored when P = 1.
 *   d_result      [P][m] doubles: row r = process r's reduction result.  May
 *                 be d_contrib itself (in place); must not overlap it
 *                 otherwise (ECC_ERR_ARG).
 *   d_result_clock [P] int32 or NULL: the clock of each result, the oldest
 *                 clock of the data it contains.
 *   d_outcome     [P][d] bytes or NULL: 0 the slot's last message was reused,
 *                 1 this call's message had landed, 2 the slot was older than
 *                 the slack and the process waited, 3 first receipt (waited
 *                 for a slot that had never been written).
 * The results are bitwise reproducible: the same fp64 operations in the
 * same order as the sequential definition. */
ecc_status_t ecc_allreduce_ssp(ecc_hypercube_t h, const double *d_contrib,
                               const uint8_t *d_delivered, double *d_result,
                               int32_t *d_result_clock, uint8_t *d_outcome);

/* Synchronises the stream.  clock: calls so far; waits_total: waits for a
 * too-old slot (outcome 2) summed over processes and steps; h_slot_clock
 * [P][d] (host, or NULL): clock of each slot's last message (INT32_MIN when
 * never written); h_waits [P][d] (host, or NULL): waits per slot. */
ecc_status_t ecc_hypercube_stats(ecc_hypercube_t h, int64_t *clock, uint64_t *waits_total,
                                 int32_t *h_slot_clock, uint64_t *h_waits);

/* ---------------------------------------------------------------------------
 * Eventually consistent Broadcast and Reduce with a threshold (Section
 * III-B; threshold and status parameters of Section III), and the partial
 * allreduce that drops what did not arrive.
 *
 * Binomial spanning tree over P processes numbered relative to the root
 * (q = (p - root) mod P): the children of q are q + 2^i for every i above
 * q's highest set bit (every i for the root) with q + 2^i < P; stage s
 * involves min(2^s, P) processes.  All sums are fp64, in the order stated,
 * and bitwise reproducible.  The calls are enqueued on hip_stream; the status
 * outputs are computed on the host and valid on return.
 * ------------------------------------------------------------------------- */

#define ECC_THRESHOLD_DATA 0   /* reduce the first ceil(theta * m) elements  */
#define ECC_THRESHOLD_PROCS 1  /* reduce whole vectors of the first stages   */

/* Broadcast of the first k = ceil(theta * m) elements (theta in [0, 1]) of
 * the root's vector d_src to every other process: d_dst[p][0, k) = d_src[0,
 * k) for p != root; elements beyond k keep what they held (the eventually
 * consistent part).  d_dst is a device array of P device pointers (entry
 * root is not used); the buffers must not overlap d_src[0, k) or each other
 * (not checked).  *h_count (host, may be NULL) receives k.  ECC_ERR_ARG for
 * P < 1, root outside [0, P), m < 0 or theta outside [0, 1]. */
ecc_status_t ecc_bcast_threshold(int32_t P, int32_t root, int64_t m, double theta,
                                 const double *d_src, double *const *d_dst, int64_t *h_count,
                                 void *hip_stream);

/* Reduce (sum) to the root over the binomial spanning tree, 1 <= P <= 4096.
 *   mode ECC_THRESHOLD_DATA:  theta in [0, 1]; the first k = ceil(theta * m)
 *     elements of all P processes are reduced; d_result[k, m) untouched.
 *   mode ECC_THRESHOLD_PROCS: theta in (0, 1]; the full vectors (k = m) of
 *     relative ranks 0 .. n-1 are reduced, n = min(P, the smallest power of
 *     two >= ceil(theta * P)): whole stages, at least ceil(theta * P)
 *     processes; the leaves far from the root drop out.
 * Order: a parent adds its children's partial sums leaves first -- stage by
 * stage from the last, q += partial(q + 2^s) for every q < 2^s -- so
 * d_result[i] is the partial of relative rank 0.  d_src is a device array
 * of P device pointers (process p's vector); d_result must not overlap them.
 * h_elements / h_processes (host, may be NULL) receive k and n: the status
 * of the call.  ECC_ERR_ARG for a bad P, root, m, theta or mode. */
ecc_status_t ecc_reduce_threshold(int32_t P, int32_t root, int64_t m, double theta, int32_t mode,
                                  const double *const *d_src, double *d_result,
                                  int64_t *h_elements, int32_t *h_processes, void *hip_stream);

/* Partial allreduce that drops the contributions that did not arrive:
 * d_result[i] = +0.0 + sum over p with d_arrived[p] != 0, in rank order, of
 * d_fresh[p][i] (+0.0 when nothing arrived).  No slot, clock or version is
 * kept: this is the stateless counterpart of ecc_allreduce_partial.
 * d_fresh: device array of P device pointers; d_arrived: device array of P
 * bytes; d_count (device int32, may be NULL) receives the number of ranks
 * that arrived.  ECC_ERR_ARG for P < 1, m < 0 or a NULL required array. */
ecc_status_t ecc_allreduce_drop(int32_t P, int64_t m, const double *const *d_fresh,
                                const uint8_t *d_arrived, double *d_result, int32_t *d_count,
                                void *hip_stream);

/* ---------------------------------------------------------------------------
 * Data-parallel matrix factorisation by minibatch stochastic gradient
 * descent over the partial allreduce: the workload of the paper's
 * allreduce_SSP experiment (Section IV), P workers, each holding a shard of
 * the ratings and a replica of the model W = [U; V] ((n_users + n_items)
 * rows of `rank` doubles, row-major, U first).  Ratings k < N are
 * (d_users[k], d_items[k], d_ratings[k]); worker p's shard is k in
 * [N p / P, N (p + 1) / P), of L ratings, and its minibatch b (0 <= b < K)
 * the shard's ratings [L b / K, L (b + 1) / K).
 * --------------------------------------------------------------------------- */

/* Build the gradient index on the host, by counting sorts: for every
 * (worker, minibatch), the ratings of every row in storage order, stored as
 * the other factor's row index and the rating value (12 bytes per rating
 * and side), and the rows of all n_users + n_items entities sorted by their
 * number of ratings (12 bytes per row: 12 P K (n_users + n_items) bytes in
 * all).  The state also keeps a copy of the ratings (16 bytes each) for
 * ecc_mf_error; the caller may free or change its arrays afterwards.
 * rank: a power of two in [1, 64]; K >= 1 minibatches per shard (1: full
 * batches); N in [1, 2^30).  ECC_ERR_ARG for bad sizes or an out-of-range
 * user/item index; ECC_ERR_RANGE when P exceeds 65535 or P K (n_users +
 * n_items) reaches 2^40; ECC_ERR_ALLOC on allocation failure.  Synchronous. */
ecc_status_t ecc_mf_create(int32_t n_users, int32_t n_items, int32_t rank, int32_t P, int32_t K,
                           int64_t N, const int32_t *d_users, const int32_t *d_items,
                           const double *d_ratings, ecc_mf_t *out);
ecc_status_t ecc_mf_destroy(ecc_mf_t h);

/* One iteration, enqueued on the plan's stream (the plan has P ranks and
 * carries the slack and the clock); worker p uses minibatch d_batch[p]
 * (device array of P int32 in [0, K), read on the device; a value outside
 * is clamped into it):
 *   e_k = r_k - U[u_k] . V[i_k]        (products added for j = 0 .. rank-1)
 *     for the ratings of every worker's minibatch;
 *   *d_rmse = sqrt(sum e_k^2 / (ratings of those minibatches))  (the error
 *     at the model on entry);
 *   g_p := worker p's gradient of the sum over its minibatch of e_k^2:
 *     row U[u] accumulates (-2 e_k) V[i_k] and row V[i] accumulates
 *     (-2 e_k) U[u_k] over the minibatch's ratings in storage order (0 for
 *     rows without), written into d_slots[p] when the allreduce takes
 *     worker p at this clock (eff[p] of Algorithm 1's rule, from the plan's
 *     versions and d_arrived), else into d_grads[p];
 *   d_G := ecc_allreduce_partial(plan, m, g, d_slots, ..., d_arrived,
 *     d_eff_out) with m = (n_users + n_items) * rank (stale gradients
 *     substituted from the slots; the plan's clock advances), the taken
 *     gradients read in place from their slots;
 *   W := W - eta * (G * c_row + 2 lam W), c_row = K / max(1, ratings of
 *     the row).
 * d_grads, d_slots: device arrays of P device pointers to m doubles each;
 * no gradient buffer may alias a slot, and d_G aliases neither. */
ecc_status_t ecc_mf_iterate(ecc_mf_t h, ecc_plan_t plan, double eta, double lam, double *d_W,
                            double *const *d_grads, double *const *d_slots, double *d_G,
                            const uint8_t *d_arrived, const int32_t *d_batch, double *d_rmse,
                            uint8_t *d_eff_out);

/* The training error at model d_W over every rating: *d_rmse = sqrt(sum_k
 * e_k^2 / N), enqueued on hip_stream.  It shares the state's partial sums
 * with ecc_mf_iterate: the two must not overlap on different streams. */
ecc_status_t ecc_mf_error(ecc_mf_t h, const double *d_W, double *d_rmse, void *hip_stream);

/* ---------------------------------------------------------------------------
 * Plain streaming copy d_dst[i] = d_src[i], 0 <= i < n, enqueued on
 * hip_stream.  Both buffers 8-byte aligned and not overlapping
 * (ECC_ERR_ARG otherwise); 16-byte accesses when both are 16-byte aligned.
 * Used to restart an iteration from a resident initial vector, as the copy
 * ceiling of the device memory, and to calibrate hardware byte counters.
 * ------------------------------------------------------------------------- */
ecc_status_t ecc_stream_copy(double *d_dst, const double *d_src, int64_t n, void *hip_stream);

/* Gather-rate ceiling of an index stream (measurement): the sum of
 * d_x[d_idx[k]] over 0 <= k < n, eight consecutive indices per thread and
 * one workgroup per ECC_GATHER_CHUNK indices, added per workgroup in a fixed
 * order into d_out[0 .. ceil(n / ECC_GATHER_CHUNK) - 1] (n_out doubles
 * available, ECC_ERR_ARG if fewer), enqueued on hip_stream.  Indices outside
 * [0, n_x) are skipped.  It does what a sweep's gathers do -- read an index
 * stream and gather one vector -- without values, rows or results, so its
 * rate bounds a sweep over the same columns. */
#define ECC_GATHER_CHUNK 2048
ecc_status_t ecc_gather_probe(const int32_t *d_idx, int64_t n, const double *d_x, int64_t n_x,
                              double *d_out, int64_t n_out, void *hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* LIBECC_H */
