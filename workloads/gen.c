/*
 * Seeded synthetic input generators for the eventually consistent
 * collective data path and the iterations it feeds.
 *
 * This file holds no arithmetic of the method itself (no staleness rule,
 * no assembly, no reduction, no iteration).  It only produces inputs:
 * counter-based random numbers, stencil matrices in CSR form, R-MAT edge
 * lists and the PageRank transition matrix built from them.  Both the
 * oracle and the GPU path consume these arrays.
 *
 * Random numbers: SplitMix64 (Steele, Lea, Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used as a counter-based
 * generator: output k of the SplitMix64 sequence started at state s is
 * mix(s + k * GOLDEN), so any element can be produced independently.
 *
 * Built with -ffp-contract=off so that every floating-point value here is
 * the same whichever compiler optimisations are on.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GOLDEN 0x9e3779b97f4a7c15ULL

/* SplitMix64 output function (the "mix" applied to the advanced state). */
static inline uint64_t sm64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* Output number k (k >= 1) of SplitMix64 started at `state`. */
static inline uint64_t sm64_nth(uint64_t state, uint64_t k) {
    return sm64_mix(state + k * GOLDEN);
}

/* Key of one named stream: output (stream + 1) of SplitMix64(seed). */
uint64_t gen_stream_key(uint64_t seed, uint64_t stream) {
    return sm64_nth(seed, stream + 1);
}

/* 64 random bits for (seed, stream, counter): output (counter + 1) of
 * SplitMix64 started at the stream key. */
uint64_t gen_u64(uint64_t seed, uint64_t stream, uint64_t ctr) {
    return sm64_nth(gen_stream_key(seed, stream), ctr + 1);
}

/* U[0,1) with 53 random bits: (bits >> 11) * 2^-53 (exact in binary64). */
static inline double u01_from_key(uint64_t key, uint64_t ctr) {
    return (double)(sm64_nth(key, ctr + 1) >> 11) * 0x1.0p-53;
}

/* First `n` outputs of SplitMix64 started at `state` (test vector check). */
void gen_splitmix64_sequence(uint64_t state, int64_t n, uint64_t *out) {
    for (int64_t i = 0; i < n; ++i) out[i] = sm64_nth(state, (uint64_t)i + 1);
}

/* out[i] = U[0,1)(seed, stream, ctr0 + i). */
void gen_uniform(uint64_t seed, uint64_t stream, uint64_t ctr0, int64_t n,
                 double *out) {
    const uint64_t key = gen_stream_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = u01_from_key(key, ctr0 + (uint64_t)i);
}

/* out[i] = lo + (hi - lo) * U[0,1)(seed, stream, ctr0 + i).  For [-1, 1)
 * the value 2u - 1 is exact. */
void gen_uniform_range(uint64_t seed, uint64_t stream, uint64_t ctr0, int64_t n,
                       double lo, double hi, double *out) {
    const uint64_t key = gen_stream_key(seed, stream);
    const double w = hi - lo;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = lo + w * u01_from_key(key, ctr0 + (uint64_t)i);
}

/* Uniform values at arbitrary counters: out[i] = lo + (hi-lo) * U(ctr[i]). */
void gen_uniform_at(uint64_t seed, uint64_t stream, int64_t n, const uint64_t *ctr,
                    double lo, double hi, double *out) {
    const uint64_t key = gen_stream_key(seed, stream);
    const double w = hi - lo;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = lo + w * u01_from_key(key, ctr[i]);
}

/* Standard normals by the Box-Muller transform (Box & Muller 1958):
 * z_i = sqrt(-2 ln(1 - u1)) cos(2 pi u2) with u1 = U(2i), u2 = U(2i + 1). */
void gen_normal(uint64_t seed, uint64_t stream, int64_t n, double *out) {
    const uint64_t key = gen_stream_key(seed, stream);
    const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const double u1 = u01_from_key(key, 2 * (uint64_t)i);
        const double u2 = u01_from_key(key, 2 * (uint64_t)i + 1);
        out[i] = sqrt(-2.0 * log(1.0 - u1)) * cos(two_pi * u2);
    }
}

/* Bernoulli arrival table, row-major [T][P]:
 * mask[t][p] = U(seed, stream, t*P + p) < q[p].  Row 0 is all ones: every
 * block is delivered by the initial exchange. */
void gen_arrival_mask(uint64_t seed, uint64_t stream, int64_t T, int32_t P,
                      const double *q, uint8_t *mask) {
    const uint64_t key = gen_stream_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t)
        for (int32_t p = 0; p < P; ++p) {
            const uint64_t c = (uint64_t)t * (uint64_t)P + (uint64_t)p;
            mask[t * P + p] = (t == 0) ? 1 : (u01_from_key(key, c) < q[p] ? 1 : 0);
        }
}

/* ---------------------------------------------------------------------------
 * Stencil matrices.  Grid points are numbered lexicographically with x
 * fastest: i = x + N*y (+ N*N*z).  Homogeneous Dirichlet boundary: neighbours
 * outside the grid are dropped.  Every row lists its columns in ascending
 * order, so the 2-D row is (i-N, i-1, i, i+1, i+N) and the 3-D row is
 * (i-N^2, i-N, i-1, i, i+1, i+N, i+N^2).  Off-diagonal value -1, diagonal
 * `diag`.
 * ------------------------------------------------------------------------- */

static inline int stencil_row(int dim, int64_t N, int64_t i, int64_t *cols) {
    int k = 0;
    if (dim == 1) {
        if (i > 0) cols[k++] = i - 1;
        cols[k++] = i;
        if (i + 1 < N) cols[k++] = i + 1;
    } else if (dim == 2) {
        const int64_t x = i % N, y = i / N;
        if (y > 0) cols[k++] = i - N;
        if (x > 0) cols[k++] = i - 1;
        cols[k++] = i;
        if (x + 1 < N) cols[k++] = i + 1;
        if (y + 1 < N) cols[k++] = i + N;
    } else {
        const int64_t NN = N * N;
        const int64_t x = i % N, y = (i / N) % N, z = i / NN;
        if (z > 0) cols[k++] = i - NN;
        if (y > 0) cols[k++] = i - N;
        if (x > 0) cols[k++] = i - 1;
        cols[k++] = i;
        if (x + 1 < N) cols[k++] = i + 1;
        if (y + 1 < N) cols[k++] = i + N;
        if (z + 1 < N) cols[k++] = i + NN;
    }
    return k;
}

/* Number of rows and nonzeros of the dim-dimensional stencil on N^dim points. */
void gen_stencil_size(int dim, int64_t N, int64_t *n_rows, int64_t *nnz) {
    int64_t n = N;
    for (int d = 1; d < dim; ++d) n *= N;
    *n_rows = n;
    /* (2 dim + 1) n minus two missing neighbours per boundary face line */
    if (dim == 1) *nnz = 3 * N - 2;
    else if (dim == 2) *nnz = 5 * N * N - 4 * N;
    else *nnz = 7 * N * N * N - 6 * N * N;
}

/* Fill row_ptr[n+1], col[nnz], val[nnz] (int32 indices).  Returns nnz, or
 * -1 if nnz does not fit in int32. */
int64_t gen_stencil_csr(int dim, int64_t N, double diag, int32_t *row_ptr,
                        int32_t *col, double *val) {
    int64_t n, nnz;
    gen_stencil_size(dim, N, &n, &nnz);
    if (nnz >= ((int64_t)1 << 31)) return -1;
    /* row lengths, then an exclusive scan */
    row_ptr[0] = 0;
    int64_t acc = 0;
    for (int64_t i = 0; i < n; ++i) {
        int64_t cols[8];
        acc += stencil_row(dim, N, i, cols);
        row_ptr[i + 1] = (int32_t)acc;
    }
    if (acc != nnz) return -2;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t cols[8];
        const int k = stencil_row(dim, N, i, cols);
        int64_t o = row_ptr[i];
        for (int j = 0; j < k; ++j) {
            col[o + j] = (int32_t)cols[j];
            val[o + j] = (cols[j] == i) ? diag : -1.0;
        }
    }
    return nnz;
}

/* ---------------------------------------------------------------------------
 * R-MAT (Chakrabarti, Zhan, Faloutsos, SDM 2004).  Edge e picks one quadrant
 * per level, most significant bit first, from u = U(seed, stream, e*scale+l):
 * u < t1 -> (0,0); u < t2 -> (0,1); u < t3 -> (1,0); else (1,1), where the
 * pair is (source bit, destination bit) and t1, t2, t3 are the cumulative
 * probabilities a, a+b, a+b+c.  No noise, no vertex permutation; duplicate
 * edges and self loops are kept.
 * ------------------------------------------------------------------------- */
void gen_rmat_edges(uint64_t seed, uint64_t stream, int scale, int64_t n_edges,
                    double t1, double t2, double t3, int32_t *src, int32_t *dst) {
    const uint64_t key = gen_stream_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n_edges; ++e) {
        uint32_t s = 0, d = 0;
        for (int l = 0; l < scale; ++l) {
            const double u = u01_from_key(key, (uint64_t)e * (uint64_t)scale + (uint64_t)l);
            uint32_t sb, db;
            if (u < t1) { sb = 0; db = 0; }
            else if (u < t2) { sb = 0; db = 1; }
            else if (u < t3) { sb = 1; db = 0; }
            else { sb = 1; db = 1; }
            s = (s << 1) | sb;
            d = (d << 1) | db;
        }
        src[e] = (int32_t)s;
        dst[e] = (int32_t)d;
    }
}

/* Out-degree of every vertex (multi-edges counted). */
void gen_out_degree(int64_t n, int64_t n_edges, const int32_t *src, int32_t *outdeg) {
    memset(outdeg, 0, (size_t)n * sizeof(int32_t));
    for (int64_t e = 0; e < n_edges; ++e) outdeg[src[e]]++;
}

/* PageRank transition matrix W = A^T D^-1 in "pull" CSR: row j lists the
 * sources i of the edges i -> j in ascending order of i (one entry per edge,
 * so duplicates stay separate entries), with value 1/outdeg(i).  Built with
 * two stable counting sorts: by source, then by destination. */
int gen_pull_csr(int64_t n, int64_t n_edges, const int32_t *src, const int32_t *dst,
                 int32_t *row_ptr, int32_t *col, double *val) {
    if (n_edges >= ((int64_t)1 << 31)) return -1;
    int64_t *cnt = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
    int32_t *order = (int32_t *)malloc((size_t)n_edges * sizeof(int32_t));
    int32_t *outdeg = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    if (!cnt || !order || !outdeg) { free(cnt); free(order); free(outdeg); return -2; }
    gen_out_degree(n, n_edges, src, outdeg);
    /* stable counting sort of edge ids by source */
    for (int64_t e = 0; e < n_edges; ++e) cnt[src[e] + 1]++;
    for (int64_t v = 0; v < n; ++v) cnt[v + 1] += cnt[v];
    for (int64_t e = 0; e < n_edges; ++e) order[cnt[src[e]]++] = (int32_t)e;
    /* stable counting sort of that order by destination */
    memset(cnt, 0, ((size_t)n + 1) * sizeof(int64_t));
    for (int64_t e = 0; e < n_edges; ++e) cnt[dst[e] + 1]++;
    for (int64_t v = 0; v < n; ++v) cnt[v + 1] += cnt[v];
    for (int64_t v = 0; v <= n; ++v) row_ptr[v] = (int32_t)cnt[v];
    for (int64_t k = 0; k < n_edges; ++k) {
        const int32_t e = order[k];
        const int64_t pos = cnt[dst[e]]++;
        col[pos] = src[e];
        val[pos] = 1.0 / (double)outdeg[src[e]];
    }
    free(cnt);
    free(order);
    free(outdeg);
    return 0;
}
