"""Seeded synthetic inputs for the eventually consistent collective data path.

This package produces inputs only: random numbers, block partitions,
arrival schedules, stencil and R-MAT matrices.  It holds none of the
method's arithmetic (no staleness rule, no assembly, no reduction, no
iteration), so it can feed both the oracle and the GPU path without either
of them depending on the other.

Every workload is a pure function of (config id, sizes); the seed of config c
is ``2203170630 + c`` and each kind of draw uses its own named stream.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libgen.so")
_GPU_SRC = os.path.join(_HERE, "gen_gpu.hip")
_GPU_LIB = os.path.join(_HERE, "libgen_gpu.so")

# Named random streams (one per kind of draw).
STREAM_PARTITION = 0
STREAM_B = 1
STREAM_Q = 2
STREAM_ARRIVAL = 3
STREAM_EDGES = 4
STREAM_COUNTS = 5
STREAM_PAYLOAD = 6
STREAM_PAYLOAD_REDUCE = 7
STREAM_PAYLOAD_HC = 8
STREAM_DELIVERY = 9
STREAM_PAYLOAD_THR = 10
STREAM_MF_USERS = 11
STREAM_MF_ITEMS = 12
STREAM_MF_NOISE = 13
STREAM_MF_TRUTH = 14
STREAM_MF_INIT = 15
STREAM_MF_PERM = 16
STREAM_MF_BATCH = 17

SEED_BASE = 2203170630

# R-MAT quadrant probabilities (Graph500 values) and their cumulative sums.
RMAT_A, RMAT_B, RMAT_C, RMAT_D = 0.57, 0.19, 0.19, 0.05
RMAT_T1, RMAT_T2, RMAT_T3 = 0.57, 0.76, 0.95

UNBOUNDED = 0x7FFFFFFF


def seed_of(config: int) -> int:
    return SEED_BASE + int(config)


def build(force: bool = False) -> str:
    """Compile gen.c into libgen.so with gcc, and gen_gpu.hip into
    libgen_gpu.so with hipcc for gfx950 (both without floating-point
    contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC",
                               "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    if force or not os.path.exists(_GPU_LIB) or \
            os.path.getmtime(_GPU_LIB) < os.path.getmtime(_GPU_SRC):
        tmp = _GPU_LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), "-O3",
                               "--offload-arch=gfx950", "-ffp-contract=off", "-fPIC", "-shared",
                               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                               "-o", tmp, _GPU_SRC])
        os.replace(tmp, _GPU_LIB)
    return _LIB


_gpu_lib = None


def gpu_lib():
    """The device-side uniform generator (gen_gpu.hip); raises if not built."""
    global _gpu_lib
    if _gpu_lib is None:
        if not os.path.exists(_GPU_LIB):
            raise RuntimeError("libgen_gpu.so is not built; run workloads.build()")
        L = ctypes.CDLL(_GPU_LIB)
        L.gen_uniform_range_device.restype = ctypes.c_int
        L.gen_uniform_range_device.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                               ctypes.c_int64, ctypes.c_double, ctypes.c_double,
                                               ctypes.c_void_p, ctypes.c_void_p]
        _gpu_lib = L
    return _gpu_lib


def uniform_device(seed: int, stream: int, n: int, d_out: int, ctr0: int = 0,
                   lo: float = 0.0, hi: float = 1.0, hip_stream: int = 0) -> None:
    """Writes uniform(seed, stream, n, ctr0, lo, hi) into device memory at
    d_out (asynchronous on hip_stream)."""
    e = gpu_lib().gen_uniform_range_device(seed, stream, ctr0, n, lo, hi, d_out, hip_stream)
    if e != 0:
        raise RuntimeError("gen_uniform_range_device failed: HIP error %d" % e)


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        u64, i64, i32, dbl, vp = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_double, ctypes.c_void_p)
        L.gen_stream_key.restype = u64
        L.gen_stream_key.argtypes = [u64, u64]
        L.gen_u64.restype = u64
        L.gen_u64.argtypes = [u64, u64, u64]
        L.gen_splitmix64_sequence.argtypes = [u64, i64, vp]
        L.gen_uniform.argtypes = [u64, u64, u64, i64, vp]
        L.gen_uniform_range.argtypes = [u64, u64, u64, i64, dbl, dbl, vp]
        L.gen_uniform_at.argtypes = [u64, u64, i64, vp, dbl, dbl, vp]
        L.gen_normal.argtypes = [u64, u64, i64, vp]
        L.gen_arrival_mask.argtypes = [u64, u64, i64, i32, vp, vp]
        L.gen_stencil_size.argtypes = [ctypes.c_int, i64, vp, vp]
        L.gen_stencil_csr.restype = i64
        L.gen_stencil_csr.argtypes = [ctypes.c_int, i64, dbl, vp, vp, vp]
        L.gen_rmat_edges.argtypes = [u64, u64, ctypes.c_int, i64, dbl, dbl, dbl, vp, vp]
        L.gen_out_degree.argtypes = [i64, i64, vp, vp]
        L.gen_pull_csr.restype = ctypes.c_int
        L.gen_pull_csr.argtypes = [i64, i64, vp, vp, vp, vp, vp]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ----------------------------------------------------------------------------
# random numbers
# ----------------------------------------------------------------------------

def splitmix64_sequence(state: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.uint64)
    lib().gen_splitmix64_sequence(state, n, _p(out))
    return out


def u64(seed: int, stream: int, ctr: int) -> int:
    return int(lib().gen_u64(seed, stream, ctr))


def uniform(seed: int, stream: int, n: int, ctr0: int = 0, lo: float = 0.0,
            hi: float = 1.0) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    if n:
        if lo == 0.0 and hi == 1.0:
            lib().gen_uniform(seed, stream, ctr0, n, _p(out))
        else:
            lib().gen_uniform_range(seed, stream, ctr0, n, lo, hi, _p(out))
    return out


def uniform_at(seed: int, stream: int, ctrs: np.ndarray, lo: float = 0.0,
               hi: float = 1.0) -> np.ndarray:
    ctrs = np.ascontiguousarray(ctrs, dtype=np.uint64)
    out = np.empty(ctrs.shape[0], dtype=np.float64)
    if ctrs.shape[0]:
        lib().gen_uniform_at(seed, stream, ctrs.shape[0], _p(ctrs), lo, hi, _p(out))
    return out


def normal(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    if n:
        lib().gen_normal(seed, stream, n, _p(out))
    return out


def arrival_mask(seed: int, T: int, q: np.ndarray) -> np.ndarray:
    """[T][P] uint8 table; row 0 is all ones (initial exchange)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    P = q.shape[0]
    out = np.empty((T, P), dtype=np.uint8)
    lib().gen_arrival_mask(seed, STREAM_ARRIVAL, T, P, _p(q), _p(out))
    return out


# ----------------------------------------------------------------------------
# partitions
# ----------------------------------------------------------------------------

def dirichlet_partition(n: int, P: int, seed: int) -> np.ndarray:
    """Block sizes from a flat Dirichlet(1) draw.

    w_p = -ln(1 - U_p) (Exp(1)); the normalised weights give ideal sizes
    w_p / sum(w) * n; sizes are their floors plus one for the largest
    remainders (ties to the lower rank); a size of 0 then takes one element
    from the largest block (lowest rank among ties)."""
    u = uniform(seed, STREAM_PARTITION, P)
    w = np.array([-math.log(1.0 - float(x)) for x in u])
    W = math.fsum(w)
    ideal = [float(wp) / W * n for wp in w]
    sizes = [int(math.floor(x)) for x in ideal]
    rem = n - sum(sizes)
    order = sorted(range(P), key=lambda p: (-(ideal[p] - sizes[p]), p))
    for p in order[:rem]:
        sizes[p] += 1
    for p in range(P):
        if sizes[p] == 0:
            big = max(range(P), key=lambda r: (sizes[r], -r))
            sizes[big] -= 1
            sizes[p] = 1
    assert sum(sizes) == n and min(sizes) >= 1
    return np.array(sizes, dtype=np.int64)


def lognormal_counts(P: int, seed: int, mean: float = 65536.0, sigma: float = 1.0) -> np.ndarray:
    """counts_p = max(1, round-half-even(exp(mu + sigma z_p))) with
    mu = ln(mean) - sigma^2/2 so that E[X] = mean; z_p standard normal by
    Box-Muller from the counts stream."""
    z = normal(seed, STREAM_COUNTS, P)
    mu = math.log(mean) - 0.5 * sigma * sigma
    return np.array([max(1, int(round(math.exp(mu + sigma * float(zp))))) for zp in z],
                    dtype=np.int64)


def exclusive_scan(counts: np.ndarray) -> np.ndarray:
    d = np.zeros(len(counts), dtype=np.int64)
    if len(counts) > 1:
        d[1:] = np.cumsum(counts[:-1])
    return d


def edge_balanced_partition(row_ptr: np.ndarray, P: int) -> np.ndarray:
    """Contiguous row ranges balanced by nonzeros: r_p = min{i : row_ptr[i]*P >= p*nnz},
    r_P = n.  Returns the block sizes."""
    n = row_ptr.shape[0] - 1
    nnz = int(row_ptr[-1])
    rp = row_ptr.astype(np.int64)
    starts = [int(np.searchsorted(rp * P, p * nnz, side="left")) for p in range(P)]
    starts[0] = 0
    bounds = starts + [n]
    return np.diff(np.array(bounds, dtype=np.int64))


# ----------------------------------------------------------------------------
# matrices
# ----------------------------------------------------------------------------

@dataclass
class CSR:
    n_rows: int
    n_cols: int
    row_ptr: np.ndarray  # int32 [n+1]
    col: np.ndarray      # int32 [nnz]
    val: np.ndarray      # float64 [nnz]

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def to_dense(self) -> np.ndarray:
        A = np.zeros((self.n_rows, self.n_cols))
        for i in range(self.n_rows):
            for k in range(self.row_ptr[i], self.row_ptr[i + 1]):
                A[i, self.col[k]] += self.val[k]
        return A


def stencil_size(dim: int, N: int):
    n = ctypes.c_int64()
    nnz = ctypes.c_int64()
    lib().gen_stencil_size(dim, N, ctypes.byref(n), ctypes.byref(nnz))
    return n.value, nnz.value


def stencil_csr(dim: int, N: int, diag: float) -> CSR:
    n, nnz = stencil_size(dim, N)
    row_ptr = np.empty(n + 1, dtype=np.int32)
    col = np.empty(nnz, dtype=np.int32)
    val = np.empty(nnz, dtype=np.float64)
    got = lib().gen_stencil_csr(dim, N, diag, _p(row_ptr), _p(col), _p(val))
    if got != nnz:
        raise ValueError("stencil too large for int32 indices (dim=%d N=%d)" % (dim, N))
    return CSR(n, n, row_ptr, col, val)


def rmat_edges(seed: int, scale: int, n_edges: int):
    src = np.empty(n_edges, dtype=np.int32)
    dst = np.empty(n_edges, dtype=np.int32)
    lib().gen_rmat_edges(seed, STREAM_EDGES, scale, n_edges, RMAT_T1, RMAT_T2, RMAT_T3,
                         _p(src), _p(dst))
    return src, dst


def out_degree(n: int, src: np.ndarray) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    lib().gen_out_degree(n, src.shape[0], _p(src), _p(out))
    return out


def pull_csr(n: int, src: np.ndarray, dst: np.ndarray) -> CSR:
    E = src.shape[0]
    row_ptr = np.empty(n + 1, dtype=np.int32)
    col = np.empty(E, dtype=np.int32)
    val = np.empty(E, dtype=np.float64)
    rc = lib().gen_pull_csr(n, E, _p(src), _p(dst), _p(row_ptr), _p(col), _p(val))
    if rc != 0:
        raise RuntimeError("gen_pull_csr failed (%d)" % rc)
    return CSR(n, n, row_ptr, col, val)


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------

@dataclass
class Iterative:
    """One of the iterative configurations: T iterations of select/assemble,
    a block-row sweep and a residual norm."""
    name: str
    kind: str                 # "jacobi" or "power"
    A: CSR
    counts: np.ndarray        # int64 [P] block sizes, tiling [0, n) in rank order
    displs: np.ndarray        # int64 [P]
    S: int                    # maximum staleness
    mask: np.ndarray          # uint8 [T][P]
    T: int
    x0: np.ndarray
    b: Optional[np.ndarray] = None
    alpha: float = 0.0
    beta: float = 0.0
    tol: float = 0.0          # stop after the first t with rho_t < tol (0: never)
    norm: int = 2             # 2: L2 of the Jacobi residual, 1: L1 of the update
    meta: dict = field(default_factory=dict)

    @property
    def P(self) -> int:
        return int(self.counts.shape[0])

    @property
    def n(self) -> int:
        return self.A.n_rows


def jacobi_1d() -> Iterative:
    """1-D tridiag(-1, 4, -1), n = 4096, b ~ U[0,1), P = 4 Dirichlet(1) blocks,
    every block arrives every iteration, S = 0, 50 iterations."""
    seed = seed_of(1)
    n = 4096
    A = stencil_csr(1, n, 4.0)
    counts = dirichlet_partition(n, 4, seed)
    T = 50
    return Iterative("jacobi-1d", "jacobi", A, counts, exclusive_scan(counts), 0,
                     np.ones((T, 4), dtype=np.uint8), T, np.zeros(n),
                     b=uniform(seed, STREAM_B, n), norm=2,
                     meta={"dim": 1, "N": n, "diag": 4.0, "q": 1.0})


def jacobi_2d(N: int = 1024, T: int = 200) -> Iterative:
    """2-D 5-point Laplacian N x N with the diagonal shifted by +4 (diag 8),
    b ~ N(0,1), P = 16 uneven blocks, Bernoulli(0.9) arrivals, S = 3."""
    seed = seed_of(2)
    A = stencil_csr(2, N, 8.0)
    n = A.n_rows
    P = 16
    counts = dirichlet_partition(n, P, seed)
    q = np.full(P, 0.9)
    return Iterative("jacobi-2d", "jacobi", A, counts, exclusive_scan(counts), 3,
                     arrival_mask(seed, T, q), T, np.zeros(n), b=normal(seed, STREAM_B, n),
                     norm=2, meta={"dim": 2, "N": N, "diag": 8.0, "q": 0.9})


def pagerank_rmat(scale: int = 22, edge_factor: int = 16, T: int = 100, P: int = 64) -> Iterative:
    """PageRank power iteration x <- 0.85 W x + 0.15/n on an R-MAT graph
    (2^scale vertices, edge_factor * 2^scale edges), W = A^T D^-1 in pull CSR,
    P edge-balanced blocks, Bernoulli(0.8) arrivals, S = 4, stop at
    ||dx||_1 < 1e-10 or after T iterations."""
    seed = seed_of(3)
    n = 1 << scale
    E = edge_factor * n
    src, dst = rmat_edges(seed, scale, E)
    W = pull_csr(n, src, dst)
    del src, dst
    counts = edge_balanced_partition(W.row_ptr, P)
    q = np.full(P, 0.8)
    return Iterative("pagerank-rmat", "power", W, counts, exclusive_scan(counts), 4,
                     arrival_mask(seed, T, q), T, np.full(n, 1.0 / n), alpha=0.85,
                     beta=0.15 / n, tol=1e-10, norm=1,
                     meta={"scale": scale, "edges": E, "q": 0.8})


def jacobi_3d(N: int = 400, T: int = 100, P: int = 512) -> Iterative:
    """3-D 7-point Laplacian N^3 with the diagonal shifted by +6 (diag 12),
    b ~ U[0,1), P uneven blocks, per-rank arrival probability q_p ~ U[0.6, 0.95],
    S = 5."""
    seed = seed_of(5)
    A = stencil_csr(3, N, 12.0)
    n = A.n_rows
    counts = dirichlet_partition(n, P, seed)
    q = 0.6 + 0.35 * uniform(seed, STREAM_Q, P)
    return Iterative("jacobi-3d", "jacobi", A, counts, exclusive_scan(counts), 5,
                     arrival_mask(seed, T, q), T, np.zeros(n), b=uniform(seed, STREAM_B, n),
                     norm=2, meta={"dim": 3, "N": N, "diag": 12.0, "q": "U[0.6,0.95]"})


@dataclass
class Allgatherv:
    """Collective data path alone: P ranks, lognormal counts, prefix-sum
    displacements, a packed send arena at the same offsets, every rank
    arriving every repetition."""
    counts: np.ndarray
    displs: np.ndarray
    send: np.ndarray
    reps: int
    mask: np.ndarray
    S: int = UNBOUNDED

    @property
    def P(self) -> int:
        return int(self.counts.shape[0])


def allgatherv_lognormal(P: int = 256, reps: int = 1000, mean: float = 65536.0) -> Allgatherv:
    seed = seed_of(4)
    counts = lognormal_counts(P, seed, mean=mean)
    displs = exclusive_scan(counts)
    E = int(counts.sum())
    send = uniform(seed, STREAM_PAYLOAD, E, lo=-1.0, hi=1.0)
    return Allgatherv(counts, displs, send, reps, np.ones((reps, P), dtype=np.uint8))


@dataclass
class Allreduce:
    """Partial allreduce-sum of P vectors of m elements; rank p's contribution
    at repetition r is U[-1,1) from its own payload stream at counters
    (r*P + p)*m + i; Bernoulli(q) arrivals; stale contributions substituted."""
    P: int
    m: int
    reps: int
    mask: np.ndarray
    S: int
    seed: int
    q: float

    def fresh_ctr0(self, p: int, r: int) -> int:
        return (r * self.P + p) * self.m

    def fresh(self, p: int, r: int) -> np.ndarray:
        return uniform(self.seed, STREAM_PAYLOAD_REDUCE, self.m, ctr0=self.fresh_ctr0(p, r),
                       lo=-1.0, hi=1.0)

    def fresh_at(self, p: int, r: int, idx: np.ndarray) -> np.ndarray:
        ctr = np.uint64(self.fresh_ctr0(p, r)) + np.asarray(idx, dtype=np.uint64)
        return uniform_at(self.seed, STREAM_PAYLOAD_REDUCE, ctr, lo=-1.0, hi=1.0)


def partial_allreduce(P: int = 256, m: int = 1 << 22, reps: int = 1000, q: float = 0.7,
             S: int = UNBOUNDED) -> Allreduce:
    seed = seed_of(4)
    return Allreduce(P, m, reps, arrival_mask(seed, reps, np.full(P, q)), S, seed, q)


@dataclass
class HypercubeSSP:
    """SSP hypercube allreduce (Algorithm 1) for P = 2^d processes: process
    p's contribution at call t is U[-1,1) from its payload stream at
    counters (t*P + p)*m + i; the message of step k of call t reaches process
    r's slot k in time with probability q (Bernoulli, independent per call,
    process and step; call 0 of every slot included)."""
    P: int
    m: int
    calls: int
    slack: int
    q: float
    seed: int
    delivered: np.ndarray     # bool [calls][P][d]

    @property
    def d(self) -> int:
        return int(self.P).bit_length() - 1

    def contrib(self, t: int) -> np.ndarray:
        return uniform(self.seed, STREAM_PAYLOAD_HC, self.P * self.m, ctr0=t * self.P * self.m,
                       lo=-1.0, hi=1.0).reshape(self.P, self.m)


def hypercube_ssp(P: int = 32, m: int = 1 << 21, calls: int = 100, slack: int = 2,
                  q: float = 0.8) -> HypercubeSSP:
    """32 processes as in the paper's allreduce_SSP run; slack 2, one of the
    paper's settings; 16 MB vectors (the paper's model size is not stated)."""
    seed = seed_of(6)
    d = int(P).bit_length() - 1
    u = uniform(seed, STREAM_DELIVERY, calls * P * max(d, 1)).reshape(calls, P, max(d, 1))
    return HypercubeSSP(P, m, calls, slack, q, seed, (u < q)[:, :, :d])


@dataclass
class ThresholdCollectives:
    """Threshold Broadcast and Reduce (Section III-B) over P processes with
    vectors of m doubles, U[-1,1) from process p's payload stream at counters
    p*m + i; theta is the data (or process) fraction."""
    P: int
    m: int
    theta: float
    reps: int
    seed: int

    def vector(self, p: int) -> np.ndarray:
        return uniform(self.seed, STREAM_PAYLOAD_THR, self.m, ctr0=p * self.m, lo=-1.0, hi=1.0)


def threshold_collectives(P: int = 32, m: int = 1 << 23, theta: float = 0.5,
                          reps: int = 100) -> ThresholdCollectives:
    """32 processes; 8,388,608 doubles, the largest message size of the
    paper's experiments; half of the data."""
    return ThresholdCollectives(P, m, theta, reps, seed_of(7))


@dataclass
class MFProblem:
    """Matrix factorisation by minibatch stochastic gradient descent, data
    parallel over P workers (the paper's allreduce_SSP experiment, Section
    IV, on synthetic ratings).

    Ratings (users[k], items[k], ratings[k]), k < N, are stored in shard order:
    worker p holds k in [p*N/P, (p+1)*N/P), cut into K minibatches of
    consecutive ratings (batch b: offsets [L b / K, L (b+1) / K) of the
    shard's L ratings).  The model W = [U; V] is (n_users + n_items) x rank
    doubles, row-major, U first.  One iteration t at model W: worker p takes
    minibatch batch[t][p] and computes the gradient of its squared error
    sum_k (r_k - U[u_k].V[i_k])^2; the partial allreduce combines the workers'
    gradients (stale ones substituted, slack S, arrivals `mask`); the step is
    W := W - eta * (G_row K / n_row + 2 lam W), n_row = the row's number of
    ratings (1 if none).  batch[t][p] runs through a seeded permutation of
    the K minibatches in every epoch of K iterations."""
    n_users: int
    n_items: int
    rank: int
    P: int
    users: np.ndarray        # int32 [N]
    items: np.ndarray        # int32 [N]
    ratings: np.ndarray      # float64 [N], centred
    W0: np.ndarray           # float64 [(n_users + n_items) * rank]
    eta: float
    lam: float
    S: int
    mask: np.ndarray         # uint8 [T][P]
    T: int
    K: int = 1               # minibatches per shard
    batch: np.ndarray = None  # int32 [T][P]: the minibatch of worker p at iteration t
    meta: dict = field(default_factory=dict)

    @property
    def N(self) -> int:
        return int(self.ratings.shape[0])

    def batch_range(self, p: int, b: int):
        """Ratings [lo, hi) of minibatch b of worker p's shard."""
        a, c = self.shard(p)
        L = c - a
        return a + L * b // self.K, a + L * (b + 1) // self.K

    @property
    def m(self) -> int:
        return (self.n_users + self.n_items) * self.rank

    def shard(self, p: int):
        return self.N * p // self.P, self.N * (p + 1) // self.P


def _zipf_pick(seed: int, stream: int, n_draws: int, n: int, s: float) -> np.ndarray:
    """Indices in [0, n) drawn with probability proportional to 1/(k+1)^s,
    then relabelled by a seeded permutation (popularity is not id order)."""
    w = 1.0 / np.power(np.arange(1, n + 1, dtype=np.float64), s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    k = np.searchsorted(cdf, uniform(seed, stream, n_draws), side="right")
    k = np.minimum(k, n - 1)
    perm = np.argsort(uniform(seed, STREAM_MF_PERM, n, ctr0=stream * (1 << 32)), kind="stable")
    return perm[k].astype(np.int32)


def batch_schedule(seed: int, T: int, P: int, K: int) -> np.ndarray:
    """[T][P] minibatch indices: for worker p and epoch e (iterations e K ..
    e K + K - 1) a seeded permutation of 0 .. K-1 (the order of K uniforms
    at counters (p * 2^32 + e) * K + j, ties to the lower j)."""
    out = np.empty((T, P), dtype=np.int32)
    for p in range(P):
        for e in range((T + K - 1) // K):
            u = uniform(seed, STREAM_MF_BATCH, K, ctr0=((p << 32) + e) * K)
            perm = np.argsort(u, kind="stable").astype(np.int32)
            n = min(K, T - e * K)
            out[e * K:e * K + n, p] = perm[:n]
    return out


def mf_problem(n_users: int = 160_000, n_items: int = 60_000, n_ratings: int = 25_000_000,
               rank: int = 16, P: int = 32, S: int = 2, q: float = 0.8, T: int = 100,
               eta: float = 0.3, lam: float = 1e-4, true_rank: int = 8, seed: int = None,
               K: int = 8) -> MFProblem:
    """Synthetic ratings shaped like a large movie-rating set (25M ratings;
    Zipf user activity, exponent 0.5, and item popularity, exponent 0.6):
    half-star ratings in [0.5, 5] from a planted rank-`true_rank` model plus
    noise, centred; drawn independently, so consecutive ratings form uniform
    shards and minibatches; P equal shards of K minibatches, each minibatch
    stored by user then item; the model starts at N(0, 0.1^2).  The step size
    0.3 keeps the training error falling through the first 100 iterations
    (from 0.5 on, it reaches the minibatches' noise floor before then)."""
    seed = seed_of(8) if seed is None else seed
    users = _zipf_pick(seed, STREAM_MF_USERS, n_ratings, n_users, 0.5)
    items = _zipf_pick(seed, STREAM_MF_ITEMS, n_ratings, n_items, 0.6)
    tu = normal(seed, STREAM_MF_TRUTH, (n_users + n_items) * true_rank) / np.sqrt(true_rank)
    tU = tu[:n_users * true_rank].reshape(n_users, true_rank)
    tV = tu[n_users * true_rank:].reshape(n_items, true_rank)
    raw = 3.5 + np.einsum("kj,kj->k", tU[users], tV[items]) + 0.5 * normal(seed, STREAM_MF_NOISE,
                                                                         n_ratings)
    r = np.clip(np.round(raw * 2.0) / 2.0, 0.5, 5.0)
    ratings = r - r.mean()
    # within each minibatch of each worker's shard, ratings are stored by
    # user, then item
    for p in range(P):
        a, b = n_ratings * p // P, n_ratings * (p + 1) // P
        for j in range(K):
            lo, hi = a + (b - a) * j // K, a + (b - a) * (j + 1) // K
            o = np.lexsort((items[lo:hi], users[lo:hi]))
            users[lo:hi], items[lo:hi], ratings[lo:hi] = (users[lo:hi][o], items[lo:hi][o],
                                                          ratings[lo:hi][o])
    W0 = 0.1 * normal(seed, STREAM_MF_INIT, (n_users + n_items) * rank)
    mask = arrival_mask(seed, T, np.full(P, q))
    return MFProblem(n_users, n_items, rank, P, users, items, ratings, W0, eta, lam, S, mask, T,
                     K=K, batch=batch_schedule(seed, T, P, K),
                     meta={"q": q, "true_rank": true_rank, "rating_mean": float(r.mean())})
