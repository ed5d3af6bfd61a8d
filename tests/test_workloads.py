"""Pins of the input generators: published test vectors, independent
constructions of the same matrices, and distribution statistics."""
import math

import numpy as np
import pytest
import scipy.sparse

import workloads as W


def test_splitmix64_reference_vector(golden):
    g = golden("splitmix64_vectors.json")
    out = W.splitmix64_sequence(g["state"], len(g["outputs"]))
    assert [int(x) for x in out] == [int(s) for s in g["outputs"]]


def test_uniform_is_indexable_and_in_range():
    a = W.uniform(7, W.STREAM_B, 1000)
    b = W.uniform(7, W.STREAM_B, 10, ctr0=500)
    assert np.array_equal(a[500:510], b)
    c = W.uniform_at(7, W.STREAM_B, np.array([3, 999, 0], dtype=np.uint64))
    assert np.array_equal(c, a[[3, 999, 0]])
    assert a.min() >= 0.0 and a.max() < 1.0
    assert abs(a.mean() - 0.5) < 0.05
    r = W.uniform(7, W.STREAM_B, 1000, lo=-1.0, hi=1.0)
    assert np.array_equal(r, 2.0 * a - 1.0)          # exact affine map


def test_normal_moments():
    z = W.normal(3, W.STREAM_B, 200000)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1.0) < 0.01


def _laplacian_kron(dim, N, diag):
    T = scipy.sparse.diags([-np.ones(N - 1), 2 * np.ones(N), -np.ones(N - 1)], [-1, 0, 1])
    I = scipy.sparse.identity(N)
    if dim == 1:
        L = T
    elif dim == 2:
        L = scipy.sparse.kron(I, T) + scipy.sparse.kron(T, I)
    else:
        L = (scipy.sparse.kron(I, scipy.sparse.kron(I, T)) +
             scipy.sparse.kron(I, scipy.sparse.kron(T, I)) +
             scipy.sparse.kron(T, scipy.sparse.kron(I, I)))
    return (L + (diag - 2 * dim) * scipy.sparse.identity(N ** dim)).toarray()


@pytest.mark.parametrize("dim,N,diag", [(1, 9, 4.0), (2, 7, 8.0), (3, 5, 12.0), (2, 1, 8.0)])
def test_stencil_matches_kronecker_sum(dim, N, diag):
    A = W.stencil_csr(dim, N, diag)
    assert np.array_equal(A.to_dense(), _laplacian_kron(dim, N, diag))
    for i in range(A.n_rows):                         # ascending columns per row
        c = A.col[A.row_ptr[i]:A.row_ptr[i + 1]]
        assert np.all(np.diff(c) > 0)


def test_stencil_nnz_formulas():
    assert W.stencil_size(1, 4096) == (4096, 3 * 4096 - 2)
    assert W.stencil_size(2, 1024) == (1 << 20, 5 * 1024 ** 2 - 4 * 1024)
    assert W.stencil_size(3, 400) == (64_000_000, 447_040_000)


def test_rmat_quadrant_statistics():
    scale, E = 12, 1 << 18
    src, dst = W.rmat_edges(W.seed_of(3), scale, E)
    msb = 1 << (scale - 1)
    s0 = (src & msb) == 0
    d0 = (dst & msb) == 0
    sd = 3 * math.sqrt(0.25 / E) * 2
    assert abs(s0.mean() - (W.RMAT_A + W.RMAT_B)) < sd
    assert abs(d0.mean() - (W.RMAT_A + W.RMAT_C)) < sd
    assert abs((s0 & d0).mean() - W.RMAT_A) < sd
    assert abs((~s0 & ~d0).mean() - W.RMAT_D) < sd
    assert src.min() >= 0 and src.max() < (1 << scale)


def test_pull_csr_matches_dense_transition_matrix():
    scale = 6
    n = 1 << scale
    src, dst = W.rmat_edges(11, scale, 16 * n)
    Wm = W.pull_csr(n, src, dst)
    outdeg = np.bincount(src, minlength=n)
    D = np.zeros((n, n))
    for i, j in zip(src, dst):
        D[j, i] += 1.0 / outdeg[i]
    assert np.allclose(Wm.to_dense(), D, rtol=1e-15, atol=0)
    for j in range(n):                                # ascending sources per row
        c = Wm.col[Wm.row_ptr[j]:Wm.row_ptr[j + 1]]
        assert np.all(np.diff(c) >= 0)
    assert Wm.nnz == 16 * n
    colsum = D.sum(axis=0)
    assert np.allclose(colsum[outdeg > 0], 1.0) and np.all(colsum[outdeg == 0] == 0)


def test_partitions():
    c = W.dirichlet_partition(1 << 20, 16, W.seed_of(2))
    assert c.sum() == 1 << 20 and c.min() >= 1
    c = W.dirichlet_partition(20, 16, 5)               # forces the zero-size fix-up
    assert c.sum() == 20 and c.min() >= 1
    lc = W.lognormal_counts(4096, 99)
    assert lc.min() >= 1 and 0.85 * 65536 < lc.mean() < 1.15 * 65536
    rp = np.array([0, 5, 5, 6, 20, 21, 30], dtype=np.int32)
    bc = W.edge_balanced_partition(rp, 3)
    assert bc.sum() == 6 and list(bc) == [4, 0, 2]     # r_p = min{i : rp[i]*3 >= p*30}


def test_arrival_mask_rate():
    q = np.array([0.9, 0.2, 0.7])
    m = W.arrival_mask(1, 20000, q)
    assert (m[0] == 1).all()
    assert np.all(np.abs(m[1:].mean(axis=0) - q) < 0.02)
