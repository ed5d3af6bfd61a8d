"""Pins of the oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: values the
paper states in its worked examples, hand computations with exact values,
closed forms of the staleness rule, brute force over every arrival schedule
on tiny inputs, library solvers (LAPACK through numpy/scipy) for fixed
points, and convergence bounds for bounded-delay iterations.
"""
import dataclasses
import itertools
import math

import numpy as np
import pytest
import scipy.linalg
import scipy.sparse
import scipy.sparse.linalg

import oracle
import workloads as W

UNB = oracle.UNBOUNDED


# ----------------------------------------------------------------------------
# helpers
# ----------------------------------------------------------------------------

def dense_csr(A: np.ndarray) -> W.CSR:
    n = A.shape[0]
    rp, cols, vals = [0], [], []
    for i in range(n):
        for j in range(n):
            if A[i, j] != 0.0:
                cols.append(j)
                vals.append(A[i, j])
        rp.append(len(cols))
    return W.CSR(n, n, np.array(rp, dtype=np.int32), np.array(cols, dtype=np.int32),
                 np.array(vals, dtype=np.float64))


def iterative(A, b, counts, S, mask, kind="jacobi", x0=None, alpha=0.85, beta=None, tol=0.0):
    n = A.n_rows
    counts = np.asarray(counts, dtype=np.int64)
    x0 = np.zeros(n) if x0 is None else x0
    if kind == "jacobi":
        return W.Iterative("t", "jacobi", A, counts, W.exclusive_scan(counts), S,
                           np.asarray(mask, dtype=np.uint8), len(mask), x0, b=b, norm=2, tol=tol)
    return W.Iterative("t", "power", A, counts, W.exclusive_scan(counts), S,
                       np.asarray(mask, dtype=np.uint8), len(mask), x0, alpha=alpha,
                       beta=(1 - alpha) / n if beta is None else beta, norm=1, tol=tol)


def select_history(S, mask):
    P = mask.shape[1]
    version = np.full(P, -1, dtype=np.int32)
    effs, ages, forced = [], [], []
    for t in range(mask.shape[0]):
        e, a, f = oracle.select(S, t, mask[t], version)
        effs.append(e)
        ages.append(a)
        forced.append(f)
    return np.array(effs), np.array(ages), np.array(forced), version


# ----------------------------------------------------------------------------
# staleness decision (Algorithm 1's acceptance test)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("case", ["slack_example", "figure2_walkthrough"])
def test_select_paper_examples(golden, case):
    g = golden("paper_staleness_examples.json")[case]
    version = np.array(g["versions_before"], dtype=np.int32)
    eff, age, forced = oracle.select(g["S"], g["t"], np.array(g["arrived"]), version)
    assert eff.tolist() == g["expect_eff"]
    assert age.tolist() == g["expect_age"]
    assert forced == g["expect_forced"]
    if "expect_version" in g:
        assert version.tolist() == g["expect_version"]


def test_min_clock_example(golden):
    g = golden("paper_staleness_examples.json")["min_clock_example"]
    assert oracle.result_clock(np.array(g["versions"], dtype=np.int32)) == g["expect_result_clock"]


@pytest.mark.parametrize("S", [0, 1, 2, 5])
def test_select_closed_form_no_arrivals(S):
    """With no arrival ever, a block is forced exactly at t = 0 mod (S+1) (after
    the initial exchange at t = 0): age_t = t mod (S+1), floor((T-1)/(S+1)) forced
    arrivals per rank."""
    T, P = 23, 3
    mask = np.zeros((T, P), dtype=np.uint8)
    eff, age, forced, version = select_history(S, mask)
    for t in range(T):
        assert (eff[t] == (1 if t % (S + 1) == 0 else 0)).all()
        assert (age[t] == t % (S + 1)).all()
    assert forced.sum() == P * ((T - 1) // (S + 1))


def test_select_closed_form_synchronous():
    rng = np.random.default_rng(0)
    mask = rng.integers(0, 2, size=(30, 5)).astype(np.uint8)
    eff, age, forced, _ = select_history(0, mask)         # S = 0: always fresh
    assert (eff == 1).all() and (age == 0).all()
    eff, age, forced, _ = select_history(3, np.ones_like(mask))  # everything arrives
    assert (eff == 1).all() and (age == 0).all() and forced.sum() == 0


def test_select_unbounded_never_forces():
    rng = np.random.default_rng(1)
    mask = rng.integers(0, 2, size=(40, 7)).astype(np.uint8)
    mask[0] = 0
    eff, age, forced, _ = select_history(UNB, mask)
    assert forced.sum() == 0
    assert (eff[0] == 1).all()
    assert (eff[1:] == mask[1:]).all()


@pytest.mark.parametrize("S", [0, 1, 3])
def test_select_invariants_random(S):
    rng = np.random.default_rng(10 + S)
    T, P = 60, 9
    mask = (rng.random((T, P)) < 0.4).astype(np.uint8)
    eff, age, forced, version = select_history(S, mask)
    assert (age >= 0).all() and (age <= S).all()
    assert (eff >= mask).all()                      # an arrival is always taken
    for t in range(T):
        for p in range(P):
            last = max(tau for tau in range(t + 1) if eff[tau, p])
            assert age[t, p] == t - last
    # forced = taken without arriving, after the initial exchange
    assert forced.sum() == int(((eff == 1) & (mask == 0))[1:].sum())


# ----------------------------------------------------------------------------
# allgatherv assembly
# ----------------------------------------------------------------------------

def test_allgatherv_prefix_displs_is_concatenation():
    rng = np.random.default_rng(2)
    counts = np.array([3, 0, 5, 1, 7], dtype=np.int64)
    displs = W.exclusive_scan(counts)
    send = [rng.standard_normal(c) for c in counts]
    recv = np.full(int(counts.sum()), np.nan)
    oracle.allgatherv(counts, displs, np.ones(5, dtype=np.uint8), send, recv)
    assert np.array_equal(recv, np.concatenate(send))


def test_allgatherv_gaps_and_unsorted_displs_keep_canaries():
    rng = np.random.default_rng(3)
    counts = np.array([4, 2, 0, 3], dtype=np.int64)
    displs = np.array([11, 0, 5, 4], dtype=np.int64)     # unsorted, with gaps
    send = [rng.standard_normal(c) for c in counts]
    canary = -12345.0
    recv = np.full(16, canary)
    eff = np.array([1, 1, 1, 0], dtype=np.uint8)
    oracle.allgatherv(counts, displs, eff, send, recv)
    expect = np.full(16, canary)
    for p in range(4):
        if eff[p]:
            expect[displs[p]:displs[p] + counts[p]] = send[p]
    assert np.array_equal(recv, expect)


# ----------------------------------------------------------------------------
# brute force: every arrival schedule on tiny problems.  The assembled view is
# rebuilt from the stored history of iterates and the version vector, a
# different formulation from the oracle's incremental copies.
# ----------------------------------------------------------------------------

def _history_view(xs, version, counts, t):
    """x_hat at iteration t rebuilt from the iterate history: block p holds
    x^{version_p} restricted to block p."""
    displs = W.exclusive_scan(counts)
    v = np.empty_like(xs[0])
    for p in range(len(counts)):
        sl = slice(displs[p], displs[p] + counts[p])
        v[sl] = xs[version[t][p]][sl]
    return v


@pytest.mark.parametrize("P,T,S", [(2, 4, 0), (2, 5, 1), (3, 4, 1), (3, 4, 2), (2, 5, 2)])
def test_bruteforce_jacobi_all_masks(P, T, S):
    n = 5
    A = np.diag(np.full(n, 4.0)) + np.diag(np.full(n - 1, -1.0), 1) + \
        np.diag(np.full(n - 1, -1.0), -1)
    A[0, n - 1] = A[n - 1, 0] = -0.5          # a long-range coupling across blocks
    Acsr = dense_csr(A)
    b = np.linspace(0.3, 1.1, n)
    counts = {2: [2, 3], 3: [2, 1, 2]}[P]
    displs = W.exclusive_scan(np.array(counts))
    owner = np.repeat(np.arange(P), counts)
    for bits in itertools.product([0, 1], repeat=P * (T - 1)):
        mask = np.ones((T, P), dtype=np.uint8)
        mask[1:] = np.array(bits, dtype=np.uint8).reshape(T - 1, P)
        prob = iterative(Acsr, b, counts, S, mask)
        h = oracle.run_iterative(prob, keep_x=set(range(T)))
        xs = [h["kept"][t][0] for t in range(T)]
        # versions after each step's decision, from the eff history
        ver = np.zeros((T, P), dtype=np.int64)
        for t in range(T):
            for p in range(P):
                ver[t, p] = max(tau for tau in range(t + 1) if h["eff"][tau, p])
        for t in range(T):
            view = _history_view(xs, ver, np.array(counts), t)
            assert np.array_equal(h["kept"][t][1], view)
            # one Jacobi row at a time from the dense matrix on each rank's view
            x_own = xs[t]
            x_next = xs[t + 1] if t + 1 < T else h["x"]
            for i in range(n):
                p = owner[i]
                y = view.copy()
                sl = slice(displs[p], displs[p] + counts[p])
                y[sl] = x_own[sl]
                s = sum(A[i, j] * y[j] for j in range(n) if j != i)
                assert abs(x_next[i] - (b[i] - s) / A[i, i]) <= 1e-15 * max(1.0, abs(x_next[i]))


# ----------------------------------------------------------------------------
# partial allreduce
# ----------------------------------------------------------------------------

def test_allreduce_hand_example(golden):
    g = golden("hand_examples.json")["allreduce_p3"]
    mask = np.array(g["mask"], dtype=np.uint8)
    h = oracle.run_allreduce(3, g["S"], mask, lambda p, r: np.array([10.0 * p + r]), 1)
    version = np.full(3, -1, dtype=np.int32)
    slots = [np.zeros(1) for _ in range(3)]
    for r, e in enumerate(g["expect"]):
        assert h["eff"][r].tolist() == e["eff"]
        assert h["result"][r][0] == e["sum"]
        assert h["clock"][r] == e["result_clock"]
        eff, _, forced = oracle.select(g["S"], r, mask[r], version)
        assert forced == e["forced"]
        oracle.allreduce(eff, [np.array([10.0 * p + r]) for p in range(3)], slots)
        assert [s[0] for s in slots] == e["slots"]


def test_allreduce_rank_order_hand_example(golden):
    """Values whose rounding depends on the order of the additions: the
    result is the rank-order sum of the held contributions, a stale rank's
    taken from its slot (the second step keeps rank 0's first value)."""
    g = golden("hand_examples.json")["allreduce_rank_order"]
    slots = [np.zeros(2) for _ in range(3)]
    for st in g["steps"]:
        fresh = [np.array(f, dtype=np.float64) for f in st["fresh"]]
        out = oracle.allreduce(np.array(st["eff"], dtype=np.uint8), fresh, slots)
        assert out.tolist() == st["expect"]


@pytest.mark.parametrize("S", [0, 2, UNB])
def test_allreduce_equals_sum_of_last_versions(S):
    """After every step each slot holds the contribution of the rank's last
    arrival, so the result is sum_p fresh_p^(version_p).  Integer-valued
    contributions make every sum exact, so any summation order agrees."""
    rng = np.random.default_rng(5)
    P, m, R = 6, 11, 15
    vals = rng.integers(-1000, 1000, size=(R, P, m)).astype(np.float64)
    mask = (rng.random((R, P)) < 0.5).astype(np.uint8)
    h = oracle.run_allreduce(P, S, mask, lambda p, r: vals[r, p].copy(), m)
    for r in range(R):
        last = [max(tau for tau in range(r + 1) if h["eff"][tau, p]) for p in range(P)]
        expect = np.sum([vals[last[p], p] for p in range(P)], axis=0)
        assert np.array_equal(h["result"][r], expect)
        assert h["clock"][r] == min(last)


def test_allreduce_synchronous_and_single_rank():
    rng = np.random.default_rng(6)
    vals = rng.integers(-50, 50, size=(4, 5, 9)).astype(np.float64)
    h = oracle.run_allreduce(5, 3, np.ones((4, 5), dtype=np.uint8), lambda p, r: vals[r, p].copy(), 9)
    for r in range(4):
        assert np.array_equal(h["result"][r], vals[r].sum(axis=0))
        assert h["clock"][r] == r
    x = rng.standard_normal((6, 1, 13))
    h = oracle.run_allreduce(1, 1, np.ones((6, 1), dtype=np.uint8),
                             lambda p, r: x[r, p].copy(), 13)
    for r in range(6):
        assert np.array_equal(h["result"][r], x[r, 0])     # P = 1: identity


# ----------------------------------------------------------------------------
# iterations
# ----------------------------------------------------------------------------

def test_jacobi_2x2_hand_example(golden):
    g = golden("hand_examples.json")["jacobi_2x2"]
    A = dense_csr(np.array(g["A"]))
    prob = iterative(A, np.array(g["b"]), g["counts"], g["S"], g["mask"])
    h = oracle.run_iterative(prob, keep_x={0, 1, 2})
    for e in g["expect"]:
        t = e["t"]
        assert h["eff"][t].tolist() == e["eff"]
        assert h["age"][t].tolist() == e["age"]
        assert h["forced"][t] == e["forced"]
        assert h["kept"][t][1].tolist() == e["x_hat"]
        assert h["rho"][t] == e["rho"]
        if t + 1 < 3:
            assert h["kept"][t + 1][0].tolist() == e["x_next"]
    assert h["x"].tolist() == g["expect"][-1]["x_next"]
    sync = iterative(A, np.array(g["b"]), g["counts"], g["S"], np.ones((3, 2)))
    assert oracle.run_iterative(sync)["x"].tolist() == g["synchronous_x3"]


@pytest.mark.parametrize("tol,iters", [(1.5, 1), (math.sqrt(2.0), 2), (0.3, 2), (0.3125, 2),
                                       (0.25, 3), (0.2, 3), (0.0, 3)])
def test_stop_rule_on_the_2x2_hand_example(golden, tol, iters):
    """Loop control (stop after the first iteration t whose norm is below the
    tolerance) on the hand-computed norms sqrt(2), 1/4, 5/16: the run length is
    that t + 1, a tolerance equal to a norm does not stop there (the test is
    strict), the norm of the stopping iteration is kept, and the state is the
    one after that iteration.  tol = 0 means no tolerance."""
    g = golden("hand_examples.json")["jacobi_2x2"]
    A = dense_csr(np.array(g["A"]))
    prob = iterative(A, np.array(g["b"]), g["counts"], g["S"], g["mask"], tol=tol)
    h = oracle.run_iterative(prob)
    assert h["iters"] == iters
    assert h["rho"].tolist() == [e["rho"] for e in g["expect"][:iters]]
    assert h["x"].tolist() == g["expect"][iters - 1]["x_next"]
    assert h["eff"].shape[0] == iters and h["forced"].sum() == (1 if iters == 3 else 0)


@pytest.mark.parametrize("pick", [0, 1, 2])
def test_stop_rule_first_iteration_below_tolerance(pick):
    """PageRank on a scale-8 R-MAT graph under staleness: with a tolerance set
    between two norms of the run without one, the run stops after the first
    iteration whose norm is below it; with the tolerance equal to a norm, not
    at that iteration."""
    prob = W.pagerank_rmat(scale=8, T=120, P=4)
    full = oracle.run_iterative(dataclasses.replace(prob, tol=0.0))
    rho = full["rho"]
    assert full["iters"] == prob.T
    k = [10, 35, 60][pick]
    for tol, strict in [((rho[k] + rho[k + 1]) / 2, False), (rho[k], True)]:
        below = np.nonzero(rho < tol)[0]
        want = int(below[0]) + 1 if below.size else prob.T
        h = oracle.run_iterative(dataclasses.replace(prob, tol=tol))
        assert h["iters"] == want
        assert np.array_equal(h["rho"], rho[:want])
        assert np.array_equal(h["eff"], full["eff"][:want])
        if strict:
            assert rho[want - 1] < tol and np.all(rho[:want - 1] >= tol)


def test_jacobi_1d_fixed_point_thomas():
    """The synchronous 1-D Jacobi workload after 50 sweeps is within rho(M)^50 sqrt(n) of the
    exact solution from a banded LAPACK solve (rho(M) = cos(pi/(n+1))/2)."""
    prob = W.jacobi_1d()
    h = oracle.run_iterative(prob)
    n = prob.n
    ab = np.zeros((3, n))
    ab[0, 1:] = -1.0
    ab[1, :] = 4.0
    ab[2, :-1] = -1.0
    xstar = scipy.linalg.solve_banded((1, 1), ab, prob.b)
    err = np.abs(h["x"] - xstar).max()
    assert err <= 1e-13 * np.abs(xstar).max()
    # residual ratios tend to the spectral radius of the iteration matrix
    rho = h["rho"]
    ratios = rho[11:31] / rho[10:30]
    assert np.all(np.abs(ratios - 0.5 * math.cos(math.pi / (n + 1))) < 2e-3)


@pytest.mark.parametrize("S,q", [(1, 0.6), (3, 0.9), (5, 0.3)])
def test_jacobi_stale_bound_and_fixed_point(S, q):
    """Bounded-delay (chaotic) relaxation, Chazan & Miranker 1969: with
    ||M||_inf = 1/2 and delays at most S, ||e_t||_inf <= (1/2)^floor(t/(S+1)) ||e_0||_inf,
    and the iteration reaches the same fixed point as the synchronous one."""
    N = 12
    A = W.stencil_csr(2, N, 8.0)
    n = A.n_rows
    rng = np.random.default_rng(int(q * 100) + S)
    b = rng.standard_normal(n)
    counts = W.dirichlet_partition(n, 5, 7)
    T = 120
    mask = (rng.random((T, 5)) < q).astype(np.uint8)
    mask[0] = 1
    prob = iterative(A, b, counts, S, mask)
    keep = set(range(T))
    h = oracle.run_iterative(prob, keep_x=keep)
    xstar = scipy.sparse.linalg.spsolve(
        scipy.sparse.csr_matrix((A.val, A.col, A.row_ptr), shape=(n, n)).tocsc(), b)
    e0 = np.abs(xstar).max()
    for t in range(T):
        et = np.abs(h["kept"][t][0] - xstar).max()
        assert et <= 0.5 ** (t // (S + 1)) * e0 * (1 + 1e-12) + 1e-14
    assert np.abs(h["x"] - xstar).max() <= 1e-13 * e0


def test_single_rank_is_mask_independent():
    A = W.stencil_csr(2, 9, 8.0)
    b = np.linspace(-1, 1, A.n_rows)
    rng = np.random.default_rng(4)
    m1 = (rng.random((20, 1)) < 0.3).astype(np.uint8)
    h1 = oracle.run_iterative(iterative(A, b, [A.n_rows], 2, m1))
    h2 = oracle.run_iterative(iterative(A, b, [A.n_rows], 2, np.ones((20, 1))))
    assert np.array_equal(h1["x"], h2["x"]) and np.array_equal(h1["rho"], h2["rho"])


def _rmat_W(scale, ef=16):
    n = 1 << scale
    src, dst = W.rmat_edges(W.seed_of(3), scale, ef * n)
    return W.pull_csr(n, src, dst), src


def test_pagerank_fixed_point_dense_solve():
    """Synchronous power iteration converges to the solution of
    (I - alpha W) x = beta 1 (dense LU)."""
    Wm, _ = _rmat_W(8)
    n = Wm.n_rows
    T = 400
    prob = iterative(Wm, None, [n], 0, np.ones((T, 1)), kind="power", x0=np.full(n, 1.0 / n))
    h = oracle.run_iterative(prob)
    xstar = np.linalg.solve(np.eye(n) - 0.85 * Wm.to_dense(), np.full(n, 0.15 / n))
    assert np.abs(h["x"] - xstar).max() <= 1e-13 * np.abs(xstar).max()


def test_pagerank_mass_identity_and_stale_fixed_point():
    Wm, src = _rmat_W(9)
    n = Wm.n_rows
    outdeg = W.out_degree(n, src)
    x = np.full(n, 1.0 / n)
    bs = oracle.block_starts([n])
    for _ in range(5):
        xn, d = oracle.power_sweep(Wm, bs, 0.85, 0.15 / n, x, x)
        lhs = math.fsum(xn)
        rhs = 0.85 * math.fsum(x[outdeg > 0]) + 0.15
        assert abs(lhs - rhs) <= 64 * n * 2.0 ** -53
        x = xn
    # stale schedule, 4 ranks, S = 4: same fixed point
    counts = W.edge_balanced_partition(Wm.row_ptr, 4)
    rng = np.random.default_rng(9)
    T = 400
    mask = (rng.random((T, 4)) < 0.5).astype(np.uint8)
    mask[0] = 1
    h = oracle.run_iterative(iterative(Wm, None, counts, 4, mask, kind="power",
                                       x0=np.full(n, 1.0 / n)))
    xstar = np.linalg.solve(np.eye(n) - 0.85 * Wm.to_dense(), np.full(n, 0.15 / n))
    assert np.abs(h["x"] - xstar).max() <= 1e-12 * np.abs(xstar).max()


def test_pagerank_stale_view_bruteforce():
    """Each step of the stale power iteration equals a dense product on the
    view rebuilt from the iterate history."""
    Wm, _ = _rmat_W(5)
    n = Wm.n_rows
    Wd = Wm.to_dense()
    counts = W.edge_balanced_partition(Wm.row_ptr, 3)
    rng = np.random.default_rng(11)
    T, S = 9, 2
    mask = (rng.random((T, 3)) < 0.3).astype(np.uint8)
    mask[0] = 1
    h = oracle.run_iterative(iterative(Wm, None, counts, S, mask, kind="power",
                                       x0=np.full(n, 1.0 / n)), keep_x=set(range(T)))
    xs = [h["kept"][t][0] for t in range(T)] + [h["x"]]
    displs = W.exclusive_scan(counts)
    owner = np.repeat(np.arange(3), counts)
    for t in range(T):
        ver = [max(tau for tau in range(t + 1) if h["eff"][tau, p]) for p in range(3)]
        for j in range(n):
            p = owner[j]
            y = np.concatenate([xs[t if q == p else ver[q]][displs[q]:displs[q] + counts[q]]
                                for q in range(3)])
            expect = 0.85 * math.fsum(Wd[j] * y) + 0.15 / n
            assert abs(xs[t + 1][j] - expect) <= 1e-14 * max(abs(expect), 1.0 / n)
        assert abs(h["rho"][t] - math.fsum(np.abs(xs[t + 1] - xs[t]))) <= 4e-16 * h["rho"][t]


def test_norms_against_exact_sums():
    rng = np.random.default_rng(12)
    v = rng.standard_normal(100003) * np.exp(rng.uniform(-30, 30, 100003))
    exact2 = math.sqrt(math.fsum(float(x) * float(x) for x in v))
    exact1 = math.fsum(abs(float(x)) for x in v)
    assert abs(oracle.norm(v, 2) - exact2) <= 2 * np.spacing(exact2)
    assert abs(oracle.norm(v, 1) - exact1) <= np.spacing(exact1)
