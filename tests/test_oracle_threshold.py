"""Pins of the threshold Broadcast / Reduce and dropping-allreduce oracle
(Section III-B): the binomial spanning tree of the paper's children formula,
exact sums on integer data, an independent stage-by-stage formulation of the
reduction order, and the paper's stage observation for 32 processes."""
import math

import numpy as np
import pytest

from oracle import threshold as TH


def test_bst_of_eight_nodes():
    """Children of p0 are p0 + 2^i for i above p0's highest bit (Section III-B,
    Fig. 3 with eight nodes): 0 -> 1, 2, 4; 1 -> 3, 5; 2 -> 6; 3 -> 7."""
    P = 8
    assert TH.children(0, P) == [1, 2, 4]
    assert TH.children(1, P) == [3, 5]
    assert TH.children(2, P) == [6]
    assert TH.children(3, P) == [7]
    assert all(TH.children(q, P) == [] for q in range(4, 8))
    # the number of processes involved doubles at every stage
    assert [sum(TH.stage(q) <= s for q in range(P)) for s in range(4)] == [1, 2, 4, 8]


@pytest.mark.parametrize("P", list(range(1, 70)) + [128, 1000])
def test_bst_is_a_spanning_tree(P):
    seen = [0]
    for q in range(P):
        for c in TH.children(q, P):
            assert TH.parent(c) == q
            assert TH.stage(c) > TH.stage(q)
            seen.append(c)
    assert sorted(seen) == list(range(P))


def _stage_fold(xs_rel, n):
    """The same reduction written stage by stage: at stage s (from the last
    to the first) every q < 2^s adds the partial of q + 2^s."""
    S = max(0, (n - 1).bit_length())
    part = [x.copy() for x in xs_rel[:n]]
    for s in range(S - 1, -1, -1):
        for q in range(min(1 << s, n)):
            if q + (1 << s) < n:
                part[q] = part[q] + part[q + (1 << s)]
    return part[0]


@pytest.mark.parametrize("P", [1, 2, 3, 5, 8, 13, 32, 33, 64, 70])
def test_reduce_order_equals_stage_fold(P):
    rng = np.random.default_rng(P)
    xs = [rng.standard_normal(50) * 10.0 ** rng.integers(-8, 8) for _ in range(P)]
    res = np.full(50, np.nan)
    k, n = TH.reduce(P, 0, 1.0, TH.DATA, xs, res)
    assert (k, n) == (50, P)
    assert np.array_equal(res, _stage_fold(xs, P))
    for theta in (0.1, 0.3, 0.6):
        res = np.full(50, np.nan)
        k, n = TH.reduce(P, 0, theta, TH.PROCS, xs, res)
        assert np.array_equal(res, _stage_fold(xs, n))


@pytest.mark.parametrize("P,root", [(1, 0), (7, 3), (32, 0), (32, 31), (50, 17)])
@pytest.mark.parametrize("theta", [0.0, 0.25, 0.5, 0.999, 1.0])
def test_reduce_data_threshold_integer_exact(P, root, theta):
    """Integer data: every order gives the exact sum; the tail is untouched."""
    m = 37
    rng = np.random.default_rng(P + root)
    xs = [rng.integers(-10**6, 10**6, m).astype(np.float64) for _ in range(P)]
    res = np.full(m, -7.5)
    k, n = TH.reduce(P, root, theta, TH.DATA, xs, res)
    assert k == math.ceil(theta * m) and n == P
    assert np.array_equal(res[:k], np.sum(xs, axis=0)[:k])
    assert (res[k:] == -7.5).all()


@pytest.mark.parametrize("P,root", [(32, 0), (32, 5), (20, 19), (64, 1)])
def test_reduce_process_threshold_excludes_far_leaves(P, root):
    m = 11
    rng = np.random.default_rng(P * root + 1)
    xs = [rng.integers(-1000, 1000, m).astype(np.float64) for _ in range(P)]
    for theta in (0.01, 0.2, 0.5, 0.75, 1.0):
        res = np.zeros(m)
        k, n = TH.reduce(P, root, theta, TH.PROCS, xs, res)
        assert k == m and n >= theta * P
        keep = [(q + root) % P for q in range(n)]       # relative ranks 0 .. n-1
        assert np.array_equal(res, np.sum([xs[p] for p in keep], axis=0))


def test_paper_stage_observation_32_processes():
    """Section IV (Reduce on the full data with a fraction of the processes):
    75 % and 100 % involve the same processes, because stages double."""
    assert TH.involved(0.75, 32) == TH.involved(1.0, 32) == 32
    assert TH.involved(0.5, 32) == 16
    assert TH.involved(0.25, 32) == 8
    for P in range(1, 80):
        for theta in (0.05, 0.3, 0.5, 0.9, 1.0):
            n = TH.involved(theta, P)
            assert n >= theta * P - 1e-12 and n <= P
            assert n == P or (n & (n - 1)) == 0


@pytest.mark.parametrize("theta", [0.0, 0.1, 0.5, 1.0])
def test_bcast_prefix_and_untouched_tails(theta):
    P, m, root = 9, 101, 4
    rng = np.random.default_rng(3)
    src = rng.standard_normal(m)
    bufs = [np.full(m, float(p)) for p in range(P)]
    k = TH.bcast(P, root, theta, src, bufs)
    assert k == math.ceil(theta * m)
    for p in range(P):
        if p == root:
            assert (bufs[p] == p).all()
        else:
            assert np.array_equal(bufs[p][:k], src[:k]) and (bufs[p][k:] == p).all()


def test_allreduce_drop_sums_only_arrivals():
    P, m = 12, 19
    rng = np.random.default_rng(5)
    fresh = [rng.integers(-100, 100, m).astype(np.float64) for _ in range(P)]
    arrived = rng.random(P) < 0.5
    got = TH.allreduce_drop(arrived, fresh)
    assert np.array_equal(got, np.sum([f for f, a in zip(fresh, arrived) if a], axis=0))
    none = TH.allreduce_drop(np.zeros(P, dtype=bool), [-np.zeros(m)] * P)
    assert (none == 0).all() and not np.signbit(none).any()   # +0.0 when nothing arrived
    neg = TH.allreduce_drop([1], [np.array([-0.0])])
    assert not np.signbit(neg[0])                              # +0.0 + -0.0 = +0.0
