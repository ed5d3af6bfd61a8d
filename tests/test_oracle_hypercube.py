"""Pins of the hypercube allreduce_SSP oracle (Algorithm 1, Section III-A)
against the paper's worked example, a hand-worked table, a closed form and
invariants that hold for every delivery schedule."""
import numpy as np
import pytest

from oracle import hypercube as H

FIRST, DELIVERED, STALE, WAITED = H.FIRST, H.DELIVERED, H.STALE, H.WAITED


def _tree_sum(c):
    """Balanced pairwise sum of the rows of c: left half + right half."""
    if c.shape[0] == 1:
        return c[0].copy()
    h = c.shape[0] // 2
    return _tree_sum(c[:h]) + _tree_sum(c[h:])


def test_figure2_walkthrough():
    """Process 0 of 8 at clock 3 with slack 1: the step-0 message of this call
    has landed; the step-1 slot holds data from clock 2, which is accepted;
    the step-2 slot holds data from clock 1, too old, so it waits there and
    only there."""
    P, d, T = 8, 3, 4
    delivered = np.ones((T, P, d), dtype=bool)
    delivered[2, 0, 2] = False      # step 2 last landed at call 1
    delivered[3, 0, 1] = False      # step 1 last landed at call 2
    delivered[3, 0, 2] = False
    contribs = np.random.default_rng(0).standard_normal((T, P, 5))
    res, clk, out, h = H.run(P, 1, contribs, delivered)
    # call 2: process 0 reuses step-2 data of clock 1 (1 >= 2 - 1)
    assert list(out[2, 0]) == [DELIVERED, DELIVERED, STALE]
    # call 3: fresh at step 0, accepted clock-2 data at step 1, waits at step 2
    assert list(out[3, 0]) == [DELIVERED, STALE, WAITED]
    assert h.waits[0].tolist() == [0, 0, 1]
    assert h.waits.sum() == 1
    # its result carries the oldest clock it used: 2
    assert clk[3, 0] == 2
    # the data: own partial over ranks 0-3 of call 3 plus ranks 4-7 of call 3
    # (the waited message) -- with ranks 2,3 taken from call 2
    lo = _tree_sum(np.stack([contribs[3, 0], contribs[3, 1]])) + \
        _tree_sum(np.stack([contribs[2, 2], contribs[2, 3]]))
    hi = _tree_sum(contribs[3, 4:8])
    assert np.array_equal(res[3, 0], lo + hi)


def test_hand_example_p2(golden):
    g = golden("hand_examples.json")["hypercube_p2"]
    res, clk, out, h = H.run(2, g["slack"], np.array(g["contrib"]),
                             np.array(g["delivered"], dtype=bool))
    assert np.array_equal(res, np.array(g["expect_result"]))
    assert np.array_equal(clk, np.array(g["expect_clock"]))
    assert np.array_equal(out, np.array(g["expect_outcome"]))
    assert np.array_equal(h.waits, np.array(g["expect_waits"]))


@pytest.mark.parametrize("P", [1, 2, 4, 8, 16, 32, 64])
def test_all_delivered_is_the_tree_sum_on_every_process(P):
    """With every message on time the collective is the plain hypercube
    allreduce: all processes hold the same balanced pairwise sum, of clock t."""
    d = H.dims(P)
    rng = np.random.default_rng(P)
    T, m = 3, 17
    contribs = rng.standard_normal((T, P, m))
    res, clk, out, _ = H.run(P, 0, contribs, np.ones((T, P, d), dtype=bool))
    for t in range(T):
        ref = _tree_sum(contribs[t])
        for r in range(P):
            assert np.array_equal(res[t, r], ref)
        assert (clk[t] == t).all()
    assert (out == DELIVERED).all()


def test_first_call_without_messages_waits_for_all_first_receipts():
    P, d = 8, 3
    contribs = np.random.default_rng(1).standard_normal((1, P, 4))
    res, clk, out, h = H.run(P, 5, contribs, np.zeros((1, P, d), dtype=bool))
    assert (out == FIRST).all()
    assert h.waits.sum() == 0
    for r in range(P):
        assert np.array_equal(res[0, r], _tree_sum(contribs[0]))


def test_unbounded_slack_without_messages_reuses_the_first_call():
    """Closed form: after call 0 no message ever lands and nothing is too
    old, so process r gets its own new contribution plus every other
    process's call-0 contribution, with clock 0."""
    P, d, T = 16, 4, 6
    rng = np.random.default_rng(2)
    contribs = rng.integers(-1000, 1000, (T, P, 3)).astype(np.float64)
    delivered = np.zeros((T, P, d), dtype=bool)
    delivered[0] = True
    res, clk, out, h = H.run(P, H.UNBOUNDED, contribs, delivered)
    for t in range(1, T):
        for r in range(P):
            others = contribs[0].sum(axis=0) - contribs[0, r]
            assert np.array_equal(res[t, r], contribs[t, r] + others)   # integers: exact
        assert (clk[t] == 0).all()
        assert (out[t] == STALE).all()
    assert h.waits.sum() == 0


@pytest.mark.parametrize("slack", [0, 1, 3, H.UNBOUNDED])
@pytest.mark.parametrize("q", [0.3, 0.7])
def test_provenance_invariants_random_schedules(slack, q):
    """Contributions encode (process, call) as (t + 1) * 64^p, exact in fp64,
    so every result can be decoded into the call each process's data came
    from.  For every schedule: each process's data enters exactly once, the
    process's own data is from this call, nothing is older than the slack,
    and the result clock is the oldest call used (the minimum-clock rule)."""
    P, d, T = 8, 3, 40
    rng = np.random.default_rng(int(q * 10) + (slack % 97))
    calls = np.arange(T, dtype=np.float64)[:, None] + 1.0
    contribs = (calls * (64.0 ** np.arange(P))[None, :])[:, :, None]     # [T][P][1]
    delivered = rng.random((T, P, d)) < q
    res, clk, out, h = H.run(P, slack, contribs, delivered)
    waits = 0
    for t in range(T):
        for r in range(P):
            v = int(res[t, r, 0])
            digits = []
            for p in range(P):
                digits.append(v % 64)
                v //= 64
            assert v == 0
            used = np.array(digits) - 1          # call each process's data is from
            assert (used >= 0).all() and (used <= t).all()
            assert used[r] == t
            if slack != H.UNBOUNDED:
                assert (t - used <= slack).all()
            assert clk[t, r] == used.min()
        waits += int((out[t] == WAITED).sum())
    assert waits == h.waits.sum()
    if slack == 0:
        assert (out[1:] != STALE).all()
