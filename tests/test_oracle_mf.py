"""Pins of the matrix-factorisation oracle (data-parallel gradient steps over
the partial allreduce, Section IV): gradients against central finite
differences of the squared error, the accumulation order against explicit
loops, descent of the preconditioned step, and the allreduce wiring against a
direct sum of the workers' gradients."""
import numpy as np
import pytest

import workloads as W
from oracle import mf as M


def _tiny(P=2, S=0, q=1.0, T=6, eta=0.5, seed=11, n_ratings=300, rank=3):
    return W.mf_problem(n_users=20, n_items=9, n_ratings=n_ratings, rank=rank, P=P, S=S, q=q,
                        T=T, eta=eta, seed=seed)


def _shard_loss(prob, Wv, p):
    a, b = prob.shard(p)
    e = M.errors(prob, Wv, a, b)
    return float(np.sum(e * e))


@pytest.mark.parametrize("p", [0, 1])
def test_worker_gradient_matches_finite_differences(p):
    prob = _tiny()
    Wv = prob.W0 * 5.0
    e = M.errors(prob, Wv)
    g = M.worker_gradient(prob, Wv, e, p)
    h = 1e-6
    for x in range(prob.m):
        d = np.zeros(prob.m)
        d[x] = h
        fd = (_shard_loss(prob, Wv + d, p) - _shard_loss(prob, Wv - d, p)) / (2 * h)
        assert abs(g[x] - fd) <= 1e-6 * (1.0 + abs(fd)), (x, g[x], fd)


def test_errors_and_gradient_accumulate_in_order():
    """The vectorised oracle equals explicit loops: products added for
    j = 0 .. rank-1, rows accumulating rating by rating in shard order."""
    prob = _tiny(n_ratings=120, rank=4)
    Wv = prob.W0 * 3.0
    U, V = M.split(prob, Wv)
    e = M.errors(prob, Wv)
    for k in range(prob.N):
        acc = 0.0
        for j in range(prob.rank):
            acc = acc + U[prob.users[k], j] * V[prob.items[k], j]
        assert e[k] == prob.ratings[k] - acc
    for p in range(prob.P):
        a, b = prob.shard(p)
        g = M.worker_gradient(prob, Wv, e, p)
        ref = np.zeros(prob.m)
        gU = ref[:prob.n_users * prob.rank].reshape(prob.n_users, prob.rank)
        gV = ref[prob.n_users * prob.rank:].reshape(prob.n_items, prob.rank)
        for k in range(a, b):
            t = -2.0 * e[k]
            for j in range(prob.rank):
                gU[prob.users[k], j] += t * V[prob.items[k], j]
                gV[prob.items[k], j] += t * U[prob.users[k], j]
        assert np.array_equal(g, ref)


def test_preconditioned_step_descends():
    """With every worker fresh (S = 0) and a small step, the regularised
    squared error decreases at every iteration: -c * gradient with c > 0 per
    row is a descent direction."""
    prob = _tiny(P=3, T=12, eta=0.05, n_ratings=600)
    res = M.run(prob, keep_W=tuple(range(13)))

    def loss(Wv):
        e = M.errors(prob, Wv)
        return float(np.sum(e * e)) + prob.lam * prob.N * float(np.sum(Wv * Wv))

    vals = [loss(res["kept"][t]) for t in range(13)]
    assert all(b < a for a, b in zip(vals, vals[1:])), vals


def test_synchronous_run_equals_direct_sum_of_gradients():
    """S = 0, everyone arrives: the allreduce result is the rank-order sum of
    the workers' gradients, and the step uses it."""
    prob = _tiny(P=4, T=5, n_ratings=500)
    res = M.run(prob, keep_W=(5,))
    Wv = prob.W0.copy()
    scale = M.row_scale(prob)
    for t in range(5):
        e = M.errors(prob, Wv)
        G = np.zeros(prob.m)
        for p in range(prob.P):
            G = G + M.worker_gradient(prob, Wv, e, p)
        Wv = M.step(prob, Wv, G, scale)
    assert np.array_equal(Wv, res["kept"][5])


def test_stale_run_respects_the_slack_and_converges():
    prob = W.mf_problem(n_users=400, n_items=150, n_ratings=20000, P=8, S=3, q=0.5, T=40,
                        eta=1.0, seed=3)
    res = M.run(prob)
    assert (res["age"] <= 3).all() and res["forced"].sum() > 0
    assert res["rmse"][-1] < 0.9 * res["rmse"][0]
