"""Pins of the matrix-factorisation oracle (data-parallel minibatch SGD over
the partial allreduce, Section IV): minibatch gradients against central
finite differences of the minibatch's squared error, the accumulation order
against explicit loops, the minibatch gradients adding up to the shard's
gradient, full batches (K = 1) against a separately written full-batch
gradient iteration, the allreduce wiring against a direct sum of the
workers' gradients, and the slack bound under random arrivals."""
import numpy as np
import pytest

import workloads as W
from oracle import mf as M


def _tiny(P=2, S=0, q=1.0, T=6, eta=0.5, seed=11, n_ratings=300, rank=3, K=4):
    return W.mf_problem(n_users=20, n_items=9, n_ratings=n_ratings, rank=rank, P=P, S=S, q=q,
                        T=T, eta=eta, seed=seed, K=K)


def _batch_loss(prob, Wv, lo, hi):
    e = M.errors(prob, Wv, lo, hi)
    return float(np.sum(e * e))


@pytest.mark.parametrize("p,b", [(0, 0), (0, 3), (1, 2)])
def test_minibatch_gradient_matches_finite_differences(p, b):
    prob = _tiny()
    lo, hi = prob.batch_range(p, b)
    assert hi - lo > 10
    Wv = prob.W0 * 5.0
    e = M.errors(prob, Wv)
    g = M.worker_gradient(prob, Wv, e, p, lo, hi)
    h = 1e-6
    for x in range(prob.m):
        d = np.zeros(prob.m)
        d[x] = h
        fd = (_batch_loss(prob, Wv + d, lo, hi) - _batch_loss(prob, Wv - d, lo, hi)) / (2 * h)
        assert abs(g[x] - fd) <= 1e-6 * (1.0 + abs(fd)), (x, g[x], fd)


def test_errors_and_gradient_accumulate_in_order():
    """The vectorised oracle equals explicit loops: products added for
    j = 0 .. rank-1, rows accumulating rating by rating in storage order,
    over each minibatch."""
    prob = _tiny(n_ratings=120, rank=4, K=3)
    Wv = prob.W0 * 3.0
    U, V = M.split(prob, Wv)
    e = M.errors(prob, Wv)
    for k in range(prob.N):
        acc = 0.0
        for j in range(prob.rank):
            acc = acc + U[prob.users[k], j] * V[prob.items[k], j]
        assert e[k] == prob.ratings[k] - acc
    for p in range(prob.P):
        for b in range(prob.K):
            lo, hi = prob.batch_range(p, b)
            g = M.worker_gradient(prob, Wv, e, p, lo, hi)
            ref = np.zeros(prob.m)
            gU = ref[:prob.n_users * prob.rank].reshape(prob.n_users, prob.rank)
            gV = ref[prob.n_users * prob.rank:].reshape(prob.n_items, prob.rank)
            for k in range(lo, hi):
                t = -2.0 * e[k]
                for j in range(prob.rank):
                    gU[prob.users[k], j] += t * V[prob.items[k], j]
                    gV[prob.items[k], j] += t * U[prob.users[k], j]
            assert np.array_equal(g, ref)


def test_minibatches_partition_the_shard_and_their_gradients_add_up():
    """The K minibatches tile the shard, and their gradients add up to the
    shard's gradient (within rounding: the additions are grouped
    differently)."""
    prob = _tiny(n_ratings=2003, K=5)
    Wv = prob.W0 * 4.0
    e = M.errors(prob, Wv)
    for p in range(prob.P):
        a, b = prob.shard(p)
        edges = [prob.batch_range(p, j) for j in range(prob.K)]
        assert edges[0][0] == a and edges[-1][1] == b
        assert all(edges[j][1] == edges[j + 1][0] for j in range(prob.K - 1))
        total = sum(M.worker_gradient(prob, Wv, e, p, lo, hi) for lo, hi in edges)
        full = M.worker_gradient(prob, Wv, e, p)
        assert np.allclose(total, full, rtol=1e-12, atol=1e-12 * np.abs(full).max())


def test_batch_schedule_is_a_permutation_per_epoch():
    prob = W.mf_problem(n_users=30, n_items=10, n_ratings=500, P=6, T=23, K=4)
    for p in range(prob.P):
        for e in range(5):
            col = prob.batch[e * 4:(e + 1) * 4, p]
            if e < 5 and col.shape[0] == 4:
                assert sorted(col.tolist()) == [0, 1, 2, 3]
    assert not np.array_equal(prob.batch[:4, 0], prob.batch[:4, 1])  # per worker


def test_full_batches_are_full_gradient_descent():
    """K = 1: every iteration is the full-shard gradient step, checked
    against a separately written loop over ratings (errors at W, every
    worker's gradient row by row, the rank-order sum, the preconditioned
    step)."""
    prob = _tiny(P=3, T=4, n_ratings=150, K=1, eta=0.3)
    res = M.run(prob, keep_W=(4,))
    Wv = prob.W0.copy()
    r = prob.rank
    cnt = np.zeros(prob.n_users + prob.n_items)
    for k in range(prob.N):
        cnt[prob.users[k]] += 1
        cnt[prob.n_users + prob.items[k]] += 1
    for t in range(4):
        grads = []
        for p in range(prob.P):
            a, b = prob.shard(p)
            g = np.zeros(prob.m)
            for k in range(a, b):
                u, i = prob.users[k], prob.items[k]
                d = 0.0
                for j in range(r):
                    d = d + Wv[u * r + j] * Wv[(prob.n_users + i) * r + j]
                ek = prob.ratings[k] - d
                for j in range(r):
                    g[u * r + j] += -2.0 * ek * Wv[(prob.n_users + i) * r + j]
                    g[(prob.n_users + i) * r + j] += -2.0 * ek * Wv[u * r + j]
            grads.append(g)
        G = grads[0]
        for g in grads[1:]:
            G = G + g
        c = np.repeat(1.0 / np.maximum(cnt, 1.0), r)
        Wv = Wv - prob.eta * (G * c + (2.0 * prob.lam) * Wv)
    assert np.allclose(Wv, res["kept"][4], rtol=1e-13, atol=1e-15)


def test_synchronous_run_equals_direct_sum_of_minibatch_gradients():
    """S = 0, everyone arrives: the allreduce result is the rank-order sum of
    the workers' minibatch gradients, and the step scales it by K / n_row."""
    prob = _tiny(P=4, T=5, n_ratings=500, K=3)
    res = M.run(prob, keep_W=(5,))
    Wv = prob.W0.copy()
    scale = M.row_scale(prob)
    for t in range(5):
        e = M.errors(prob, Wv)
        G = np.zeros(prob.m)
        for p in range(prob.P):
            lo, hi = prob.batch_range(p, int(prob.batch[t][p]))
            G = G + M.worker_gradient(prob, Wv, e, p, lo, hi)
        Wv = M.step(prob, Wv, G, scale)
    assert np.array_equal(Wv, res["kept"][5])


def test_full_batch_step_descends():
    """K = 1, every worker fresh and a small step: the regularised squared
    error decreases at every iteration (-c * gradient with c > 0 per row is a
    descent direction)."""
    prob = _tiny(P=3, T=12, eta=0.05, n_ratings=600, K=1)
    res = M.run(prob, keep_W=tuple(range(13)))

    def loss(Wv):
        e = M.errors(prob, Wv)
        return float(np.sum(e * e)) + prob.lam * prob.N * float(np.sum(Wv * Wv))

    vals = [loss(res["kept"][t]) for t in range(13)]
    assert all(b < a for a, b in zip(vals, vals[1:])), vals


def test_stale_sgd_respects_the_slack_and_converges():
    prob = W.mf_problem(n_users=400, n_items=150, n_ratings=20000, P=8, S=3, q=0.5, T=40,
                        eta=0.5, seed=3, K=4)
    res = M.run(prob, keep_W=(0, 40))
    assert (res["age"] <= 3).all() and res["forced"].sum() > 0
    assert M.full_rmse(prob, res["kept"][40]) < 0.9 * M.full_rmse(prob, res["kept"][0])
