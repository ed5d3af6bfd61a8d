"""ORACLE -- test infrastructure only.

Plain CPU statement of data-parallel matrix factorisation by minibatch
stochastic gradient descent over the eventually consistent partial allreduce:
the paper's allreduce_SSP experiment (Section IV, "Eventually consistent
Allreduce"; the reduction of Algorithm 1 with slack), on synthetic ratings.
Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use it; it shares no code with the GPU library.

Iteration t, in the algorithm's order:
- every worker p takes its minibatch b = batch[t][p] -- the ratings [lo, hi)
  of its shard (``prob.batch_range``) -- and evaluates, at the model W, the
  error of each of those ratings, e_k = r_k - U[u_k] . V[i_k] (products
  added for j = 0 .. rank-1 in order), and its gradient of
  sum_{k in batch} e_k^2: for each rating in storage order, row U[u_k]
  accumulates (-2 e_k) V[i_k] and row V[i_k] accumulates (-2 e_k) U[u_k]
  (every row starts at 0; rows without ratings in the batch stay 0);
- the staleness decision and the partial allreduce of the workers' gradients
  (stale ones substituted from each worker's slot) give G (``oracle.select``
  and ``oracle.allreduce``);
- W := W - eta * (G * c + (2 lam) * W), elementwise, where c is K over the
  number of ratings of the element's row (K for rows without ratings): each
  rating lies in one of the K minibatches, so K times a minibatch gradient
  estimates the full-shard gradient, and each row's gradient is averaged over
  its ratings (a diagonal preconditioning; rows of a skewed rating set
  differ in their number of ratings by orders of magnitude).
With K = 1 a minibatch is the whole shard and this is full-batch gradient
descent.  The error reported for iteration t is the square root of the mean
of e_k^2 over the minibatches of that iteration (every rating when K = 1);
``full_rmse`` gives the mean over all ratings at any model.
"""
from __future__ import annotations

import numpy as np

import oracle as _orc


def split(prob, W):
    r = prob.rank
    U = W[:prob.n_users * r].reshape(prob.n_users, r)
    V = W[prob.n_users * r:].reshape(prob.n_items, r)
    return U, V


def errors(prob, W, lo=0, hi=None):
    """e_k for ratings k in [lo, hi)."""
    hi = prob.N if hi is None else hi
    U, V = split(prob, W)
    u, i = prob.users[lo:hi], prob.items[lo:hi]
    acc = np.zeros(hi - lo)
    for j in range(prob.rank):
        acc = acc + U[u, j] * V[i, j]
    return prob.ratings[lo:hi] - acc


def worker_gradient(prob, W, e, p, lo=None, hi=None):
    """Gradient of the squared error over ratings [lo, hi) of worker p's
    shard (the whole shard by default); e holds the errors of those ratings
    at their global indices.  Rows accumulate in storage order (np.bincount
    adds its weights in index order)."""
    a, b = prob.shard(p)
    lo = a if lo is None else lo
    hi = b if hi is None else hi
    assert a <= lo <= hi <= b
    U, V = split(prob, W)
    r = prob.rank
    g = np.zeros(prob.m)
    gU = g[:prob.n_users * r].reshape(prob.n_users, r)
    gV = g[prob.n_users * r:].reshape(prob.n_items, r)
    t = -2.0 * e[lo:hi]
    u, i = prob.users[lo:hi], prob.items[lo:hi]
    for j in range(r):
        gU[:, j] = np.bincount(u, weights=t * V[i, j], minlength=prob.n_users)
        gV[:, j] = np.bincount(i, weights=t * U[u, j], minlength=prob.n_items)
    return g


def row_scale(prob):
    """K / (number of ratings of the row), K for rows without ratings, one
    value per model element (rows of U, then rows of V)."""
    cu = np.bincount(prob.users, minlength=prob.n_users).astype(np.float64)
    ci = np.bincount(prob.items, minlength=prob.n_items).astype(np.float64)
    c = np.concatenate([cu, ci])
    return np.repeat(prob.K / np.maximum(c, 1.0), prob.rank)


def step(prob, W, G, scale):
    return W - prob.eta * (G * scale + (2.0 * prob.lam) * W)


def full_rmse(prob, W):
    """sqrt(mean of e_k^2 over every rating) at model W."""
    e = errors(prob, W)
    return float(np.sqrt(np.sum(e * e) / prob.N))


def run(prob, T=None, keep_W=()):
    """T iterations from prob.W0.  Returns dict with rmse [T] (over each
    iteration's minibatches), eff [T][P], age [T][P], forced [T], W (final),
    kept {t: W^t}."""
    T = prob.T if T is None else T
    P = prob.P
    W = prob.W0.copy()
    version = np.full(P, -1, dtype=np.int32)
    slots = [np.zeros(prob.m) for _ in range(P)]
    rmse = np.zeros(T)
    effs = np.zeros((T, P), dtype=np.uint8)
    ages = np.zeros((T, P), dtype=np.int32)
    forced = np.zeros(T, dtype=np.int64)
    kept = {}
    scale = row_scale(prob)
    for t in range(T):
        if t in keep_W:
            kept[t] = W.copy()
        # every worker's minibatch errors at W
        ranges = [prob.batch_range(p, int(prob.batch[t][p])) for p in range(P)]
        e = np.zeros(prob.N)
        for lo, hi in ranges:
            e[lo:hi] = errors(prob, W, lo, hi)
        used = np.concatenate([e[lo:hi] for lo, hi in ranges])
        rmse[t] = np.sqrt(np.sum(used * used) / used.shape[0])
        eff, age, f = _orc.select(prob.S, t, prob.mask[t], version)
        fresh = [worker_gradient(prob, W, e, p, *ranges[p]) if eff[p] else None
                 for p in range(P)]
        G = _orc.allreduce(eff, [f_ if f_ is not None else slots[p] for p, f_ in enumerate(fresh)],
                           slots)
        W = step(prob, W, G, scale)
        effs[t], ages[t], forced[t] = eff, age, f
    if T in keep_W:
        kept[T] = W.copy()
    return {"rmse": rmse, "eff": effs, "age": ages, "forced": forced, "W": W, "kept": kept}
