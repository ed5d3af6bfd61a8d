"""ORACLE -- test infrastructure only.

Plain CPU statement of data-parallel matrix factorisation by gradient steps
over the eventually consistent partial allreduce: the paper's allreduce_SSP
experiment (Section IV, "Eventually consistent Allreduce"; the reduction of
Algorithm 1 with slack), on synthetic ratings.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it; it shares no code with the GPU library.

Iteration t, in the algorithm's order:
- every worker p evaluates, at the model W, the error of each rating of its
  shard, e_k = r_k - U[u_k] . V[i_k] (products added for j = 0 .. rank-1 in
  order), and its gradient of sum_k e_k^2: for each rating in shard order,
  row U[u_k] accumulates (-2 e_k) V[i_k] and row V[i_k] accumulates
  (-2 e_k) U[u_k] (every row starts at 0; rows without ratings stay 0);
- the staleness decision and the partial allreduce of the workers' gradients
  (stale ones substituted from each worker's slot) give G (``oracle.select``
  and ``oracle.allreduce``);
- W := W - eta * (G * c + (2 lam) * W), elementwise, where c is 1 over the
  number of ratings of the element's row (1 for rows without ratings): the
  gradient of each row averaged over its ratings, a diagonal preconditioning
  of the full-batch step (rows of a skewed rating set differ in their number
  of ratings by orders of magnitude).
The error reported for iteration t is sqrt(mean e_k^2) at the model W^t.
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


def worker_gradient(prob, W, e, p):
    """Gradient of worker p's shard; e holds the errors of every rating.
    Rows accumulate in shard order (np.bincount adds its weights in index
    order)."""
    a, b = prob.shard(p)
    U, V = split(prob, W)
    r = prob.rank
    g = np.zeros(prob.m)
    gU = g[:prob.n_users * r].reshape(prob.n_users, r)
    gV = g[prob.n_users * r:].reshape(prob.n_items, r)
    t = -2.0 * e[a:b]
    u, i = prob.users[a:b], prob.items[a:b]
    for j in range(r):
        gU[:, j] = np.bincount(u, weights=t * V[i, j], minlength=prob.n_users)
        gV[:, j] = np.bincount(i, weights=t * U[u, j], minlength=prob.n_items)
    return g


def row_scale(prob):
    """1 / (number of ratings of the row), 1 for rows without ratings, one
    value per model element (rows of U, then rows of V)."""
    cu = np.bincount(prob.users, minlength=prob.n_users).astype(np.float64)
    ci = np.bincount(prob.items, minlength=prob.n_items).astype(np.float64)
    c = np.concatenate([cu, ci])
    return np.repeat(1.0 / np.maximum(c, 1.0), prob.rank)


def step(prob, W, G, scale):
    return W - prob.eta * (G * scale + (2.0 * prob.lam) * W)


def run(prob, T=None, keep_W=()):
    """T iterations from prob.W0.  Returns dict with rmse [T], eff [T][P],
    age [T][P], forced [T], W (final), kept {t: W^t}."""
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
        e = errors(prob, W)
        rmse[t] = np.sqrt(np.sum(e * e) / prob.N)
        eff, age, f = _orc.select(prob.S, t, prob.mask[t], version)
        fresh = [worker_gradient(prob, W, e, p) if eff[p] else None for p in range(P)]
        G = _orc.allreduce(eff, [f_ if f_ is not None else slots[p] for p, f_ in enumerate(fresh)],
                           slots)
        W = step(prob, W, G, scale)
        effs[t], ages[t], forced[t] = eff, age, f
    if T in keep_W:
        kept[T] = W.copy()
    return {"rmse": rmse, "eff": effs, "age": ages, "forced": forced, "W": W, "kept": kept}
