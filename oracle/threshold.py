"""ORACLE -- test infrastructure only.

Plain CPU statement of the eventually consistent Broadcast and Reduce with a
threshold (Iakymchuk et al., "Efficient and Eventually Consistent Collective
Operations", Section III-B and the threshold/status parameters introduced in
Section III), and of the partial allreduce that drops the contributions that
did not arrive.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may use it; it shares no code with the GPU
library.

Binomial spanning tree (BST) over P processes, numbered relative to the root
(q = (p - root) mod P): the children of q are q + 2^i for every i above the
highest set bit of q (every i >= 0 for the root) with q + 2^i < P, so the
parent of q > 0 is q with its highest set bit cleared and q joins at stage
floor(log2 q) + 1; stage s doubles the processes involved, to min(2^s, P).

Readings (listed in the design notes):
- Broadcast with threshold theta delivers the first ceil(theta * m) elements
  of the root's vector to every other process; the rest of each receive
  buffer keeps what it held (the status reports the count);
- Reduce with a data threshold reduces the first ceil(theta * m) elements of
  every process; the root's result beyond them is untouched;
- Reduce with a process threshold reduces the full vectors of the processes
  of the first stages of the tree, as many stages as needed to involve at
  least ceil(theta * P) processes (the leaves far from the root drop out);
- a parent adds its children's partial sums as they complete, leaves first:
  partial(q) = x_q, then + partial(child) for the children from the largest
  offset 2^i to the smallest, in fp64;
- the dropping partial allreduce sums, in rank order starting from +0.0, the
  contributions of the ranks that arrived in this step, and nothing else.
"""
from __future__ import annotations

import math

import numpy as np

DATA = 0    # reduce the first ceil(theta * m) elements of every process
PROCS = 1   # reduce full vectors of the first stages, >= ceil(theta * P) processes


def children(q: int, P: int):
    """Children of relative rank q, in order of increasing offset."""
    i = 0 if q == 0 else q.bit_length()
    out = []
    while q + (1 << i) < P:
        out.append(q + (1 << i))
        i += 1
    return out


def parent(q: int) -> int:
    return q - (1 << (q.bit_length() - 1))


def stage(q: int) -> int:
    """Stage at which relative rank q receives (0 for the root)."""
    return q.bit_length()


def prefix_len(theta: float, m: int) -> int:
    if not 0.0 <= theta <= 1.0:
        raise ValueError("theta must lie in [0, 1]")
    return min(m, int(math.ceil(theta * m)))


def involved(theta: float, P: int) -> int:
    """Processes of the first stages, at least ceil(theta * P) of them."""
    if not 0.0 < theta <= 1.0:
        raise ValueError("theta must lie in (0, 1]")
    need = max(1, int(math.ceil(theta * P)))
    n = 1
    while n < need:
        n *= 2
    return min(n, P)


def bcast(P: int, root: int, theta: float, src: np.ndarray, bufs) -> int:
    """bufs[p] (p != root) receive src[:k]; returns k."""
    k = prefix_len(theta, src.shape[0])
    for p in range(P):
        if p != root:
            bufs[p][:k] = src[:k]
    return k


def _tree_sum(q: int, n: int, xs_rel):
    """partial(q) over the tree restricted to relative ranks < n."""
    acc = xs_rel[q].copy()
    for c in reversed(children(q, n)):
        acc = acc + _tree_sum(c, n, xs_rel)
    return acc


def reduce(P: int, root: int, theta: float, mode: int, xs, result: np.ndarray):
    """Writes the reduction into result (root's buffer); returns
    (elements reduced, processes involved)."""
    m = result.shape[0]
    if mode == DATA:
        k, n = prefix_len(theta, m), P
    elif mode == PROCS:
        k, n = m, involved(theta, P)
    else:
        raise ValueError("unknown mode")
    xs_rel = [np.asarray(xs[(q + root) % P], dtype=np.float64)[:k] for q in range(P)]
    if k > 0:
        result[:k] = _tree_sum(0, n, xs_rel)
    return k, n


def allreduce_drop(arrived, fresh_list) -> np.ndarray:
    """Sum of the contributions of the ranks with arrived[p] != 0, in rank
    order starting from +0.0."""
    m = fresh_list[0].shape[0] if fresh_list else 0
    acc = np.zeros(m)
    for p, a in enumerate(arrived):
        if a:
            acc = acc + fresh_list[p]
    return acc
