"""ORACLE -- test infrastructure only.

Plain CPU statement of the SSP hypercube allreduce (Iakymchuk et al.,
"Efficient and Eventually Consistent Collective Operations", Section III-A,
Algorithm 1 and Fig. 2), emulated for P = 2^d processes with one view per
receiver.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may use it; it shares no code with the GPU library.

Per call (one iteration of every process), in the algorithm's order:
- the process clock advances; the contribution computed in this call carries
  it, and data older than ``clock - slack`` is not accepted;
- the partial reduction starts as the process's own new contribution;
- for each hypercube dimension k = 0 .. d-1 the process sends its partial
  reduction (with its clock) to the partner ``rank XOR 2^k`` -- the message
  lands in the partner's dedicated receive slot for step k (``rcv_data_vec``
  in the paper), overwriting what was there -- then reads its own slot k;
- if the slot is too old it waits for the partner's message of this call;
- it reduces: partial := partial + received, whose clock is the smaller of
  the two clocks (Section III-A: a reduction carries the minimum clock).

Emulation choices (readings of the paper, listed in the design notes):
- all processes run the steps of a call in lock step, so the message a
  process can receive at step k of call t is its partner's partial reduction
  at step k of the same call;
- whether that message has landed before the receiver reads its slot is an
  input (``delivered[r][k]``); when it has not, the slot still holds the last
  message that did land;
- a slot that has never received anything cannot be used: the process waits
  for the message (a first receipt, reported apart from the waits).
"""
from __future__ import annotations

import numpy as np

UNBOUNDED = 0x7FFFFFFF
NEVER = np.iinfo(np.int64).min // 4   # clock of a slot that has never been written

# per (process, step) outcome of a call
STALE = 0      # the slot's last message was recent enough and is reused
DELIVERED = 1  # the partner's message of this call had landed
WAITED = 2     # the slot was too old: the process waited for this call's message
FIRST = 3      # the slot had never been written: the process waited for it


def dims(P: int) -> int:
    d = int(P).bit_length() - 1
    if P < 1 or (1 << d) != P:
        raise ValueError("P must be a power of two")
    return d


class HypercubeSSP:
    """State of every process: its clock and its d receive slots (data and
    clock of the last message that landed)."""

    def __init__(self, P: int, m: int, slack: int):
        self.P, self.m, self.slack = int(P), int(m), int(slack)
        self.d = dims(P)
        self.clock = 0                      # calls completed so far
        self.slot = np.zeros((self.P, self.d, self.m))
        self.slot_clock = np.full((self.P, self.d), NEVER, dtype=np.int64)
        self.waits = np.zeros((self.P, self.d), dtype=np.int64)

    def call(self, contrib: np.ndarray, delivered: np.ndarray):
        """One allreduce_SSP call of every process.

        contrib   [P][m] float64: each process's new contribution.
        delivered [P][d] bool: whether the partner's message of this call
                  reaches slot k of process r before r reads it.
        Returns (result [P][m], result_clock [P], outcome [P][d])."""
        P, d = self.P, self.d
        contrib = np.asarray(contrib, dtype=np.float64).reshape(P, self.m)
        delivered = np.asarray(delivered).reshape(P, d).astype(bool)
        t = self.clock
        min_clock_accepted = t - self.slack if self.slack != UNBOUNDED else NEVER + 1
        part = contrib.copy()
        part_clock = np.full(P, t, dtype=np.int64)
        outcome = np.zeros((P, d), dtype=np.uint8)
        for k in range(d):
            # messages sent at step k: every process's current partial reduction
            sent, sent_clock = part.copy(), part_clock.copy()
            for r in range(P):
                q = r ^ (1 << k)
                if delivered[r, k]:
                    how = DELIVERED
                elif self.slot_clock[r, k] == NEVER:
                    how = FIRST
                elif self.slot_clock[r, k] < min_clock_accepted:
                    how = WAITED
                    self.waits[r, k] += 1
                else:
                    how = STALE
                if how != STALE:
                    self.slot[r, k] = sent[q]
                    self.slot_clock[r, k] = sent_clock[q]
                outcome[r, k] = how
                part[r] = part[r] + self.slot[r, k]
                part_clock[r] = min(part_clock[r], self.slot_clock[r, k])
        self.clock = t + 1
        return part, part_clock, outcome


def run(P: int, slack: int, contribs, delivered):
    """Calls t = 0 .. T-1 with contribs[t] [P][m] and delivered[t] [P][d].
    Returns per-call results, result clocks and outcomes stacked on axis 0,
    and the final state."""
    contribs = np.asarray(contribs, dtype=np.float64)
    T, m = contribs.shape[0], contribs.shape[2]
    h = HypercubeSSP(P, m, slack)
    res, clk, out = [], [], []
    for t in range(T):
        r, c, o = h.call(contribs[t], delivered[t])
        res.append(r)
        clk.append(c)
        out.append(o)
    return np.stack(res), np.stack(clk), np.stack(out), h
