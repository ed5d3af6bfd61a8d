"""Planted mistakes in the oracle, to show that its pins catch them.

Each mutant reproduces one plausible slip in one oracle function exactly --
an acceptance boundary off by one, a sign, a dropped term, an operand read
from the wrong vector, a comparison that is not strict, a summation order --
by wrapping the function (or rebinding a name its code looks up), never by
changing the oracle's files.  ``install(name)`` applies one of them to the
imported oracle modules; the test suite activates it in a separate process
(environment variable ORACLE_MUTANT, read by conftest.py) and requires the
oracle's pin tests to fail.
"""
import math
import types

import numpy as np

import oracle
from oracle import hypercube as H
from oracle import mf as M
from oracle import threshold as TH

PIN_FILES = {
    "core": ["tests/test_oracle_pins.py"],
    "hypercube": ["tests/test_oracle_hypercube.py"],
    "threshold": ["tests/test_oracle_threshold.py"],
    "mf": ["tests/test_oracle_mf.py"],
}


def _wrap(module, name, make):
    setattr(module, name, make(getattr(module, name)))


# --- staleness decision (Algorithm 1's acceptance test) ----------------------

def _select_boundary(orig):
    # data of age S forces an arrival (>= instead of >): the rule with slack S - 1
    def select(S, t, arrived, version):
        return orig(S - 1 if 0 < S < oracle.UNBOUNDED else S, t, arrived, version)
    return select


def _select_no_first_receipt(orig):
    # a block never received is not taken unless it arrives
    def select(S, t, arrived, version):
        before = version.copy()
        eff, age, forced = orig(S, t, arrived, version)
        skip = (before < 0) & (np.asarray(arrived) == 0)
        eff = eff.copy()
        eff[skip] = 0
        version[skip] = before[skip]
        age = age.copy()
        age[skip] = t - before[skip]
        return eff, age, forced
    return select


def _select_forced_counts_arrivals(orig):
    # every taken block counted as a forced arrival
    def select(S, t, arrived, version):
        eff, age, forced = orig(S, t, arrived, version)
        return eff, age, int(np.sum(eff))
    return select


def _select_forced_keeps_version(orig):
    # a forced arrival is used but its version is not advanced
    def select(S, t, arrived, version):
        before = version.copy()
        eff, age, forced = orig(S, t, arrived, version)
        keep = (eff != 0) & (np.asarray(arrived) == 0) & (before >= 0)
        version[keep] = before[keep]
        return eff, age, forced
    return select


# --- assembly and partial allreduce -----------------------------------------

def _allgatherv_ignores_eff(orig):
    def allgatherv(counts, displs, eff, send_list, recv):
        return orig(counts, displs, np.ones_like(np.asarray(eff, dtype=np.uint8)), send_list,
                    recv)
    return allgatherv


def _allgatherv_packed_displs(orig):
    # blocks written back to back, ignoring the displacements
    def allgatherv(counts, displs, eff, send_list, recv):
        c = np.asarray(counts, dtype=np.int64)
        packed = np.concatenate([[0], np.cumsum(c)[:-1]]).astype(np.int64)
        return orig(counts, packed, eff, send_list, recv)
    return allgatherv


def _allreduce_ignores_staleness(orig):
    def allreduce(eff, fresh_list, slot_list):
        return orig(np.ones_like(np.asarray(eff, dtype=np.uint8)), fresh_list, slot_list)
    return allreduce


def _allreduce_no_slot_refresh(orig):
    def allreduce(eff, fresh_list, slot_list):
        return orig(eff, fresh_list, [s.copy() for s in slot_list])
    return allreduce


def _allreduce_reverse_order(orig):
    # the same contributions summed from the last rank down
    def allreduce(eff, fresh_list, slot_list):
        out = orig(eff, fresh_list, slot_list)
        rev = [slot_list[p] for p in range(len(slot_list) - 1, -1, -1)]
        acc = rev[0].copy()
        for v in rev[1:]:
            acc = acc + v
        out[:] = acc
        return out
    return allreduce


def _result_clock_newest(orig):
    # the result's clock is the newest version instead of the oldest
    def result_clock(version):
        return int(np.max(np.asarray(version)))
    return result_clock


# --- sweeps and norms --------------------------------------------------------

def _diag(A):
    d = np.zeros(A.n_rows)
    for i in range(A.n_rows):
        for k in range(A.row_ptr[i], A.row_ptr[i + 1]):
            if A.col[k] == i:
                d[i] = A.val[k]
    return d


def _jacobi_fresh_everywhere(orig):
    # every column read from the current iterate: no stale view
    def jacobi_sweep(A, bstart, b, x_own, x_hat, threads=1):
        return orig(A, bstart, b, x_own, x_own, threads)
    return jacobi_sweep


def _jacobi_own_block_stale(orig):
    # the rank's own block read from the assembled vector as well
    def jacobi_sweep(A, bstart, b, x_own, x_hat, threads=1):
        view = np.where(np.isnan(x_hat), x_own, x_hat)
        xn, _ = orig(A, bstart, b, view, x_hat, threads)
        _, r = orig(A, bstart, b, x_own, x_hat, threads)
        return xn, r
    return jacobi_sweep


def _jacobi_sign(orig):
    # x_next = (b + s) / a_ii
    def jacobi_sweep(A, bstart, b, x_own, x_hat, threads=1):
        xn, r = orig(A, bstart, b, x_own, x_hat, threads)
        d = _diag(A)
        bs = r + d * x_own          # b - s
        s = b - bs
        return (b + s) / d, r
    return jacobi_sweep


def _jacobi_residual_of_new_iterate(orig):
    # r = (b - s) - a_ii x_next instead of a_ii x_own
    def jacobi_sweep(A, bstart, b, x_own, x_hat, threads=1):
        xn, r = orig(A, bstart, b, x_own, x_hat, threads)
        d = _diag(A)
        return xn, (r + d * x_own) - d * xn
    return jacobi_sweep


def _power_drops_beta(orig):
    def power_sweep(W, bstart, alpha, beta, x_own, x_hat, threads=1):
        return orig(W, bstart, alpha, 0.0, x_own, x_hat, threads)
    return power_sweep


def _power_alpha_twice(orig):
    def power_sweep(W, bstart, alpha, beta, x_own, x_hat, threads=1):
        return orig(W, bstart, alpha * alpha, beta, x_own, x_hat, threads)
    return power_sweep


def _power_stale_own_block(orig):
    def power_sweep(W, bstart, alpha, beta, x_own, x_hat, threads=1):
        view = np.where(np.isnan(x_hat), x_own, x_hat)
        xn, _ = orig(W, bstart, alpha, beta, view, x_hat, threads)
        return xn, np.abs(xn - x_own)
    return power_sweep


def _norm_l2_without_sqrt(orig):
    def norm(v, which):
        x = orig(v, which)
        return x * x if which == 2 else x
    return norm


def _norm_l1_as_l2(orig):
    def norm(v, which):
        return orig(v, 2 if which == 1 else which)
    return norm


# --- loop control ------------------------------------------------------------

def _stop_not_strict(orig):
    # stop at the first norm <= tol
    def run_iterative(prob, T=None, threads=1, keep_x=()):
        if prob.tol > 0:
            import dataclasses
            prob = dataclasses.replace(prob, tol=float(np.nextafter(prob.tol, np.inf)))
        return orig(prob, T, threads, keep_x)
    return run_iterative


# --- hypercube allreduce_SSP --------------------------------------------------

def _hc_max_clock():
    # the result clock takes the newest input instead of the oldest
    H.min = max


def _hc_slack_boundary(orig_init):
    # a slot of clock t - slack counted as too old (<= instead of <): the
    # rule with slack - 1
    def __init__(self, P, m, slack):
        orig_init(self, P, m, slack - 1 if 0 < slack < oracle.UNBOUNDED else slack)
    return __init__


def _hc_ignores_deliveries(orig_call):
    def call(self, contrib, delivered):
        return orig_call(self, contrib, np.zeros_like(np.asarray(delivered), dtype=bool))
    return call


# --- threshold collectives ----------------------------------------------------

def _thr_children_forward():
    # children added nearest first instead of leaves first
    TH.reversed = lambda seq: list(seq)


def _thr_prefix_floor():
    TH.math = types.SimpleNamespace(ceil=math.floor)


def _thr_involved_unrounded(orig):
    def involved(theta, P):
        return min(P, max(1, int(math.ceil(theta * P))))
    return involved


def _thr_bcast_whole(orig):
    # the whole vector broadcast whatever the threshold
    def bcast(P, root, theta, src, bufs):
        orig(P, root, 1.0, src, bufs)
        return TH.prefix_len(theta, np.asarray(src).shape[0])
    return bcast


def _thr_drop_keeps_all(orig):
    # contributions that did not arrive are added too
    def allreduce_drop(arrived, fresh_list):
        return orig(np.ones(len(fresh_list), dtype=np.uint8), fresh_list)
    return allreduce_drop


# --- matrix factorisation -----------------------------------------------------

def _mf_gradient_sign(orig):
    def worker_gradient(prob, W, e, p, lo=None, hi=None):
        return -orig(prob, W, e, p, lo, hi)
    return worker_gradient


def _mf_gradient_half(orig):
    def worker_gradient(prob, W, e, p, lo=None, hi=None):
        return 0.5 * orig(prob, W, e, p, lo, hi)
    return worker_gradient


def _mf_error_sign(orig):
    def errors(prob, W, lo=0, hi=None):
        return -orig(prob, W, lo, hi)
    return errors


def _mf_scale_without_k(orig):
    def row_scale(prob):
        return orig(prob) / prob.K
    return row_scale


def _mf_decay_sign(orig):
    def step(prob, W, G, scale):
        return W - prob.eta * (G * scale - (2.0 * prob.lam) * W)
    return step


MUTANTS = {
    # name: (pin files, installer)
    "select_boundary": ("core", lambda: _wrap(oracle, "select", _select_boundary)),
    "select_no_first_receipt": ("core", lambda: _wrap(oracle, "select", _select_no_first_receipt)),
    "select_forced_counts_arrivals": ("core", lambda: _wrap(oracle, "select",
                                                            _select_forced_counts_arrivals)),
    "select_forced_keeps_version": ("core", lambda: _wrap(oracle, "select",
                                                          _select_forced_keeps_version)),
    "allgatherv_ignores_eff": ("core", lambda: _wrap(oracle, "allgatherv", _allgatherv_ignores_eff)),
    "allgatherv_packed_displs": ("core", lambda: _wrap(oracle, "allgatherv",
                                                       _allgatherv_packed_displs)),
    "allreduce_ignores_staleness": ("core", lambda: _wrap(oracle, "allreduce",
                                                          _allreduce_ignores_staleness)),
    "allreduce_no_slot_refresh": ("core", lambda: _wrap(oracle, "allreduce",
                                                        _allreduce_no_slot_refresh)),
    "allreduce_reverse_order": ("core", lambda: _wrap(oracle, "allreduce", _allreduce_reverse_order)),
    "result_clock_newest": ("core", lambda: _wrap(oracle, "result_clock", _result_clock_newest)),
    "jacobi_fresh_everywhere": ("core", lambda: _wrap(oracle, "jacobi_sweep",
                                                      _jacobi_fresh_everywhere)),
    "jacobi_own_block_stale": ("core", lambda: _wrap(oracle, "jacobi_sweep",
                                                     _jacobi_own_block_stale)),
    "jacobi_sign": ("core", lambda: _wrap(oracle, "jacobi_sweep", _jacobi_sign)),
    "jacobi_residual_of_new_iterate": ("core", lambda: _wrap(oracle, "jacobi_sweep",
                                                             _jacobi_residual_of_new_iterate)),
    "power_drops_beta": ("core", lambda: _wrap(oracle, "power_sweep", _power_drops_beta)),
    "power_alpha_twice": ("core", lambda: _wrap(oracle, "power_sweep", _power_alpha_twice)),
    "power_stale_own_block": ("core", lambda: _wrap(oracle, "power_sweep", _power_stale_own_block)),
    "norm_l2_without_sqrt": ("core", lambda: _wrap(oracle, "norm", _norm_l2_without_sqrt)),
    "norm_l1_as_l2": ("core", lambda: _wrap(oracle, "norm", _norm_l1_as_l2)),
    "stop_not_strict": ("core", lambda: _wrap(oracle, "run_iterative", _stop_not_strict)),
    "hypercube_max_clock": ("hypercube", _hc_max_clock),
    "hypercube_slack_boundary": ("hypercube", lambda: setattr(
        H.HypercubeSSP, "__init__", _hc_slack_boundary(H.HypercubeSSP.__init__))),
    "hypercube_ignores_deliveries": ("hypercube", lambda: setattr(
        H.HypercubeSSP, "call", _hc_ignores_deliveries(H.HypercubeSSP.call))),
    "threshold_children_forward": ("threshold", _thr_children_forward),
    "threshold_prefix_floor": ("threshold", _thr_prefix_floor),
    "threshold_involved_unrounded": ("threshold", lambda: _wrap(TH, "involved",
                                                                _thr_involved_unrounded)),
    "threshold_bcast_whole": ("threshold", lambda: _wrap(TH, "bcast", _thr_bcast_whole)),
    "threshold_drop_keeps_all": ("threshold", lambda: _wrap(TH, "allreduce_drop",
                                                            _thr_drop_keeps_all)),
    "mf_gradient_sign": ("mf", lambda: _wrap(M, "worker_gradient", _mf_gradient_sign)),
    "mf_gradient_half": ("mf", lambda: _wrap(M, "worker_gradient", _mf_gradient_half)),
    "mf_error_sign": ("mf", lambda: _wrap(M, "errors", _mf_error_sign)),
    "mf_scale_without_k": ("mf", lambda: _wrap(M, "row_scale", _mf_scale_without_k)),
    "mf_decay_sign": ("mf", lambda: _wrap(M, "step", _mf_decay_sign)),
}


def install(name):
    MUTANTS[name][1]()
