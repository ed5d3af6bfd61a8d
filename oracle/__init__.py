"""ORACLE -- test infrastructure only.

Plain sequential CPU statement of the eventually consistent collective data
path (Iakymchuk et al., "Efficient and Eventually Consistent Collective
Operations", Section III-A, Algorithm 1) and of the iterations it feeds.
Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it.  It shares no code with the GPU library; both
take their inputs from the ``workloads`` package.

The per-element work is plain C (``oracle.c``, no floating-point
contraction); the loop control below follows Algorithm 1's order: advance
the clock, decide which contributions are fresh enough, take the newest
data, reduce/iterate.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

UNBOUNDED = 0x7FFFFFFF


def build(force: bool = False) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC",
                               "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        i32, i64, dbl, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
        L.orc_select.restype = i64
        L.orc_select.argtypes = [i32, i64, i64, vp, vp, vp, vp]
        L.orc_allgatherv.argtypes = [i32, vp, vp, vp, vp, vp]
        L.orc_allreduce.argtypes = [i32, i64, vp, vp, vp, vp]
        L.orc_result_clock.restype = i64
        L.orc_result_clock.argtypes = [i32, vp]
        L.orc_jacobi_sweep.argtypes = [i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_int]
        L.orc_power_sweep.argtypes = [i32, vp, vp, vp, vp, dbl, dbl, vp, vp, vp, vp,
                                      ctypes.c_int]
        L.orc_norm.restype = dbl
        L.orc_norm.argtypes = [i64, vp, i32]
        _lib = L
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _ptrs(arrs):
    return np.array([a.ctypes.data for a in arrs], dtype=np.uint64)


# ----------------------------------------------------------------------------
# one step of each operation
# ----------------------------------------------------------------------------

def select(S: int, t: int, arrived: np.ndarray, version: np.ndarray):
    """Staleness decision for iteration t.  Updates ``version`` in place and
    returns (eff, age, forced)."""
    assert version.dtype == np.int32 and version.flags.c_contiguous
    arrived = np.ascontiguousarray(arrived, dtype=np.uint8)
    P = version.shape[0]
    eff = np.empty(P, dtype=np.uint8)
    age = np.empty(P, dtype=np.int32)
    forced = lib().orc_select(P, S, t, _p(arrived), _p(version), _p(eff), _p(age))
    return eff, age, int(forced)


def allgatherv(counts, displs, eff, send_list, recv: np.ndarray) -> None:
    counts = np.ascontiguousarray(counts, dtype=np.int64)
    displs = np.ascontiguousarray(displs, dtype=np.int64)
    eff = np.ascontiguousarray(eff, dtype=np.uint8)
    send_list = [np.ascontiguousarray(s, dtype=np.float64) for s in send_list]
    ptrs = _ptrs(send_list)
    lib().orc_allgatherv(len(counts), _p(counts), _p(displs), _p(eff), _p(ptrs), _p(recv))


def allreduce(eff, fresh_list, slot_list) -> np.ndarray:
    """One partial allreduce; ``slot_list`` arrays are updated in place."""
    P = len(fresh_list)
    m = fresh_list[0].shape[0]
    eff = np.ascontiguousarray(eff, dtype=np.uint8)
    for a in list(fresh_list) + list(slot_list):
        assert a.dtype == np.float64 and a.flags.c_contiguous and a.shape[0] == m
    out = np.empty(m, dtype=np.float64)
    lib().orc_allreduce(P, m, _p(eff), _p(_ptrs(fresh_list)), _p(_ptrs(slot_list)), _p(out))
    return out


def result_clock(version: np.ndarray) -> int:
    version = np.ascontiguousarray(version, dtype=np.int32)
    return int(lib().orc_result_clock(version.shape[0], _p(version)))


def block_starts(counts) -> np.ndarray:
    bs = np.zeros(len(counts) + 1, dtype=np.int64)
    bs[1:] = np.cumsum(np.asarray(counts, dtype=np.int64))
    return bs


def jacobi_sweep(A, bstart, b, x_own, x_hat, threads: int = 1):
    n = A.n_rows
    x_next = np.empty(n)
    r = np.empty(n)
    lib().orc_jacobi_sweep(len(bstart) - 1, _p(bstart), _p(A.row_ptr), _p(A.col), _p(A.val),
                           _p(b), _p(x_own), _p(x_hat), _p(x_next), _p(r), threads)
    return x_next, r


def power_sweep(W, bstart, alpha, beta, x_own, x_hat, threads: int = 1):
    n = W.n_rows
    x_next = np.empty(n)
    d = np.empty(n)
    lib().orc_power_sweep(len(bstart) - 1, _p(bstart), _p(W.row_ptr), _p(W.col), _p(W.val),
                          alpha, beta, _p(x_own), _p(x_hat), _p(x_next), _p(d), threads)
    return x_next, d


def norm(v: np.ndarray, which: int) -> float:
    v = np.ascontiguousarray(v, dtype=np.float64)
    return float(lib().orc_norm(v.shape[0], _p(v), which))


# ----------------------------------------------------------------------------
# whole runs
# ----------------------------------------------------------------------------

def run_iterative(prob, T: int | None = None, threads: int = 1, keep_x=()):
    """Run an iterative workload (``workloads.Iterative``) step by step.

    Per iteration t (loop control of the data path):
      1. staleness decision for every block (Algorithm 1's acceptance test);
      2. assembly: blocks that arrive are copied from the owner's current
         iterate into the assembled vector; the others keep the last version
         received;
      3. block-row sweep on each rank's view (own block current, the rest
         assembled);
      4. residual norm rho_t;
      5. the new iterate replaces the old one; stop after the first t with
         rho_t < tol when a tolerance is set.
    Returns a dict of the full history."""
    T = prob.T if T is None else T
    P, n = prob.P, prob.n
    bstart = block_starts(prob.counts)
    displs = bstart[:-1]
    version = np.full(P, -1, dtype=np.int32)
    x_own = prob.x0.astype(np.float64).copy()
    x_hat = np.full(n, np.nan)
    effs, ages, rhos, forced_hist = [], [], [], []
    kept = {}
    forced_total = 0
    for t in range(T):
        eff, age, forced = select(prob.S, t, prob.mask[t], version)
        forced_total += forced
        for p in range(P):
            if eff[p]:
                x_hat[displs[p]:displs[p] + prob.counts[p]] = \
                    x_own[displs[p]:displs[p] + prob.counts[p]]
        if t in keep_x:
            kept[t] = (x_own.copy(), x_hat.copy())
        if prob.kind == "jacobi":
            x_next, r = jacobi_sweep(prob.A, bstart, prob.b, x_own, x_hat, threads)
            rho = norm(r, 2)
        else:
            x_next, r = power_sweep(prob.A, bstart, prob.alpha, prob.beta, x_own, x_hat,
                                    threads)
            rho = norm(r, 1)
        effs.append(eff)
        ages.append(age)
        rhos.append(rho)
        forced_hist.append(forced)
        x_own = x_next
        if prob.tol > 0 and rho < prob.tol:
            break
    return {
        "eff": np.array(effs, dtype=np.uint8),
        "age": np.array(ages, dtype=np.int32),
        "rho": np.array(rhos),
        "forced": np.array(forced_hist, dtype=np.int64),
        "forced_total": forced_total,
        "version": version,
        "x": x_own,
        "x_hat": x_hat,
        "iters": len(rhos),
        "kept": kept,
    }


def run_allgatherv(counts, displs, send_list, recv_init: np.ndarray, mask, S: int):
    """Repeated allgatherv assembly with staleness; returns the history of
    (eff, age) and the final receive buffer."""
    P = len(counts)
    version = np.full(P, -1, dtype=np.int32)
    recv = recv_init.copy()
    effs, ages, forced_total = [], [], 0
    for t in range(mask.shape[0]):
        eff, age, forced = select(S, t, mask[t], version)
        forced_total += forced
        allgatherv(counts, displs, eff, send_list, recv)
        effs.append(eff)
        ages.append(age)
    return {"recv": recv, "eff": np.array(effs), "age": np.array(ages),
            "version": version, "forced_total": forced_total}


def run_allreduce(P: int, S: int, mask, fresh_fn, m: int, slots_init=None):
    """Repeated partial allreduce.  ``fresh_fn(p, r)`` returns rank p's new
    contribution at repetition r.  Returns per-repetition results, result
    clocks, eff/age histories and the final slots."""
    version = np.full(P, -1, dtype=np.int32)
    slots = [np.zeros(m) if slots_init is None else slots_init[p].copy() for p in range(P)]
    results, clocks, effs, ages, forced_total = [], [], [], [], 0
    for t in range(mask.shape[0]):
        eff, age, forced = select(S, t, mask[t], version)
        forced_total += forced
        fresh = [fresh_fn(p, t) for p in range(P)]
        res = allreduce(eff, fresh, slots)
        results.append(res)
        clocks.append(result_clock(version))
        effs.append(eff)
        ages.append(age)
    return {"result": results, "clock": clocks, "eff": np.array(effs),
            "age": np.array(ages), "slots": slots, "version": version,
            "forced_total": forced_total}
