#!/usr/bin/env python3
"""Benchmark of the eventually consistent collective data path on one MI355X.

Default workload: 3-D 7-point Laplacian 400^3 (n = 64,000,000, diagonal 12),
512 uneven block-row ranks, per-rank arrival probability q_p ~ U[0.6, 0.95],
maximum staleness 5, 100 Jacobi iterations -- the largest configuration that
fits one GPU.  One step = one complete solve (plan reset, x0 loaded, then
100 x [staleness decision + allgatherv assembly -> block-row sweep ->
residual norm]) on inputs already resident in HBM.

Metric: assembled+iterated GB/s (algorithmic bytes of assembly + sweep + norm,
each distinct element counted once) and iterations/s, with the dominant
kernel's achieved bandwidth against the HBM roofline and against the
measured copy ceiling.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--config NAME]

NAME: jacobi-3d (the default above), jacobi-1d (tridiagonal, n = 4096, 4
ranks, synchronous), jacobi-2d (5-point 1024^2, 16 ranks), pagerank-rmat
(R-MAT scale 22, 64 ranks), allgatherv (256 lognormal blocks, 16.5M
elements), allreduce (partial allreduce of 256 x 4M), hypercube
(allreduce_SSP, 32 x 16 MB), threshold (Broadcast + Reduce, 32 x 8M), mf
(matrix factorisation, 25M ratings, 32 workers).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, AMD specification
METRIC = "assembled+iterated GB/s and iterations/s at 1 GPU; % of HBM peak"
PROFILES = os.path.join(ROOT, "profiles")


def sweep_bytes(n, nnz):
    """Algorithmic bytes of one sweep: col + val per nonzero, row_ptr, the x
    view, b (or x_own for the update norm), the written iterate.  This is the
    model of the method's data (CSR), whatever layout the library sweeps."""
    return 12 * nnz + 28 * n + 4


def format_sweep_bytes(n, nnz, form, row_class):
    """The same for the bytes the library's copy of the matrix holds: the
    diagonal form reads values by diagonal (row_class per row, absent ones
    included) and a mask byte per row, and no column indices or row
    pointers; the column-value form one value per column in place of one
    per nonzero.  The general form: the CSR model."""
    if form == "diagonals":
        return 8 * row_class * n + n + 24 * n
    if form == "column values":
        return 4 * nnz + 4 * (n + 1) + 8 * n + 24 * n
    return sweep_bytes(n, nnz)


def kernel_source_digest(names):
    h = hashlib.sha256()
    for nm in names:
        with open(os.path.join(ROOT, "paper_2203_17063_amd", "csrc", nm), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel_tag, digest):
    """Fabric bytes per launch (calibrated FETCH_SIZE + WRITE_SIZE: L2 to
    Infinity Fabric requests, Infinity Cache hits included) from the
    committed rocprofv3 counter summary, or None when absent or taken on other
    kernel sources."""
    path = os.path.join(PROFILES, "%s.counters.txt" % kernel_tag)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_digest") != digest:
        return None
    try:
        return float(kv["fabric_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------

def build_workload(cfg):
    import workloads as W
    if cfg == "jacobi-1d":
        return W.jacobi_1d()
    if cfg == "jacobi-2d":
        return W.jacobi_2d()
    if cfg == "pagerank-rmat":
        return W.pagerank_rmat()
    if cfg == "jacobi-3d":
        return W.jacobi_3d()
    if cfg == "allgatherv":
        return W.allgatherv_lognormal()
    if cfg == "allreduce":
        return W.partial_allreduce()
    if cfg == "hypercube":
        return W.hypercube_ssp()
    if cfg == "threshold":
        return W.threshold_collectives()
    if cfg == "mf":
        return W.mf_problem()
    raise ValueError(cfg)


def describe(cfg, prob):
    if cfg in ("jacobi-1d", "jacobi-2d", "jacobi-3d"):
        dims = {"jacobi-1d": "1-D tridiagonal", "jacobi-2d": "2-D 5-point", "jacobi-3d": "3-D 7-point"}[cfg]
        return {"workload": "jacobi %s Laplacian n=%d, P=%d block-row ranks, S=%d, %s arrivals, "
                            "%d iterations" % (dims, prob.n, prob.P, prob.S,
                                               "all" if cfg == "jacobi-1d" else "Bernoulli",
                                               prob.T),
                "n": prob.n, "nnz": prob.A.nnz, "P": prob.P, "max_staleness": prob.S,
                "iterations": prob.T, "name": cfg}
    if cfg == "pagerank-rmat":
        return {"workload": "pagerank power iteration on R-MAT scale %d (%d edges), P=%d, S=%d, "
                            "Bernoulli(0.8), <=%d iterations or L1 < 1e-10"
                            % (prob.meta["scale"], prob.A.nnz, prob.P, prob.S, prob.T),
                "n": prob.n, "nnz": prob.A.nnz, "P": prob.P, "max_staleness": prob.S,
                "iterations": prob.T, "name": cfg}
    if cfg == "allgatherv":
        return {"workload": "allgatherv assembly, P=%d lognormal counts, %d elements, %d reps"
                            % (prob.P, int(prob.counts.sum()), prob.reps),
                "P": prob.P, "elements": int(prob.counts.sum()), "reps": prob.reps,
                "name": cfg}
    if cfg == "mf":
        return {"workload": "data-parallel matrix factorisation by minibatch SGD over the partial "
                            "allreduce: %d synthetic ratings (%d users x %d items), rank %d, P=%d "
                            "workers of %d minibatches, slack %d, Bernoulli(%.1f) arrivals, %d "
                            "iterations"
                            % (prob.N, prob.n_users, prob.n_items, prob.rank, prob.P, prob.K,
                               prob.S, prob.meta["q"], prob.T),
                "N": prob.N, "n_users": prob.n_users, "n_items": prob.n_items, "rank": prob.rank,
                "P": prob.P, "minibatches": prob.K, "slack": prob.S, "iterations": prob.T,
                "name": cfg}
    if cfg == "threshold":
        return {"workload": "threshold broadcast + reduce over a binomial tree, P=%d processes x "
                            "%d elements, data fraction %.2f, %d repetitions"
                            % (prob.P, prob.m, prob.theta, prob.reps),
                "P": prob.P, "m": prob.m, "theta": prob.theta, "reps": prob.reps,
                "name": cfg}
    if cfg == "hypercube":
        return {"workload": "hypercube allreduce_SSP with per-receiver views, P=%d processes x "
                            "%d elements, slack %d, Bernoulli(%.1f) message delivery, %d calls"
                            % (prob.P, prob.m, prob.slack, prob.q, prob.calls),
                "P": prob.P, "m": prob.m, "slack": prob.slack, "calls": prob.calls,
                "name": cfg}
    return {"workload": "partial allreduce-sum, P=%d x %d elements, Bernoulli(%.1f), stale "
                        "substitution, %d reps" % (prob.P, prob.m, prob.q, prob.reps),
            "P": prob.P, "m": prob.m, "reps": prob.reps, "name": cfg}


# ----------------------------------------------------------------------------
# GPU legs
# ----------------------------------------------------------------------------

def run_iterative_gpu(cfg, prob, steps, warmup):
    import torch
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R

    mem0 = torch.cuda.mem_get_info()[0]
    run = R.Iterative(prob.n, prob.A.row_ptr, prob.A.col, prob.A.val, prob.counts, prob.S,
                      prob.mask, prob.kind, b=prob.b, alpha=prob.alpha, beta=prob.beta,
                      x0=prob.x0)
    torch.cuda.synchronize()
    footprint = mem0 - torch.cuda.mem_get_info()[0]
    # one untimed solve records the eff history (bytes of the assembly)
    iters = run.solve(tol=prob.tol, histories=True)
    eff_hist = run.eff_hist.cpu().numpy()[:iters]
    for _ in range(warmup):
        run.solve(tol=prob.tol)
    # timed region: K solves, bracketed by device synchronisation and by two
    # HIP events on the plan's stream (torch's current stream)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(steps):
        it = run.solve(tol=prob.tol)
        assert it == iters
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    region_ms = ev0.elapsed_time(ev1)
    # the per-step work that is not a sweep: the solve's set-up (plan reset,
    # x0 copy, loop-control reset and read-back: a solve of 0 iterations) ...
    ev2, ev3 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev2.record()
    for _ in range(steps):
        run.solve(T=0)
    ev3.record()
    torch.cuda.synchronize()
    setup_ms = ev2.elapsed_time(ev3) / steps
    # ... and the separate assembly / norm launches, timed by HIP events
    # around every launch over a second region of the same K steps (the
    # events add a little time per launch)
    E.ecc_plan_set_timing(run.plan.handle, True)
    for k in (E.ECC_TIMING_ASSEMBLE, E.ECC_TIMING_SWEEP, E.ECC_TIMING_NORM):
        E.ecc_plan_timing(run.plan.handle, k, reset=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(steps):
        run.solve(tol=prob.tol)
    torch.cuda.synchronize()
    wall_events = time.perf_counter() - t1
    times = {k: E.ecc_plan_timing(run.plan.handle, getattr(E, "ECC_TIMING_" + k))
             for k in ("ASSEMBLE", "SWEEP", "NORM")}
    E.ecc_plan_set_timing(run.plan.handle, False)
    rho = run.d_rho.cpu().numpy()[:iters]
    n_part = int(run.d_partials.numel())
    layout, slots = E.ecc_matrix_layout(run.mat)
    schedule = E.ecc_matrix_schedule(run.mat)
    tiling = E.ecc_matrix_tiling(run.mat)
    form_id, offsets = E.ecc_matrix_form(run.mat)
    form = {E.ECC_FORM_GENERAL: "general", E.ECC_FORM_COLUMN_VALUES: "column values",
            E.ECC_FORM_DIAGONALS: "diagonals"}[form_id]
    probe = None
    if layout in (E.ECC_LAYOUT_SORTED, E.ECC_LAYOUT_RANGES):
        probe = gather_probe(prob, run, slots if layout == E.ECC_LAYOUT_RANGES else 1)
    run.close()

    counts = prob.counts
    eff_elems = np.array([int(counts[eff_hist[t] == 1].sum()) for t in range(iters)])
    # one fused launch per iteration: the sweep plus the write of the arrived
    # blocks into the assembled vector (their read is the sweep's own x read);
    # otherwise a separate assembly reads and writes every arrived element
    fused = times["SWEEP"][1] > 0 and times["ASSEMBLE"][1] == 0
    per_elem = 8.0 if fused else 16.0
    b_assemble = per_elem * eff_elems + 14.0 * prob.P
    b_sweep = float(sweep_bytes(prob.n, prob.A.nnz))
    b_sweep_form = float(format_sweep_bytes(prob.n, prob.A.nnz, form,
                                            slots if layout == E.ECC_LAYOUT_SHORT else 0))
    b_norm = 16.0 * n_part                 # partials written, then read by the second pass
    bytes_per_step = float(np.sum(b_assemble)) + iters * (b_sweep + b_norm)
    dom = b_sweep + b_norm + (float(np.mean(b_assemble)) if fused else 0.0)
    # the sweep's average duration from the uninstrumented region: its time
    # minus the set-up and the other launches, per sweep launch
    other_ms = setup_ms + (times["ASSEMBLE"][0] + times["NORM"][0]) / steps
    sweeps = times["SWEEP"][1] / steps
    dom_ms = (region_ms / steps - other_ms) / sweeps
    dom_timing = ("HIP events on the plan's stream around the timed region; the sweep's share "
                  "is that time minus a 0-iteration solve's (set-up) and the other launches' "
                  "(events around each), divided by the sweep launches")
    if schedule == E.ECC_SCHEDULE_SINGLE:
        # one launch per solve, bracketed by the solve's own synchronisation:
        # the events around that launch
        dom_ms = times["SWEEP"][0] / max(times["SWEEP"][1], 1)
        dom_timing = "HIP events on the plan's stream around the single launch of each solve"
    if probe:
        best = max(v["gathers_per_s"] for v in probe.values())
        probe["sweep_gathers_per_s"] = round(prob.A.nnz / (dom_ms / 1e3), 0)
        probe["sweep_over_probe"] = round(prob.A.nnz / (dom_ms / 1e3) / best, 4)
    return {
        "iters": iters, "wall": wall, "wall_events": wall_events, "times": times,
        "bytes_per_step": bytes_per_step, "dominant": "sweep",
        "dominant_bytes": dom, "footprint": footprint, "rho_last": float(rho[-1]),
        "dominant_format_bytes": dom - b_sweep + b_sweep_form,
        "unit_per_step": iters, "fused": fused, "dom_ms": dom_ms,
        "dom_timing": dom_timing,
        "dom_events_avg_us": round(times["SWEEP"][0] / max(times["SWEEP"][1], 1) * 1e3, 3),
        "extra": {"layout": {0: "stream", 1: "sorted", 2: "short", 3: "ranges"}[layout],
                  "schedule": {E.ECC_SCHEDULE_STATIC: "static", E.ECC_SCHEDULE_QUEUE: "queue",
                               E.ECC_SCHEDULE_SINGLE: "single launch"}[schedule],
                  "plane_tiling": {"plane_rows": tiling[0], "tile_rows": tiling[1]},
                  "matrix_form": form, "diagonal_offsets": offsets,
                  "gather_probe": probe,
                  "assembly_bytes_per_arrived_element": per_elem},
    }


def gather_probe(prob, run, n_ranges, reps=20):
    """The gather-rate ceiling of the matrix's columns (ecc_gather_probe: the
    index stream read, one vector gathered, nothing else), over the CSR
    order and over the order of its column ranges (entries grouped by range,
    CSR order within a range, as the range layout sweeps them), with HIP
    events around `reps` probes of each."""
    import torch
    from paper_2203_17063_amd import capi as E
    n, nnz = prob.n, prob.A.nnz
    col = prob.A.col
    orders = {"csr": None}
    if n_ranges > 1:
        rng_of = (col.astype(np.int64) * n_ranges) // n
        orders["ranges"] = np.argsort(rng_of, kind="stable")
    out = torch.empty((nnz + E.ECC_GATHER_CHUNK - 1) // E.ECC_GATHER_CHUNK, dtype=torch.float64,
                      device="cuda")
    x = run.d_x
    res = {}
    for name, order in orders.items():
        d_idx = run.d_col if order is None else torch.from_numpy(col[order]).cuda()
        E.ecc_gather_probe(d_idx, nnz, x, n, out, out.numel())
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            E.ecc_gather_probe(d_idx, nnz, x, n, out, out.numel())
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        res[name] = {"us": round(us, 2), "gathers_per_s": round(nnz / us * 1e6, 0)}
        del d_idx
    return res


def run_allgatherv_gpu(prob, steps, warmup):
    import torch
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R

    mem0 = torch.cuda.mem_get_info()[0]
    send = torch.from_numpy(prob.send).cuda()
    recv = torch.empty_like(send)
    d_mask = torch.from_numpy(prob.mask).cuda()
    plan = R.Plan(prob.P, prob.counts, prob.displs, prob.S)
    torch.cuda.synchronize()
    footprint = mem0 - torch.cuda.mem_get_info()[0]

    def step():
        plan.reset()
        for r in range(prob.reps):
            E.ecc_allgatherv_assemble_packed(plan.handle, send, recv, d_mask[r].data_ptr())

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    E.ecc_plan_set_timing(plan.handle, True)
    E.ecc_plan_timing(plan.handle, E.ECC_TIMING_ASSEMBLE, reset=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall_events = time.perf_counter() - t1
    times = {"ASSEMBLE": E.ecc_plan_timing(plan.handle, E.ECC_TIMING_ASSEMBLE)}
    E.ecc_plan_set_timing(plan.handle, False)
    assert torch.equal(recv, send)
    per_rep = 16.0 * float(prob.counts.sum()) + 14 * prob.P
    # the same repetitions over four send/receive buffer sets used in turn:
    # a working set of about 1 GB, four times the 256 MB Infinity Cache, so
    # that every repetition streams from HBM
    sets = [(send.clone(), torch.empty_like(send)) for _ in range(4)]
    del recv

    def step_rot():
        plan.reset()
        for r in range(prob.reps):
            sd, rv = sets[r & 3]
            E.ecc_allgatherv_assemble_packed(plan.handle, sd, rv, d_mask[r].data_ptr())

    step_rot()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(steps):
        step_rot()
    ev1.record()
    torch.cuda.synchronize()
    rot_ms = ev0.elapsed_time(ev1) / steps
    for sd, rv in sets:
        assert torch.equal(rv, sd)
    plan.close()
    rot = {"value": round(per_rep * prob.reps / rot_ms / 1e6, 3), "unit": "GB/s",
           "ms_per_step": round(rot_ms, 4),
           "avg_rep_us": round(rot_ms / prob.reps * 1e3, 3),
           "hbm_peak_frac": round(per_rep * prob.reps / rot_ms / 1e6 / HBM_PEAK_GBS, 4),
           "note": "repetition r reads and writes buffer set r mod 4 (4 x 264 MB); HIP "
                   "events around the K steps on the plan's stream"}
    return {"iters": prob.reps, "wall": wall, "wall_events": wall_events, "times": times,
            "bytes_per_step": per_rep * prob.reps, "dominant": "assemble",
            "dominant_bytes": per_rep, "footprint": footprint, "unit_per_step": prob.reps,
            "extra": {"rotated_4_buffer_sets": rot}}


def run_allreduce_gpu(prob, steps, warmup):
    import torch
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R

    mem0 = torch.cuda.mem_get_info()[0]
    P, m = prob.P, prob.m
    # every repetition reuses rank p's repetition-0 contribution (same bytes moved)
    fresh = [torch.from_numpy(prob.fresh(p, 0)).cuda() for p in range(P)]
    slots = [torch.empty(m, dtype=torch.float64, device="cuda") for _ in range(P)]
    result = torch.empty(m, dtype=torch.float64, device="cuda")
    d_fresh, d_slots = R.ptr_array(fresh), R.ptr_array(slots)
    d_mask = torch.from_numpy(prob.mask).cuda()
    plan = R.Plan(P, None, None, prob.S)
    eff = torch.empty((prob.reps, P), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    footprint = mem0 - torch.cuda.mem_get_info()[0]

    def step(record=False):
        plan.reset()
        for r in range(prob.reps):
            E.ecc_allreduce_partial(plan.handle, m, d_fresh, d_slots, result,
                                    d_mask[r].data_ptr(), eff[r] if record else None)

    step(record=True)
    n_eff = eff.sum(dim=1).cpu().numpy().astype(np.int64)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    E.ecc_plan_set_timing(plan.handle, True)
    E.ecc_plan_timing(plan.handle, E.ECC_TIMING_ALLREDUCE, reset=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall_events = time.perf_counter() - t1
    times = {"ALLREDUCE": E.ecc_plan_timing(plan.handle, E.ECC_TIMING_ALLREDUCE)}
    E.ecc_plan_set_timing(plan.handle, False)
    plan.close()
    per_rep = [8.0 * m * (P + int(a) + 1) + 14 * P for a in n_eff]
    return {"iters": prob.reps, "wall": wall, "wall_events": wall_events, "times": times,
            "bytes_per_step": float(sum(per_rep)), "dominant": "allreduce",
            "dominant_bytes": float(np.mean(per_rep)), "footprint": footprint,
            "unit_per_step": prob.reps}


def run_hypercube_gpu(prob, steps, warmup):
    """One step = a reset and prob.calls calls of every process.  Two
    contribution sets alternate between calls (the bytes moved do not depend
    on the values)."""
    import torch
    from paper_2203_17063_amd import capi as E

    mem0 = torch.cuda.mem_get_info()[0]
    P, m, d = prob.P, prob.m, prob.d
    contrib = [torch.from_numpy(prob.contrib(t)).cuda() for t in range(2)]
    result = torch.empty((P, m), dtype=torch.float64, device="cuda")
    d_del = torch.from_numpy(prob.delivered.astype(np.uint8)).cuda()
    stream = torch.cuda.current_stream().cuda_stream
    h = E.ecc_hypercube_create(P, m, prob.slack, stream)
    torch.cuda.synchronize()
    footprint = mem0 - torch.cuda.mem_get_info()[0]

    def step(events=None):
        E.ecc_hypercube_reset(h)
        for t in range(prob.calls):
            if events is not None:
                events[t][0].record()
            E.ecc_allreduce_ssp(h, contrib[t & 1], d_del[t], result)
            if events is not None:
                events[t][1].record()

    for _ in range(max(warmup, 1)):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # the same steps with events around every call (one kernel launch each)
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(prob.calls)] for _ in range(steps)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for s_ in range(steps):
        step(ev[s_])
    torch.cuda.synchronize()
    wall_events = time.perf_counter() - t1
    ms = sum(a.elapsed_time(b) for row in ev for a, b in row)
    _, waits, _, _ = E.ecc_hypercube_stats(h, P)
    E.ecc_hypercube_destroy(h)
    per_call = 8.0 * m * P * (d + 2) + 2.0 * P * d
    return {"iters": prob.calls, "wall": wall, "wall_events": wall_events,
            "times": {"ALLREDUCE_SSP": (ms, steps * prob.calls)},
            "bytes_per_step": per_call * prob.calls, "dominant": "allreduce_ssp",
            "dominant_bytes": per_call, "footprint": footprint, "unit_per_step": prob.calls,
            "waits_per_step": waits}


def run_threshold_gpu(prob, steps, warmup):
    """One step = prob.reps x [threshold broadcast from process 0, then
    threshold reduce to process 0, both with data fraction theta]."""
    import torch
    from paper_2203_17063_amd import capi as E

    mem0 = torch.cuda.mem_get_info()[0]
    P, m, theta = prob.P, prob.m, prob.theta
    vecs = [torch.from_numpy(prob.vector(p)).cuda() for p in range(P)]
    result = torch.empty(m, dtype=torch.float64, device="cuda")
    d_vecs = torch.tensor([v.data_ptr() for v in vecs], dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    torch.cuda.synchronize()
    footprint = mem0 - torch.cuda.mem_get_info()[0]
    k_b = k_r = n_r = 0

    def step(ev=None):
        nonlocal k_b, k_r, n_r
        for r in range(prob.reps):
            if ev is not None:
                ev[r][0].record()
            k_b = E.ecc_bcast_threshold(P, 0, m, theta, vecs[0], d_vecs, stream)
            if ev is not None:
                ev[r][1].record()
            k_r, n_r = E.ecc_reduce_threshold(P, 0, m, theta, E.ECC_THRESHOLD_DATA, d_vecs,
                                              result, stream)
            if ev is not None:
                ev[r][2].record()

    for _ in range(max(warmup, 1)):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(prob.reps)]
          for _ in range(steps)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for s_ in range(steps):
        step(ev[s_])
    torch.cuda.synchronize()
    wall_events = time.perf_counter() - t1
    ms_b = sum(e[0].elapsed_time(e[1]) for row in ev for e in row)
    ms_r = sum(e[1].elapsed_time(e[2]) for row in ev for e in row)
    bytes_b = 8.0 * k_b * P                 # the root's prefix read once, P - 1 copies written
    bytes_r = 8.0 * k_r * (n_r + 1)         # n prefixes read, the result written
    return {"iters": prob.reps, "wall": wall, "wall_events": wall_events,
            "times": {"REDUCE": (ms_r, steps * prob.reps), "BCAST": (ms_b, steps * prob.reps)},
            "bytes_per_step": (bytes_b + bytes_r) * prob.reps, "dominant": "reduce",
            "dominant_bytes": bytes_r, "footprint": footprint, "unit_per_step": prob.reps}


def mf_bytes(prob):
    """Algorithmic bytes of one factorisation iteration, per kernel."""
    N, m, P = prob.N, prob.m, prob.P
    rows = prob.n_users + prob.n_items
    return {"MF_GRAD": 24.0 * N / prob.K + 12.0 * P * rows + 8.0 * m + 8.0 * m * P,
            # 2 x (other row, rating) per rating of the minibatches, (row,
            # start, length) per (worker, row), the model, P gradients written
            # the P slots read (the gradients of the workers taken this
            # iteration were written into their slots), the result written
            "ALLREDUCE": 8.0 * m * (P + 1),
            "MF_STEP": 24.0 * m + 8.0 * rows}


def run_mf_gpu(prob, steps, warmup):
    """One step = a reset and prob.T iterations.  Afterwards, a slack study:
    the iterations needed at slack 0 / 2 / 32 / 64 to reach the full training
    error that slack 0 reaches after prob.T iterations (same arrival
    probability and minibatch schedule)."""
    import dataclasses
    import torch
    import workloads as W
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R

    mem0 = torch.cuda.mem_get_info()[0]
    run = R.MatrixFactorization(prob)
    torch.cuda.synchronize()
    footprint = mem0 - torch.cuda.mem_get_info()[0]
    run.run()
    torch.cuda.synchronize()
    arrivals = run.d_eff.sum(dim=1).cpu().numpy().astype(np.int64)
    rmse_T = float(run.d_rmse[prob.T - 1].item())
    for _ in range(warmup):
        run.run(record=False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run.run(record=False)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ph = run.plan.handle
    E.ecc_plan_set_timing(ph, True)
    kinds = {"MF_GRAD": E.ECC_TIMING_MF_GRAD, "ALLREDUCE": E.ECC_TIMING_ALLREDUCE,
             "MF_STEP": E.ECC_TIMING_MF_STEP}
    for k in kinds.values():
        E.ecc_plan_timing(ph, k, reset=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(steps):
        run.run(record=False)
    torch.cuda.synchronize()
    wall_events = time.perf_counter() - t1
    times = {name: E.ecc_plan_timing(ph, k) for name, k in kinds.items()}
    E.ecc_plan_set_timing(ph, False)
    run.close()
    per = mf_bytes(prob)
    # slack study, 3 x T iterations each, arrivals Bernoulli(q) per (iteration,
    # worker), the same minibatch schedule; the full training error before
    # every iteration (err[t] = error of W^t) and after the last
    T3 = 3 * prob.T
    study = {}
    target = None
    for S in (0, 2, 32, 64):
        pS = dataclasses.replace(prob, S=S, T=T3,
                                 mask=W.arrival_mask(W.seed_of(8), T3, np.full(prob.P, prob.meta["q"])),
                                 batch=W.batch_schedule(W.seed_of(8), T3, prob.P, prob.K))
        rs = R.MatrixFactorization(pS)
        rs.run(errors=True)
        torch.cuda.synchronize()
        err = rs.d_err.cpu().numpy()[:T3 + 1]
        _, forced, _, _ = rs.plan.stats()
        if target is None:
            target = float(err[prob.T])
        hit = np.nonzero(err[1:] <= target)[0]
        # time to the target: the iterations it takes, run again without the
        # error evaluations
        ms_to_target = None
        if hit.size:
            n_it = int(hit[0]) + 1
            rs.run(T=n_it, record=False)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            rs.run(T=n_it, record=False)
            e1.record()
            torch.cuda.synchronize()
            ms_to_target = round(e0.elapsed_time(e1), 3)
        rs.close()
        study[str(S)] = {"iterations_to_target": int(hit[0]) + 1 if hit.size else None,
                         "gpu_ms_to_target": ms_to_target,
                         "forced_arrivals_in_%d" % T3: int(forced),
                         "error_after_%d" % prob.T: round(float(err[prob.T]), 6)}
    return {"iters": prob.T, "wall": wall, "wall_events": wall_events, "times": times,
            "bytes_per_step": sum(per.values()) * prob.T, "dominant": "mf_grad",
            "dominant_bytes": per["MF_GRAD"], "footprint": footprint, "unit_per_step": prob.T,
            "extra": {"minibatch_rmse_at_T": round(rmse_T, 6), "target_error": round(target, 6),
                      "workers_taken_per_iteration": round(float(arrivals.mean()), 3),
                      "minibatches_per_worker": prob.K, "eta": prob.eta,
                      "slack_study": study,
                      "kernel_bytes": {k: round(v) for k, v in per.items()}}}


# ----------------------------------------------------------------------------
# CPU baseline: the oracle as it stands, on a bounded sample
# ----------------------------------------------------------------------------

def host_cpu():
    """Cores this process may run on, and the CPU model."""
    cores = len(os.sched_getaffinity(0))
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cores, model


def cpu_baseline(cfg, prob, res, budget_s=12.0):
    import oracle
    cores = 1
    n_cores, model = host_cpu()
    if cfg in ("jacobi-1d", "jacobi-2d", "pagerank-rmat", "jacobi-3d"):
        # whole iterations of the oracle (sample = the first k iterations), on
        # one thread and on every core of this host: its row loops run on
        # OpenMP threads, one row per thread in the same order, so both give
        # the same bits
        per_iter_bytes = res["bytes_per_step"] / res["iters"]
        sample_iters = res["iters"] if cfg in ("jacobi-1d", "jacobi-2d") else min(res["iters"], 8)

        def timed(threads, budget):
            t0 = time.perf_counter()
            k = done_iters = 0
            while True:
                oracle.run_iterative(prob, T=sample_iters, threads=threads)
                done_iters += sample_iters
                k += 1
                if time.perf_counter() - t0 >= budget:
                    break
            dt = time.perf_counter() - t0
            return per_iter_bytes * done_iters / dt / 1e9, done_iters, k, dt

        g1, i1, k1, d1 = timed(1, budget_s / 2)
        gn, i_n, kn, dn = timed(n_cores, budget_s / 2)
        return {"value": round(gn, 4), "unit": "GB/s", "cores": n_cores, "kind": "oracle",
                "value_1_thread": round(g1, 4), "cpu_model": model,
                "iterations_per_s": round(i_n / dn, 4),
                "iterations_per_s_1_thread": round(i1 / d1, 4),
                "sample": "runs of the first %d oracle iterations of this workload: %d run(s) "
                          "on %d threads in %.1f s, %d run(s) on 1 thread in %.1f s"
                          % (sample_iters, kn, n_cores, dn, k1, d1)}
    if cfg == "allgatherv":
        version = np.full(prob.P, -1, dtype=np.int32)
        recv = np.empty_like(prob.send)
        sends = [prob.send[d:d + c] for d, c in zip(prob.displs, prob.counts)]
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < budget_s and reps < prob.reps:
            eff, _, _ = oracle.select(prob.S, reps, prob.mask[reps], version)
            oracle.allgatherv(prob.counts, prob.displs, eff, sends, recv)
            reps += 1
        dt = time.perf_counter() - t0
        per_rep = res["bytes_per_step"] / res["iters"]
        return {"value": round(per_rep * reps / dt / 1e9, 4), "unit": "GB/s", "cores": cores,
                "kind": "oracle", "cpu_model": model,
                "sample": "%d of %d repetitions, 1 thread (the oracle has no threaded loop here), %.1f s"
                                            % (reps, prob.reps, dt)}
    if cfg == "mf":
        # workers' shares of the iterations in order (iteration t's minibatch
        # of worker p, at the initial model), one after another: the errors
        # and gradient of each worker's minibatch, until the time is used
        from oracle import mf as MFO
        e = np.zeros(prob.N)
        t0 = time.perf_counter()
        done = 0
        while done < prob.P * prob.T and (done == 0 or time.perf_counter() - t0 < budget_s):
            t, p = divmod(done, prob.P)
            lo, hi = prob.batch_range(p, int(prob.batch[t][p]))
            e[lo:hi] = MFO.errors(prob, prob.W0, lo, hi)
            MFO.worker_gradient(prob, prob.W0, e, p, lo, hi)
            done += 1
        dt = time.perf_counter() - t0
        # per worker: its share of the index and ratings, the model read,
        # its gradient written
        rows = prob.n_users + prob.n_items
        per_worker = (24.0 * prob.N / prob.K + 12.0 * prob.P * rows) / prob.P + 16.0 * prob.m
        return {"value": round(per_worker * done / dt / 1e9, 4), "unit": "GB/s", "cores": cores,
                "kind": "oracle", "cpu_model": model,
                "sample": "the errors and gradients of %d worker minibatches of the first "
                          "iterations' schedule (%d per iteration, 1/%d of the ratings each) at "
                          "the initial model, 1 thread, %.1f s"
                          % (done, prob.P, prob.P * prob.K, dt)}
    if cfg == "threshold":
        from oracle import threshold as THO
        P, m = prob.P, prob.m
        vecs = [prob.vector(p) for p in range(P)]
        bufs = [v.copy() for v in vecs]
        result = np.zeros(m)
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < budget_s and reps < prob.reps:
            THO.bcast(P, 0, prob.theta, vecs[0], bufs)
            THO.reduce(P, 0, prob.theta, THO.DATA, vecs, result)
            reps += 1
        dt = time.perf_counter() - t0
        per_rep = res["bytes_per_step"] / res["iters"]
        return {"value": round(per_rep * reps / dt / 1e9, 4), "unit": "GB/s", "cores": cores,
                "kind": "oracle", "cpu_model": model,
                "sample": "%d of %d repetitions, 1 thread (the oracle has no threaded loop here), %.1f s"
                                            % (reps, prob.reps, dt)}
    if cfg == "hypercube":
        # whole calls of the oracle over the full vectors, from a reset
        from oracle import hypercube as HC
        P, m, d = prob.P, prob.m, prob.d
        contrib = [prob.contrib(t) for t in range(2)]
        st = HC.HypercubeSSP(P, m, prob.slack)
        t0 = time.perf_counter()
        calls = 0
        while time.perf_counter() - t0 < budget_s and calls < prob.calls:
            st.call(contrib[calls & 1], prob.delivered[calls])
            calls += 1
        dt = time.perf_counter() - t0
        per_call = res["bytes_per_step"] / res["iters"]
        return {"value": round(per_call * calls / dt / 1e9, 4), "unit": "GB/s", "cores": cores,
                "kind": "oracle", "cpu_model": model,
                "sample": "the first %d of %d calls, 1 thread, %.1f s"
                                            % (calls, prob.calls, dt)}
    # 4b: a few repetitions over stored vectors
    P, m = prob.P, prob.m
    fresh = [prob.fresh(p, 0) for p in range(P)]
    slots = [np.zeros(m) for _ in range(P)]
    version = np.full(P, -1, dtype=np.int32)
    t0 = time.perf_counter()
    reps = 0
    nbytes = 0.0
    while time.perf_counter() - t0 < budget_s and reps < prob.reps:
        eff, _, _ = oracle.select(prob.S, reps, prob.mask[reps], version)
        oracle.allreduce(eff, fresh, slots)
        nbytes += 8.0 * m * (P + int(eff.sum()) + 1)
        reps += 1
    dt = time.perf_counter() - t0
    return {"value": round(nbytes / dt / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "cpu_model": model,
            "sample": "%d of %d repetitions over stored vectors, 1 thread, "
                                        "%.1f s" % (reps, prob.reps, dt)}


def copy_probe(n_doubles=1 << 29, reps=10):
    """Measured copy ceiling: a plain 16-byte streaming copy of 4 GiB (far
    beyond the 256 MB Infinity Cache) with libecc's ecc_stream_copy, and the
    runtime's own device-to-device copy for comparison; read + write bytes per
    second."""
    import torch
    from paper_2203_17063_amd import capi as E
    x = torch.empty(n_doubles, dtype=torch.float64, device="cuda").fill_(1.0)
    y = torch.empty_like(x)
    stream = torch.cuda.current_stream().cuda_stream
    out = {}
    for name, fn in (("ecc_stream_copy", lambda: E.ecc_stream_copy(y, x, n_doubles, stream)),
                     ("runtime_copy", lambda: y.copy_(x))):
        fn()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(reps):
            fn()
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / reps
        nbytes = 2 * 8 * n_doubles
        out[name] = {"bytes_per_copy": nbytes, "avg_ms": round(ms, 4),
                     "gbs": round(nbytes / ms / 1e6, 2),
                     "frac_of_peak": round(nbytes / ms / 1e6 / HBM_PEAK_GBS, 4)}
    assert torch.equal(x, y)
    return {"copy_probe": out}


# ----------------------------------------------------------------------------

def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="jacobi-3d",
                    choices=["jacobi-1d", "jacobi-2d", "pagerank-rmat", "jacobi-3d", "allgatherv",
                             "allreduce", "hypercube", "threshold", "mf"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-ceiling", action="store_true",
                    help="skip the 4 GiB copy that measures the copy ceiling")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only measure a plain 4 GiB device copy (copy ceiling)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the data path runs P virtual ranks inside one "
              "GPU's HBM and the library has no multi-GPU path (requested --gpus %d)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    from paper_2203_17063_amd import capi
    capi.lib()
    if args.copy_probe:
        print(json.dumps(copy_probe()), flush=True)
        return

    cfg = args.config
    print("[bench] generating workload %s" % cfg, file=sys.stderr, flush=True)
    prob = build_workload(cfg)
    print("[bench] running on GPU", file=sys.stderr, flush=True)
    if cfg in ("jacobi-1d", "jacobi-2d", "pagerank-rmat", "jacobi-3d"):
        res = run_iterative_gpu(cfg, prob, args.steps, args.warmup)
        digest = kernel_source_digest(["sweep.hip", "tiny.hip", "ecc_common.h"])
        tag = "sweep_" + cfg.replace("-", "_")
        dom_ms, dom_n = res["times"]["SWEEP"]
    elif cfg == "allgatherv":
        res = run_allgatherv_gpu(prob, args.steps, args.warmup)
        digest = kernel_source_digest(["collectives.hip", "ecc_common.h"])
        tag = "assemble_allgatherv"
        dom_ms, dom_n = res["times"]["ASSEMBLE"]
    elif cfg == "mf":
        res = run_mf_gpu(prob, args.steps, args.warmup)
        digest = kernel_source_digest(["mf.hip", "ecc_common.h"])
        tag = "mf_grad_p32"
        dom_ms, dom_n = res["times"]["MF_GRAD"]
    elif cfg == "threshold":
        res = run_threshold_gpu(prob, args.steps, args.warmup)
        digest = kernel_source_digest(["threshold.hip", "ecc_common.h"])
        tag = "reduce_threshold_p32"
        dom_ms, dom_n = res["times"]["REDUCE"]
    elif cfg == "hypercube":
        res = run_hypercube_gpu(prob, args.steps, args.warmup)
        digest = kernel_source_digest(["hypercube.hip", "ecc_common.h"])
        tag = "allreduce_ssp_p32"
        dom_ms, dom_n = res["times"]["ALLREDUCE_SSP"]
    else:
        res = run_allreduce_gpu(prob, args.steps, args.warmup)
        digest = kernel_source_digest(["collectives.hip", "ecc_common.h"])
        tag = "allreduce_partial"
        dom_ms, dom_n = res["times"]["ALLREDUCE"]

    steps = args.steps
    wall = res["wall"]
    ms_per_step = wall / steps * 1e3
    gbs = res["bytes_per_step"] * steps / wall / 1e9
    iters_per_s = res["unit_per_step"] * steps / wall
    if "dom_ms" in res:
        avg_dom_s = res["dom_ms"] / 1e3
        timing = res["dom_timing"]
    else:
        avg_dom_s = dom_ms / max(dom_n, 1) / 1e3
        timing = "HIP events on the launching stream around every launch, over a second " \
                 "region of the same K steps"
    achieved = res["dominant_bytes"] / avg_dom_s / 1e9 if avg_dom_s > 0 else None
    traffic = read_traffic(tag, digest)
    ceiling = None
    if not args.no_copy_ceiling:
        print("[bench] copy ceiling", file=sys.stderr, flush=True)
        ceiling = copy_probe(n_doubles=1 << 29, reps=5)["copy_probe"]["ecc_stream_copy"]["gbs"]
    line = {
        "metric": METRIC,
        "value": round(gbs, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic (seeded generators; no dataset)",
        "config": describe(cfg, prob),
        "iterations_per_s": round(iters_per_s, 2),
        "hbm_peak_frac": round(gbs / HBM_PEAK_GBS, 4),
        "copy_ceiling_gbs": ceiling,
        "copy_ceiling_frac": round(gbs / ceiling, 4) if ceiling else None,
        "ms_per_step_with_kernel_events": round(res["wall_events"] / steps * 1e3, 4),
        "peak_hbm_footprint_gb": round(res["footprint"] / 1e9, 3),
        "kernel_avg_us": {k.lower(): round(v[0] / max(v[1], 1) * 1e3, 3)
                          for k, v in res["times"].items()},
        "roofline": {
            "kernel": tag,
            "bound": "hbm",
            "achieved": round(achieved, 2) if achieved else None,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None,
            "frac_of_copy_ceiling": round(achieved / ceiling, 4) if (achieved and ceiling)
            else None,
            "traffic": traffic,
            "traffic_kind": "fabric bytes per launch: calibrated FETCH_SIZE + WRITE_SIZE (L2 to "
                            "Infinity Fabric requests, Infinity Cache hits included)",
            "algorithmic_bytes_per_launch": res["dominant_bytes"],
            "algorithmic_model": "the method's data as its definition holds it (CSR for the "
                                 "iterations), each element counted once",
            "avg_launch_us": round(avg_dom_s * 1e6, 3),
            "launches_timed": dom_n,
            "timing": timing,
        },
    }
    if "dom_events_avg_us" in res:
        line["roofline"]["avg_launch_us_with_events"] = res["dom_events_avg_us"]
    if "dominant_format_bytes" in res and achieved:
        # the same launch against the bytes the library's copy of the matrix
        # holds (compact forms drop column indices or per-entry values)
        fb = res["dominant_format_bytes"]
        line["roofline"]["format_bytes_per_launch"] = round(fb)
        line["roofline"]["achieved_format"] = round(fb / avg_dom_s / 1e9, 2)
        line["roofline"]["frac_format"] = round(fb / avg_dom_s / 1e9 / HBM_PEAK_GBS, 4)
    if "extra" in res:
        line.update(res["extra"])
    if not args.no_cpu_baseline:
        print("[bench] oracle CPU baseline", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(cfg, prob, res)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
