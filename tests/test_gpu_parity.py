"""GPU parity: the HIP path through the C ABI against the oracle.

Collectives (assembly, partial allreduce) and all staleness bookkeeping are
compared bit for bit.  Iterates are compared normwise within 1e-12 of the
oracle, norms within 1e-12 relative plus 32 units of rounding of the
problem's scale; stencil sweeps sum every row on one lane in CSR order, so
their iterates are also checked bit for bit.
"""

import dataclasses
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle                                             # noqa: E402
import workloads as W                                     # noqa: E402
from gpu_common import (UNB, announce, assert_iterates_close,  # noqa: E402
                        assert_rho_close)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2203_17063_amd import capi
    capi.lib()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _capi():
    from paper_2203_17063_amd import capi
    return capi


def _runner():
    from paper_2203_17063_amd import runner
    return runner


# ----------------------------------------------------------------------------
# allgatherv assembly
# ----------------------------------------------------------------------------

def _layout(kind, P, rng):
    if kind == "prefix":
        counts = rng.integers(0, 5000, P)
        displs = W.exclusive_scan(counts)
    elif kind == "gapped_unsorted":
        counts = rng.integers(0, 3000, P)
        counts[rng.random(P) < 0.2] = 0
        order = rng.permutation(P)
        displs = np.zeros(P, dtype=np.int64)
        pos = int(rng.integers(0, 7))
        for p in order:
            displs[p] = pos
            pos += int(counts[p]) + int(rng.integers(0, 9))   # odd gaps
    else:  # tiny blocks
        counts = rng.integers(0, 4, P)
        displs = W.exclusive_scan(counts) + np.arange(P)      # one-element gaps
    return counts.astype(np.int64), displs.astype(np.int64)


@pytest.mark.parametrize("P,layout,S,misalign", [
    (1, "prefix", 0, False),
    (2, "gapped_unsorted", 1, True),
    (3, "tiny", 2, False),
    (7, "gapped_unsorted", 5, True),
    (64, "prefix", 3, False),
    (512, "gapped_unsorted", UNB, True),
    (512, "tiny", 1, True),
])
def test_assemble_parity(P, layout, S, misalign):
    E, R = _capi(), _runner()
    rng = np.random.default_rng(P * 31 + S % 97)
    counts, displs = _layout(layout, P, rng)
    extent = int((displs + counts).max()) if P else 0
    T = 12
    mask = (rng.random((T, P)) < 0.5).astype(np.uint8)
    announce("assemble", P, layout, S, misalign, extent)
    # each rank's send block in its own allocation, some starting at an odd
    # element so that source and destination alignments differ
    host_send = [rng.standard_normal(int(c)) for c in counts]
    dev_store = []
    send = []
    for p in range(P):
        off = int(rng.integers(0, 2)) if misalign else 0
        buf = torch.empty(int(counts[p]) + 2, dtype=torch.float64, device="cuda")
        view = buf[off:off + int(counts[p])]
        view.copy_(torch.from_numpy(host_send[p]))
        dev_store.append(buf)
        send.append(view)
    d_send = R.ptr_array(send)
    canary = -7.25
    recv = torch.full((extent + 3,), canary, dtype=torch.float64, device="cuda")
    plan = R.Plan(P, counts, displs, S)
    d_mask = torch.from_numpy(mask).cuda()
    eff_d = torch.empty(P, dtype=torch.uint8, device="cuda")
    age_d = torch.empty(P, dtype=torch.int32, device="cuda")
    ref_recv = np.full(extent + 3, canary)
    version = np.full(P, -1, dtype=np.int32)
    forced_total = 0
    for t in range(T):
        # new contents every step so that stale blocks are distinguishable
        for p in range(P):
            host_send[p] = host_send[p] + 1.0
            send[p].copy_(torch.from_numpy(host_send[p]))
        E.ecc_allgatherv_assemble(plan.handle, d_send, recv, d_mask[t].data_ptr(), eff_d, age_d)
        eff, age, forced = oracle.select(S, t, mask[t], version)
        forced_total += forced
        oracle.allgatherv(counts, displs, eff, host_send, ref_recv)
        torch.cuda.synchronize()
        assert np.array_equal(eff_d.cpu().numpy(), eff), t
        assert np.array_equal(age_d.cpu().numpy(), age), t
        got = recv.cpu().numpy()
        assert np.array_equal(got, ref_recv), (t, np.nonzero(got != ref_recv)[0][:8])
    clock, forced_dev, ver_dev, age_dev = plan.stats()
    assert clock == T and forced_dev == forced_total
    assert np.array_equal(ver_dev, version)
    plan.close()


def test_assemble_packed_and_empty():
    E, R = _capi(), _runner()
    prob = W.allgatherv_lognormal(P=256, reps=6, mean=700.0)
    announce("assemble_packed 4a-small", prob.counts.sum())
    E_tot = int(prob.counts.sum())
    send = torch.from_numpy(prob.send).cuda()
    recv = torch.full((E_tot,), np.nan, dtype=torch.float64, device="cuda")
    plan = R.Plan(prob.P, prob.counts, prob.displs, prob.S)
    d_mask = torch.from_numpy(prob.mask).cuda()
    for t in range(prob.reps):
        E.ecc_allgatherv_assemble_packed(plan.handle, send, recv, d_mask[t].data_ptr())
    torch.cuda.synchronize()
    assert np.array_equal(recv.cpu().numpy(), prob.send)   # prefix displs: concatenation
    plan.close()
    # a plan whose blocks are all empty
    plan = R.Plan(3, [0, 0, 0], [0, 5, 9], 1)
    E.ecc_allgatherv_assemble_packed(plan.handle, send, recv, d_mask[0].data_ptr())
    assert plan.stats()[0] == 1
    plan.close()


def test_assemble_errors_leave_state():
    E, R = _capi(), _runner()
    plan = R.Plan(2, None, None, 1)
    with pytest.raises(E.EccError) as ei:
        E.ecc_allgatherv_assemble_packed(plan.handle, 1, 1, 1)
    assert ei.value.status == E.ECC_ERR_STATE
    assert plan.stats()[0] == 0
    plan.close()


# ----------------------------------------------------------------------------
# partial allreduce
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("P,m,S,aligned", [
    (1, 1000, 0, True),
    (3, 1, 1, True),
    (5, 1023, 2, True),
    (17, 4097, UNB, False),
    (256, 3000, 3, True),
    (256, 2048, UNB, True),
])
def test_allreduce_parity(P, m, S, aligned):
    E, R = _capi(), _runner()
    rng = np.random.default_rng(1000 + P + m)
    R_ = 10
    mask = (rng.random((R_, P)) < 0.6).astype(np.uint8)
    announce("allreduce", P, m, S, aligned)
    off = 0 if aligned else 1
    fresh_store = [torch.empty(m + 2, dtype=torch.float64, device="cuda") for _ in range(P)]
    slot_store = [torch.full((m + 2,), np.nan, dtype=torch.float64, device="cuda")
                  for _ in range(P)]
    fresh = [f[off:off + m] for f in fresh_store]
    slots = [s[off:off + m] for s in slot_store]
    result = torch.empty(m + 1, dtype=torch.float64, device="cuda")[off:off + m]
    d_fresh, d_slots = R.ptr_array(fresh), R.ptr_array(slots)
    d_mask = torch.from_numpy(mask).cuda()
    eff_d = torch.empty(P, dtype=torch.uint8, device="cuda")
    clk_d = torch.empty(1, dtype=torch.int32, device="cuda")
    plan = R.Plan(P, None, None, S)
    version = np.full(P, -1, dtype=np.int32)
    ref_slots = [np.zeros(m) for _ in range(P)]
    for r in range(R_):
        host_fresh = [rng.uniform(-1, 1, m) for _ in range(P)]
        for p in range(P):
            fresh[p].copy_(torch.from_numpy(host_fresh[p]))
        E.ecc_allreduce_partial(plan.handle, m, d_fresh, d_slots, result, d_mask[r].data_ptr(),
                                eff_d, clk_d)
        eff, age, _ = oracle.select(S, r, mask[r], version)
        ref = oracle.allreduce(eff, host_fresh, ref_slots)
        torch.cuda.synchronize()
        assert np.array_equal(eff_d.cpu().numpy(), eff)
        assert np.array_equal(result.cpu().numpy(), ref), r
        assert int(clk_d.item()) == oracle.result_clock(version)
        for p in range(P):
            if eff[p] or r > 0:
                assert np.array_equal(slots[p].cpu().numpy(), ref_slots[p]), (r, p)
    plan.close()


@pytest.mark.parametrize("P,m,S,aligned", [
    (6, 1023, 1, True),
    (17, 4097, UNB, False),
    (64, 3000, 0, True),
])
def test_allreduce_in_place(P, m, S, aligned):
    """Contributions that their producer wrote into the slot itself
    (fresh[p] == slots[p] for every third rank, written only where the rank
    is taken, as the matrix factorisation does) next to ordinary ones: the
    same results and slots as copying them."""
    E, R = _capi(), _runner()
    rng = np.random.default_rng(2000 + P + m)
    R_ = 10
    mask = (rng.random((R_, P)) < 0.5).astype(np.uint8)
    announce("allreduce in place", P, m, S, aligned)
    off = 0 if aligned else 1
    inplace = [p % 3 == 0 for p in range(P)]
    fresh_store = [torch.empty(m + 2, dtype=torch.float64, device="cuda") for _ in range(P)]
    slot_store = [torch.full((m + 2,), np.nan, dtype=torch.float64, device="cuda")
                  for _ in range(P)]
    slots = [s_[off:off + m] for s_ in slot_store]
    fresh = [slots[p] if inplace[p] else fresh_store[p][off:off + m] for p in range(P)]
    result = torch.empty(m + 1, dtype=torch.float64, device="cuda")[off:off + m]
    d_fresh, d_slots = R.ptr_array(fresh), R.ptr_array(slots)
    d_mask = torch.from_numpy(mask).cuda()
    eff_d = torch.empty(P, dtype=torch.uint8, device="cuda")
    clk_d = torch.empty(1, dtype=torch.int32, device="cuda")
    plan = R.Plan(P, None, None, S)
    version = np.full(P, -1, dtype=np.int32)
    ref_slots = [np.zeros(m) for _ in range(P)]
    for r in range(R_):
        host_fresh = [rng.uniform(-1, 1, m) for _ in range(P)]
        eff, _, _ = oracle.select(S, r, mask[r], version)
        for p in range(P):
            if not inplace[p] or eff[p]:
                fresh[p].copy_(torch.from_numpy(host_fresh[p]))
        E.ecc_allreduce_partial(plan.handle, m, d_fresh, d_slots, result, d_mask[r].data_ptr(),
                                eff_d, clk_d)
        ref = oracle.allreduce(eff, host_fresh, ref_slots)
        torch.cuda.synchronize()
        assert np.array_equal(eff_d.cpu().numpy(), eff)
        assert np.array_equal(result.cpu().numpy(), ref), r
        assert int(clk_d.item()) == oracle.result_clock(version)
        for p in range(P):
            assert np.array_equal(slots[p].cpu().numpy(), ref_slots[p]), (r, p)
    plan.close()


def test_partial_allreduce_full_sampled():
    """The benchmark's partial allreduce shape (256 ranks x 4M, 70% arrival, no staleness bound) for a
    few repetitions, checked at sampled indices against the last-arrival sum."""
    E, R = _capi(), _runner()
    prob = W.partial_allreduce(reps=4)
    P, m = prob.P, prob.m
    announce("allreduce 4b full-size sampled", P, m)
    fresh = [torch.empty(m, dtype=torch.float64, device="cuda") for _ in range(P)]
    slots = [torch.empty(m, dtype=torch.float64, device="cuda") for _ in range(P)]
    result = torch.empty(m, dtype=torch.float64, device="cuda")
    d_fresh, d_slots = R.ptr_array(fresh), R.ptr_array(slots)
    d_mask = torch.from_numpy(prob.mask).cuda()
    plan = R.Plan(P, None, None, prob.S)
    version = np.full(P, -1, dtype=np.int32)
    rng = np.random.default_rng(4)
    idx = np.sort(rng.choice(m, 4096, replace=False))
    idx[0], idx[-1] = 0, m - 1
    last = np.zeros(P, dtype=np.int64)
    for r in range(prob.reps):
        for p in range(P):
            fresh[p].copy_(torch.from_numpy(prob.fresh(p, r)))
        E.ecc_allreduce_partial(plan.handle, m, d_fresh, d_slots, result, d_mask[r].data_ptr())
        eff, _, _ = oracle.select(prob.S, r, prob.mask[r], version)
        last[eff == 1] = r
        torch.cuda.synchronize()
        got = result.cpu().numpy()[idx]
        # oracle: slots hold each rank's last arrival; rank-ordered sum
        cols = [prob.fresh_at(p, int(last[p]), idx) for p in range(P)]
        ref = oracle.allreduce(np.zeros(P, dtype=np.uint8), [np.zeros(idx.size)] * P,
                               [c.copy() for c in cols])
        assert np.array_equal(got, ref), r
    plan.close()


# ----------------------------------------------------------------------------
# iterations
# ----------------------------------------------------------------------------

def _floor(prob, x):
    if prob.kind == "jacobi":
        A = prob.A
        absAx = np.zeros(prob.n)
        rows = np.repeat(np.arange(prob.n), np.diff(A.row_ptr))
        np.add.at(absAx, rows, np.abs(A.val) * np.abs(x[A.col]))
        return float(np.sqrt(np.sum((np.abs(prob.b) + absAx) ** 2)))
    Wm = prob.A
    rows = np.repeat(np.arange(prob.n), np.diff(Wm.row_ptr))
    wx = np.zeros(prob.n)
    np.add.at(wx, rows, np.abs(Wm.val) * np.abs(x[Wm.col]))
    return float(np.sum(prob.alpha * wx + prob.beta + np.abs(x)))


def _iterative(prob, range_bytes=0, tile_rows=0, schedule=0, compact=0):
    """The problem resident on the GPU; range_bytes / tile_rows / schedule /
    compact are the matrix set-up options (0: the library's choice)."""
    return _runner().Iterative(prob.n, prob.A.row_ptr, prob.A.col, prob.A.val, prob.counts,
                               prob.S, prob.mask, prob.kind, b=prob.b, alpha=prob.alpha,
                               beta=prob.beta, x0=prob.x0, range_bytes=range_bytes,
                               tile_rows=tile_rows, schedule=schedule, compact=compact)


def _solve_and_compare(prob, bitwise, threads=8, layout=None, range_bytes=0, tile_rows=0,
                       tiling=None, schedule=0, expect_schedule=None, solves=1, compact=0,
                       form=None):
    announce("solve", prob.name, prob.n, prob.A.nnz, prob.P, prob.T)
    run = _iterative(prob, range_bytes, tile_rows, schedule, compact)
    if form is not None:  # the form of the copy the set-up must choose
        assert _capi().ecc_matrix_form(run.mat)[0] == form
    if tiling is not None:  # (plane rows, tile rows) the set-up must choose
        assert _capi().ecc_matrix_tiling(run.mat) == tiling
    if expect_schedule is not None:
        assert _capi().ecc_matrix_schedule(run.mat) == expect_schedule
    for _ in range(solves - 1):  # earlier solves of the same handle change nothing
        run.solve(tol=prob.tol)
    if layout is not None:  # the layout by name: "SHORT", "STREAM" or "SORTED"
        E = _capi()
        assert E.ecc_matrix_layout(run.mat)[0] == getattr(E, "ECC_LAYOUT_" + layout)
    iters = run.solve(tol=prob.tol, histories=True)
    torch.cuda.synchronize()
    x = run.d_x.cpu().numpy()
    rho = run.d_rho.cpu().numpy()[:iters]
    eff = run.eff_hist.cpu().numpy()[:iters]
    age = run.age_hist.cpu().numpy()[:iters]
    clock, forced, version, _ = run.plan.stats()
    run.close()
    ref = oracle.run_iterative(prob, threads=threads)
    n_cmp = min(iters, ref["iters"])
    if iters != ref["iters"]:
        # a different stopping iteration only if rho sits at the tolerance
        t = n_cmp - 1
        assert abs(ref["rho"][t] - prob.tol) <= 1e-12 * prob.tol * 10, (iters, ref["iters"])
    assert clock == iters
    assert np.array_equal(eff[:n_cmp], ref["eff"][:n_cmp])
    assert np.array_equal(age[:n_cmp], ref["age"][:n_cmp])
    assert forced == int(ref["forced"][:iters].sum())
    if iters == ref["iters"]:
        assert np.array_equal(version, ref["version"])
        err = assert_iterates_close(x, ref["x"])
        if bitwise:
            assert np.array_equal(x, ref["x"]), "max |dx| = %.3e" % err
    assert_rho_close(rho[:n_cmp], ref["rho"][:n_cmp], _floor(prob, ref["x"]))
    return iters


def test_solve_jacobi_1d():
    _solve_and_compare(W.jacobi_1d(), bitwise=True)


@pytest.mark.parametrize("N,T", [(33, 40), (64, 80)])
def test_solve_jacobi_2d_small(N, T):
    _solve_and_compare(W.jacobi_2d(N=N, T=T), bitwise=True)


def test_solve_jacobi_2d_full():
    _solve_and_compare(W.jacobi_2d(), bitwise=True)


@pytest.mark.parametrize("N,P", [(12, 512), (24, 512), (40, 64)])
def test_solve_jacobi_3d_small(N, P):
    _solve_and_compare(W.jacobi_3d(N=N, T=60, P=P), bitwise=True)


@pytest.mark.parametrize("scale", [8, 12, 15, 17])
def test_solve_pagerank_rmat_small(scale):
    """Scale 15 has rows summed by a whole workgroup; scale 17 also has rows
    longer than one work item, split into pieces and recombined."""
    _solve_and_compare(W.pagerank_rmat(scale=scale, T=60), bitwise=False, layout="SORTED")


def _plan_continuation(prob, split, **kw):
    """One ecc_solve of T iterations against two calls of split and T - split
    iterations without a reset in between (the second continues the plan's
    clock from the iterate and assembled vector the first left).  Returns
    both runs' (x, x_hat, rho, eff, age, clock)."""
    E = _capi()
    run = _iterative(prob, **kw)
    P, T = prob.P, prob.T
    out = []
    for parts in ((0, T), (0, split, T)):
        run.plan.reset()
        run.load_x0()
        rho = torch.zeros(T, dtype=torch.float64, device="cuda")
        eff = torch.zeros((T, P), dtype=torch.uint8, device="cuda")
        age = torch.zeros((T, P), dtype=torch.int32, device="cuda")
        for t0, t1 in zip(parts[:-1], parts[1:]):
            # the iterate of the first call is the second call's x^0
            it = E.ecc_solve(run.plan.handle, run.mat, run.d_b, run.alpha, run.beta, run.d_x,
                             run.d_x_tmp, run.d_x_hat, run.d_mask[t0:].data_ptr(), t1 - t0, 0.0,
                             rho[t0:].data_ptr(), eff[t0:].data_ptr(), age[t0:].data_ptr())
            assert it == t1 - t0
        torch.cuda.synchronize()
        out.append((run.d_x.cpu().numpy(), run.d_x_hat.cpu().numpy(), rho.cpu().numpy(),
                    eff.cpu().numpy(), age.cpu().numpy(), run.plan.stats()[0]))
    schedule = E.ecc_matrix_schedule(run.mat)
    run.close()
    return out, schedule


@pytest.mark.parametrize("which", ["jacobi1d", "jacobi2d", "jacobi3d_unfused", "pagerank"])
def test_solve_continues_plan(which):
    """ecc_solve continues a plan: two calls (the second starting where the
    first stopped, with blocks that do not arrive at its first iteration
    keeping the assembled values the first call left) equal one call of both
    lengths bit for bit -- iterate, assembled vector, norms, histories and
    clock -- in the single-launch loop, the fused loop, the loop with
    separate assembly launches and the column-value range loop."""
    E = _capi()
    if which == "jacobi1d":
        prob, kw, sched = W.jacobi_1d(), {}, E.ECC_SCHEDULE_SINGLE
        rng = np.random.default_rng(3)
        mask = (rng.random(prob.mask.shape) < 0.5).astype(np.uint8)
        mask[0] = 1
        prob = dataclasses.replace(prob, S=2, mask=mask)
    elif which == "jacobi2d":
        prob, kw, sched = W.jacobi_2d(N=64, T=30), {}, None
    elif which == "jacobi3d_unfused":
        prob, kw, sched = W.jacobi_3d(N=16, T=24, P=2048), {}, None
    else:
        prob, kw, sched = W.pagerank_rmat(scale=12, T=30), {"range_bytes": 4096}, None
    announce("solve continuation", which)
    # a block does not arrive at the continuation's first iteration
    split = next(t for t in range(prob.T // 3, prob.T) if not prob.mask[t].all())
    (a, b), schedule = _plan_continuation(prob, split, **kw)
    if sched is not None:
        assert schedule == sched
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def test_solve_many_ranks_unfused():
    """More ranks than a workgroup stages in LDS: separate assembly launches."""
    _solve_and_compare(W.jacobi_3d(N=24, T=30, P=2048), bitwise=True)


def _arrow_problem(n=40000, T=40, P=7, S=2):
    """Jacobi on an arrow matrix: row 0 and column 0 are dense, so row 0 is
    split into pieces; a few other rows are long enough for one workgroup."""
    rng = np.random.default_rng(77)
    rows = []
    for i in range(n):
        if i == 0:
            cols = np.arange(n)
        elif i % 9973 == 0:
            cols = np.unique(np.concatenate([[0, i], rng.choice(n, 5000, replace=False)]))
        else:
            cols = np.unique(np.array([0, i, max(i - 1, 0), min(i + 1, n - 1)]))
        vals = np.where(cols == i, 0.0, -rng.uniform(0.1, 1.0, cols.size))
        vals[cols == i] = 2.0 * np.abs(vals).sum() + 1.0
        rows.append((cols, vals))
    rp = np.zeros(n + 1, dtype=np.int32)
    rp[1:] = np.cumsum([c.size for c, _ in rows])
    A = W.CSR(n, n, rp, np.concatenate([c for c, _ in rows]).astype(np.int32),
              np.concatenate([v for _, v in rows]))
    counts = W.dirichlet_partition(n, P, 5)
    mask = (rng.random((T, P)) < 0.6).astype(np.uint8)
    mask[0] = 1
    return W.Iterative("arrow-jacobi", "jacobi", A, counts, W.exclusive_scan(counts), S, mask,
                       T, np.zeros(n), b=rng.standard_normal(n), norm=2)


def _banded_problem(kind, n, lmin, lmax, P=13, T=40, S=3, seed=5):
    """Rows of lmin..lmax entries (at most 64: a regular matrix) at random
    columns within a band of +-1500 around the diagonal, so that rows read
    neighbouring ranks: the LDS-staged stream layout for rows of more than
    eight entries, the short-row layout otherwise."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(lmin, lmax + 1, n)
    cols, vals = [], []
    for i in range(n):
        lo, hi = max(0, i - 1500), min(n, i + 1501)
        c = np.sort(rng.choice(np.arange(lo, hi), int(lens[i]), replace=False))
        if kind == "jacobi" and i not in c:
            c[rng.integers(0, c.size)] = i
            c = np.sort(c)
        v = rng.uniform(0.05, 1.0, c.size) / c.size
        if kind == "jacobi":
            v = -v
            v[c == i] = 2.0 * np.abs(v).sum() + 1.0
        cols.append(c)
        vals.append(v)
    rp = np.zeros(n + 1, dtype=np.int32)
    rp[1:] = np.cumsum([c.size for c in cols])
    A = W.CSR(n, n, rp, np.concatenate(cols).astype(np.int32), np.concatenate(vals))
    counts = W.dirichlet_partition(n, P, seed)
    mask = (rng.random((T, P)) < 0.7).astype(np.uint8)
    mask[0] = 1
    if kind == "jacobi":
        return W.Iterative("banded-jacobi", "jacobi", A, counts, W.exclusive_scan(counts), S,
                           mask, T, np.zeros(n), b=rng.standard_normal(n), norm=2)
    return W.Iterative("banded-power", "power", A, counts, W.exclusive_scan(counts), S, mask, T,
                       np.full(n, 1.0 / n), alpha=0.85, beta=0.15 / n, norm=1)


@pytest.mark.parametrize("kind", ["jacobi", "power"])
@pytest.mark.parametrize("lmin,lmax", [(9, 16), (20, 60)])
def test_solve_stream_layout(kind, lmin, lmax):
    """Regular rows longer than eight entries: rows of up to 16 entries are
    summed by one lane in CSR order (bitwise), longer ones by several lanes."""
    _solve_and_compare(_banded_problem(kind, 30000, lmin, lmax), bitwise=(lmax <= 16))


@pytest.mark.parametrize("kind,lmin,lmax", [
    ("jacobi", 1, 2), ("power", 0, 3), ("jacobi", 2, 4), ("power", 3, 6), ("jacobi", 5, 7),
    ("jacobi", 8, 8), ("power", 1, 8)])
def test_solve_short_layout(kind, lmin, lmax):
    """Rows of at most eight entries: the short-row layout, one lane per row
    summed in CSR order (bitwise).  The kernel holds 3, 4, 5, 7 or 8 entries
    per row after the longest row; rows may be shorter than that, or empty
    (power step)."""
    _solve_and_compare(_banded_problem(kind, 30000, lmin, lmax), bitwise=True)


@pytest.mark.parametrize("kind", ["jacobi", "power"])
@pytest.mark.parametrize("n,counts", [(1, [1]), (2, [0, 2, 0]), (255, [100, 0, 155]),
                                      (257, [257]), (513, [0, 256, 1, 256])])
def test_solve_tiny_and_ragged(kind, n, counts):
    """Matrices of one row, a few rows, and just under / over a 256-row item,
    with single-rank plans and ranks that own no rows: one-item grids, ragged
    last items and empty ranks in the short-row layout."""
    rng = np.random.default_rng(n + 7 * len(counts))
    rows = []
    for i in range(n):
        c = np.unique(np.clip(np.array([i - 1, i, i + 1, i + 37]), 0, n - 1))
        v = -rng.uniform(0.1, 1.0, c.size) / c.size
        if kind == "jacobi":
            v[c == i] = 2.0 * np.abs(v).sum() + 1.0
        rows.append((c, v))
    rp = np.zeros(n + 1, dtype=np.int32)
    rp[1:] = np.cumsum([c.size for c, _ in rows])
    A = W.CSR(n, n, rp, np.concatenate([c for c, _ in rows]).astype(np.int32),
              np.abs(np.concatenate([v for _, v in rows])) if kind == "power"
              else np.concatenate([v for _, v in rows]))
    counts = np.array(counts, dtype=np.int64)
    P, T = counts.size, 12
    mask = (rng.random((T, P)) < 0.6).astype(np.uint8)
    mask[0] = 1
    if kind == "jacobi":
        prob = W.Iterative("tiny-jacobi", "jacobi", A, counts, W.exclusive_scan(counts), 2, mask,
                           T, np.zeros(n), b=rng.standard_normal(n), norm=2)
    else:
        prob = W.Iterative("tiny-power", "power", A, counts, W.exclusive_scan(counts), 2, mask, T,
                           np.full(n, 1.0 / n), alpha=0.85, beta=0.15 / n, norm=1)
    _solve_and_compare(prob, bitwise=True)


@pytest.mark.parametrize("seed", range(20))
def test_solve_random_shapes(seed):
    """Random sizes (1-5,000 rows), row lengths (0-12 entries, so both the
    short-row and the stream layouts), rank counts (1-12, some empty),
    staleness bounds and arrival rates, Jacobi or PageRank; compared with the
    oracle at every iteration."""
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 5001))
    kind = "jacobi" if seed % 2 == 0 else "power"
    lmax = int(rng.integers(1, 13))
    band = int(rng.integers(1, max(2, n)))
    rows = []
    for i in range(n):
        ln = int(rng.integers(0 if kind == "power" else 1, lmax + 1))
        lo, hi = max(0, i - band), min(n, i + band + 1)
        c = np.sort(rng.choice(np.arange(lo, hi), min(ln, hi - lo), replace=False))
        if kind == "jacobi" and i not in c:
            c = np.sort(np.concatenate([c[1:], [i]])) if c.size else np.array([i])
        v = rng.uniform(0.05, 1.0, c.size) / max(c.size, 1)
        if kind == "jacobi":
            v = -v
            v[c == i] = 2.0 * np.abs(v).sum() + 1.0
        rows.append((c.astype(np.int64), v))
    rp = np.zeros(n + 1, dtype=np.int32)
    rp[1:] = np.cumsum([c.size for c, _ in rows])
    A = W.CSR(n, n, rp, np.concatenate([c for c, _ in rows]).astype(np.int32),
              np.concatenate([v for _, v in rows]))
    P = int(rng.integers(1, 13))
    cuts = np.sort(rng.integers(0, n + 1, P - 1))
    counts = np.diff(np.concatenate([[0], cuts, [n]])).astype(np.int64)
    T, S = 15, int(rng.integers(0, 4))
    mask = (rng.random((T, P)) < rng.uniform(0.3, 1.0)).astype(np.uint8)
    mask[0] = 1
    if kind == "jacobi":
        prob = W.Iterative("random-jacobi", "jacobi", A, counts, W.exclusive_scan(counts), S,
                           mask, T, np.zeros(n), b=rng.standard_normal(n), norm=2)
    else:
        prob = W.Iterative("random-power", "power", A, counts, W.exclusive_scan(counts), S,
                           mask, T, np.full(n, 1.0 / n), alpha=0.85, beta=0.15 / n, norm=1)
    _solve_and_compare(prob, bitwise=lmax <= 16)


def test_solve_arrow_split_rows():
    _solve_and_compare(_arrow_problem(), bitwise=False, layout="SORTED")


def _powerlaw_problem(kind, n, counts, seed, T=25, S=2, column_values=False):
    """Rows whose lengths follow a heavy tail (most hold a few entries, a few
    hold thousands, one is split into pieces) at random columns: very uneven
    rows, swept in the sorted layout.  PageRank rows may be empty.  With
    column_values every entry of column j holds the same value."""
    rng = np.random.default_rng(seed)
    col_value = rng.uniform(0.05, 1.0, n) / 64.0
    lens = np.minimum((rng.pareto(1.1, n) * 2.0).astype(np.int64), n - 1)
    lens[rng.integers(0, n)] = n - 1                       # longer than one vector item
    lens[rng.choice(n, 6, replace=False)] = rng.integers(2049, 9000, 6)  # whole-workgroup rows
    rows = []
    for i in range(n):
        c = np.sort(rng.choice(n, int(lens[i]), replace=False))
        if kind == "jacobi" and i not in c:
            c = np.sort(np.concatenate([c[1:], [i]])) if c.size else np.array([i])
        v = rng.uniform(0.05, 1.0, c.size) / max(c.size, 1)
        if column_values:
            v = col_value[c]
        if kind == "jacobi":
            v = -v
            v[c == i] = 2.0 * np.abs(v).sum() + 1.0
        rows.append((c.astype(np.int64), v))
    rp = np.zeros(n + 1, dtype=np.int32)
    rp[1:] = np.cumsum([c.size for c, _ in rows])
    A = W.CSR(n, n, rp, np.concatenate([c for c, _ in rows]).astype(np.int32),
              np.concatenate([v for _, v in rows]))
    counts = (W.dirichlet_partition(n, counts, seed) if isinstance(counts, int)
              else np.array(counts, dtype=np.int64))
    P = counts.size
    mask = (rng.random((T, P)) < 0.7).astype(np.uint8)
    mask[0] = 1
    if kind == "jacobi":
        return W.Iterative("powerlaw-jacobi", "jacobi", A, counts, W.exclusive_scan(counts), S,
                           mask, T, np.zeros(n), b=rng.standard_normal(n), norm=2)
    return W.Iterative("powerlaw-power", "power", A, counts, W.exclusive_scan(counts), S, mask, T,
                       np.full(n, 1.0 / n), alpha=0.85, beta=0.15 / n, norm=1)


@pytest.mark.parametrize("kind", ["jacobi", "power"])
@pytest.mark.parametrize("counts", [[20000], [0, 3000, 0, 9000, 1000, 7000], 9])
@pytest.mark.parametrize("range_bytes", [16384, 1])
def test_solve_range_layout(kind, counts, range_bytes):
    """Very uneven rows cut by column range into sub-rows (10 ranges of 16 KB
    of the vector, or the most, 16): each sub-row summed on its own, a row's
    sums added in range order by a second kernel, split sub-rows recombined
    first; Jacobi takes the diagonal kept at set-up."""
    prob = _powerlaw_problem(kind, 20000, counts, seed=31 + len(str(counts)))
    _solve_and_compare(prob, bitwise=False, layout="RANGES", range_bytes=range_bytes)


@pytest.mark.parametrize("scale", [12, 15, 17])
def test_solve_pagerank_rmat_ranges(scale):
    """R-MAT PageRank in the range layout (scale 15 has sub-rows summed by a
    whole workgroup, scale 17 split sub-rows)."""
    _solve_and_compare(W.pagerank_rmat(scale=scale, T=60), bitwise=False, layout="RANGES",
                       range_bytes=4096)


@pytest.mark.parametrize("seed", range(8))
def test_irregular_random(seed):
    """R-MAT PageRank of random scale (8-16), rank count (1-128), staleness
    bound (0-4), arrival rate (0.3-1) and range size (unsplit or 2 KB-64 KB
    ranges): the sorted or range layout in the column-value form (with its
    copy of the most gathered columns) against the oracle at every
    iteration, and bit for bit against the general form of the same layout."""
    import dataclasses
    E = _capi()
    rng = np.random.default_rng(5000 + seed)
    scale = int(rng.integers(8, 17))
    base = W.pagerank_rmat(scale=scale, T=20,
                           P=max(1, min(int(rng.integers(1, 129)), (1 << scale) // 4)))
    mask = (rng.random((base.T, base.P)) < rng.uniform(0.3, 1.0)).astype(np.uint8)
    mask[0] = 1
    prob = dataclasses.replace(base, S=int(rng.integers(0, 5)), mask=mask, tol=0.0)
    rb = int(rng.choice([0, 2048, 4096, 16384, 65536]))
    _solve_and_compare(prob, bitwise=False, range_bytes=rb)
    it1, x1, xh1, _, f1 = _solve_x_rho(prob, range_bytes=rb)
    it2, x2, xh2, _, f2 = _solve_x_rho(prob, range_bytes=rb, compact=E.ECC_COMPACT_NONE)
    assert (f1, f2) == (E.ECC_FORM_COLUMN_VALUES, E.ECC_FORM_GENERAL)
    assert it1 == it2 and np.array_equal(x1, x2) and np.array_equal(xh1, xh2)


def test_solve_arrow_ranges():
    _solve_and_compare(_arrow_problem(), bitwise=False, layout="RANGES", range_bytes=8192)


def _solve_x_rho(prob, range_bytes=0, compact=0):
    run = _iterative(prob, range_bytes, compact=compact)
    iters = run.solve(tol=prob.tol, histories=True)
    torch.cuda.synchronize()
    out = (iters, run.d_x.cpu().numpy(), run.d_x_hat.cpu().numpy(),
           run.d_rho.cpu().numpy()[:iters], _capi().ecc_matrix_form(run.mat)[0])
    run.close()
    return out


@pytest.mark.parametrize("which", ["rmat12", "rmat15", "rmat17", "powerlaw"])
@pytest.mark.parametrize("range_bytes", [0, 4096])
def test_column_values_match_general_form(which, range_bytes):
    """A matrix whose every column holds one value (the PageRank matrix, and
    heavy-tailed rows with whole-workgroup rows and split rows) is swept from
    the column values and the scaled views: iterate and assembled vector equal
    the general form's bit for bit at every iteration count, in the sorted
    and the range layout, and match the oracle (checked by
    _solve_and_compare).  The residuals agree to rounding: the column-value
    kernel holds no values in LDS, so more of its workgroups fit on a CU and
    the sweep's per-workgroup partial sums group the rows differently."""
    prob = (W.pagerank_rmat(scale=int(which[4:]), T=40) if which.startswith("rmat")
            else _powerlaw_problem("power", 20000, 9, seed=77, column_values=True))
    layout = "RANGES" if range_bytes else "SORTED"
    E = _capi()
    _solve_and_compare(prob, bitwise=False, layout=layout, range_bytes=range_bytes,
                       form=E.ECC_FORM_COLUMN_VALUES)
    a = _solve_x_rho(prob, range_bytes, compact=E.ECC_COMPACT_AUTO)
    g = _solve_x_rho(prob, range_bytes, compact=E.ECC_COMPACT_NONE)
    assert a[4] == E.ECC_FORM_COLUMN_VALUES and g[4] == E.ECC_FORM_GENERAL
    assert a[0] == g[0]
    assert np.array_equal(a[1], g[1]) and np.array_equal(a[2], g[2])
    assert np.allclose(a[3], g[3], rtol=1e-12, atol=0.0)


def test_column_values_choice():
    """Only power matrices in the sorted or range layout whose columns each
    hold one value, bit for bit, take the column-value form: one entry off by
    one unit in the last place, a general heavy-tailed matrix, a Jacobi
    matrix, a short-row matrix and the caller's ECC_COMPACT_NONE keep the
    general form."""
    E = _capi()
    announce("column values choice")
    prob = W.pagerank_rmat(scale=10, T=2)

    def one(p, **kw):
        run = _iterative(p, **kw)
        v = int(E.ecc_matrix_form(run.mat)[0] == E.ECC_FORM_COLUMN_VALUES)
        run.close()
        return v

    assert one(prob) == 1
    assert one(prob, range_bytes=4096) == 1
    assert one(prob, compact=E.ECC_COMPACT_NONE) == 0
    val = prob.A.val.copy()
    k = int(np.argmax(np.bincount(prob.A.col, minlength=prob.n)[prob.A.col]))  # busiest column
    val[k] = np.nextafter(val[k], 1.0)
    bent = dataclasses.replace(prob, A=W.CSR(prob.n, prob.n, prob.A.row_ptr, prob.A.col, val))
    assert one(bent) == 0
    assert one(_powerlaw_problem("power", 12000, 3, seed=5, T=2)) == 0
    assert one(_powerlaw_problem("power", 12000, 3, seed=5, T=2, column_values=True)) == 1
    assert one(_powerlaw_problem("jacobi", 12000, 3, seed=5, T=2)) == 0
    assert one(_banded_problem("power", 3000, 6, 6, T=2)) == 0
    with pytest.raises(E.EccError) as ei:
        _iterative(prob, compact=7)
    assert ei.value.status == E.ECC_ERR_ARG


@pytest.mark.parametrize("which", ["sorted", "ranges", "ranges_general", "powerlaw_sorted",
                                   "powerlaw_ranges"])
def test_reordered_layouts_every_iterate(which):
    """Layouts that add a row's entries in another order than CSR (the
    sorted copy with rows on several lanes, the range layout's per-range
    sub-row sums): through the separate calls, the assembled vector and the
    new iterate of every iteration against the oracle's, normwise within
    1e-12, and every norm within its bound."""
    E = _capi()
    if which == "sorted":
        prob, kw = W.pagerank_rmat(scale=13, T=30), {}
    elif which == "ranges":
        prob, kw = W.pagerank_rmat(scale=13, T=30), {"range_bytes": 4096}
    elif which == "ranges_general":
        prob, kw = W.pagerank_rmat(scale=13, T=30), {"range_bytes": 4096,
                                                     "compact": E.ECC_COMPACT_NONE}
    elif which == "powerlaw_sorted":
        prob, kw = _powerlaw_problem("jacobi", 20000, 9, seed=40, T=20), {}
    else:
        prob, kw = _powerlaw_problem("jacobi", 20000, 9, seed=40, T=20), {"range_bytes": 8192}
    announce("every iterate", which)
    ref = oracle.run_iterative(prob, threads=8, keep_x=tuple(range(prob.T)))
    assert ref["iters"] == prob.T
    run = _iterative(prob, **kw)
    layout = E.ecc_matrix_layout(run.mat)[0]
    assert layout == (E.ECC_LAYOUT_SORTED if "sorted" in which else E.ECC_LAYOUT_RANGES)
    run.plan.reset()
    a = torch.from_numpy(prob.x0.copy()).cuda()
    b = torch.empty_like(a)
    rhos = []
    for t in range(prob.T):
        rhos.append(run.step(t, a, b))
        assert_iterates_close(run.d_x_hat.cpu().numpy(), ref["kept"][t][1])
        expect = ref["kept"][t + 1][0] if t + 1 < prob.T else ref["x"]
        assert_iterates_close(b.cpu().numpy(), expect)
        a, b = b, a
    assert_rho_close(np.array(rhos), ref["rho"], _floor(prob, ref["x"]))
    run.close()


def _form(prob, **kw):
    run = _iterative(prob, **kw)
    f = _capi().ecc_matrix_form(run.mat)
    run.close()
    return f


def test_diagonal_form_choice():
    """Short-row matrices whose sorted rows lie on at most R offsets col - row
    (R: the row class) take the diagonal form, with those offsets ascending;
    random columns within a band, a row out of column order, a
    caller's ECC_COMPACT_NONE and the longer rows of other layouts do not."""
    E = _capi()
    announce("diagonal form choice")
    D, G = E.ECC_FORM_DIAGONALS, E.ECC_FORM_GENERAL
    assert _form(W.jacobi_1d()) == (D, [-1, 0, 1])
    assert _form(W.jacobi_2d(N=33, T=2)) == (D, [-33, -1, 0, 1, 33])
    assert _form(W.jacobi_3d(N=12, T=2, P=8)) == (D, [-144, -12, -1, 0, 1, 12, 144])
    assert _form(W.jacobi_2d(N=33, T=2), compact=E.ECC_COMPACT_NONE) == (G, [])
    assert _form(_banded_problem("jacobi", 3000, 4, 4, T=2))[0] == G
    assert _form(_banded_problem("jacobi", 3000, 9, 16, T=2))[0] == G   # stream layout
    # one row with its entries out of column order
    prob = W.jacobi_2d(N=33, T=2)
    rp, col, val = prob.A.row_ptr, prob.A.col.copy(), prob.A.val.copy()
    k0 = int(rp[40])
    col[k0], col[k0 + 1] = col[k0 + 1], col[k0]
    val[k0], val[k0 + 1] = val[k0 + 1], val[k0]
    bent = dataclasses.replace(prob, A=W.CSR(prob.n, prob.n, rp, col, val))
    assert _form(bent)[0] == G


def _offset_subset_problem(kind, n, offsets, P, seed, T=30, S=2):
    """Rows holding a random subset of a fixed set of offsets col - row (the
    diagonal always, for Jacobi; possibly none at all, for the power step),
    in increasing column order: the diagonal form with gaps in every row's
    mask."""
    rng = np.random.default_rng(seed)
    rows_c, rows_v = [], []
    for i in range(n):
        keep = rng.random(len(offsets)) < 0.6
        c = np.array([i + d for d, k in zip(offsets, keep) if k and 0 <= i + d < n], dtype=np.int64)
        if kind == "jacobi" and i not in c:
            c = np.sort(np.append(c, i))
        v = -rng.uniform(0.05, 1.0, c.size)
        if kind == "jacobi":
            v[c == i] = 2.0 * np.abs(v).sum() + 1.0
        else:
            v = np.abs(v) / len(offsets)
        rows_c.append(c)
        rows_v.append(v)
    rp = np.zeros(n + 1, dtype=np.int32)
    rp[1:] = np.cumsum([c.size for c in rows_c])
    A = W.CSR(n, n, rp, np.concatenate(rows_c).astype(np.int32), np.concatenate(rows_v))
    counts = W.dirichlet_partition(n, P, seed)
    mask = (rng.random((T, P)) < 0.7).astype(np.uint8)
    mask[0] = 1
    if kind == "jacobi":
        return W.Iterative("offsets-jacobi", "jacobi", A, counts, W.exclusive_scan(counts), S,
                           mask, T, np.zeros(n), b=rng.standard_normal(n), norm=2)
    return W.Iterative("offsets-power", "power", A, counts, W.exclusive_scan(counts), S, mask, T,
                       rng.random(n), alpha=0.85, beta=0.15 / n, norm=1)


@pytest.mark.parametrize("kind,offsets,n,P", [
    ("jacobi", [-700, -3, -1, 0, 2, 650, 1800], 20000, 9),
    ("power", [-1500, -40, -1, 0, 1, 40, 1500], 20000, 5),
    ("power", [-5, 0, 7], 3001, 3),        # the single-launch solve
    ("jacobi", [-64, -1, 0, 1, 64], 700, 2),
])
def test_diagonal_form_with_gaps(kind, offsets, n, P):
    """Every row a random subset of the offsets (the power step's rows may be
    empty): the diagonal form, bitwise against the oracle and the general
    form, through the loop and the separate calls."""
    E = _capi()
    prob = _offset_subset_problem(kind, n, offsets, P, seed=n + P)
    announce("diagonal form with gaps", kind, offsets, n, P)
    assert _form(prob) == (E.ECC_FORM_DIAGONALS, sorted(offsets))
    _solve_and_compare(prob, bitwise=True, form=E.ECC_FORM_DIAGONALS)
    outs = []
    for compact in (E.ECC_COMPACT_AUTO, E.ECC_COMPACT_NONE):
        run = _iterative(prob, compact=compact)
        run.solve(histories=True)
        torch.cuda.synchronize()
        outs.append((run.d_x.cpu().numpy(), run.d_x_hat.cpu().numpy(),
                     run.d_rho.cpu().numpy()[:prob.T]))
        run.close()
    for u, v in zip(*outs):
        assert np.array_equal(u, v)
    _step_api_matches_solve((prob,))


@pytest.mark.parametrize("which", ["jacobi1d", "jacobi2d", "jacobi3d", "jacobi3d_tiled",
                                   "power_stencil"])
def test_diagonal_form_matches_general_form(which):
    """The diagonal form (values by diagonal, one mask byte per row) gives
    the iterate, assembled vector and every residual of the general form bit
    for bit, and the oracle's (checked by _solve_and_compare): the
    single-launch loop, the fused loop (static and queue schedules), plane
    tiles, and the power step on a stencil."""
    E = _capi()
    kw = {}
    if which == "jacobi1d":
        prob = W.jacobi_1d()
    elif which == "jacobi2d":
        prob = W.jacobi_2d(N=64, T=30)
    elif which == "jacobi3d":
        prob = W.jacobi_3d(N=24, T=20, P=512)
        kw = {"schedule": E.ECC_SCHEDULE_QUEUE}
    elif which == "jacobi3d_tiled":
        prob = W.jacobi_3d(N=40, T=12, P=64)
        kw = {"tile_rows": 256}
    else:
        base = W.jacobi_2d(N=48, T=20)
        A = base.A
        val = np.abs(A.val) / 8.0
        rng = np.random.default_rng(5)
        x0 = rng.random(base.n)
        prob = W.Iterative("power-stencil", "power", W.CSR(base.n, base.n, A.row_ptr, A.col, val),
                           base.counts, base.displs, base.S, base.mask, base.T, x0,
                           alpha=0.85, beta=0.15 / base.n, norm=1)
    _solve_and_compare(prob, bitwise=True, form=E.ECC_FORM_DIAGONALS, **kw)
    run_a = _iterative(prob, compact=E.ECC_COMPACT_AUTO, **kw)
    run_g = _iterative(prob, compact=E.ECC_COMPACT_NONE, **kw)
    outs = []
    for run in (run_a, run_g):
        iters = run.solve(tol=prob.tol, histories=True)
        torch.cuda.synchronize()
        outs.append((iters, run.d_x.cpu().numpy(), run.d_x_hat.cpu().numpy(),
                     run.d_rho.cpu().numpy()[:iters]))
        run.close()
    assert outs[0][0] == outs[1][0]
    for u, v in zip(outs[0][1:], outs[1][1:]):
        assert np.array_equal(u, v)


@pytest.mark.parametrize("kind", ["jacobi", "power"])
@pytest.mark.parametrize("counts", [[20000], [0, 3000, 0, 9000, 1000, 7000], 9])
def test_solve_sorted_layout(kind, counts):
    """Very uneven rows: each rank's rows are swept in order of decreasing
    length from a copy, and every result goes back to its own row (Jacobi
    finds each row's diagonal by the row's index).  One rank, ranks that own
    no rows, and nine uneven ranks."""
    prob = _powerlaw_problem(kind, 20000, counts, seed=31 + len(str(counts)))
    _solve_and_compare(prob, bitwise=False, layout="SORTED")


def test_solve_pagerank_rmat_tolerance_stop():
    prob = W.pagerank_rmat(scale=10, T=200)
    iters = _solve_and_compare(prob, bitwise=False)
    assert iters < 200


def test_step_api_matches_solve():
    """assemble -> iterate -> residual through the separate calls reproduce the
    loop-control call bit for bit (fused single-launch loop, the loop with a
    second pass per iteration, and split rows)."""
    _step_api_matches_solve((W.jacobi_2d(N=40, T=25), W.pagerank_rmat(scale=11, T=25),
                             _arrow_problem(T=12)))


@pytest.mark.parametrize("N,P,tile", [(24, 7, 256), (24, 1, 512), (30, 5, 768), (17, 33, 256)])
def test_solve_jacobi_3d_plane_tiles(N, P, tile):
    """3-D stencils swept in plane tiles (items ordered tile by tile, plane by
    plane; the entries copied in that order): iterates bitwise equal to the
    oracle.  A plane of N^2 rows cut into tiles of `tile` rows, with a ragged
    last tile (24^2 = 576 = 2 x 256 + 64; 30^2 = 900 = 768 + 132; 17^2 = 289),
    ranks cut across tiles
    and planes, and one rank."""
    prob = W.jacobi_3d(N=N, T=30, P=P)
    run = _iterative(prob, tile_rows=tile)
    E = _capi()
    assert E.ecc_matrix_tiling(run.mat) == (N * N, tile)
    run.close()
    _solve_and_compare(prob, bitwise=True, layout="SHORT", tile_rows=tile)


def test_plane_tiles_not_taken():
    """Row order where tiling does not apply: no option (the plane is small),
    a negative tile size, tiles as wide as the plane (3-D and 2-D stencils),
    and a banded matrix whose columns spread over the whole band."""
    E = _capi()
    for prob, tile in [(W.jacobi_3d(N=16, T=2, P=3), 0), (W.jacobi_3d(N=16, T=2, P=3), -1),
                       (W.jacobi_3d(N=16, T=2, P=3), 256), (W.jacobi_2d(N=64, T=2), 256),
                       (_banded_problem("jacobi", 6000, 4, 4, T=2), 256)]:
        run = _iterative(prob, tile_rows=tile)
        assert E.ecc_matrix_tiling(run.mat) == (0, 0), (prob.name, tile)
        run.close()


def test_step_api_matches_solve_plane_tiles():
    _step_api_matches_solve((W.jacobi_3d(N=20, T=15, P=6),), tile_rows=256)


def _queue_cases():
    return [("jacobi-1d", lambda: W.jacobi_1d(), 0),
            ("jacobi-2d-48", lambda: W.jacobi_2d(N=48, T=40), 0),
            ("jacobi-3d-24-tiled", lambda: W.jacobi_3d(N=24, T=30, P=7), 256),
            ("jacobi-3d-20", lambda: W.jacobi_3d(N=20, T=30, P=40), 0),
            ("banded-power-0-3", lambda: _banded_problem("power", 3000, 0, 3), 0),
            ("banded-jacobi-8", lambda: _banded_problem("jacobi", 3000, 8, 8), 0)]


@pytest.mark.parametrize("case", range(6))
def test_solve_queue_schedule(case):
    """Items claimed from the run-time queue (forced on small problems): every
    item swept exactly once, iterates bitwise equal to the oracle, the
    per-item norm partials within tolerance; three solves of one handle (the
    ticket counters start from zero at every launch)."""
    name, make, tile = _queue_cases()[case]
    E = _capi()
    _solve_and_compare(make(), bitwise=True, layout="SHORT", tile_rows=tile,
                       schedule=E.ECC_SCHEDULE_QUEUE, expect_schedule=E.ECC_SCHEDULE_QUEUE,
                       solves=3)


@pytest.mark.parametrize("seed", range(6))
def test_short_layout_random(seed):
    """3-D stencils of random size (6-47 per side; random rank counts and
    plane tiles) and 2-D ones (8-199), random staleness bounds and arrival
    rates, the static or the queue schedule: the diagonal-form short layout
    bitwise against the oracle over two solves of one handle."""
    import dataclasses
    E = _capi()
    rng = np.random.default_rng(9000 + seed)
    if seed % 3 != 0:
        N = int(rng.integers(6, 48))
        base = W.jacobi_3d(N=N, T=12, P=int(rng.integers(1, 80)))
        tile = int(rng.choice([0, 256, 512, 768, 1024]))
        tile = tile if tile < N * N else 0
    else:
        base = W.jacobi_2d(N=int(rng.integers(8, 200)), T=12)
        tile = 0
    S = int(rng.integers(0, 6))
    mask = (rng.random((base.T, base.P)) < rng.uniform(0.3, 1.0)).astype(np.uint8)
    mask[0] = 1
    sch = int(rng.choice([E.ECC_SCHEDULE_STATIC, E.ECC_SCHEDULE_QUEUE]))
    _solve_and_compare(dataclasses.replace(base, S=S, mask=mask), bitwise=True, layout="SHORT",
                       tile_rows=tile, schedule=sch, expect_schedule=sch, solves=2)


def test_step_api_matches_solve_queue():
    E = _capi()
    _step_api_matches_solve((W.jacobi_2d(N=40, T=25), W.jacobi_3d(N=20, T=15, P=6)),
                            tile_rows=256, schedule=E.ECC_SCHEDULE_QUEUE)


def test_schedule_choice():
    """A problem of at most 2,048 rows (4,096 rows of at most 3 entries) is
    solved by one launch; a larger one with few items per workgroup walks them
    statically; either can be forced."""
    E = _capi()
    small, big = W.jacobi_2d(N=40, T=2), W.jacobi_2d(N=64, T=2)
    for prob, sch, want in [(small, 0, E.ECC_SCHEDULE_SINGLE),
                            (small, E.ECC_SCHEDULE_STATIC, E.ECC_SCHEDULE_STATIC),
                            (small, E.ECC_SCHEDULE_QUEUE, E.ECC_SCHEDULE_QUEUE),
                            (small, E.ECC_SCHEDULE_SINGLE, E.ECC_SCHEDULE_SINGLE),
                            (big, 0, E.ECC_SCHEDULE_STATIC),
                            (big, E.ECC_SCHEDULE_SINGLE, E.ECC_SCHEDULE_STATIC)]:
        run = _iterative(prob, schedule=sch)
        assert E.ecc_matrix_schedule(run.mat) == want, (prob.n, sch)
        run.close()
    with pytest.raises(E.EccError):
        _iterative(small, schedule=7)


def _single_cases():
    def power_tol():
        prob = _banded_problem("power", 3000, 0, 3, T=80)
        rho = oracle.run_iterative(prob)["rho"]
        return dataclasses.replace(prob, tol=float(rho[37]) * (1 + 1e-9))
    return [("jacobi-1d", lambda: W.jacobi_1d()),
            ("jacobi-2d-33", lambda: W.jacobi_2d(N=33, T=40)),
            ("jacobi-2d-45", lambda: W.jacobi_2d(N=45, T=30)),
            ("jacobi-3d-12", lambda: W.jacobi_3d(N=12, T=30, P=40)),
            ("banded-jacobi-8", lambda: _banded_problem("jacobi", 2000, 8, 8)),
            ("power-tol", power_tol)]


@pytest.mark.parametrize("case", range(6))
def test_single_launch_matches_launch_loop(case):
    """The whole loop as one single-workgroup launch (vectors in LDS) against
    the launch-per-iteration loop (queue schedule) on the same problem:
    iterates, assembled vector, eff/age histories, versions, forced arrivals
    and clock bit for bit, norms within tolerance (the queue path adds them
    per work item); against the separate calls on the same matrix, norms bit
    for bit too (both reduce one partial per row); a tolerance that stops the
    run midway; and the oracle."""
    E = _capi()
    name, make = _single_cases()[case]
    prob = make()
    announce("single", name, prob.n, prob.P, prob.T)
    out = []
    for sch in (E.ECC_SCHEDULE_SINGLE, E.ECC_SCHEDULE_QUEUE):
        run = _iterative(prob, schedule=sch)
        assert E.ecc_matrix_schedule(run.mat) == sch
        iters = run.solve(tol=prob.tol, histories=True)
        torch.cuda.synchronize()
        out.append((iters, run.d_x.cpu().numpy(), run.d_x_hat.cpu().numpy(),
                    run.d_rho.cpu().numpy()[:iters], run.eff_hist.cpu().numpy()[:iters],
                    run.age_hist.cpu().numpy()[:iters], run.plan.stats()))
        if sch == E.ECC_SCHEDULE_SINGLE:
            # the separate calls over the same matrix: assemble, sweep, norm
            run.plan.reset()
            xa = torch.from_numpy(prob.x0.copy()).cuda()
            xb = torch.empty_like(xa)
            rhos = []
            for t in range(iters):
                rhos.append(run.step(t, xa, xb))
                xa, xb = xb, xa
            assert np.array_equal(np.array(rhos), out[0][3])
            assert np.array_equal(xa.cpu().numpy(), out[0][1])
        run.close()
    (i1, x1, h1, r1, e1, a1, s1), (i2, x2, h2, r2, e2, a2, s2) = out
    assert i1 == i2
    assert np.array_equal(x1, x2) and np.array_equal(h1, h2)
    assert np.all(np.abs(r1 - r2) <= 1e-12 * np.abs(r2) + 1e-300)
    assert np.array_equal(e1, e2) and np.array_equal(a1, a2)
    assert s1[0] == s2[0] and s1[1] == s2[1]
    assert np.array_equal(s1[2], s2[2]) and np.array_equal(s1[3], s2[3])
    if prob.tol > 0:
        assert i1 < prob.T
    _solve_and_compare(prob, bitwise=True, expect_schedule=E.ECC_SCHEDULE_SINGLE, solves=2)


def test_step_api_matches_solve_ranges():
    """The same for the range layout (sub-row sums, then rows)."""
    _step_api_matches_solve((W.pagerank_rmat(scale=11, T=25), _arrow_problem(T=12)),
                            range_bytes=2048)


def _step_api_matches_solve(problems, range_bytes=0, tile_rows=0, schedule=0):
    for prob in problems:
        announce("step api", prob.name)
        run = _iterative(prob, range_bytes, tile_rows, schedule)
        run.solve()
        x_solve = run.d_x.cpu().numpy()
        rho_solve = run.d_rho.cpu().numpy()
        run.plan.reset()
        a = torch.from_numpy(prob.x0.copy()).cuda()
        b = torch.empty_like(a)
        rhos = []
        for t in range(prob.T):
            rhos.append(run.step(t, a, b))
            a, b = b, a
        assert np.array_equal(a.cpu().numpy(), x_solve)
        assert np.array_equal(np.array(rhos), rho_solve)
        run.close()


def test_layout_choice():
    """The layout each kind of matrix gets: rows of at most 8 entries the
    short-row layout (entries held per row after the longest row), regular
    longer rows the stream layout, power-law rows the sorted layout, or over a
    vector of several column ranges the range layout."""
    E, R = _capi(), _runner()
    cases = [(W.jacobi_1d(), E.ECC_LAYOUT_SHORT, 3), (W.jacobi_2d(N=33, T=2), E.ECC_LAYOUT_SHORT, 5),
             (W.jacobi_3d(N=12, T=2, P=8), E.ECC_LAYOUT_SHORT, 7),
             (_banded_problem("jacobi", 3000, 4, 4, T=2), E.ECC_LAYOUT_SHORT, 4),
             (_banded_problem("power", 3000, 6, 6, T=2), E.ECC_LAYOUT_SHORT, 7),
             (_banded_problem("jacobi", 3000, 9, 16, T=2), E.ECC_LAYOUT_STREAM, 0),
             (W.pagerank_rmat(scale=10, T=2), E.ECC_LAYOUT_SORTED, 0)]
    for prob, layout, slots in cases:
        _check_layout(R, E, prob, layout, slots)
    # 8 KB of vector per range: two column ranges
    _check_layout(R, E, W.pagerank_rmat(scale=10, T=2), E.ECC_LAYOUT_RANGES, 2, range_bytes=4096)


def _check_layout(R, E, prob, layout, slots, range_bytes=0):
    announce("layout", prob.name)
    run = _iterative(prob, range_bytes)
    assert E.ecc_matrix_layout(run.mat) == (layout, slots), prob.name
    run.close()


def test_matrix_checks():
    E, R = _capi(), _runner()
    prob = W.jacobi_2d(N=8, T=2)
    announce("matrix checks")
    run = R.Iterative(prob.n, prob.A.row_ptr, prob.A.col, prob.A.val, prob.counts, prob.S,
                      prob.mask, "jacobi", b=prob.b)
    # zero one diagonal entry: Jacobi must refuse the matrix
    val = prob.A.val.copy()
    row5 = np.arange(prob.A.row_ptr[5], prob.A.row_ptr[6])
    val[row5[prob.A.col[row5] == 5]] = 0.0
    d_val = torch.from_numpy(val).cuda()
    bad = E.make_csr(prob.n, prob.n, prob.A.nnz, run.d_row_ptr, run.d_col, d_val)
    with pytest.raises(E.EccError) as ei:
        E.ecc_matrix_create(run.plan.handle, bad, E.ECC_KIND_JACOBI)
    assert ei.value.status == E.ECC_ERR_ARG
    # an out-of-range column index is refused for both kinds
    col = prob.A.col.copy()
    col[7] = prob.n + 3
    d_col = torch.from_numpy(col).cuda()
    bad = E.make_csr(prob.n, prob.n, prob.A.nnz, run.d_row_ptr, d_col, run.d_val)
    with pytest.raises(E.EccError):
        E.ecc_matrix_create(run.plan.handle, bad, E.ECC_KIND_POWER)
    # a plan that does not tile the rows
    plan = R.Plan(2, [3, 3], [0, 4], 0)
    with pytest.raises(E.EccError) as ei:
        E.ecc_matrix_create(plan.handle, run.csr, E.ECC_KIND_JACOBI)
    assert ei.value.status == E.ECC_ERR_STATE
    plan.close()
    run.close()


def test_matrix_checks_long_rows():
    """Rows longer than 256 entries are checked by a workgroup each: a zero
    or doubled diagonal entry and an out-of-range column in such a row are
    refused, as in short rows; the unchanged arrow matrix is accepted."""
    E, R = _capi(), _runner()
    prob = _arrow_problem(n=5000, T=2)
    announce("matrix checks, long rows")
    rp, col, val = prob.A.row_ptr, prob.A.col, prob.A.val
    run = _iterative(prob)
    row0 = np.arange(rp[0], rp[1])
    assert row0.size > 256 and (col[row0] == 0).sum() == 1

    def refused(c, v, kind):
        d_c, d_v = torch.from_numpy(c).cuda(), torch.from_numpy(v).cuda()
        csr = E.make_csr(prob.n, prob.n, prob.A.nnz, run.d_row_ptr, d_c, d_v)
        with pytest.raises(E.EccError) as ei:
            E.ecc_matrix_create(run.plan.handle, csr, kind)
        return ei.value.status

    v = val.copy()
    v[row0[col[row0] == 0]] = 0.0
    assert refused(col, v, E.ECC_KIND_JACOBI) == E.ECC_ERR_ARG
    c = col.copy()
    c[row0[-1]] = 0                        # a second diagonal entry in row 0
    assert refused(c, val, E.ECC_KIND_JACOBI) == E.ECC_ERR_ARG
    c = col.copy()
    c[row0[-1]] = prob.n                   # a column one past the end
    assert refused(c, val, E.ECC_KIND_POWER) == E.ECC_ERR_ARG
    run.close()


@pytest.mark.parametrize("n", [0, 1, 2047, 2048, 2049, 100003])
def test_gather_probe(n):
    """ecc_gather_probe: per-workgroup sums of x[idx[k]] over chunks of 2,048
    indices (compared with exact sums of the same chunks within rounding),
    indices outside [0, n_x) skipped, and a too-small output refused."""
    E = _capi()
    announce("gather probe", n)
    rng = np.random.default_rng(n + 3)
    n_x = 5000
    idx = rng.integers(-3, n_x + 3, n).astype(np.int32)   # a few out of range
    x = rng.standard_normal(n_x)
    chunks = max(1, (n + E.ECC_GATHER_CHUNK - 1) // E.ECC_GATHER_CHUNK)
    out = torch.full((chunks + 1,), np.nan, dtype=torch.float64, device="cuda")
    d_idx, d_x = torch.from_numpy(idx).cuda(), torch.from_numpy(x).cuda()
    E.ecc_gather_probe(d_idx, n, d_x, n_x, out, out.numel())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ok = (idx >= 0) & (idx < n_x)
    vals = np.where(ok, x[np.clip(idx, 0, n_x - 1)], 0.0)
    for c in range((n + E.ECC_GATHER_CHUNK - 1) // E.ECC_GATHER_CHUNK):
        part = vals[c * E.ECC_GATHER_CHUNK:(c + 1) * E.ECC_GATHER_CHUNK]
        ref = math.fsum(part)
        assert abs(got[c] - ref) <= 1e-13 * np.abs(part).sum(), (c, got[c], ref)
    if n == 0:
        assert np.isnan(got).all()                      # nothing written
    else:
        assert np.isnan(got[(n + E.ECC_GATHER_CHUNK - 1) // E.ECC_GATHER_CHUNK:]).all()
        with pytest.raises(E.EccError) as ei:
            E.ecc_gather_probe(d_idx, n, d_x, n_x, out, 0)
        assert ei.value.status == E.ECC_ERR_ARG


@pytest.mark.parametrize("n,off", [(0, 0), (1, 0), (3, 0), (1001, 0), (1001, 1), (65536 * 3 + 5, 0),
                                   (65536 * 3 + 5, 1)])
def test_stream_copy(n, off):
    """ecc_stream_copy: exact copy for odd lengths and 8-byte (not 16-byte)
    aligned buffers; nothing outside [0, n) is written."""
    E, R = _capi(), _runner()
    announce("stream copy", n, off)
    src = torch.randn(n + 4, dtype=torch.float64, device="cuda")
    dst = torch.full((n + 4,), float("nan"), dtype=torch.float64, device="cuda")
    E.ecc_stream_copy(dst[off:], src[off:], n, R.current_stream())
    torch.cuda.synchronize()
    assert torch.equal(dst[off:off + n], src[off:off + n])
    assert bool(torch.isnan(dst[:off]).all()) and bool(torch.isnan(dst[off + n:]).all())
    if n > 1:
        with pytest.raises(E.EccError) as ei:
            E.ecc_stream_copy(src[1:], src, n, R.current_stream())
        assert ei.value.status == E.ECC_ERR_ARG
