"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (ecc_solve / the collective calls), against the oracle run
on the host's cores.  Minutes of host time: marked both gpu and slow."""
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle                                             # noqa: E402
import workloads as W                                     # noqa: E402
from gpu_common import announce                           # noqa: E402
from test_gpu_parity import _solve_and_compare            # noqa: E402

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.empty_cache()


def test_pagerank_rmat_full():
    """PageRank on R-MAT scale 22 (2^26 edges), 64 ranks, S = 4: the range
    layout in 2 column ranges, in the column-value form, against the oracle
    (normwise); then, both over 4 ranges of 8 MiB, the column-value form and
    the general form give bitwise equal iterates."""
    from paper_2203_17063_amd import capi as E
    from test_gpu_parity import _iterative, _solve_x_rho
    prob = W.pagerank_rmat()
    run = _iterative(prob)
    assert E.ecc_matrix_layout(run.mat) == (E.ECC_LAYOUT_RANGES, 2)
    assert E.ecc_matrix_form(run.mat)[0] == E.ECC_FORM_COLUMN_VALUES
    run.close()
    _solve_and_compare(prob, bitwise=False, threads=THREADS)
    rb = 8 << 20
    a = _solve_x_rho(prob, rb, compact=E.ECC_COMPACT_AUTO)
    g = _solve_x_rho(prob, rb, compact=E.ECC_COMPACT_NONE)
    assert a[4] == E.ECC_FORM_COLUMN_VALUES and g[4] == E.ECC_FORM_GENERAL and a[0] == g[0]
    assert np.array_equal(a[1], g[1]) and np.array_equal(a[2], g[2])
    assert np.allclose(a[3], g[3], rtol=1e-12, atol=0.0)


def test_jacobi_3d_full():
    """3-D Jacobi, n = 64,000,000, 447,040,000 nonzeros, 512 ranks, S = 5:
    iterates bitwise equal to the oracle.  The set-up sweeps it in plane
    tiles (planes of 400^2 rows, tiles of 64 x 400 rows)."""
    from paper_2203_17063_amd import capi as E
    _solve_and_compare(W.jacobi_3d(), bitwise=True, threads=THREADS, tiling=(160000, 25600),
                       expect_schedule=E.ECC_SCHEDULE_QUEUE)


def test_allgatherv_full():
    """allgatherv of 256 lognormal blocks (16.5M elements), 1,000 repetitions."""
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R
    prob = W.allgatherv_lognormal()
    announce("4a full", int(prob.counts.sum()), prob.reps)
    send = torch.from_numpy(prob.send).cuda()
    recv = torch.full_like(send, float("nan"))
    d_mask = torch.from_numpy(prob.mask).cuda()
    eff = torch.empty((prob.reps, prob.P), dtype=torch.uint8, device="cuda")
    plan = R.Plan(prob.P, prob.counts, prob.displs, prob.S)
    for r in range(prob.reps):
        E.ecc_allgatherv_assemble_packed(plan.handle, send, recv, d_mask[r].data_ptr(), eff[r])
    torch.cuda.synchronize()
    assert torch.equal(recv, send)                        # prefix displacements: concatenation
    assert bool((eff == 1).all())
    clock, forced, version, age = plan.stats()
    assert clock == prob.reps and forced == 0
    assert (version == prob.reps - 1).all() and (age == 0).all()
    plan.close()


def test_hypercube_full_sampled():
    """allreduce_SSP at the benchmark's shape: 32 processes x 16 MB, slack 2,
    Bernoulli(0.8) delivery, all 100 calls with the benchmark's two
    contribution sets alternating.  Element j of every result depends only on
    element j of the contributions and of the slots (the decisions only on
    clocks), so the oracle runs on 4,096 sampled elements; those results, the
    result clocks, the slot outcomes and the wait count match bit for bit."""
    from oracle import hypercube as H
    from paper_2203_17063_amd import capi as E
    prob = W.hypercube_ssp()
    P, m, d, T = prob.P, prob.m, prob.d, prob.calls
    announce("hypercube full", P, m, prob.slack, T)
    rng = np.random.default_rng(11)
    idx = np.unique(np.concatenate([[0, m - 1], rng.choice(m, 4094, replace=False)]))
    c_h = [prob.contrib(t) for t in range(2)]
    ref_res, ref_clk, ref_out, ref_state = H.run(
        P, prob.slack, np.stack([c_h[t & 1][:, idx] for t in range(T)]), prob.delivered[:T])
    contrib = [torch.from_numpy(c).cuda() for c in c_h]
    del c_h
    stream = torch.cuda.current_stream().cuda_stream
    result = torch.empty((P, m), dtype=torch.float64, device="cuda")
    d_idx = torch.from_numpy(idx).cuda()
    d_del = torch.from_numpy(prob.delivered.astype(np.uint8)).cuda()
    d_clk = torch.empty(P, dtype=torch.int32, device="cuda")
    d_out = torch.empty((P, d), dtype=torch.uint8, device="cuda")
    h = E.ecc_hypercube_create(P, m, prob.slack, stream)
    try:
        for t in range(T):
            E.ecc_allreduce_ssp(h, contrib[t & 1], d_del[t], result, d_clk, d_out)
            got = result[:, d_idx].cpu().numpy()
            assert np.array_equal(got, ref_res[t]), (t, np.abs(got - ref_res[t]).max())
            assert np.array_equal(d_clk.cpu().numpy(), ref_clk[t]), t
            assert np.array_equal(d_out.cpu().numpy(), ref_out[t]), t
        clock, waits, _, _ = E.ecc_hypercube_stats(h, P)
        assert clock == T and waits == int(ref_state.waits.sum())
    finally:
        E.ecc_hypercube_destroy(h)


def test_threshold_full():
    """Threshold Broadcast then Reduce at the benchmark's shape (32
    processes, 8,388,608 doubles, data fraction 0.5, root 0), two repetitions
    in the benchmark's order: the broadcast overwrites every receiver's
    prefix, which the reduce then sums.  Bit for bit with the oracle on the
    full vectors, the untouched tail of the result included."""
    from oracle import threshold as TH
    from paper_2203_17063_amd import capi as E
    prob = W.threshold_collectives()
    P, m, theta = prob.P, prob.m, prob.theta
    announce("threshold full", P, m, theta)
    xs_h = [prob.vector(p) for p in range(P)]
    res_h = np.full(m, -2.5)
    vecs = [torch.from_numpy(x).cuda() for x in xs_h]
    result = torch.full((m,), -2.5, dtype=torch.float64, device="cuda")
    d_vecs = torch.tensor([v.data_ptr() for v in vecs], dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    for r in range(2):
        k_ref = TH.bcast(P, 0, theta, xs_h[0], xs_h)
        kr_ref, n_ref = TH.reduce(P, 0, theta, TH.DATA, xs_h, res_h)
        k = E.ecc_bcast_threshold(P, 0, m, theta, vecs[0], d_vecs, stream)
        k_r, n_r = E.ecc_reduce_threshold(P, 0, m, theta, E.ECC_THRESHOLD_DATA, d_vecs, result,
                                          stream)
        torch.cuda.synchronize()
        assert k == k_ref and (k_r, n_r) == (kr_ref, n_ref), r
        assert np.array_equal(result.cpu().numpy(), res_h), r
        for p in (0, 1, 17, P - 1):
            assert np.array_equal(vecs[p].cpu().numpy(), xs_h[p]), (r, p)


def test_mf_full():
    """The factorisation at the benchmark's shape (25M ratings, 160,000 users,
    60,000 items, rank 16, 32 workers of 8 minibatches, slack 2,
    Bernoulli(0.8) arrivals), two iterations: the model bit for bit, the
    decisions exactly, the errors within 1e-12."""
    from test_gpu_mf import _compare
    _compare(W.mf_problem(T=2))


def test_partial_allreduce_full_every_repetition():
    """The partial allreduce at the benchmark's shape: 256 ranks x 2^22
    elements, Bernoulli(0.7) arrivals, no staleness bound, 1,000 repetitions,
    each rank's contribution at repetition r regenerated on the device from
    its counters.  Every repetition: eff, result clock and the result at 4,096
    sampled indices (first and last included) bit for bit against the oracle's
    rank-ordered sum of each rank's last arrival; repetitions 0-9 and 999:
    the whole result vector, by chunks of the index range; at the end, every
    slot at the sampled indices."""
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R
    prob = W.partial_allreduce()
    P, m = prob.P, prob.m
    announce("4b full, every repetition", P, m, prob.reps)
    fresh = torch.empty((P, m), dtype=torch.float64, device="cuda")
    slots = torch.empty((P, m), dtype=torch.float64, device="cuda")
    result = torch.empty(m, dtype=torch.float64, device="cuda")
    d_fresh = R.ptr_array([fresh[p] for p in range(P)])
    d_slots = R.ptr_array([slots[p] for p in range(P)])
    d_mask = torch.from_numpy(prob.mask).cuda()
    eff_d = torch.empty((prob.reps, P), dtype=torch.uint8, device="cuda")
    clk_d = torch.empty(prob.reps, dtype=torch.int32, device="cuda")
    plan = R.Plan(P, None, None, prob.S)
    stream = torch.cuda.current_stream().cuda_stream
    rng = np.random.default_rng(44)
    idx = np.sort(rng.choice(m, 4096, replace=False))
    idx[0], idx[-1] = 0, m - 1
    d_idx = torch.from_numpy(idx).cuda()
    version = np.full(P, -1, dtype=np.int32)
    full = set(range(10)) | {prob.reps - 1}
    chunk = 1 << 18
    for r in range(prob.reps):
        # rank p's contribution of repetition r: counters (r P + p) m + i
        W.uniform_device(prob.seed, W.STREAM_PAYLOAD_REDUCE, P * m, fresh.data_ptr(),
                         ctr0=prob.fresh_ctr0(0, r), lo=-1.0, hi=1.0, hip_stream=stream)
        E.ecc_allreduce_partial(plan.handle, m, d_fresh, d_slots, result, d_mask[r].data_ptr(),
                                eff_d[r], clk_d[r:r + 1])
        eff, _, _ = oracle.select(prob.S, r, prob.mask[r], version)
        got = result[d_idx].cpu().numpy()
        cols = [prob.fresh_at(p, int(version[p]), idx) for p in range(P)]
        ref = oracle.allreduce(np.zeros(P, dtype=np.uint8), [np.zeros(idx.size)] * P, cols)
        assert np.array_equal(got, ref), r
        assert np.array_equal(eff_d[r].cpu().numpy(), eff), r
        assert int(clk_d[r].item()) == oracle.result_clock(version), r
        if r in full:
            res = result.cpu().numpy()
            for a in range(0, m, chunk):
                parts = [W.uniform(prob.seed, W.STREAM_PAYLOAD_REDUCE, chunk,
                                   ctr0=prob.fresh_ctr0(p, int(version[p])) + a, lo=-1.0, hi=1.0)
                         for p in range(P)]
                ref = oracle.allreduce(np.zeros(P, dtype=np.uint8), [np.zeros(chunk)] * P, parts)
                assert np.array_equal(res[a:a + chunk], ref), (r, a)
    for p in range(P):
        assert np.array_equal(slots[p][d_idx].cpu().numpy(),
                              prob.fresh_at(p, int(version[p]), idx)), p
    plan.close()


def test_allgatherv_full_stale():
    """allgatherv of the 256 lognormal blocks (16.5M elements) with Bernoulli(0.7)
    arrivals and maximum staleness 3, 1,000 repetitions, the send arena of
    repetition r regenerated on the device (counters r E + i): eff and ages
    bit for bit at every repetition, and the receive vector bit for bit
    against the oracle's assembly (oracle.select then oracle.allgatherv over
    the same arena) every 25 repetitions, at 4,096 sampled indices at every
    other one."""
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R
    base = W.allgatherv_lognormal()
    P, reps, S = base.P, base.reps, 3
    seed = W.seed_of(4)
    mask = W.arrival_mask(seed + 100, reps, np.full(P, 0.7))
    counts, displs = base.counts, base.displs
    Etot = int(counts.sum())
    announce("4a full, stale", P, Etot, reps, S)
    send = torch.empty(Etot, dtype=torch.float64, device="cuda")
    recv = torch.full((Etot,), float("nan"), dtype=torch.float64, device="cuda")
    d_mask = torch.from_numpy(mask).cuda()
    eff_d = torch.empty(P, dtype=torch.uint8, device="cuda")
    age_d = torch.empty(P, dtype=torch.int32, device="cuda")
    plan = R.Plan(P, counts, displs, S)
    stream = torch.cuda.current_stream().cuda_stream
    version = np.full(P, -1, dtype=np.int32)
    h_recv = np.full(Etot, np.nan)
    rng = np.random.default_rng(45)
    idx = np.sort(rng.choice(Etot, 4096, replace=False))
    d_idx = torch.from_numpy(idx).cuda()
    sends = None
    forced_total = 0
    for r in range(reps):
        W.uniform_device(seed, W.STREAM_PAYLOAD, Etot, send.data_ptr(), ctr0=r * Etot,
                         lo=-1.0, hi=1.0, hip_stream=stream)
        E.ecc_allgatherv_assemble_packed(plan.handle, send, recv, d_mask[r].data_ptr(), eff_d,
                                         age_d)
        eff, age, forced = oracle.select(S, r, mask[r], version)
        forced_total += forced
        assert np.array_equal(eff_d.cpu().numpy(), eff), r
        assert np.array_equal(age_d.cpu().numpy(), age), r
        # the oracle's receive vector: every repetition's arena, arrived blocks copied
        arena = W.uniform(seed, W.STREAM_PAYLOAD, Etot, ctr0=r * Etot, lo=-1.0, hi=1.0)
        sends = [arena[d:d + c] for d, c in zip(displs, counts)]
        oracle.allgatherv(counts, displs, eff, sends, h_recv)
        if r % 25 == 0 or r == reps - 1:
            assert np.array_equal(recv.cpu().numpy(), h_recv), r
        else:
            assert np.array_equal(recv[d_idx].cpu().numpy(), h_recv[idx]), r
    clock, forced, ver, _ = plan.stats()
    assert clock == reps and forced == forced_total > 0 and np.array_equal(ver, version)
    plan.close()
