"""GPU parity of the data-parallel matrix factorisation by minibatch SGD over
the partial allreduce (Section IV's workload) through the C ABI against the
oracle: the model after every iteration and the staleness decisions bit for
bit, the minibatch error and the full training error within 1e-12 (their
sums are reduced in another order)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import workloads as W                                     # noqa: E402
from oracle import mf as M                                # noqa: E402
from gpu_common import announce                           # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _compare(prob, clobber_inputs=False):
    from paper_2203_17063_amd import runner as R
    announce("mf", prob.n_users, prob.n_items, prob.N, prob.rank, prob.P, prob.S, prob.T)
    ref = M.run(prob, keep_W=tuple(range(prob.T + 1)))
    run = R.MatrixFactorization(prob)
    if clobber_inputs:
        # the state keeps its own copy of the ratings: the caller's arrays
        # may change after ecc_mf_create
        run.d_users.fill_(0)
        run.d_items.fill_(0)
        run.d_ratings.fill_(-1.0)
    try:
        run.reset()
        for t in range(prob.T):
            run.iterate(t, error=True)
            torch.cuda.synchronize()
            got = run.d_W.cpu().numpy()
            assert np.array_equal(got, ref["kept"][t + 1]), \
                (t, np.abs(got - ref["kept"][t + 1]).max())
            err = float(run.d_err[t].item())
            assert abs(err - M.full_rmse(prob, ref["kept"][t])) <= 1e-12 * err, t
        rmse = run.d_rmse.cpu().numpy()[:prob.T]
        assert np.allclose(rmse, ref["rmse"], rtol=1e-12, atol=0)
        assert np.array_equal(run.d_eff.cpu().numpy()[:prob.T], ref["eff"])
        clock, forced, _, _ = run.plan.stats()
        assert clock == prob.T and forced == int(ref["forced"].sum())
    finally:
        run.close()


@pytest.mark.parametrize("rank,K", [(1, 1), (4, 4), (16, 8), (32, 3)])
def test_mf_synchronous(rank, K):
    """Every worker fresh; full batches (K = 1) and minibatches."""
    _compare(W.mf_problem(n_users=300, n_items=120, n_ratings=20011, rank=rank, P=8, S=0, q=1.0,
                          T=6, eta=0.5, seed=rank, K=K))


@pytest.mark.parametrize("S,q,K", [(0, 0.5, 8), (2, 0.6, 8), (5, 0.3, 2)])
def test_mf_stale(S, q, K):
    """32 workers, stale gradients substituted; more iterations than
    minibatches (several epochs of the schedule)."""
    _compare(W.mf_problem(n_users=700, n_items=250, n_ratings=40009, rank=16, P=32, S=S, q=q,
                          T=20, eta=0.5, seed=7 + S, K=K))


@pytest.mark.parametrize("rank", [1, 16, 64])
def test_mf_long_rows(rank):
    """Few users and items: every (worker, minibatch, row) holds hundreds to
    thousands of ratings, so each row is summed by a whole workgroup over
    several chunks of its ratings."""
    _compare(W.mf_problem(n_users=60, n_items=25, n_ratings=50021, rank=rank, P=2, S=1, q=0.7,
                          T=4, eta=0.5, seed=11 + rank, K=2))


@pytest.mark.parametrize("rank", [2, 8, 16])
def test_mf_long_and_short_rows(rank):
    """Item rows of hundreds of ratings next to user rows of a few: both
    row paths in one launch."""
    _compare(W.mf_problem(n_users=2000, n_items=40, n_ratings=60013, rank=rank, P=4, S=2, q=0.6,
                          T=5, eta=0.5, seed=23 + rank, K=2))


def test_mf_inputs_copied_at_create():
    _compare(W.mf_problem(n_users=400, n_items=90, n_ratings=30011, rank=8, P=4, S=1, q=0.7,
                          T=4, eta=0.5, seed=31, K=4), clobber_inputs=True)


def test_mf_one_worker_and_idle_rows():
    """P = 1; many users and items without ratings, in the minibatch or at
    all (their rows only decay)."""
    _compare(W.mf_problem(n_users=5000, n_items=3000, n_ratings=3001, rank=8, P=1, S=0, q=1.0,
                          T=4, eta=0.5, seed=2, K=5))


def test_mf_empty_minibatches():
    """Fewer ratings per shard than minibatches: some workers' minibatches
    are empty (their lists hold only rows without ratings), though never
    all of one iteration's."""
    prob = W.mf_problem(n_users=40, n_items=25, n_ratings=20, rank=4, P=4, S=1, q=0.7, T=8,
                        eta=0.5, seed=1, K=8)
    N, P, K = prob.N, prob.P, prob.K
    used = np.zeros((prob.T, P), dtype=np.int64)
    for t in range(prob.T):
        for p in range(P):
            L = N * (p + 1) // P - N * p // P
            b = prob.batch[t][p]
            used[t, p] = L * (b + 1) // K - L * b // K
    assert (used == 0).sum() > 3 and (used.sum(axis=1) > 0).all()
    _compare(prob)


@pytest.mark.parametrize("seed", range(6))
def test_mf_random(seed):
    """Random worker counts (1-64, multiples of 8 and not, so with and
    without the XCD pinning), ranks, minibatch counts, sizes, staleness
    bounds and arrival rates."""
    rng = np.random.default_rng(7000 + seed)
    P = int(rng.choice([1, 2, 3, 8, 16, 24, 32, 40, 64]))
    rank = int(rng.choice([1, 2, 4, 8, 16, 32, 64]))
    K = int(rng.integers(1, 9))
    nu, ni = int(rng.integers(20, 3000)), int(rng.integers(10, 800))
    nr = int(rng.integers(P * 2, 60000))
    _compare(W.mf_problem(n_users=nu, n_items=ni, n_ratings=nr, rank=rank, P=P,
                          S=int(rng.integers(0, 6)), q=float(rng.uniform(0.2, 1.0)), T=8,
                          eta=0.3, seed=100 + seed, K=K))


def test_mf_errors():
    from paper_2203_17063_amd import capi as E
    announce("mf errors")
    u = torch.zeros(10, dtype=torch.int32, device="cuda")
    i = torch.zeros(10, dtype=torch.int32, device="cuda")
    r = torch.zeros(10, dtype=torch.float64, device="cuda")
    for args in [(4, 4, 3, 2, 1, 10), (4, 4, 128, 2, 1, 10), (0, 4, 4, 2, 1, 10),
                 (4, 4, 4, 0, 1, 10), (4, 4, 4, 2, 0, 10)]:
        with pytest.raises(E.EccError) as ei:
            E.ecc_mf_create(*args, u, i, r)
        assert ei.value.status == E.ECC_ERR_ARG
    bad = u.clone()
    bad[7] = 4
    with pytest.raises(E.EccError) as ei:
        E.ecc_mf_create(4, 4, 4, 2, 1, 10, bad, i, r)
    assert ei.value.status == E.ECC_ERR_ARG
