"""The allocation-free sweep entry point: ecc_iterate_jacobi_noalloc against
ecc_iterate_jacobi + ecc_residual (the existing entry points, with a caller
workspace) and against the oracle's sweep.  Two calls in a row, the second on
a smaller problem, with each schedule of the short-row layout and with the
stream layout; the partial sums of every call live in the library's one
static array per GPU."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle                                             # noqa: E402
import workloads as W                                     # noqa: E402
from gpu_common import announce                           # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield


def _banded(n, seed):
    """Rows of 9-12 entries within a band (the stream layout)."""
    rng = np.random.default_rng(seed)
    cols, vals = [], []
    for i in range(n):
        lo, hi = max(0, i - 300), min(n, i + 301)
        c = np.sort(rng.choice(np.arange(lo, hi), int(rng.integers(9, 13)), replace=False))
        if i not in c:
            c[0] = i
            c = np.sort(c)
        v = -rng.uniform(0.05, 1.0, c.size) / c.size
        v[c == i] = 2.0 * np.abs(v).sum() + 1.0
        cols.append(c)
        vals.append(v)
    rp = np.zeros(n + 1, dtype=np.int32)
    rp[1:] = np.cumsum([c.size for c in cols])
    A = W.CSR(n, n, rp, np.concatenate(cols).astype(np.int32), np.concatenate(vals))
    counts = W.dirichlet_partition(n, 5, seed)
    mask = np.ones((2, 5), dtype=np.uint8)
    return W.Iterative("banded", "jacobi", A, counts, W.exclusive_scan(counts), 1, mask, 2,
                       np.zeros(n), b=rng.standard_normal(n), norm=2)


def _one_call(prob, schedule, seed):
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R
    announce("noalloc", prob.name, prob.n, schedule)
    run = R.Iterative(prob.n, prob.A.row_ptr, prob.A.col, prob.A.val, prob.counts, prob.S,
                      prob.mask, prob.kind, b=prob.b, schedule=schedule)
    rng = np.random.default_rng(seed)
    x_own = rng.standard_normal(prob.n)
    x_hat = rng.standard_normal(prob.n)
    d_own = torch.from_numpy(x_own).cuda()
    d_hat = torch.from_numpy(x_hat).cuda()
    nx_ref = torch.full_like(d_own, float("nan"))
    nx = torch.full_like(d_own, float("nan"))
    rho = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
    ph = run.plan.handle
    # the existing entry points, with the caller's workspace
    E.ecc_iterate_jacobi(ph, run.mat, run.d_b, d_own, d_hat, nx_ref, run.d_partials)
    rho_ref = E.ecc_residual(ph, run.d_partials, run.d_partials.numel(), E.ECC_NORM_L2)
    # the allocation-free variant
    E.ecc_iterate_jacobi_noalloc(ph, run.mat, run.d_b, d_own, d_hat, nx, rho)
    torch.cuda.synchronize()
    assert torch.equal(nx, nx_ref)
    assert rho.item() == rho_ref
    # and the definition: the oracle's sweep of the same view
    bstart = oracle.block_starts(prob.counts)
    xo, r = oracle.jacobi_sweep(prob.A, bstart, prob.b, x_own, x_hat, threads=4)
    assert np.array_equal(nx.cpu().numpy(), xo)        # one lane per row, CSR order
    ro = oracle.norm(r, 2)
    assert abs(rho.item() - ro) <= 1e-12 * ro
    run.close()


@pytest.mark.parametrize("schedule", [0, 2])
def test_noalloc_two_calls_second_smaller(schedule):
    _one_call(W.jacobi_3d(N=40, T=2, P=9), schedule, 1)
    _one_call(W.jacobi_2d(N=24, T=2), schedule, 2)


def test_noalloc_stream_layout_then_short():
    _one_call(_banded(6000, 3), 0, 3)
    _one_call(W.jacobi_1d(), 0, 4)


def test_noalloc_rejects_missing_output():
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R
    prob = W.jacobi_2d(N=8, T=2)
    run = R.Iterative(prob.n, prob.A.row_ptr, prob.A.col, prob.A.val, prob.counts, prob.S,
                      prob.mask, prob.kind, b=prob.b)
    x = torch.zeros(prob.n, dtype=torch.float64, device="cuda")
    y = torch.zeros_like(x)
    with pytest.raises(E.EccError):
        E.ecc_iterate_jacobi_noalloc(run.plan.handle, run.mat, run.d_b, x, x, y, None)
    run.close()
