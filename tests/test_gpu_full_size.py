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


def test_config3_full():
    """PageRank on R-MAT scale 22 (2^26 edges), 64 ranks, S = 4."""
    _solve_and_compare(W.config3(), bitwise=False, threads=THREADS)


def test_config5_full():
    """3-D Jacobi, n = 64,000,000, 447,040,000 nonzeros, 512 ranks, S = 5:
    iterates bitwise equal to the oracle."""
    _solve_and_compare(W.config5(), bitwise=True, threads=THREADS)


def test_config4a_full():
    """allgatherv of 256 lognormal blocks (16.5M elements), 1,000 repetitions."""
    from paper_2203_17063_amd import capi as E
    from paper_2203_17063_amd import runner as R
    prob = W.config4a()
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
