"""GPU parity of the threshold Broadcast / Reduce and of the dropping
allreduce (Section III-B) through the C ABI against the oracle, bit for bit,
with the status outputs."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import threshold as TH                        # noqa: E402
from gpu_common import announce                           # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _E():
    from paper_2203_17063_amd import capi
    return capi


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _ptrs(ts):
    return torch.tensor([t.data_ptr() for t in ts], dtype=torch.int64, device="cuda")


@pytest.mark.parametrize("P,root", [(1, 0), (2, 1), (7, 3), (32, 0), (33, 20)])
@pytest.mark.parametrize("m,theta", [(0, 0.5), (1, 1.0), (1001, 0.1), (70001, 0.5), (4096 * 3 + 1, 1.0),
                                     (5000, 0.0)])
def test_bcast(P, root, m, theta):
    E = _E()
    announce("bcast", P, root, m, theta)
    rng = np.random.default_rng(P * 31 + m)
    src_h = rng.standard_normal(m)
    # every other receive buffer starts one element into its allocation: 8-byte aligned only
    bufs_h = [np.full(m, float(p) + 0.5) for p in range(P)]
    k_ref = TH.bcast(P, root, theta, src_h, bufs_h)
    src = torch.from_numpy(src_h).cuda()
    store = [torch.full((m + 1,), float(p) + 0.5, dtype=torch.float64, device="cuda")
             for p in range(P)]
    bufs = [s[(p & 1):(p & 1) + m] for p, s in enumerate(store)]
    k = E.ecc_bcast_threshold(P, root, m, theta, src, _ptrs(bufs), _stream())
    torch.cuda.synchronize()
    assert k == k_ref
    for p in range(P):
        assert np.array_equal(bufs[p].cpu().numpy(), bufs_h[p]), p


@pytest.mark.parametrize("P,root", [(1, 0), (2, 0), (3, 2), (8, 5), (13, 0), (32, 0), (33, 7),
                                    (64, 63)])
@pytest.mark.parametrize("mode,theta", [(TH.DATA, 1.0), (TH.DATA, 0.37), (TH.PROCS, 0.5),
                                        (TH.PROCS, 0.75), (TH.PROCS, 0.01)])
def test_reduce(P, root, mode, theta):
    E = _E()
    m = 20011
    announce("reduce", P, root, mode, theta, m)
    rng = np.random.default_rng(P + 100 * root)
    xs_h = [rng.standard_normal(m) * 10.0 ** rng.integers(-6, 6) for _ in range(P)]
    res_h = np.full(m, -3.25)
    k_ref, n_ref = TH.reduce(P, root, theta, mode, xs_h, res_h)
    xs = [torch.from_numpy(x).cuda() for x in xs_h]
    res = torch.full((m,), -3.25, dtype=torch.float64, device="cuda")
    k, n = E.ecc_reduce_threshold(P, root, m, theta, mode, _ptrs(xs), res, _stream())
    torch.cuda.synchronize()
    assert (k, n) == (k_ref, n_ref)
    got = res.cpu().numpy()
    assert np.array_equal(got, res_h), np.abs(got - res_h).max()


@pytest.mark.parametrize("P,root", [(65, 0), (100, 99), (128, 5), (257, 100), (1000, 1),
                                    (4096, 4095)])
@pytest.mark.parametrize("mode,theta", [(TH.DATA, 1.0), (TH.DATA, 0.4), (TH.PROCS, 0.3),
                                        (TH.PROCS, 0.6)])
def test_reduce_many_processes(P, root, mode, theta):
    """More than 64 processes: the tree's pairwise form, relative ranks
    missing from the top of the tree (P and the involved count not powers
    of two) and processes of the first stages only."""
    E = _E()
    m = 2053
    announce("reduce many", P, root, mode, theta, m)
    rng = np.random.default_rng(P + 7 * root)
    scale = 10.0 ** rng.integers(-6, 6, size=P)
    xs_h = [rng.standard_normal(m) * scale[p] for p in range(P)]
    res_h = np.full(m, -3.25)
    k_ref, n_ref = TH.reduce(P, root, theta, mode, xs_h, res_h)
    xs = [torch.from_numpy(x).cuda() for x in xs_h]
    res = torch.full((m,), -3.25, dtype=torch.float64, device="cuda")
    k, n = E.ecc_reduce_threshold(P, root, m, theta, mode, _ptrs(xs), res, _stream())
    torch.cuda.synchronize()
    assert (k, n) == (k_ref, n_ref)
    got = res.cpu().numpy()
    assert np.array_equal(got, res_h), np.abs(got - res_h).max()


@pytest.mark.parametrize("m", [0, 1, 7, 300007])
def test_reduce_lengths(m):
    E = _E()
    announce("reduce lengths", m)
    P = 32
    rng = np.random.default_rng(m)
    xs_h = [rng.standard_normal(m) for _ in range(P)]
    res_h = np.zeros(m)
    TH.reduce(P, 0, 0.5, TH.DATA, xs_h, res_h)
    xs = [torch.from_numpy(x).cuda() for x in xs_h]
    res = torch.zeros(m, dtype=torch.float64, device="cuda")
    E.ecc_reduce_threshold(P, 0, m, 0.5, TH.DATA, _ptrs(xs) if m else None, res if m else None,
                           _stream())
    torch.cuda.synchronize()
    assert np.array_equal(res.cpu().numpy(), res_h)


@pytest.mark.parametrize("P,q", [(1, 1.0), (5, 0.5), (17, 0.3), (64, 0.9), (300, 0.5), (9, 0.0)])
def test_allreduce_drop(P, q):
    E = _E()
    m = 10007
    announce("allreduce drop", P, q, m)
    rng = np.random.default_rng(P)
    fresh_h = [rng.standard_normal(m) for _ in range(P)]
    arrived_h = (rng.random(P) < q).astype(np.uint8)
    ref = TH.allreduce_drop(arrived_h, fresh_h)
    fresh = [torch.from_numpy(f).cuda() for f in fresh_h]
    arrived = torch.from_numpy(arrived_h).cuda()
    res = torch.full((m,), np.nan, dtype=torch.float64, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    E.ecc_allreduce_drop(P, m, _ptrs(fresh), arrived, res, cnt, _stream())
    torch.cuda.synchronize()
    got = res.cpu().numpy()
    assert np.array_equal(got, ref)
    assert not np.signbit(got[got == 0]).any()
    assert int(cnt.item()) == int(arrived_h.sum())


@pytest.mark.parametrize("seed", range(4))
def test_reduce_random(seed):
    """Random process counts (up to 64, or up to 4,096), roots, modes,
    fractions and lengths (a one-off run of 30 such cases passed as well)."""
    E = _E()
    rng = np.random.default_rng(12000 + seed)
    P = int(rng.integers(1, 4097)) if seed % 2 else int(rng.integers(1, 65))
    root = int(rng.integers(0, P))
    mode = int(rng.choice([TH.DATA, TH.PROCS]))
    theta = float(rng.choice([0.0, 0.1, 0.37, 0.5, 0.75, 1.0]))
    if mode == TH.PROCS and theta == 0.0:
        theta = 0.05
    m = int(rng.integers(0, 20000)) if P <= 256 else int(rng.integers(0, 1500))
    announce("reduce random", P, root, mode, theta, m)
    xs_h = [rng.standard_normal(m) * 10.0 ** rng.integers(-6, 6) for _ in range(P)]
    res_h = np.full(m, -3.25)
    k_ref, n_ref = TH.reduce(P, root, theta, mode, xs_h, res_h)
    xs = [torch.from_numpy(x).cuda() for x in xs_h]
    res = torch.full((m,), -3.25, dtype=torch.float64, device="cuda")
    k, n = E.ecc_reduce_threshold(P, root, m, theta, mode, _ptrs(xs), res, _stream())
    torch.cuda.synchronize()
    assert (k, n) == (k_ref, n_ref)
    assert np.array_equal(res.cpu().numpy(), res_h)


def test_threshold_errors():
    E = _E()
    announce("threshold errors")
    x = torch.zeros(4, dtype=torch.float64, device="cuda")
    p = _ptrs([x] * 65)
    for args in [(4097, 0, 4, 1.0, TH.DATA), (0, 0, 4, 1.0, TH.DATA), (4, 4, 4, 1.0, TH.DATA), (4, 0, 4, 1.5, TH.DATA),
                 (4, 0, 4, 0.0, TH.PROCS), (4, 0, 4, 0.5, 7), (4, 0, -1, 0.5, TH.DATA)]:
        with pytest.raises(E.EccError) as ei:
            E.ecc_reduce_threshold(*args, p, x, _stream())
        assert ei.value.status == E.ECC_ERR_ARG
    for args in [(0, 0, 4, 0.5), (4, -1, 4, 0.5), (4, 0, 4, -0.1)]:
        with pytest.raises(E.EccError) as ei:
            E.ecc_bcast_threshold(*args, x, p, _stream())
        assert ei.value.status == E.ECC_ERR_ARG
    with pytest.raises(E.EccError):
        E.ecc_allreduce_drop(4, 4, p, None, x, None, _stream())
