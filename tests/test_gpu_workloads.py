"""The device-side input generator (workloads/gen_gpu.hip) against the host
generator: the same counter-based uniforms, bit for bit, at large counters,
odd lengths and both ranges the workloads use."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import workloads as W                                     # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield


@pytest.mark.parametrize("stream,ctr0,n,lo,hi", [
    (W.STREAM_PAYLOAD_REDUCE, 0, 1, -1.0, 1.0),
    (W.STREAM_PAYLOAD_REDUCE, 12345, 100003, -1.0, 1.0),
    (W.STREAM_PAYLOAD_REDUCE, (999 * 256 + 255) << 22, 1 << 22, -1.0, 1.0),
    (W.STREAM_PAYLOAD, 3 << 40, 65537, 0.0, 1.0),
    (W.STREAM_B, 7, 4099, 0.0, 1.0)])
def test_device_uniform_matches_host(stream, ctr0, n, lo, hi):
    seed = W.seed_of(4)
    ref = W.uniform(seed, stream, n, ctr0=ctr0, lo=lo, hi=hi)
    d = torch.full((n,), float("nan"), dtype=torch.float64, device="cuda")
    W.uniform_device(seed, stream, n, d.data_ptr(), ctr0=ctr0, lo=lo, hi=hi,
                     hip_stream=torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert np.array_equal(d.cpu().numpy(), ref)
