"""The calibration read (gleam_read_stream): it reads every byte exactly once, so its
XOR fold equals the fold computed on the host; misaligned input is refused."""

import numpy as np
import pytest
import torch

import paper_2607_23115_amd as g
from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    torch.cuda.init()


def host_fold(a: np.ndarray) -> int:
    w = a.view(np.uint64)
    return int(np.bitwise_xor.reduce(w)) if w.size else 0


@pytest.mark.parametrize("nbytes", [0, 16, 4096 + 48, (1 << 20), (3 << 20) + 16 * 1001, (37 << 20) + 4096])
def test_read_stream_fold(nbytes):
    say("read_stream", nbytes)
    rng = np.random.default_rng(nbytes)
    a = rng.integers(0, 256, size=max(nbytes, 16), dtype=np.uint8)
    d = torch.from_numpy(a).to("cuda")
    sink = torch.zeros(1, dtype=torch.int64, device="cuda")
    g.read_stream(d, nbytes, sink)
    torch.cuda.synchronize()
    assert int(g.as_u64(sink)[0]) == host_fold(a[:nbytes])


def test_read_stream_rejects_misaligned():
    d = torch.zeros(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(g.GleamError):
        g.read_stream(d[1:], 32)
    with pytest.raises(g.GleamError):
        g.read_stream(d, 24)
