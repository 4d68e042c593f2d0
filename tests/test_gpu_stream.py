"""tl_stream_read, the HBM read ceiling the GEMM kernels are measured against:
every byte is read -- the XOR of the buffer's 32-bit words, computed on the
host by numpy, comes back XORed into the caller's word -- for sizes with and
without a partial 4 KB piece, and the empty buffer."""
import numpy as np
import pytest

import paper_2607_04031_amd as tl
from tests._gpu import banner

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield


@pytest.mark.parametrize("nbytes", [0, 16, 4096, 3 * 4096 + 48, (1 << 20) + 7 * 16, 4096 * 1024 * 16 + 4080,
                                    (256 << 20)])
def test_stream_read_checksum(nbytes):
    import torch
    banner(f"stream read {nbytes} bytes")
    rng = np.random.default_rng(nbytes % 1000 + 1)
    words = rng.integers(0, 1 << 32, size=max(nbytes // 4, 1), dtype=np.uint32)[: nbytes // 4]
    buf = torch.from_numpy(words.view(np.int32)).cuda() if nbytes else torch.zeros(4, dtype=torch.int32,
                                                                                       device="cuda")
    ck = torch.full((1,), 12345, dtype=torch.int32, device="cuda")     # XORed into
    tl.tl_stream_read(buf, nbytes, ck)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(words) if nbytes else np.uint32(0)
    assert np.uint32(ck.cpu().numpy().view(np.uint32)[0]) == np.uint32(want) ^ np.uint32(12345)
