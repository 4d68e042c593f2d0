"""GPU: tl_view_load (the TMA-like box load whose source addresses the
TileLens-HW generator computes on the device, Section 4.3) against the
oracle's gather -- bit-exact bytes -- on the paper's view and Case-2
examples, random views of random memory-tile layouts (both the 16-byte and
the per-element copy), and a box of a full-size Llama weight."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_u8, host_bits
from tests.test_view_host import _random_view

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.synchronize()


def _tile_major(N, K, s, G, br, seed):
    """Random bytes as an N x K weight, repacked on the GPU (checked against the oracle's repack)."""
    raw = synth.random_bytes(N * K * s, seed=seed).reshape(N, K * s)
    src = dev_u8(raw)
    dst = dev_u8(np.zeros_like(raw))
    tl.tl_repack(src, dst, N, K, s, G, br)
    tm = host_bits(dst).reshape(-1)
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[s]
    assert np.array_equal(tm, oracle.repack(raw.view(dt).reshape(N, K), G, br).view(np.uint8).reshape(-1))
    return dst, tm


def _load_and_check(d_tm, tm, strides, coords, box, K, N, s, G, br):
    import torch
    n = int(np.prod(box))
    out = torch.zeros(n * s + 16, dtype=torch.uint8, device="cuda")
    tl.tl_view_load(d_tm, tl.view(strides, coords, box), K, N, s, G, br, out)
    torch.cuda.synchronize()
    got = host_bits(out)
    want = oracle.view_gather(tm, strides, coords, box, K, s, G, br)
    assert np.array_equal(got[:n * s], want), (strides, coords, box)
    assert np.all(got[n * s:] == 0)                       # nothing written past the box


def test_paper_view_example_on_gpu():
    K, N = 384, 128
    banner("view load: paper 2-D/3-D/4-D example")
    d_tm, tm = _tile_major(N, K, 1, 4096, 64, seed=1)
    for strides, coords, box in (([1, K], [256, 64], [128, 64]), ([1, K, 128], [0, 64, 2], [128, 64, 1]),
                                 ([1, K, 128, 64 * K], [0, 0, 2, 1], [128, 64, 1, 1])):
        _load_and_check(d_tm, tm, strides, coords, box, K, N, 1, 4096, 64)


def test_paper_case2_on_gpu():
    K, N = 512, 64
    banner("view load: Case 2 (32 x 32 box, 128 x 32 FP8 memory tile)")
    d_tm, tm = _tile_major(N, K, 1, 4096, 32, seed=2)
    for t in range(4):
        _load_and_check(d_tm, tm, [1, K], [32 * t, 32], [32, 32], K, N, 1, 4096, 32)


@pytest.mark.parametrize("s,G,br", [(1, 4096, 64), (2, 4096, 32), (2, 4096, 8), (2, 1024, 16), (4, 4096, 16),
                                    (2, 512, 8), (1, 16384, 128), (2, 16384, 64)])
def test_random_views_on_gpu(s, G, br):
    rng = np.random.default_rng(7 * s + G + br)
    a = G // (s * br)
    K, N = a * int(rng.integers(2, 7)), br * int(rng.integers(2, 7))
    banner(f"view load random: s={s} G={G} br={br} K={K} N={N}")
    d_tm, tm = _tile_major(N, K, s, G, br, seed=G + br + s)
    for _ in range(25):
        strides, coords, box = _random_view(rng, K, N, a, br)
        _load_and_check(d_tm, tm, strides, coords, box, K, N, s, G, br)


def test_llama_weight_box():
    """A 128 x 256 (K x N) box of the gate+up weight at a compute-tile
    position, bf16, (64, 32) memory tiles: the compute tile of Section 6.5."""
    import torch
    N, K, s, G, br = 57344, 8192, 2, 4096, 32
    banner("view load: gate_up 128 x 256 box")
    raw = torch.randint(0, 256, (N, K * s), dtype=torch.uint8, device="cuda",
                        generator=torch.Generator(device="cuda").manual_seed(3))
    d_tm = torch.empty_like(raw)
    tl.tl_repack(raw, d_tm, N, K, s, G, br)
    strides, coords, box = [1, K], [4096, 30720], [128, 256]
    out = torch.zeros(128 * 256 * s, dtype=torch.uint8, device="cuda")
    tl.tl_view_load(d_tm, tl.view(strides, coords, box), K, N, s, G, br, out)
    torch.cuda.synchronize()
    # element (col c, row r) of the box is W[30720 + c][4096 + r] of the row-major original
    want = raw[30720:30720 + 256].view(torch.int16)[:, 4096:4096 + 128]
    assert torch.equal(out.view(torch.int16).view(256, 128), want)
