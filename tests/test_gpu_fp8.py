"""GPU parity of the weight-only FP8 decode (tl_gemm_w8 / tl_gemm with
elem_bytes 1): OCP E4M3 weights in 64 x 64 (4 KB) memory tiles, bf16
activations, against the oracle's W8 GEMM; exact cases bit for bit; the
fetch tally; full-size Llama shapes on sampled outputs."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, dev_u8, host_f32, parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.synchronize()


def fp8_layout(G=4096, br=64, **kw):
    return tl.layout(elem_bytes=1, G=G, block_rows=br, **kw)


def run_w8(A_bits, W8, scales, desc, fetch=tl.TL_FETCH_BLOCK):
    import torch
    M, K = A_bits.shape
    N = W8.shape[0]
    W = dev_u8(W8)
    if desc.kind == tl.TL_LAYOUT_TILE:
        Wt = torch.empty_like(W)
        tl.tl_repack(W, Wt, N, K, 1, desc.G, desc.block_rows)
        W = Wt
    sc = None if scales is None else torch.from_numpy(np.ascontiguousarray(scales, dtype=np.float32)).cuda()
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    tl.tl_gemm_w8(dev_bf16(A_bits), W, sc, C, M, N, K, desc, fetch)
    torch.cuda.synchronize()
    return C


@pytest.mark.parametrize("M", [1, 8, 16, 32, 64])
@pytest.mark.parametrize("scaled", [False, True])
def test_w8_parity(M, scaled):
    N, K = 512, 2048
    banner(f"fp8 decode M={M} scaled={scaled}")
    A = synth.normal_bf16((M, K), seed=300 + M)
    W8, sc = synth.fp8_weights((N, K), seed=301)
    scales = sc if scaled else None
    parity(host_f32(run_w8(A, W8, scales, fp8_layout())), oracle.gemm_w8_f64(A, W8, scales), "fp8")


@pytest.mark.parametrize("kind,G,br", [(tl.TL_LAYOUT_TILE, 4096, 32), (tl.TL_LAYOUT_TILE, 16384, 64),
                                       (tl.TL_LAYOUT_TILE, 1024, 64), (tl.TL_LAYOUT_NK_ROW, 4096, 64)])
def test_w8_layouts(kind, G, br):
    N, K = 256, 4096
    banner(f"fp8 decode layout kind={kind} G={G} br={br}")
    A = synth.normal_bf16((8, K), seed=310)
    W8, sc = synth.fp8_weights((N, K), seed=311)
    d = tl.layout(kind=kind, elem_bytes=1, G=G, block_rows=br)
    fetch = tl.TL_FETCH_NATIVE if kind == tl.TL_LAYOUT_NK_ROW else tl.TL_FETCH_BLOCK
    parity(host_f32(run_w8(A, W8, sc, d, fetch)), oracle.gemm_w8_f64(A, W8, sc), "fp8 layout")


@pytest.mark.parametrize("split_k", [1, 4])
def test_w8_small_integers_exact(split_k):
    import torch
    M, N, K = 8, 256, 4096
    A = synth.small_int_bf16((M, K), seed=320)
    Wi = np.random.default_rng(321).integers(-8, 9, size=(N, K)).astype(np.float32)
    W8 = torch.from_numpy(Wi).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    banner(f"fp8 exact split_k={split_k}")
    got = host_f32(run_w8(A, W8, None, fp8_layout(split_k=split_k))).astype(np.float64)
    assert np.array_equal(got, oracle.gemm_w8_f64(A, W8))


def test_w8_through_tl_gemm_and_fetch_counter():
    """tl_gemm with an FP8 descriptor is the unscaled W8 GEMM; the tally is
    the weight's N * K bytes."""
    import torch
    M, N, K = 8, 1024, 2048
    A = synth.normal_bf16((M, K), seed=330)
    W8, _ = synth.fp8_weights((N, K), seed=331)
    banner("fp8 via tl_gemm + counter")
    W = dev_u8(W8)
    Wt = torch.empty_like(W)
    tl.tl_repack(W, Wt, N, K, 1, 4096, 64)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    tl.tl_fetch_counter_read()
    tl.tl_gemm(dev_bf16(A), Wt, C, M, N, K, fp8_layout(), tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    assert tl.tl_fetch_counter_read() == N * K
    parity(host_f32(C), oracle.gemm_w8_f64(A, W8), "tl_gemm fp8")


@pytest.mark.parametrize("i,name,N,K", [(i, *s) for i, s in enumerate(synth.LLAMA70B)])
def test_w8_llama_full_size(i, name, N, K):
    """The FP8 layer the bench times (64 x 64 FP8 memory tiles, per-channel
    scales) at M = 1, 8 and 32: every output element against the oracle."""
    banner(f"fp8 llama full {name}")
    W8, sc = synth.fp8_weights((N, K), seed=synth.llama_weight_seed(i))
    for M in synth.LLAMA_DECODE_M:
        A = synth.normal_bf16((M, K), seed=synth.llama_decode_act_seed(i, M))
        C = run_w8(A, W8, sc, fp8_layout())
        parity(host_f32(C), oracle.gemm_w8_f64(A, W8, sc), f"fp8 {name} M={M}")
