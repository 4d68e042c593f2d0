"""GPU parity of tl_gemm over a weight stored [K][N] row-major (N contiguous:
TL_LAYOUT_KN_ROW, the paper's "row-major" layout), through the C ABI, against
the fp64 oracle on the logical [N][K] weight: ragged M and N, split-K, fp32
and bf16 output, exact (small-integer and one-hot) inputs bit-exact, the
block-granular fetch whose counted bytes equal tl_read_amp's and the oracle's
brute-force count, and the four Llama-70B decode shapes element by element."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, host_bits, host_f32, parity, parity_bf16_out

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.synchronize()


def run_kn(A_bits, W_bits, desc, fetch=tl.TL_FETCH_NATIVE):
    """C = A W^T with W (logically [N][K]) uploaded as its [K][N] transpose."""
    import torch
    M, K = A_bits.shape
    N = W_bits.shape[0]
    W_kn = dev_bf16(np.ascontiguousarray(W_bits.T))
    dt = torch.bfloat16 if desc.out_dtype == tl.TL_OUT_BF16 else torch.float32
    C = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
    tl.tl_gemm(dev_bf16(A_bits), W_kn, C, M, N, K, desc, fetch)
    torch.cuda.synchronize()
    return C


KN = tl.TL_LAYOUT_KN_ROW
CASES = [
    # M, N, K, split_k (0 = the library's plan)
    (1, 1024, 4096, 0), (5, 512, 2048, 0), (8, 4096, 1024, 0), (16, 256, 8192, 0), (17, 1000, 512, 0),
    (24, 2048, 2048, 3), (32, 64, 64, 0), (33, 520, 1024, 0), (48, 1024, 4096, 4), (64, 8192, 256, 1),
    (8, 1024, 8192, 16), (3, 8, 128, 0),
]


@pytest.mark.parametrize("M,N,K,S", CASES)
def test_kn_row_decode_random(M, N, K, S):
    d = tl.layout(kind=KN, split_k=S)
    plan = tl.tl_gemm_plan(M, N, K, d, tl.TL_FETCH_NATIVE)
    banner(f"KN_ROW decode M={M} N={N} K={K} plan={plan}")
    assert plan["kernel"] == 1 and plan["tile_n"] == 64 and plan["tile_k"] == 64
    A = synth.normal_bf16((M, K), seed=1100 + M)
    W = synth.normal_bf16((N, K), seed=1200 + N, sigma=synth.W_SIGMA)
    parity(host_f32(run_kn(A, W, d)), oracle.gemm_f64(A, W), f"KN_ROW M={M} N={N} K={K}")


@pytest.mark.parametrize("M,N,K,S", [(8, 1024, 2048, 4), (32, 2048, 4096, 1), (64, 512, 1024, 3), (1, 4096, 8192, 0)])
def test_kn_row_exact_inputs_bit_exact(M, N, K, S):
    """Small integers: every partial sum is exact in fp32, so any summation
    order gives the exact result; repeated calls are bitwise identical."""
    banner(f"KN_ROW exact M={M} N={N} K={K} S={S}")
    A = synth.small_int_bf16((M, K), seed=1300 + M)
    W = synth.small_int_bf16((N, K), seed=1301 + N)
    d = tl.layout(kind=KN, split_k=S)
    C1 = host_f32(run_kn(A, W, d))
    C2 = host_f32(run_kn(A, W, d))
    assert np.array_equal(C1, oracle.gemm_f64(A, W).astype(np.float32))
    assert np.array_equal(C1, C2)


def test_kn_row_one_hot_rows():
    """A[m] = e_{k_m}: C[m][n] = W[n][k_m] exactly -- pins which stored element
    the transposed reads deliver to which (m, n)."""
    M, N, K = 64, 1024, 2048
    banner("KN_ROW one-hot")
    ks = np.random.default_rng(5).integers(0, K, M)
    A = np.zeros((M, K), dtype=np.uint16)
    A[np.arange(M), ks] = 0x3F80                       # bf16 1.0
    W = synth.normal_bf16((N, K), seed=1400, sigma=synth.W_SIGMA)
    C = host_f32(run_kn(A, W, tl.layout(kind=KN)))
    assert np.array_equal(C, synth.bf16_bits_to_f32(W[:, ks].T))


def test_kn_row_bf16_out():
    M, N, K = 12, 2048, 4096
    banner("KN_ROW bf16 out")
    A = synth.normal_bf16((M, K), seed=1500)
    W = synth.normal_bf16((N, K), seed=1501, sigma=synth.W_SIGMA)
    C = run_kn(A, W, tl.layout(kind=KN, out_dtype=tl.TL_OUT_BF16))
    parity_bf16_out(host_bits(C), oracle.gemm_f64(A, W), "KN_ROW bf16 out")


@pytest.mark.parametrize("M,N,K,G", [(8, 1024, 2048, 4096), (8, 512, 1024, 512), (1, 256, 1024, 16384),
                                     (16, 64, 2048, 4096), (32, 128, 512, 256), (5, 192, 640, 128)])
def test_kn_row_block_fetch_counted(M, N, K, G):
    """[K][N] weight read in whole G-byte blocks: same result, and the bytes
    the kernel counts while it loads them equal tl_read_amp's fetched bytes
    for the kernel's tile and the oracle's brute-force enumeration (several
    k-rows share a block when N * 2 < G)."""
    banner(f"KN_ROW block fetch M={M} N={N} K={K} G={G}")
    A = synth.normal_bf16((M, K), seed=1600 + M)
    W = synth.normal_bf16((N, K), seed=1601, sigma=synth.W_SIGMA)
    d = tl.layout(kind=KN, G=G)
    tl.tl_fetch_counter_read()
    C = run_kn(A, W, d, fetch=tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    got = tl.tl_fetch_counter_read()
    parity(host_f32(C), oracle.gemm_f64(A, W), f"KN_ROW block G={G}")
    p = tl.tl_gemm_plan(M, N, K, d, tl.TL_FETCH_BLOCK)
    amp = tl.tl_read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], d, G)
    want = oracle.read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], oracle.KN_ROW, G)
    assert got == amp["fetched_bytes"] == want["fetched_bytes"], (got, amp, want)


def test_kn_row_native_count():
    """Native fetch: the tally is the bytes the 64-column tiles load, N * K * 2
    when 64 divides N."""
    M, N, K = 8, 2048, 4096
    banner("KN_ROW native count")
    A = synth.normal_bf16((M, K), seed=1700)
    W = synth.normal_bf16((N, K), seed=1701, sigma=synth.W_SIGMA)
    tl.tl_fetch_counter_read()
    run_kn(A, W, tl.layout(kind=KN), fetch=tl.TL_FETCH_NATIVE | tl.TL_FETCH_COUNT)
    assert tl.tl_fetch_counter_read() == N * K * 2


@pytest.mark.parametrize("i,name,N,K", [(i, *s) for i, s in enumerate(synth.LLAMA70B)])
def test_kn_row_llama_full_size(i, name, N, K):
    """The bench's row-major layout case: the Llama-70B shapes at M = 8 with the
    weight stored [K][N], every output element against the oracle."""
    import torch
    banner(f"KN_ROW llama {name}")
    W = synth.normal_bf16((N, K), seed=synth.llama_weight_seed(i), sigma=synth.W_SIGMA)
    M = 8
    A = synth.normal_bf16((M, K), seed=synth.llama_decode_act_seed(i, M))
    Wd = dev_bf16(W)
    W_kn = Wd.t().contiguous()
    del Wd
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    tl.tl_gemm(dev_bf16(A), W_kn, C, M, N, K, tl.layout(kind=KN), tl.TL_FETCH_NATIVE)
    torch.cuda.synchronize()
    parity(host_f32(C), oracle.gemm_f64(A, W), f"KN_ROW {name}")
