"""Parity of the decode kernel that stages the activations in LDS (17 <= M <= 64
on whole tile-major strips; the planner's default when its T tiles x S K
ranges per workgroup cover the CUs in whole rounds, or at least 7/8 of one
round above 32 rows) against the oracle:
every (T, S) the Llama-70B shapes use, ragged M, bf16 output, memory-tile
shapes, exact inputs (bit-exact), reproducibility and the fetch tally."""
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
    torch.cuda.empty_cache()


def lds_plan(M, N, K, d):
    """The plan, asserting it is the LDS-staged kernel (8 waves, 32-row tiles,
    one workgroup per CU per round)."""
    p = tl.tl_gemm_plan(M, N, K, d)
    assert p["kernel"] == 1 and p["waves"] == 8 and p["tile_n"] == 32 and p["workgroups"] % 256 == 0, p
    return p


def run(A_bits, W_bits, d, fetch=tl.TL_FETCH_BLOCK):
    import torch
    M, K = A_bits.shape
    N = W_bits.shape[0]
    W = dev_bf16(W_bits)
    Wt = torch.empty(tl.padded_shape(N, K, 2, d.G, d.block_rows), dtype=torch.bfloat16, device="cuda")
    tl.tl_repack(W, Wt, N, K, 2, d.G, d.block_rows)
    out_dt = torch.bfloat16 if d.out_dtype == tl.TL_OUT_BF16 else torch.float32
    C = torch.full((M, N), float("nan"), dtype=out_dt, device="cuda")
    tl.tl_gemm(dev_bf16(A_bits), Wt, C, M, N, K, d, fetch)
    torch.cuda.synchronize()
    return C


# (M, N, K): tiles per workgroup T and K splits S the planner picks
LDS_SHAPES = [
    (32, 32768, 2048),     # T = 4, S = 1
    (17, 8192, 16384),     # T = 4, S = 4, 8 chunks per split
    (24, 10240, 8192),     # T = 5, S = 4 (Llama QKV)
    (32, 57344, 2048),     # T = 7, S = 1 (Llama gate+up rows)
    (20, 8192, 28672),     # T = 4, S = 4, 14 chunks per split (Llama down)
]


@pytest.mark.parametrize("M,N,K", LDS_SHAPES)
def test_lds_decode_parity(M, N, K):
    d = tl.layout()
    p = lds_plan(M, N, K, d)
    banner(f"lds decode M={M} N={N} K={K} split_k={p['split_k']} wgs={p['workgroups']}")
    A = synth.normal_bf16((M, K), seed=300 + M)
    W = synth.normal_bf16((N, K), seed=301 + N % 97, sigma=synth.W_SIGMA)
    parity(host_f32(run(A, W, d)), oracle.gemm_f64(A, W), f"lds M={M} N={N} K={K}")


@pytest.mark.parametrize("M", [17, 25, 32])
def test_lds_decode_exact_inputs_and_reproducible(M):
    """Small integers: every partial sum is an exact fp32 integer, so the
    result equals the oracle bit for bit (split-K partials included); one-hot
    rows pick single weights; two runs are bitwise identical."""
    N, K = 8192, 16384
    d = tl.layout()
    lds_plan(M, N, K, d)
    banner(f"lds decode exact M={M}")
    Ai = synth.small_int_bf16((M, K), seed=310 + M)
    Wi = synth.small_int_bf16((N, K), seed=311)
    C1 = host_f32(run(Ai, Wi, d))
    assert np.array_equal(C1.astype(np.float64), oracle.gemm_f64(Ai, Wi))
    assert np.array_equal(host_f32(run(Ai, Wi, d)), C1)
    Ah, _ = synth.one_hot_bf16(M, K, seed=312 + M)
    W = synth.normal_bf16((N, K), seed=313, sigma=synth.W_SIGMA)
    assert np.array_equal(host_f32(run(Ah, W, d)).astype(np.float64), oracle.gemm_f64(Ah, W))


def test_lds_decode_bf16_output():
    M, N, K = 32, 8192, 16384
    d = tl.layout(out_dtype=tl.TL_OUT_BF16)
    lds_plan(M, N, K, d)
    banner("lds decode bf16 out")
    A = synth.normal_bf16((M, K), seed=320)
    W = synth.normal_bf16((N, K), seed=321, sigma=synth.W_SIGMA)
    parity_bf16_out(host_bits(run(A, W, d)), oracle.gemm_f64(A, W), "lds bf16")


@pytest.mark.parametrize("G,br", [(4096, 8), (4096, 16), (16384, 32), (1024, 8), (512, 4), (512, 32), (1024, 16)])
def test_lds_decode_memory_tile_shapes(G, br):
    """Memory tiles narrower or wider than a 64-column step (block_cols 256,
    128, 256, 64, 64, 8, 32): a 32-row tile spans 32 / block_rows strips, and
    a step spans several memory tiles when block_cols < 64."""
    M, N, K = 32, 32768, 2048
    d = tl.layout(G=G, block_rows=br)
    lds_plan(M, N, K, d)
    banner(f"lds decode G={G} br={br}")
    A = synth.normal_bf16((M, K), seed=330)
    W = synth.normal_bf16((N, K), seed=331, sigma=synth.W_SIGMA)
    parity(host_f32(run(A, W, d)), oracle.gemm_f64(A, W), f"lds G={G} br={br}")


def test_lds_decode_fetch_tally_equals_read_amp():
    """Every weight byte is fetched once: the kernel's tally equals the exact
    count for the plan's tile."""
    import torch
    M, N, K = 32, 10240, 8192
    d = tl.layout()
    p = lds_plan(M, N, K, d)
    banner("lds decode fetch tally")
    A = synth.normal_bf16((M, K), seed=340)
    W = synth.normal_bf16((N, K), seed=341, sigma=synth.W_SIGMA)
    tl.tl_fetch_counter_read()
    run(A, W, d, tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    got = tl.tl_fetch_counter_read()
    amp = tl.tl_read_amp(16, N, K, 16, p["tile_n"], p["tile_k"], d, 4096)
    assert got == amp["fetched_bytes"] == 2 * N * K
    torch.cuda.synchronize()


# 33 <= M <= 64: four M tiles, T = 4 tiles per workgroup, 64 KB chunks of A
# (M, N, K, G, block_rows, split_k, workgroups): 64 groups x 4 K ranges,
# 80 groups x 3 uneven ranges (13 chunks: 4, 4, 5), 224 groups unsplit, a
# ragged M with 16-row memory tiles of 1 KB (block_cols 32: a step spans two)
# and one with 256-column memory tiles.
LDS64_SHAPES = [(33, 8192, 8192, 4096, 32, 4, 256), (64, 10240, 6656, 4096, 32, 3, 240),
                (48, 28672, 2048, 4096, 32, 1, 224), (37, 8192, 8192, 1024, 16, 4, 256),
                (57, 16384, 4096, 16384, 32, 2, 256)]


@pytest.mark.parametrize("M,N,K,G,br,S,wgs", LDS64_SHAPES)
def test_lds_decode_four_m_tiles(M, N, K, G, br, S, wgs):
    d = tl.layout(G=G, block_rows=br)
    p = tl.tl_gemm_plan(M, N, K, d)
    banner(f"lds decode four M tiles M={M} N={N} K={K} G={G} br={br} plan={p}")
    assert (p["kernel"], p["tile_m"], p["tile_n"], p["waves"], p["split_k"], p["workgroups"]) == (1, 64, 32, 8, S, wgs)
    A = synth.normal_bf16((M, K), seed=350 + M)
    W = synth.normal_bf16((N, K), seed=351, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    C1 = host_f32(run(A, W, d))
    parity(C1, y_ref, f"lds four M tiles M={M}")
    assert np.array_equal(C1, host_f32(run(A, W, d)))       # fixed-order sums: bitwise reproducible
    db = tl.layout(G=G, block_rows=br, out_dtype=tl.TL_OUT_BF16)
    parity_bf16_out(host_bits(run(A, W, db)), y_ref, f"lds four M tiles M={M} bf16")
    Ai = synth.small_int_bf16((M, K), seed=352 + M)
    Wi = synth.small_int_bf16((N, K), seed=353)
    assert np.array_equal(host_f32(run(Ai, Wi, d)).astype(np.float64), oracle.gemm_f64(Ai, Wi))


def test_lds_decode_four_m_tiles_fetch_tally():
    import torch
    M, N, K = 64, 8192, 8192
    d = tl.layout()
    p = tl.tl_gemm_plan(M, N, K, d)
    assert p["tile_n"] == 32 and p["waves"] == 8
    banner("lds decode four M tiles fetch tally")
    A = synth.normal_bf16((M, K), seed=360)
    W = synth.normal_bf16((N, K), seed=361, sigma=synth.W_SIGMA)
    tl.tl_fetch_counter_read()
    run(A, W, d, tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    got = tl.tl_fetch_counter_read()
    assert got == 2 * N * K
    torch.cuda.synchronize()
