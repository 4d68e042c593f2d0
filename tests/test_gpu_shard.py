"""Tensor-parallel shards of tile-major weights against the oracle.  A row
shard (output rows [r N/TP, (r+1) N/TP)) of a tile-major weight is a
zero-copy byte range of the whole copy, because a strip of block_rows rows is
contiguous: tl_gemm on that range must equal the oracle on those rows of the
row-major weight.  A column shard (input columns [r K/TP, (r+1) K/TP)) is
repacked on its own; the ranks' partial outputs summed (the all-reduce, here
on the host in fp64) must equal the oracle on the whole weight.  Shapes are
one GPU's share of the Llama-70B projections at TP = 2, 4 and 8 -- tile
counts that do not divide the CUs, which the planner fills one round of the
CUs with -- at M = 1, 8 and 32; small-integer inputs make both bit-exact."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, host_f32, parity

pytestmark = pytest.mark.gpu
G, BR = 4096, 32


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.empty_cache()


def repacked(W_bits):
    import torch
    N, K = W_bits.shape
    Wt = torch.empty((N, K), dtype=torch.bfloat16, device="cuda")
    tl.tl_repack(dev_bf16(W_bits), Wt, N, K, 2, G, BR)
    return Wt


def gemm(A_bits, W_dev, N, K):
    import torch
    M = A_bits.shape[0]
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    tl.tl_gemm(dev_bf16(A_bits), W_dev, C, M, N, K, tl.layout(G=G, block_rows=BR), tl.TL_FETCH_BLOCK)
    torch.cuda.synchronize()
    return host_f32(C)


# (TP, rows of one shard, K): QKV and gate+up shards; the whole weight holds
# the first two or three ranks' shards
ROW_CASES = [(4, 2560, 8192), (8, 1280, 8192), (2, 5120, 8192), (8, 7168, 8192), (4, 14336, 8192)]


@pytest.mark.parametrize("M", [1, 8, 32])
@pytest.mark.parametrize("tp,Nr,K", ROW_CASES)
def test_row_shard_is_a_zero_copy_slice(tp, Nr, K, M):
    ranks = min(tp, 3) if Nr <= 5120 else 2
    W = synth.normal_bf16((ranks * Nr, K), seed=500 + Nr % 97, sigma=synth.W_SIGMA)
    A = synth.normal_bf16((M, K), seed=510 + M)
    Wt = repacked(W)
    p = tl.tl_gemm_plan(M, Nr, K, tl.layout(G=G, block_rows=BR))
    for r in range(ranks):
        banner(f"row shard tp={tp} rank={r} M={M} N={Nr} K={K} plan={p}")
        part = Wt.view(-1).narrow(0, r * Nr * K, Nr * K)
        parity(gemm(A, part, Nr, K), oracle.gemm_f64(A, W[r * Nr:(r + 1) * Nr]), f"row shard tp={tp} r={r} M={M}")


@pytest.mark.parametrize("M", [8, 32])
def test_row_shard_exact(M):
    tp, Nr, K = 4, 2560, 8192
    W = synth.small_int_bf16((2 * Nr, K), seed=520)
    A = synth.small_int_bf16((M, K), seed=521 + M)
    Wt = repacked(W)
    banner(f"row shard exact M={M}")
    part = Wt.view(-1).narrow(0, Nr * K, Nr * K)
    assert np.array_equal(gemm(A, part, Nr, K).astype(np.float64), oracle.gemm_f64(A, W[Nr:]))


def column_shard_outputs(A, W, tp):
    N, K = W.shape
    Kr = K // tp
    outs = []
    for r in range(tp):
        Wr = np.ascontiguousarray(W[:, r * Kr:(r + 1) * Kr])
        outs.append(gemm(np.ascontiguousarray(A[:, r * Kr:(r + 1) * Kr]), repacked(Wr), N, Kr).astype(np.float64))
    return outs


@pytest.mark.parametrize("M", [1, 8, 32])
@pytest.mark.parametrize("tp,N,K", [(8, 8192, 8192), (2, 8192, 8192), (4, 8192, 28672)])
def test_column_shards_sum_to_the_whole(tp, N, K, M):
    W = synth.normal_bf16((N, K), seed=530 + K % 89, sigma=synth.W_SIGMA)
    A = synth.normal_bf16((M, K), seed=540 + M)
    banner(f"column shards tp={tp} M={M} N={N} K={K} plan={tl.tl_gemm_plan(M, N, K // tp, tl.layout())}")
    parity(sum(column_shard_outputs(A, W, tp)), oracle.gemm_f64(A, W), f"column shards tp={tp} M={M}")


def test_column_shards_exact():
    tp, N, K, M = 8, 8192, 8192, 8
    W = synth.small_int_bf16((N, K), seed=550)
    A = synth.small_int_bf16((M, K), seed=551)
    banner("column shards exact")
    assert np.array_equal(sum(column_shard_outputs(A, W, tp)), oracle.gemm_f64(A, W))
