"""GPU parity for weights whose dimensions are not multiples of the memory
tile's sides: the copy is padded to whole memory tiles (Section 3.3).  The
repack is bit-exact against the oracle's padded copy (zeros in the padding)
and round-trips; every GEMM kernel (decode, FP8 decode, grouped, prefill)
meets the parity gate on ragged N and K, bit-exact on exact inputs; the
fetch tally of a padded weight."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, dev_u8, host_bits, host_f32, parity, parity_bf16_out

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.synchronize()


def _sync():
    import torch
    torch.cuda.synchronize()


def tile_major(W_dev, N, K, s, G, br):
    """Padded tile-major copy of a device weight, in a buffer of exactly
    tl_tile_bytes bytes."""
    import torch
    nbytes = tl.tl_tile_bytes(N, K, s, G, br)
    out = torch.empty(nbytes // W_dev.element_size(), dtype=W_dev.dtype, device="cuda")
    tl.tl_repack(W_dev, out, N, K, s, G, br)
    return out


# ---------------------------------------------------------------------------
# Repack
# ---------------------------------------------------------------------------

PADDED_REPACK = [
    # rows, cols, elem_bytes, G, block_rows
    (40, 100, 2, 4096, 32), (1000, 1000, 2, 4096, 32), (50257, 72, 2, 4096, 32),
    (7, 24, 2, 4096, 32), (33, 200, 1, 4096, 64), (100, 200, 2, 512, 8),
    (65, 264, 2, 16384, 16), (3, 5, 4, 1024, 4), (9, 13, 1, 4096, 64),   # odd row bytes: 1-byte chunks
    (130, 70, 2, 4096, 64),                                            # bc = 32
]


@pytest.mark.parametrize("rows,cols,s,G,br", PADDED_REPACK)
def test_padded_repack_bit_exact(rows, cols, s, G, br):
    import torch
    banner(f"padded repack rows={rows} cols={cols} s={s} G={G} br={br}")
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[s]
    src = synth.random_bytes(rows * cols * s, seed=rows + cols * 3 + G).view(dt).reshape(rows, cols)
    want = oracle.repack(src, G, br).view(np.uint8).reshape(-1)
    nbytes = tl.tl_tile_bytes(rows, cols, s, G, br)
    assert nbytes == want.size
    d_src = dev_u8(src.view(np.uint8).reshape(-1))
    d_dst = torch.full((nbytes,), 0xA5, dtype=torch.uint8, device="cuda")   # padding must be overwritten
    tl.tl_repack(d_src, d_dst, rows, cols, s, G, br)
    assert np.array_equal(host_bits(d_dst), want)
    d_back = torch.full((rows * cols * s,), 0x5A, dtype=torch.uint8, device="cuda")
    tl.tl_unpack(d_dst, d_back, rows, cols, s, G, br)
    assert np.array_equal(host_bits(d_back), src.view(np.uint8).reshape(-1))


# ---------------------------------------------------------------------------
# Decode (M <= 64)
# ---------------------------------------------------------------------------

def run_padded(A_bits, W_bits, desc, fetch=tl.TL_FETCH_BLOCK, tile_major_w=True):
    import torch
    M, K = A_bits.shape
    N = W_bits.shape[0]
    W = dev_bf16(W_bits)
    if tile_major_w:
        W = tile_major(W, N, K, 2, desc.G, desc.block_rows)
    out_dt = torch.bfloat16 if desc.out_dtype == tl.TL_OUT_BF16 else torch.float32
    C = torch.full((M, N), float("nan"), dtype=out_dt, device="cuda")
    tl.tl_gemm(dev_bf16(A_bits), W, C, M, N, K, desc, fetch)
    _sync()
    return C


DECODE_SHAPES = [
    # M, N, K: ragged N, ragged K (K % 8 == 0), both, K < 64, a last partial step
    (1, 100, 200), (8, 1000, 1000), (5, 33, 72), (17, 70, 4104), (64, 300, 520),
    (8, 40, 8), (32, 8200, 1032), (3, 8, 56),
]


@pytest.mark.parametrize("M,N,K", DECODE_SHAPES)
def test_decode_padded_parity(M, N, K):
    banner(f"padded decode M={M} N={N} K={K}")
    A = synth.normal_bf16((M, K), seed=M + N)
    W = synth.normal_bf16((N, K), seed=N + K, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    parity(host_f32(run_padded(A, W, tl.layout())), y_ref, f"M={M} N={N} K={K}")
    Ai = synth.small_int_bf16((M, K), seed=3)
    Wi = synth.small_int_bf16((N, K), seed=4)
    assert np.array_equal(host_f32(run_padded(Ai, Wi, tl.layout())).astype(np.float64), oracle.gemm_f64(Ai, Wi))


@pytest.mark.parametrize("G,br", [(4096, 64), (4096, 8), (512, 8), (1024, 16), (16384, 32), (4096, 16)])
@pytest.mark.parametrize("M", [4, 24])
def test_decode_padded_memory_tile_shapes(G, br, M):
    """block_cols 32 (fewer than one 64-wide step), 256 and 512; block_rows
    8 to 64; N and K ragged against every one of them."""
    N, K = 200, 1000
    banner(f"padded decode G={G} br={br} M={M}")
    A = synth.normal_bf16((M, K), seed=G + br)
    W = synth.normal_bf16((N, K), seed=br, sigma=synth.W_SIGMA)
    parity(host_f32(run_padded(A, W, tl.layout(G=G, block_rows=br))), oracle.gemm_f64(A, W), f"G={G} br={br}")


@pytest.mark.parametrize("split_k", [1, 2, 3, 7])
def test_decode_padded_split_k_exact_and_reproducible(split_k):
    """Ragged K split across workgroups (the partial step falls in the last
    split); the partials of an odd M x N are 16-byte aligned per split."""
    M, N, K = 7, 1001, 3000
    banner(f"padded decode split_k={split_k}")
    d = tl.layout(split_k=split_k)
    A = synth.normal_bf16((M, K), seed=9)
    W = synth.normal_bf16((N, K), seed=10, sigma=synth.W_SIGMA)
    C1 = host_f32(run_padded(A, W, d))
    parity(C1, oracle.gemm_f64(A, W), f"split_k={split_k}")
    assert np.array_equal(C1, host_f32(run_padded(A, W, d)))
    Ai = synth.small_int_bf16((M, K), seed=11)
    Wi = synth.small_int_bf16((N, K), seed=12)
    assert np.array_equal(host_f32(run_padded(Ai, Wi, d)).astype(np.float64), oracle.gemm_f64(Ai, Wi))


@pytest.mark.parametrize("split_k", [1, 4])
def test_decode_padded_bf16_out_and_one_hot(split_k):
    M, N, K = 9, 777, 1224
    banner(f"padded decode bf16 out / one-hot split_k={split_k}")
    A = synth.normal_bf16((M, K), seed=21)
    W = synth.normal_bf16((N, K), seed=22, sigma=synth.W_SIGMA)
    C = run_padded(A, W, tl.layout(out_dtype=tl.TL_OUT_BF16, split_k=split_k))
    parity_bf16_out(host_bits(C), oracle.gemm_f64(A, W), "bf16 out")
    A1, ks = synth.one_hot_bf16(M, K, seed=23)
    got = host_f32(run_padded(A1, W, tl.layout(split_k=split_k)))
    assert np.array_equal(got, synth.bf16_bits_to_f32(W[:, ks].T))


def test_decode_padded_row_major_native():
    M, N, K = 8, 999, 1000
    banner("padded decode row-major native")
    A = synth.normal_bf16((M, K), seed=31)
    W = synth.normal_bf16((N, K), seed=32, sigma=synth.W_SIGMA)
    C = run_padded(A, W, tl.layout(kind=tl.TL_LAYOUT_NK_ROW), fetch=tl.TL_FETCH_NATIVE, tile_major_w=False)
    parity(host_f32(C), oracle.gemm_f64(A, W), "row-major")


def test_decode_padded_fetch_tally():
    """The kernel issues whole 32 x 64 memory-tile steps over the padded copy
    of its clamped rows: tiles x steps x 4 KB."""
    import torch
    M, N, K = 8, 100, 200
    banner("padded decode fetch tally")
    A = synth.normal_bf16((M, K), seed=41)
    W = synth.normal_bf16((N, K), seed=42, sigma=synth.W_SIGMA)
    d = tl.layout(split_k=1)
    Wt = tile_major(dev_bf16(W), N, K, 2, 4096, 32)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    tl.tl_fetch_counter_read()
    tl.tl_gemm(dev_bf16(A), Wt, C, M, N, K, d, tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    got = tl.tl_fetch_counter_read()
    assert got == 4 * 4 * 4096          # ceil(100 / 32) tiles x ceil(200 / 64) steps x 4 KB
    parity(host_f32(C), oracle.gemm_f64(A, W), "tally run")


def test_gpt2_lm_head_shape():
    """A real ragged shape: GPT-2's LM head [50257, 768] at M = 8."""
    M, N, K = 8, 50257, 768
    banner("padded decode GPT-2 LM head")
    A = synth.normal_bf16((M, K), seed=51)
    W = synth.normal_bf16((N, K), seed=52, sigma=synth.W_SIGMA)
    parity(host_f32(run_padded(A, W, tl.layout())), oracle.gemm_f64(A, W), "lm head")


# ---------------------------------------------------------------------------
# FP8 decode
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("M,N,K", [(1, 100, 208), (8, 1000, 1008), (33, 70, 4112)])
@pytest.mark.parametrize("scaled", [False, True])
def test_fp8_padded_parity(M, N, K, scaled):
    import torch
    banner(f"padded fp8 M={M} N={N} K={K} scaled={scaled}")
    A = synth.normal_bf16((M, K), seed=61 + M)
    W8, sc = synth.fp8_weights((N, K), seed=62)
    scales = sc if scaled else None
    Wt = tile_major(dev_u8(W8), N, K, 1, 4096, 64)
    d_sc = None if scales is None else torch.from_numpy(np.ascontiguousarray(scales, dtype=np.float32)).cuda()
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    tl.tl_gemm_w8(dev_bf16(A), Wt, d_sc, C, M, N, K, tl.layout(elem_bytes=1, G=4096, block_rows=64),
                  tl.TL_FETCH_BLOCK)
    _sync()
    parity(host_f32(C), oracle.gemm_w8_f64(A, W8, scales), "fp8 padded")


# ---------------------------------------------------------------------------
# Grouped (stacked experts)
# ---------------------------------------------------------------------------

def test_grouped_padded_experts():
    import torch
    E, N, K = 6, 100, 200
    banner("padded grouped experts")
    Ws = [synth.normal_bf16((N, K), seed=70 + e, sigma=synth.W_SIGMA) for e in range(E)]
    stride = tl.tl_tile_bytes(N, K, 2, 4096, 32)
    stack = torch.empty((E * stride // 2,), dtype=torch.bfloat16, device="cuda")
    for e, W in enumerate(Ws):
        tl.tl_repack(dev_bf16(W), stack[e * stride // 2:(e + 1) * stride // 2], N, K, 2, 4096, 32)
    offsets = np.array([0, 3, 3, 10, 11, 30, 34], dtype=np.int32)      # an empty group, a 19-row group
    T = int(offsets[-1])
    A = synth.normal_bf16((20, K), seed=79)
    ids = np.random.default_rng(5).integers(0, 20, T).astype(np.int32)
    C = torch.full((T, N), float("nan"), dtype=torch.float32, device="cuda")
    tl.tl_gemm_grouped(dev_bf16(A), 20, torch.from_numpy(ids).cuda(), torch.from_numpy(offsets).cuda(), E, T, 19,
                       stack, stride, C, N, K, tl.layout(), tl.TL_FETCH_BLOCK)
    _sync()
    parity(host_f32(C), oracle.grouped_gemm_f64(A, ids, offsets, Ws), "grouped padded")


# ---------------------------------------------------------------------------
# Prefill (M > 64)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("M,N,K,tm,tn", [(300, 1000, 1000, 128, 128), (513, 700, 1032, 256, 128),
                                        (1024, 520, 2056, 256, 256), (100, 130, 72, 128, 128)])
def test_prefill_padded_parity(M, N, K, tm, tn):
    banner(f"padded prefill M={M} N={N} K={K} tile {tm}x{tn}")
    A = synth.normal_bf16((M, K), seed=M + 1)
    W = synth.normal_bf16((N, K), seed=N + 2, sigma=synth.W_SIGMA)
    parity(host_f32(run_padded(A, W, tl.layout(tile_m=tm, tile_n=tn))), oracle.gemm_f64(A, W),
           f"prefill {M}x{N}x{K}")
    Ai = synth.small_int_bf16((M, K), seed=5)
    Wi = synth.small_int_bf16((N, K), seed=6)
    assert np.array_equal(host_f32(run_padded(Ai, Wi, tl.layout(tile_m=tm, tile_n=tn))).astype(np.float64),
                          oracle.gemm_f64(Ai, Wi))


@pytest.mark.parametrize("G,br", [(4096, 64), (512, 8), (16384, 64)])
def test_prefill_padded_memory_tile_shapes(G, br):
    M, N, K = 256, 300, 1000
    banner(f"padded prefill G={G} br={br}")
    A = synth.normal_bf16((M, K), seed=G)
    W = synth.normal_bf16((N, K), seed=br, sigma=synth.W_SIGMA)
    C = run_padded(A, W, tl.layout(G=G, block_rows=br, out_dtype=tl.TL_OUT_BF16))
    parity_bf16_out(host_bits(C), oracle.gemm_f64(A, W), f"G={G} br={br}")


def test_prefill_padded_row_major():
    M, N, K = 200, 300, 1000
    banner("padded prefill row-major")
    A = synth.normal_bf16((M, K), seed=91)
    W = synth.normal_bf16((N, K), seed=92, sigma=synth.W_SIGMA)
    C = run_padded(A, W, tl.layout(kind=tl.TL_LAYOUT_NK_ROW), fetch=tl.TL_FETCH_NATIVE, tile_major_w=False)
    parity(host_f32(C), oracle.gemm_f64(A, W), "prefill row-major")
