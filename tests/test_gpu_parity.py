"""GPU parity: libtl's HIP kernels, called through the C ABI, against the CPU
oracle on the same seeded inputs.  Repack and amplification counts must be
bit-exact; GEMMs meet relative L2 <= 1e-3 and max abs <= 5e-3 * max|y_ref|,
and are bit-exact where the exact result is representable (one-hot and
small-integer inputs)."""
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


# ---------------------------------------------------------------------------
# Repack
# ---------------------------------------------------------------------------

REPACK_SMALL = [
    # rows, cols, elem_bytes, G, block_rows
    (1024, 1024, 2, 4096, 32),       # tiny config
    (256, 2048, 2, 512, 8), (256, 2048, 2, 512, 16), (256, 2048, 2, 512, 32), (256, 2048, 2, 512, 64),
    (256, 2048, 2, 1024, 8), (256, 2048, 2, 1024, 16), (256, 2048, 2, 1024, 32), (256, 2048, 2, 1024, 64),
    (256, 2048, 2, 4096, 8), (256, 2048, 2, 4096, 16), (256, 2048, 2, 4096, 32), (256, 2048, 2, 4096, 64),
    (256, 2048, 2, 16384, 8), (256, 2048, 2, 16384, 16), (256, 2048, 2, 16384, 32), (256, 2048, 2, 16384, 64),
    (256, 2048, 2, 512, 4), (256, 2048, 2, 1024, 4), (256, 2048, 2, 4096, 4), (256, 2048, 2, 16384, 4),   # 4-row tiles
    (192, 768, 1, 4096, 64),         # FP8-sized elements, 64 x 64 memory tile
    (64, 4096, 4, 4096, 8),
    (32, 64, 2, 4096, 32),           # a single memory tile
]


@pytest.mark.parametrize("rows,cols,s,G,br", REPACK_SMALL)
def test_repack_bit_exact_small(rows, cols, s, G, br):
    banner(f"repack rows={rows} cols={cols} s={s} G={G} br={br}")
    src = synth.random_bytes(rows * cols * s, seed=rows * 7 + cols + G + br).reshape(rows, cols * s)
    want = oracle.repack(src.view({1: np.uint8, 2: np.uint16, 4: np.uint32}[s]).reshape(rows, cols),
                         G, br).view(np.uint8).reshape(rows, cols * s)
    d_src = dev_u8(src)
    d_dst = dev_u8(np.zeros_like(src))
    tl.tl_repack(d_src, d_dst, rows, cols, s, G, br)
    got = host_bits(d_dst)
    assert np.array_equal(got, want)
    d_back = dev_u8(np.zeros_like(src))
    tl.tl_unpack(d_dst, d_back, rows, cols, s, G, br)
    assert np.array_equal(host_bits(d_back), src)


@pytest.mark.parametrize("name,N,K", synth.LLAMA70B)
def test_repack_full_size_llama(name, N, K):
    """Full Llama-70B weight shapes: exact round trip, plus 4096 sampled
    elements placed where the oracle's Eq. 2 offset says."""
    import torch
    banner(f"repack full {name} [{N},{K}]")
    W = torch.randint(-32768, 32767, (N, K), dtype=torch.int16, device="cuda",
                      generator=torch.Generator(device="cuda").manual_seed(5))
    Wt = torch.empty_like(W)
    tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
    back = torch.empty_like(W)
    tl.tl_unpack(Wt, back, N, K, 2, 4096, 32)
    assert torch.equal(back, W)
    rng = np.random.default_rng(1)
    rs = rng.integers(0, N, 4096)
    cs = rng.integers(0, K, 4096)
    offs = np.array([oracle.tm_offset(int(r), int(c), K, 2, 4096, 32) // 2 for r, c in zip(rs, cs)])
    flat = Wt.view(-1)
    got = flat[torch.from_numpy(offs).cuda()].cpu().numpy()
    want = W[torch.from_numpy(rs).cuda(), torch.from_numpy(cs).cuda()].cpu().numpy()
    assert np.array_equal(got, want)


# ---------------------------------------------------------------------------
# GEMM helpers
# ---------------------------------------------------------------------------

def run_gemm(A_bits, W_bits, desc, fetch=tl.TL_FETCH_BLOCK, tile_major=True):
    """Upload, (repack), run tl_gemm; returns the output tensor."""
    import torch
    M, K = A_bits.shape
    N = W_bits.shape[0]
    A = dev_bf16(A_bits)
    W = dev_bf16(W_bits)
    if tile_major:
        Wt = torch.empty_like(W)
        tl.tl_repack(W, Wt, N, K, 2, desc.G, desc.block_rows)
        W = Wt
    out_dt = torch.bfloat16 if desc.out_dtype == tl.TL_OUT_BF16 else torch.float32
    C = torch.full((M, N), float("nan"), dtype=out_dt, device="cuda")
    tl.tl_gemm(A, W, C, M, N, K, desc, fetch)
    _sync()
    return C


DECODE_SHAPES = [
    # M, N, K
    (16, 1024, 1024),     # tiny config
    (1, 1024, 1024), (5, 512, 2048), (8, 1024, 1024), (17, 256, 1024), (32, 512, 1024),
    (33, 256, 512), (48, 128, 4096), (64, 256, 1024),
]


@pytest.mark.parametrize("M,N,K", DECODE_SHAPES)
def test_decode_tile_major_parity(M, N, K):
    banner(f"decode tile-major M={M} N={N} K={K}")
    A = synth.normal_bf16((M, K), seed=1 + M)
    W = synth.normal_bf16((N, K), seed=2 + N, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    C = run_gemm(A, W, tl.layout())
    parity(host_f32(C), y_ref, f"decode M={M}")


@pytest.mark.parametrize("M", [1, 8, 32, 64])
@pytest.mark.parametrize("N", [8192, 16384])
def test_decode_in_workgroup_k_split(M, N):
    """256 or 512 tiles: one workgroup per tile, 16 or 8 waves splitting K."""
    K = 1024
    d = tl.layout(tile_n=32)
    p = tl.tl_gemm_plan(M, N, K, d)
    banner(f"decode M={M} N={N} waves={p['waves']} split_k={p['split_k']}")
    assert p["split_k"] == 1 and p["waves"] in (8, 16)
    A = synth.normal_bf16((M, K), seed=60 + M)
    W = synth.normal_bf16((N, K), seed=61, sigma=synth.W_SIGMA)
    parity(host_f32(run_gemm(A, W, d)), oracle.gemm_f64(A, W), f"M={M} N={N}")
    Ai = synth.small_int_bf16((M, K), seed=62)
    Wi = synth.small_int_bf16((N, K), seed=63)
    assert np.array_equal(host_f32(run_gemm(Ai, Wi, d)).astype(np.float64), oracle.gemm_f64(Ai, Wi))


# 33 <= M <= 64 on 64-row tiles (four 16-row M tiles, one K step in flight
# per wave): M, N, K, waves, split_k of the plan.  One 8-wave workgroup per
# CU with split_k 2 and 1, a 320-tile grid with 8 waves, and 4-wave
# workgroups (768 of them).
MID_M_DECODE = [(33, 8192, 2048, 8, 2), (64, 16384, 2048, 8, 1), (48, 10240, 2048, 8, 2), (40, 24576, 2048, 4, 2)]


@pytest.mark.parametrize("M,N,K,waves,S", MID_M_DECODE)
def test_decode_four_m_tiles(M, N, K, waves, S):
    d = tl.layout()
    p = tl.tl_gemm_plan(M, N, K, d)
    banner(f"decode four M tiles M={M} N={N} K={K} plan={p}")
    assert (p["kernel"], p["tile_m"], p["tile_n"], p["waves"], p["split_k"]) == (1, 64, 64, waves, S)
    A = synth.normal_bf16((M, K), seed=180 + M)
    W = synth.normal_bf16((N, K), seed=181, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    C1 = host_f32(run_gemm(A, W, d))
    parity(C1, y_ref, f"four M tiles M={M}")
    assert np.array_equal(C1, host_f32(run_gemm(A, W, d)))       # fixed-order sums: bitwise reproducible
    db = tl.layout(out_dtype=tl.TL_OUT_BF16)
    parity_bf16_out(host_bits(run_gemm(A, W, db)), y_ref, f"four M tiles M={M} bf16")
    Ai = synth.small_int_bf16((M, K), seed=182)
    Wi = synth.small_int_bf16((N, K), seed=183)
    assert np.array_equal(host_f32(run_gemm(Ai, Wi, d)).astype(np.float64), oracle.gemm_f64(Ai, Wi))


# 33 <= M <= 64 on a wide weight (N >= 32768): the prefill kernel's 128 x 128
# tiles.  M, N, K, row-major [N][K] weight; a ragged N (N % 128 = 96).
MID_M_WIDE = [(33, 32768, 512, False), (48, 32768 + 96, 1024, False), (64, 40960, 512, True), (40, 57344, 256, False)]


@pytest.mark.parametrize("M,N,K,row_major", MID_M_WIDE)
def test_mid_m_wide_weight_on_prefill_tiles(M, N, K, row_major):
    kind = tl.TL_LAYOUT_NK_ROW if row_major else tl.TL_LAYOUT_TILE
    fetch = tl.TL_FETCH_NATIVE if row_major else tl.TL_FETCH_BLOCK
    d = tl.layout(kind=kind)
    p = tl.tl_gemm_plan(M, N, K, d, fetch)
    banner(f"mid-M wide weight M={M} N={N} K={K} row_major={row_major} plan={p}")
    assert (p["kernel"], p["tile_m"], p["tile_n"], p["split_k"]) == (2, 128, 128, 1)
    assert p["workgroups"] == -(-N // 128) and p["workspace_bytes"] == 0
    A = synth.normal_bf16((M, K), seed=190 + M)
    W = synth.normal_bf16((N, K), seed=191, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    parity(host_f32(run_gemm(A, W, d, fetch=fetch, tile_major=not row_major)), y_ref, f"mid-M wide M={M}")
    db = tl.layout(kind=kind, out_dtype=tl.TL_OUT_BF16)
    parity_bf16_out(host_bits(run_gemm(A, W, db, fetch=fetch, tile_major=not row_major)), y_ref,
                    f"mid-M wide M={M} bf16")
    Ai = synth.small_int_bf16((M, K), seed=192)
    Wi = synth.small_int_bf16((N, K), seed=193)
    assert np.array_equal(host_f32(run_gemm(Ai, Wi, d, fetch=fetch, tile_major=not row_major)).astype(np.float64),
                          oracle.gemm_f64(Ai, Wi))


@pytest.mark.parametrize("split_k", [1, 2, 3, 7, 16])
def test_decode_split_k_parity_and_reproducible(split_k):
    M, N, K = 8, 512, 4096
    banner(f"decode split_k={split_k}")
    A = synth.normal_bf16((M, K), seed=3)
    W = synth.normal_bf16((N, K), seed=4, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    d = tl.layout(split_k=split_k)
    C1 = host_f32(run_gemm(A, W, d))
    C2 = host_f32(run_gemm(A, W, d))
    parity(C1, y_ref, f"split_k={split_k}")
    assert np.array_equal(C1, C2)    # fixed-order reduction: bitwise reproducible


def test_decode_split_k_interleaved_calls():
    """Split calls of different shapes and split counts, back to back on one
    stream with no synchronisation: consecutive calls share the stream's
    split-K workspace (partials, then the reduce kernel), so every call must
    equal the same call made alone."""
    banner("decode split-K interleaved calls")
    cases = [(8, 512, 4096, 3), (1, 1024, 2048, 7), (8, 512, 4096, 2), (32, 256, 8192, 16), (8, 512, 4096, 3)]
    alone = {}
    for (M, N, K, S) in cases:
        A = synth.normal_bf16((M, K), seed=M + N)
        W = synth.normal_bf16((N, K), seed=K, sigma=synth.W_SIGMA)
        alone.setdefault((M, N, K, S), host_f32(run_gemm(A, W, tl.layout(split_k=S))))
    import torch
    outs = []
    for (M, N, K, S) in cases * 2:              # no synchronisation between the calls
        A = dev_bf16(synth.normal_bf16((M, K), seed=M + N))
        W = dev_bf16(synth.normal_bf16((N, K), seed=K, sigma=synth.W_SIGMA))
        Wt = torch.empty_like(W)
        tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        tl.tl_gemm(A, Wt, C, M, N, K, tl.layout(split_k=S), tl.TL_FETCH_BLOCK)
        outs.append(((M, N, K, S), C, A, Wt))
    _sync()
    for key, C, _, _ in outs:
        assert np.array_equal(host_f32(C), alone[key]), key


@pytest.mark.parametrize("M", [1, 8, 32, 64])
def test_decode_one_hot_exact(M):
    """A[m] = e_{k_m}: every output is one weight element, exact in any order."""
    K, N = 2048, 512
    banner(f"decode one-hot M={M}")
    A, ks = synth.one_hot_bf16(M, K, seed=M)
    W = synth.normal_bf16((N, K), seed=9, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    for split_k in (1, 4):
        C = host_f32(run_gemm(A, W, tl.layout(split_k=split_k)))
        assert np.array_equal(C.astype(np.float64), y_ref)


@pytest.mark.parametrize("split_k", [1, 5])
def test_decode_small_integers_exact(split_k):
    """Integers in [-4, 4]: every partial sum is an exact fp32 integer."""
    M, N, K = 24, 256, 4096
    banner(f"decode small-int split_k={split_k}")
    A = synth.small_int_bf16((M, K), seed=5)
    W = synth.small_int_bf16((N, K), seed=6)
    y_ref = oracle.gemm_f64(A, W)
    C = host_f32(run_gemm(A, W, tl.layout(split_k=split_k)))
    assert np.array_equal(C.astype(np.float64), y_ref)


def test_decode_zero_weight():
    banner("decode zero weight")
    A = synth.normal_bf16((8, 1024), seed=7)
    W = np.zeros((256, 1024), dtype=np.uint16)
    C = host_f32(run_gemm(A, W, tl.layout(split_k=2)))
    assert np.all(C == 0.0)


@pytest.mark.parametrize("M", [1, 8, 32])
def test_decode_bf16_output(M):
    N, K = 1024, 2048
    banner(f"decode bf16-out M={M}")
    A = synth.normal_bf16((M, K), seed=11)
    W = synth.normal_bf16((N, K), seed=12, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    for split_k in (1, 4):
        C = run_gemm(A, W, tl.layout(out_dtype=tl.TL_OUT_BF16, split_k=split_k))
        parity_bf16_out(host_bits(C), y_ref, f"bf16 M={M}")


@pytest.mark.parametrize("G", [512, 1024, 4096, 16384])
@pytest.mark.parametrize("br", [4, 8, 16, 32, 64])
def test_decode_memory_tile_shapes(G, br):
    """One library binary for every memory-tile shape (runtime descriptor)."""
    M, N, K = 8, 256, 4096
    if G // (2 * br) < 8:   # memory-tile rows under 16 bytes: rejected before any device work
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_plan(M, N, K, tl.layout(G=G, block_rows=br))
        assert e.value.status == tl.TL_EUNSUPPORTED
        return
    banner(f"decode G={G} br={br}")
    A = synth.normal_bf16((M, K), seed=13)
    W = synth.normal_bf16((N, K), seed=14, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    C = host_f32(run_gemm(A, W, tl.layout(G=G, block_rows=br)))
    parity(C, y_ref, f"G={G} br={br}")


@pytest.mark.parametrize("M", [1, 8, 32])
def test_decode_row_major_native(M):
    N, K = 1024, 2048
    banner(f"decode NK_ROW native M={M}")
    A = synth.normal_bf16((M, K), seed=15)
    W = synth.normal_bf16((N, K), seed=16, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    C = host_f32(run_gemm(A, W, tl.layout(kind=tl.TL_LAYOUT_NK_ROW), fetch=tl.TL_FETCH_NATIVE,
                          tile_major=False))
    parity(C, y_ref, f"NK_ROW M={M}")


@pytest.mark.parametrize("M,N,K,G", [(8, 1024, 2048, 4096), (8, 512, 2048, 512), (1, 256, 4096, 16384),
                                     (8, 512, 1024, 4096), (32, 512, 512, 8192), (5, 256, 2048, 128)])
def test_decode_row_major_block_fetch_emulation(M, N, K, G):
    """Row-major weight read in whole G-byte blocks: same result, and the
    fetch tally equals tl_read_amp's fetched bytes for the kernel's tile
    exactly (rows share a block when K * 2 < G)."""
    banner(f"decode NK_ROW block fetch M={M} N={N} K={K} G={G}")
    A = synth.normal_bf16((M, K), seed=70 + M)
    W = synth.normal_bf16((N, K), seed=71, sigma=synth.W_SIGMA)
    d = tl.layout(kind=tl.TL_LAYOUT_NK_ROW, G=G)
    tl.tl_fetch_counter_read()
    C = run_gemm(A, W, d, fetch=tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT, tile_major=False)
    got = tl.tl_fetch_counter_read()
    parity(host_f32(C), oracle.gemm_f64(A, W), f"block fetch G={G}")
    p = tl.tl_gemm_plan(M, N, K, d, tl.TL_FETCH_BLOCK)
    amp = tl.tl_read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], d, G)
    assert got == amp["fetched_bytes"]
    want = oracle.read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], oracle.NK_ROW, G)
    assert got == want["fetched_bytes"]


def test_decode_issued_weight_bytes_equal_read_amp():
    """Construction check: on a tile-major weight the TL_FETCH_COUNT tally is
    the bytes of the weight loads of every K step the kernel issues, and it
    equals tl_read_amp's fetched bytes for the plan's tile (= N * K * 2: each
    memory tile is loaded once, whole).  The HBM bytes themselves are measured
    by the FETCH_SIZE counter (committed profile); the row- and column-major
    block emulations count the blocks they load."""
    M, N, K = 8, 1024, 2048
    banner("decode fetch counter")
    A = synth.normal_bf16((M, K), seed=17)
    W = synth.normal_bf16((N, K), seed=18, sigma=synth.W_SIGMA)
    d = tl.layout()
    tl.tl_fetch_counter_read()   # reset
    run_gemm(A, W, d, fetch=tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    got = tl.tl_fetch_counter_read()
    p = tl.tl_gemm_plan(M, N, K, d, tl.TL_FETCH_BLOCK)
    amp = tl.tl_read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], d, 4096)
    assert got == amp["fetched_bytes"] == N * K * 2


# ---------------------------------------------------------------------------
# Prefill
# ---------------------------------------------------------------------------

PREFILL_SHAPES = [
    # M, N, K, tile_m, tile_n
    (256, 1024, 1024, 128, 128), (256, 1024, 1024, 256, 128), (512, 1024, 1024, 256, 256),
    (300, 512, 2048, 128, 128), (300, 512, 2048, 256, 128),    # ragged M tail
    (300, 768, 1024, 256, 256),
    (65, 256, 512, 128, 128),                                  # just above the decode limit
    (512, 1056, 512, 256, 128), (512, 1056, 512, 256, 256),    # ragged N tail (N % 128 = 32)
    # 256 x 256 tiles (the four-wave kernel with three weight stages) at 1, 3
    # and 5 K steps: one step (no second weight tile to prefetch) and odd
    # counts, outside the persistent grid
    (300, 768, 64, 256, 256), (512, 1024, 192, 256, 256), (300, 768, 320, 256, 256),
]


@pytest.mark.parametrize("M,N,K,tm,tn", PREFILL_SHAPES)
def test_prefill_tile_major_parity(M, N, K, tm, tn):
    banner(f"prefill M={M} N={N} K={K} tile={tm}x{tn}")
    A = synth.normal_bf16((M, K), seed=21)
    W = synth.normal_bf16((N, K), seed=22, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    C = host_f32(run_gemm(A, W, tl.layout(tile_m=tm, tile_n=tn)))
    parity(C, y_ref, f"prefill {tm}x{tn}")
    Cb = run_gemm(A, W, tl.layout(tile_m=tm, tile_n=tn, out_dtype=tl.TL_OUT_BF16))
    parity_bf16_out(host_bits(Cb), y_ref, "prefill bf16")


@pytest.mark.parametrize("bf16_out", [False, True])
def test_prefill_column_split_plan(bf16_out):
    """M = 1024, N = 33024: 516 tiles of 256 x 256 would leave 252 CUs idle in a
    third round, so the plan covers columns [0, 32768) with 256 x 256 tiles
    (two full rounds) and the last 256 columns with a second launch of
    128 x 128 tiles."""
    M, N, K = 1024, 33024, 256
    plan = tl.tl_gemm_plan(M, N, K, tl.layout())
    assert plan["workgroups"] == 512 + 16
    banner(f"prefill column split bf16_out={bf16_out}")
    A = synth.normal_bf16((M, K), seed=91)
    W = synth.normal_bf16((N, K), seed=92, sigma=synth.W_SIGMA)
    d = tl.layout(out_dtype=tl.TL_OUT_BF16 if bf16_out else tl.TL_OUT_F32)
    C = run_gemm(A, W, d)
    y_ref = oracle.gemm_f64(A, W)
    if bf16_out:
        parity_bf16_out(host_bits(C), y_ref, "split bf16")
    else:
        parity(host_f32(C), y_ref, "split f32")


def test_prefill_column_split_exact():
    M, N, K = 1024, 33024, 256
    A = synth.small_int_bf16((M, K), seed=93)
    W = synth.small_int_bf16((N, K), seed=94)
    banner("prefill column split exact")
    C = run_gemm(A, W, tl.layout())
    assert np.array_equal(host_f32(C).astype(np.float64), oracle.gemm_f64(A, W))


# Columns past the whole rounds of 256 x 256 tiles, run as 256 x 256 tiles
# with K split S ways (fp32 partials, fixed-order reduce): M, N, K, S.
# M = 2000 = 7 * 256 + 208 leaves a ragged last row of tiles.
KSPLIT_REST = [(2000, 12288, 1024, 2), (2000, 10240, 2048, 4)]


@pytest.mark.parametrize("M,N,K,S", KSPLIT_REST)
def test_prefill_ksplit_rest(M, N, K, S):
    plan = tl.tl_gemm_plan(M, N, K, tl.layout())
    banner(f"prefill K-split rest M={M} N={N} K={K} plan={plan}")
    assert plan["split_k"] == S and plan["workgroups"] == 512
    assert plan["workspace_bytes"] == S * M * (N - 8192) * 4
    A = synth.normal_bf16((M, K), seed=95 + S)
    W = synth.normal_bf16((N, K), seed=96 + S, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    parity(host_f32(run_gemm(A, W, tl.layout())), y_ref, f"K-split rest S={S} f32")
    Cb = run_gemm(A, W, tl.layout(out_dtype=tl.TL_OUT_BF16))
    parity_bf16_out(host_bits(Cb), y_ref, f"K-split rest S={S} bf16")


def test_prefill_ksplit_rest_exact():
    """Small-integer inputs: exact in fp32 whatever the split, so the split
    path equals the oracle bit for bit, and two calls are identical."""
    M, N, K = 2000, 10240, 2048
    banner("prefill K-split rest exact")
    A = synth.small_int_bf16((M, K), seed=97)
    W = synth.small_int_bf16((N, K), seed=98)
    C1 = host_f32(run_gemm(A, W, tl.layout()))
    C2 = host_f32(run_gemm(A, W, tl.layout()))
    assert np.array_equal(C1.astype(np.float64), oracle.gemm_f64(A, W))
    assert np.array_equal(C1, C2)


# A persistent grid (one workgroup per CU) over more than one round of whole
# 256 x 256 tiles with bf16 output: M, N, K, tile_m/tile_n pinned or not.
#  - 512 tiles, two per workgroup;
#  - 1024 tiles (four per workgroup) next to a second launch of 128 x 128
#    tiles on the last 4096 columns (K too short for the K-split remainder);
#  - 300 pinned tiles, not a multiple of 8 (units in plain order), 1 or 2 per
#    workgroup;
#  - 2 tiles with K = 128, the fewest K steps the kernel takes (two).
PERSIST_CASES = [(1024, 32768, 512, 0), (2048, 36864, 256, 0), (256, 76800, 256, 256), (256, 512, 128, 256)]


@pytest.mark.parametrize("M,N,K,pin", PERSIST_CASES)
def test_prefill_persistent_grid(M, N, K, pin):
    d = tl.layout(tile_m=pin, tile_n=pin, out_dtype=tl.TL_OUT_BF16)
    plan = tl.tl_gemm_plan(M, N, K, d)
    banner(f"prefill persistent M={M} N={N} K={K} pin={pin} plan={plan}")
    assert plan["workgroups"] == min(256, (M // 256) * (N // 256)) + (512 if N == 36864 else 0)
    assert plan["tile_m"] == 256
    A = synth.normal_bf16((M, K), seed=130 + M // 256)
    W = synth.normal_bf16((N, K), seed=131, sigma=synth.W_SIGMA)
    parity_bf16_out(host_bits(run_gemm(A, W, d)), oracle.gemm_f64(A, W), f"persistent M={M} N={N}")


# Small and medium M, no tile requested: fewer 256 x 256 tiles than CUs, so
# the plan splits K over all the columns (S = CUs / tiles, at most 8, each
# split >= 8 K steps; fp32 partials, then the split-order reduce).  M, N, K,
# row-major [N][K] weight: ragged M with S = 8, S = 4, a row-major weight with
# S = 2; at M <= 128 the same over 128 x 128 tiles: M = 96 (S = 8) and 65
# (S = 4), 80 tiles x 3 uneven ranges (10, 11, 11 K steps), a row-major
# weight whose K has a partial last step (S = 2: 8 and 8 steps, the last 40
# wide), and a ragged M of 77.
KSPLIT_ALL = [(300, 2048, 4096, False), (512, 4096, 2048, False), (256, 1024, 1024, True),
              (96, 2048, 4096, False), (65, 1024, 2048, False), (128, 10240, 2048, False),
              (100, 1024, 1000, True), (77, 4096, 2048, False)]


@pytest.mark.parametrize("M,N,K,row_major", KSPLIT_ALL)
def test_prefill_ksplit_all_columns(M, N, K, row_major):
    kind = tl.TL_LAYOUT_NK_ROW if row_major else tl.TL_LAYOUT_TILE
    fetch = tl.TL_FETCH_NATIVE if row_major else tl.TL_FETCH_BLOCK
    d = tl.layout(kind=kind)
    plan = tl.tl_gemm_plan(M, N, K, d, fetch)
    banner(f"prefill K split over all columns M={M} N={N} K={K} row_major={row_major} plan={plan}")
    tm = 128 if M <= 128 else 256
    tiles = -(-M // tm) * (N // tm)
    S = min(256 // tiles, 8, -(-K // 64) // 8)
    assert S >= 2 and (plan["tile_m"], plan["tile_n"], plan["split_k"]) == (tm, tm, S)
    assert plan["workgroups"] == tiles * S and plan["workspace_bytes"] == S * M * N * 4
    A = synth.normal_bf16((M, K), seed=170 + S)
    W = synth.normal_bf16((N, K), seed=171, sigma=synth.W_SIGMA)
    y_ref = oracle.gemm_f64(A, W)
    C1 = host_f32(run_gemm(A, W, d, fetch=fetch, tile_major=not row_major))
    C2 = host_f32(run_gemm(A, W, d, fetch=fetch, tile_major=not row_major))
    parity(C1, y_ref, f"K split all S={S} f32")
    assert np.array_equal(C1, C2)                      # fixed-order reduce: bitwise reproducible
    db = tl.layout(kind=kind, out_dtype=tl.TL_OUT_BF16)
    assert tl.tl_gemm_plan(M, N, K, db, fetch)["split_k"] == S
    parity_bf16_out(host_bits(run_gemm(A, W, db, fetch=fetch, tile_major=not row_major)), y_ref,
                    f"K split all S={S} bf16")
    Ai = synth.small_int_bf16((M, K), seed=172)
    Wi = synth.small_int_bf16((N, K), seed=173)
    assert np.array_equal(host_f32(run_gemm(Ai, Wi, d, fetch=fetch, tile_major=not row_major)).astype(np.float64),
                          oracle.gemm_f64(Ai, Wi))


# The persistent grid at more K steps (10 and 18) with several units per
# workgroup: M, N, K, pinned tile, row-major [N][K] weight.  Four units per
# workgroup; 384 units (half the workgroups take two); a row-major weight.
PERSIST_DEEP_CASES = [(2048, 32768, 640, 0, False), (768, 32768, 1152, 256, False), (1024, 32768, 640, 0, True)]


@pytest.mark.parametrize("M,N,K,pin,row_major", PERSIST_DEEP_CASES)
def test_prefill_persistent_deeper_k(M, N, K, pin, row_major):
    kind = tl.TL_LAYOUT_NK_ROW if row_major else tl.TL_LAYOUT_TILE
    fetch = tl.TL_FETCH_NATIVE if row_major else tl.TL_FETCH_BLOCK
    d = tl.layout(kind=kind, tile_m=pin, tile_n=pin, out_dtype=tl.TL_OUT_BF16)
    plan = tl.tl_gemm_plan(M, N, K, d, fetch)
    banner(f"prefill persistent M={M} N={N} K={K} row_major={row_major} plan={plan}")
    assert (plan["tile_m"], plan["tile_n"], plan["workgroups"], plan["split_k"]) == (256, 256, 256, 1)
    assert (M // 256) * (N // 256) > 256
    A = synth.normal_bf16((M, K), seed=160 + K // 128)
    W = synth.normal_bf16((N, K), seed=161, sigma=synth.W_SIGMA)
    C = run_gemm(A, W, d, fetch=fetch, tile_major=not row_major)
    parity_bf16_out(host_bits(C), oracle.gemm_f64(A, W), f"persistent M={M} N={N} K={K}")


@pytest.mark.parametrize("K", [512, 640])
def test_prefill_persistent_exact(K):
    """Small-integer inputs through the persistent grid: every fp32 sum is
    exact, so the bf16 output equals the oracle's exact result rounded to
    bf16 (nearest even) bit for bit, and two calls are identical."""
    M, N = 1024, 32768
    banner(f"prefill persistent exact K={K}")
    A = synth.small_int_bf16((M, K), seed=132)
    W = synth.small_int_bf16((N, K), seed=133)
    d = tl.layout(out_dtype=tl.TL_OUT_BF16)
    assert tl.tl_gemm_plan(M, N, K, d)["workgroups"] == 256
    C1 = host_bits(run_gemm(A, W, d))
    C2 = host_bits(run_gemm(A, W, d))
    assert np.array_equal(C1, C2)
    assert np.array_equal(C1, oracle.round_bf16(oracle.gemm_f64(A, W)))


# 256 x 320 tiles (each wave 128 x 160 of C, the fifth 32-column tile's sums
# in VGPRs): M, N, K, memory tile (G, block_rows) or None for a row-major
# weight.  512 tiles (two per workgroup), 256 tiles (one each, 16 K steps),
# 64- and 16-row memory tiles, and [N][K] row-major.
TILES_320 = [(1024, 40960, 512, (4096, 32)), (2048, 10240, 1024, (4096, 32)), (1024, 40960, 256, (8192, 64)),
             (1024, 40960, 256, (2048, 16)), (1024, 40960, 512, None)]


@pytest.mark.parametrize("M,N,K,mt", TILES_320)
def test_prefill_tiles_256x320(M, N, K, mt):
    G, br = mt if mt else (4096, 32)
    kind = tl.TL_LAYOUT_TILE if mt else tl.TL_LAYOUT_NK_ROW
    d = tl.layout(kind=kind, G=G, block_rows=br, out_dtype=tl.TL_OUT_BF16)
    fetch = tl.TL_FETCH_BLOCK if mt else tl.TL_FETCH_NATIVE     # (block fetch on [N][K]: the emulation)
    plan = tl.tl_gemm_plan(M, N, K, d, fetch)
    banner(f"prefill 256x320 M={M} N={N} K={K} mt={mt} plan={plan}")
    assert plan["tile_n"] == 320 and plan["workgroups"] == 256 and plan["split_k"] == 1
    A = synth.normal_bf16((M, K), seed=140 + K // 256)
    W = synth.normal_bf16((N, K), seed=141 + br, sigma=synth.W_SIGMA)
    C = run_gemm(A, W, d, fetch=fetch, tile_major=mt is not None)
    parity_bf16_out(host_bits(C), oracle.gemm_f64(A, W), f"256x320 M={M} N={N} K={K} mt={mt}")


def test_prefill_tiles_256x320_exact():
    """Small integers: the bf16 output equals the oracle's exact result
    rounded to bf16 bit for bit (all five column tiles of every wave), and two
    calls are identical."""
    M, N, K = 1024, 40960, 512
    banner("prefill 256x320 exact")
    A = synth.small_int_bf16((M, K), seed=142)
    W = synth.small_int_bf16((N, K), seed=143)
    d = tl.layout(out_dtype=tl.TL_OUT_BF16)
    assert tl.tl_gemm_plan(M, N, K, d)["tile_n"] == 320
    C1 = host_bits(run_gemm(A, W, d))
    C2 = host_bits(run_gemm(A, W, d))
    assert np.array_equal(C1, C2)
    assert np.array_equal(C1, oracle.round_bf16(oracle.gemm_f64(A, W)))


# The bf16 epilogues round on the GPU (the persistent 256 x 256 and 256 x 320
# grids and the LDS-staged 256 x 256 epilogue with the hardware's packed
# conversion).  A consistency property on top of the oracle parity: the bf16
# output equals, bit for bit, the round-to-nearest-even (the oracle's
# round_bf16) of the fp32 output of a plan whose per-element sums run in the
# same order (256 x 256 tiles, no K split).  M, N, K, the bf16 plan's pinned
# tile (0: the library's) and the kernel it takes.
BF16_OF_F32_CASES = [(1024, 32768, 512, 0, "persistent 256x256"), (1024, 40960, 512, 0, "persistent 256x320"),
                     (300, 1024, 256, 256, "LDS epilogue, ragged M")]


@pytest.mark.parametrize("M,N,K,pin,what", BF16_OF_F32_CASES)
def test_prefill_bf16_out_rounds_the_fp32_sums(M, N, K, pin, what):
    d16 = tl.layout(tile_m=pin, tile_n=pin, out_dtype=tl.TL_OUT_BF16)
    d32 = tl.layout(tile_m=256, tile_n=256, out_dtype=tl.TL_OUT_F32)
    p16, p32 = tl.tl_gemm_plan(M, N, K, d16), tl.tl_gemm_plan(M, N, K, d32)
    banner(f"prefill bf16 = rne(fp32) M={M} N={N} K={K} ({what}) bf16 plan={p16} fp32 plan={p32}")
    assert p16["tile_m"] == 256 and p16["split_k"] == 1 and p32["split_k"] == 1
    assert p16["tile_n"] == (320 if "320" in what else 256)
    assert p16["workgroups"] == (256 if "persistent" in what else -(-M // 256) * (N // 256))
    A = synth.normal_bf16((M, K), seed=150 + M % 7)
    W = synth.normal_bf16((N, K), seed=151, sigma=synth.W_SIGMA)
    C16 = host_bits(run_gemm(A, W, d16))
    C32 = host_f32(run_gemm(A, W, d32))
    assert np.array_equal(C16, oracle.round_bf16(C32.astype(np.float64))), what
    parity_bf16_out(C16, oracle.gemm_f64(A, W), what)


@pytest.mark.parametrize("M,N,K,out", [(1024, 32768, 512, tl.TL_OUT_BF16), (1024, 40960, 512, tl.TL_OUT_BF16),
                                        (2048, 10240, 2048, tl.TL_OUT_F32), (512, 1024, 1024, tl.TL_OUT_BF16),
                                        (512, 1024, 512, tl.TL_OUT_BF16)])
def test_prefill_issued_weight_bytes_equal_read_amp(M, N, K, out):
    """Construction check for the prefill kernels on a tile-major weight
    (persistent 256 x 256, 256 x 320, the K-split remainder, K split over all
    columns, 128 x 128): the
    TL_FETCH_COUNT tally of the weight loads issued equals tl_read_amp's
    fetched bytes for the plan's tile and the oracle's count -- every m-tile
    loads the weight once, whole memory tiles."""
    d = tl.layout(out_dtype=out)
    p = tl.tl_gemm_plan(M, N, K, d, tl.TL_FETCH_BLOCK)
    banner(f"prefill fetch tally M={M} N={N} K={K} plan={p}")
    A = synth.normal_bf16((M, K), seed=150)
    W = synth.normal_bf16((N, K), seed=151, sigma=synth.W_SIGMA)
    tl.tl_fetch_counter_read()   # reset
    run_gemm(A, W, d, fetch=tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT)
    got = tl.tl_fetch_counter_read()
    amp = tl.tl_read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], d, 4096)
    want = oracle.read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], oracle.TILE, 4096, block_rows=32)
    assert got == amp["fetched_bytes"] == want["fetched_bytes"] == -(-M // p["tile_m"]) * N * K * 2, (got, amp, want)


def test_prefill_exact_inputs():
    M, N, K = 256, 256, 1024
    banner("prefill one-hot / small-int")
    A, _ = synth.one_hot_bf16(M, K, seed=23)
    W = synth.normal_bf16((N, K), seed=24, sigma=synth.W_SIGMA)
    assert np.array_equal(host_f32(run_gemm(A, W, tl.layout(tile_m=128))).astype(np.float64),
                          oracle.gemm_f64(A, W))
    A = synth.small_int_bf16((M, K), seed=25)
    W = synth.small_int_bf16((N, K), seed=26)
    for tn in (128, 256):
        assert np.array_equal(host_f32(run_gemm(A, W, tl.layout(tile_m=256, tile_n=tn))).astype(np.float64),
                              oracle.gemm_f64(A, W))


@pytest.mark.parametrize("G,br", [(4096, 8), (16384, 32), (1024, 16), (512, 32), (4096, 4), (16384, 4)])
def test_prefill_memory_tile_shapes(G, br):
    M, N, K = 256, 256, 2048
    banner(f"prefill G={G} br={br}")
    A = synth.normal_bf16((M, K), seed=27)
    W = synth.normal_bf16((N, K), seed=28, sigma=synth.W_SIGMA)
    parity(host_f32(run_gemm(A, W, tl.layout(G=G, block_rows=br))), oracle.gemm_f64(A, W),
           f"prefill G={G} br={br}")


def test_prefill_row_major_native():
    M, N, K = 256, 512, 1024
    banner("prefill NK_ROW")
    A = synth.normal_bf16((M, K), seed=29)
    W = synth.normal_bf16((N, K), seed=30, sigma=synth.W_SIGMA)
    C = host_f32(run_gemm(A, W, tl.layout(kind=tl.TL_LAYOUT_NK_ROW), fetch=tl.TL_FETCH_NATIVE,
                          tile_major=False))
    parity(C, oracle.gemm_f64(A, W), "prefill NK_ROW")


@pytest.mark.parametrize("M,N,K,G,tm,tn", [(256, 512, 1024, 4096, 0, 0), (300, 384, 2048, 1024, 128, 128),
                                           (512, 1024, 512, 16384, 256, 256), (129, 96, 256, 128, 256, 128),
                                           (1024, 2048, 1024, 4096, 0, 0)])
def test_prefill_row_major_block_fetch_counted(M, N, K, G, tm, tn):
    """Prefill over a row-major weight read in whole G-byte blocks: same
    result, and the bytes the kernel counts while loading the blocks equal
    tl_read_amp's fetched bytes for the plan's tile and the oracle's
    brute-force enumeration (rows share a block when K * 2 < G; a ragged last
    tile clips its rows)."""
    banner(f"prefill NK_ROW block fetch M={M} N={N} K={K} G={G} tile {tm}x{tn}")
    A = synth.normal_bf16((M, K), seed=31 + M)
    W = synth.normal_bf16((N, K), seed=32 + N, sigma=synth.W_SIGMA)
    d = tl.layout(kind=tl.TL_LAYOUT_NK_ROW, G=G, tile_m=tm, tile_n=tn)
    p = tl.tl_gemm_plan(M, N, K, d, tl.TL_FETCH_BLOCK)
    assert p["kernel"] == 2
    tl.tl_fetch_counter_read()
    C = run_gemm(A, W, d, fetch=tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT, tile_major=False)
    got = tl.tl_fetch_counter_read()
    parity(host_f32(C), oracle.gemm_f64(A, W), f"prefill block G={G}")
    amp = tl.tl_read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], d, G)
    want = oracle.read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], oracle.NK_ROW, G)
    assert got == amp["fetched_bytes"] == want["fetched_bytes"], (got, amp, want)


# ---------------------------------------------------------------------------
# Full-size workloads
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("i,name,N,K", [(i, *s) for i, s in enumerate(synth.LLAMA70B)])
def test_llama_decode_full_size(i, name, N, K):
    """The bench workload (Llama-70B shapes, M = 1, 8, 32, tile-major G = 4 KB,
    br = 32, block fetch), in the launch configuration the bench uses: every
    output element against the fp64 oracle."""
    banner(f"llama decode full {name}")
    import torch
    W_bits = synth.normal_bf16((N, K), seed=synth.llama_weight_seed(i), sigma=synth.W_SIGMA)
    W = dev_bf16(W_bits)
    Wt = torch.empty_like(W)
    tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
    del W
    for M in synth.LLAMA_DECODE_M:
        banner(f"llama decode full {name} M={M} plan={tl.tl_gemm_plan(M, N, K, tl.layout())}")
        A_bits = synth.normal_bf16((M, K), seed=synth.llama_decode_act_seed(i, M))
        A = dev_bf16(A_bits)
        C = torch.empty((M, N), dtype=torch.float32, device="cuda")
        tl.tl_gemm(A, Wt, C, M, N, K, tl.layout(), tl.TL_FETCH_BLOCK)
        _sync()
        parity(host_f32(C), oracle.gemm_f64(A_bits, W_bits), f"{name} M={M}")


def _prefill_bands(M, N):
    """Rows and columns of the prefill band checks: 32 rows, one in each
    64-row block at a varying offset, and 128 columns, one in each N/128-wide
    block at a varying offset.  The row band (those rows x every column) then
    meets every (128- or 256-row, any-column) output tile at a varying row
    inside it; the column band (every row x those columns) checks every row
    at 128 column positions spread over N."""
    rows = np.array([64 * b + (13 * b + 5) % 64 for b in range(M // 64)], dtype=np.int64)
    step = N // 128
    cols = np.array([step * b + (37 * b + 11) % step for b in range(128)], dtype=np.int64)
    return rows, cols


@pytest.mark.parametrize("i,name,N,K", [(i, *s) for i, s in enumerate(synth.LLAMA70B)])
def test_llama_prefill_full_size_bands(i, name, N, K):
    """Prefill at M = 2048 for the four Llama shapes, every tile the library
    offers and its own plan (the one bench.py times): a band of full rows and
    a band of full columns against the fp64 oracle, bf16 output.  The bands
    meet every workgroup's output tile of every plan (asserted), including
    the 256 x 320 tiles of QKV's plan."""
    banner(f"llama prefill full {name}")
    import torch
    W_bits = synth.normal_bf16((N, K), seed=synth.llama_weight_seed(i), sigma=synth.W_SIGMA)
    W = dev_bf16(W_bits)
    Wt = torch.empty_like(W)
    tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
    del W
    M = synth.LLAMA_PREFILL_M
    A_bits = synth.normal_bf16((M, K), seed=synth.llama_prefill_act_seed(i))
    A = dev_bf16(A_bits)
    rows, cols = _prefill_bands(M, N)
    want_rows = oracle.gemm_f64(A_bits[rows], W_bits)            # [32, N]
    want_cols = oracle.gemm_f64(A_bits, W_bits[cols])            # [M, 128]
    d_rows, d_cols = torch.from_numpy(rows).cuda(), torch.from_numpy(cols).cuda()
    # (0, 0): the library's plan (QKV: 256 x 320 tiles, one round)
    for tm, tn in ((128, 128), (256, 128), (256, 256), (0, 0)):
        d = tl.layout(tile_m=tm, tile_n=tn, out_dtype=tl.TL_OUT_BF16)
        plan = tl.tl_gemm_plan(M, N, K, d)
        ptm, ptn = plan["tile_m"], plan["tile_n"]
        # every (m-tile, n-tile) of the plan -- and of either kind of tile
        # past a column split -- holds row-band elements: the band has rows
        # in every 128-row block and all N columns
        assert len(np.unique(rows // 128)) == M // 128 and len(np.unique(rows // ptm)) == -(-M // ptm)
        assert ptn % 64 == 0
        banner(f"llama prefill full {name} tile {tm}x{tn} plan={plan}")
        C = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        tl.tl_gemm(A, Wt, C, M, N, K, d, tl.TL_FETCH_BLOCK)
        _sync()
        parity_bf16_out(host_bits(C[d_rows]), want_rows, f"{name} {tm}x{tn} row band")
        parity_bf16_out(host_bits(C[:, d_cols]), want_cols, f"{name} {tm}x{tn} column band")


def test_llama_prefill_o_every_element():
    """The O projection [8192, 8192] at M = 2048 with the library's plan: every
    output element against the fp64 oracle (bf16 output), and the fp32-output
    run of the same plan against the fp32 gate."""
    i, name, N, K = 1, *synth.LLAMA70B[1]
    banner(f"llama prefill {name} every element")
    import torch
    W_bits = synth.normal_bf16((N, K), seed=synth.llama_weight_seed(i), sigma=synth.W_SIGMA)
    W = dev_bf16(W_bits)
    Wt = torch.empty_like(W)
    tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
    del W
    M = synth.LLAMA_PREFILL_M
    A_bits = synth.normal_bf16((M, K), seed=synth.llama_prefill_act_seed(i))
    A = dev_bf16(A_bits)
    want = oracle.gemm_f64(A_bits, W_bits)
    C = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    tl.tl_gemm(A, Wt, C, M, N, K, tl.layout(out_dtype=tl.TL_OUT_BF16), tl.TL_FETCH_BLOCK)
    C32 = torch.empty((M, N), dtype=torch.float32, device="cuda")
    tl.tl_gemm(A, Wt, C32, M, N, K, tl.layout(), tl.TL_FETCH_BLOCK)
    _sync()
    parity_bf16_out(host_bits(C), want, f"{name} bf16 out")
    parity(host_f32(C32), want, f"{name} fp32 out")


# ---------------------------------------------------------------------------
# HIP graph capture: replays equal eager results, replay after replay
# ---------------------------------------------------------------------------

def test_graph_replay_matches_eager():
    import torch
    banner("graph capture / replay")
    side = torch.cuda.Stream()
    # M, N, K, split_k, bf16 out: decode (split or not); the LDS-staged decode
    # kernel (split-K 4 with its reduce, and unsplit; four M tiles with
    # split-K 4); 64-row streaming tiles at four M tiles (8 waves, split-K 2);
    # a wide weight at M = 48 on 128 x 128 prefill tiles; prefill through
    # 128 x 128 tiles, the persistent 256 x 256 and 256 x 320 grids, and the
    # plan whose remaining columns split K (main launch, partials and reduce)
    cases = [(8, 1024, 2048, 1, False), (8, 1024, 2048, 4, False), (32, 512, 4096, 3, False),
             (256, 512, 1024, 0, False), (32, 8192, 16384, 0, False), (24, 32768, 2048, 0, False),
             (48, 8192, 8192, 0, True), (40, 8192, 2048, 0, False), (48, 32768, 512, 0, True),
             (1024, 32768, 512, 0, True), (1024, 40960, 512, 0, True), (2000, 12288, 1024, 0, False)]
    with torch.cuda.stream(side):
        tensors = []
        for i, (M, N, K, S, bf16) in enumerate(cases):
            A = dev_bf16(synth.normal_bf16((M, K), seed=40 + i))
            W = dev_bf16(synth.normal_bf16((N, K), seed=50 + i, sigma=synth.W_SIGMA))
            Wt = torch.empty_like(W)
            tl.tl_repack(W, Wt, N, K, 2, 4096, 32)
            C = torch.zeros((M, N), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
            d = tl.layout(split_k=S, out_dtype=tl.TL_OUT_BF16 if bf16 else tl.TL_OUT_F32)
            tl.tl_gemm(A, Wt, C, M, N, K, d, tl.TL_FETCH_BLOCK)       # eager; creates the workspace
            tensors.append((A, Wt, C, d, M, N, K))
        side.synchronize()
        eager = [t[2].clone() for t in tensors]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for (A, Wt, C, d, M, N, K) in tensors:
                tl.tl_gemm(A, Wt, C, M, N, K, d, tl.TL_FETCH_BLOCK)
        for rep in range(4):
            for (_, _, C, _, _, _, _) in tensors:
                C.fill_(float("nan"))                # eager work between replays
            side.synchronize()
            g.replay()
            side.synchronize()
            for (_, _, C, _, _, _, _), want in zip(tensors, eager):
                assert torch.equal(C, want), f"replay {rep}"


# ---------------------------------------------------------------------------
# Qwen-3-30B-A3B-shaped MoE layer: per-expert GEMMs at the token counts the
# seeded top-8 routing gives, and the attention projections at M = 64
# ---------------------------------------------------------------------------

def _moe_experts_sample():
    tok = synth.tokens_per_expert(synth.moe_routing())
    counts = np.array([len(t) for t in tok])
    touched = np.nonzero(counts)[0]
    # largest, smallest and a spread of token counts
    order = touched[np.argsort(counts[touched], kind="stable")]
    pick = sorted(set(order[[0, 1, len(order) // 3, len(order) // 2, -2, -1]].tolist()))
    return tok, pick


def test_moe_expert_gemms():
    """Gate+up [1536, 2048] and down [2048, 768] of sampled experts, each at
    its own token count (rows gathered from the seeded hidden states)."""
    tok, pick = _moe_experts_sample()
    hidden = synth.normal_bf16((synth.QWEN_TOKENS, synth.QWEN_HIDDEN), seed=synth.QWEN_SEED_HIDDEN)
    total = int(sum(len(t) for t in tok))
    down_in = synth.normal_bf16((total, synth.QWEN_DOWN[1]), seed=synth.QWEN_SEED_DOWN_IN)
    starts = np.concatenate([[0], np.cumsum([len(t) for t in tok])])
    for e in pick:
        Me = len(tok[e])
        banner(f"moe expert {e}: M={Me}")
        A_gu = np.ascontiguousarray(hidden[tok[e]])
        W_gu = synth.normal_bf16(synth.QWEN_GATE_UP, seed=synth.qwen_gate_up_seed(e), sigma=synth.W_SIGMA)
        parity(host_f32(run_gemm(A_gu, W_gu, tl.layout())), oracle.gemm_f64(A_gu, W_gu), f"gate_up e={e}")
        A_d = np.ascontiguousarray(down_in[starts[e]:starts[e] + Me])
        W_d = synth.normal_bf16(synth.QWEN_DOWN, seed=synth.qwen_down_seed(e), sigma=synth.W_SIGMA)
        parity(host_f32(run_gemm(A_d, W_d, tl.layout())), oracle.gemm_f64(A_d, W_d), f"down e={e}")


@pytest.mark.parametrize("i", range(len(synth.QWEN_ATTN)))
def test_moe_attention_projections(i):
    name, N, K = synth.QWEN_ATTN[i]
    banner(f"moe attention {name} M={synth.QWEN_TOKENS} N={N} K={K}")
    seed = synth.QWEN_SEED_HIDDEN if K == synth.QWEN_HIDDEN else synth.QWEN_SEED_ATTN_O_IN
    A = synth.normal_bf16((synth.QWEN_TOKENS, K), seed=seed)
    W = synth.normal_bf16((N, K), seed=synth.qwen_attn_seed(i), sigma=synth.W_SIGMA)
    parity(host_f32(run_gemm(A, W, tl.layout())), oracle.gemm_f64(A, W), f"attn {name}")


def test_moe_attention_stacked_qkv():
    """q, k and v repacked one by one and laid end to end are the tile-major
    copy of the stacked [q; k; v] weight (each has whole strips of 32 rows),
    and one call over them equals the three projections (the bench's path)."""
    import torch
    K, M = synth.QWEN_HIDDEN, synth.QWEN_TOKENS
    banner("moe attention stacked qkv")
    Ws = [synth.normal_bf16((N, K), seed=synth.qwen_attn_seed(i), sigma=synth.W_SIGMA)
          for i, (_, N, _) in enumerate(synth.QWEN_ATTN[:3])]
    parts = []
    for W in Ws:
        Wd = dev_bf16(W)
        Wt = torch.empty_like(Wd)
        tl.tl_repack(Wd, Wt, W.shape[0], K, 2, 4096, 32)
        parts.append(Wt.reshape(-1))
    stacked = np.vstack(Ws)
    cat = torch.cat(parts).view(stacked.shape[0], K)
    _sync()
    assert np.array_equal(host_bits(cat), oracle.repack(stacked, 4096, 32))
    A = synth.normal_bf16((M, K), seed=synth.QWEN_SEED_HIDDEN)
    C = torch.empty((M, stacked.shape[0]), dtype=torch.float32, device="cuda")
    tl.tl_gemm(dev_bf16(A), cat, C, M, stacked.shape[0], K, tl.layout(), tl.TL_FETCH_BLOCK)
    _sync()
    parity(host_f32(C), oracle.gemm_f64(A, stacked), "stacked qkv")
