"""Seeded random sweeps against the oracle.  tl_gemm: shapes (ragged M, N and K,
padded tile-major copies), memory tiles, layouts, fetch modes, tiles, split
counts and output types drawn together, so that combinations the targeted
tests do not name are exercised too.  Cases the planner rejects
(TL_EUNSUPPORTED) are counted and skipped; everything it accepts must pass the
parity gate (fp32 out) or match the bf16 rounding of the oracle.  The grouped
launches: random group tables, ids, weights and memory tiles."""
import os

import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from paper_2607_04031_amd import synth
from tests._gpu import banner, dev_bf16, host_bits, host_f32, parity, parity_bf16_out

pytestmark = pytest.mark.gpu
# TL_RANDOM_SCALE=n runs n times as many draws of each sweep (further seeds)
SCALE = max(1, int(os.environ.get("TL_RANDOM_SCALE", "1")))


@pytest.fixture(scope="module", autouse=True)
def _lib():
    import torch
    assert torch.cuda.is_available()
    tl.load_library()
    yield
    torch.cuda.empty_cache()


def draw(rng, decode):
    G = int(rng.choice([512, 1024, 4096, 16384]))
    br = int(rng.choice([b for b in (4, 8, 16, 32, 64) if G // (2 * b) >= 8]))
    M = int(rng.integers(1, 65)) if decode else int(rng.integers(65, 1500))
    N = int(rng.integers(1, 3000))
    # prefill: half the draws take K % 64 = 0, which the four-wave 256 x 256
    # kernel needs (1 to 75 K steps)
    if not decode and rng.random() < 0.5:
        K = 64 * int(rng.integers(1, 76))
    else:
        K = 8 * int(rng.integers(1, 600))
    kind = tl.TL_LAYOUT_TILE if rng.random() < 0.8 else tl.TL_LAYOUT_NK_ROW
    fetch = tl.TL_FETCH_BLOCK if rng.random() < 0.7 else tl.TL_FETCH_NATIVE
    out = tl.TL_OUT_BF16 if rng.random() < 0.3 else tl.TL_OUT_F32
    tile_n = int(rng.choice([0, 0, 32, 64] if decode else [0, 0, 128, 256]))
    split_k = int(rng.choice([0, 0, 0, 1, 2, 3, 5])) if decode else 0
    d = tl.layout(kind=kind, G=G, block_rows=br, out_dtype=out, tile_n=tile_n, split_k=split_k)
    return M, N, K, d, fetch


def run_case(M, N, K, d, fetch, seed):
    import torch
    A = synth.normal_bf16((M, K), seed=seed)
    W = synth.normal_bf16((N, K), seed=seed + 1, sigma=synth.W_SIGMA)
    Wd = dev_bf16(W)
    if d.kind == tl.TL_LAYOUT_TILE:
        Wt = torch.empty(tl.padded_shape(N, K, 2, d.G, d.block_rows), dtype=torch.bfloat16, device="cuda")
        tl.tl_repack(Wd, Wt, N, K, 2, d.G, d.block_rows)
        Wd = Wt
    bf16 = d.out_dtype == tl.TL_OUT_BF16
    C = torch.full((M, N), float("nan"), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
    tl.tl_gemm(dev_bf16(A), Wd, C, M, N, K, d, fetch)
    torch.cuda.synchronize()
    y_ref = oracle.gemm_f64(A, W)
    what = f"M={M} N={N} K={K} kind={d.kind} G={d.G} br={d.block_rows} tn={d.tile_n} S={d.split_k} bf16={bf16}"
    if bf16:
        parity_bf16_out(host_bits(C), y_ref, what)
    else:
        parity(host_f32(C), y_ref, what)


@pytest.mark.parametrize("decode", [True, False])
def test_random_gemm_cases(decode):
    rng = np.random.default_rng(2024 if decode else 2025)
    ran = skipped = 0
    for case in range((60 if decode else 24) * SCALE):
        M, N, K, d, fetch = draw(rng, decode)
        try:
            p = tl.tl_gemm_plan(M, N, K, d, fetch)
        except tl.TLError as e:
            assert e.status == tl.TL_EUNSUPPORTED, (M, N, K, e)
            skipped += 1
            continue
        banner(f"random {'decode' if decode else 'prefill'} case {case}: M={M} N={N} K={K} G={d.G} "
               f"br={d.block_rows} kind={d.kind} plan={p}")
        run_case(M, N, K, d, fetch, seed=7000 + case)
        ran += 1
    assert ran >= (40 if decode else 12) * SCALE, (ran, skipped)


def draw_whole_tiles(rng):
    """Prefill shapes of whole 256-row tiles and an even number (2 to 16) of
    64-wide K steps, bf16 out (mostly): the persistent four-wave kernel --
    more tiles than CUs (several per workgroup), 256 x 320 tiles that fill
    whole rounds, or fewer tiles than CUs -- on random memory tiles or a
    row-major weight."""
    mt = int(rng.choice([4, 8]))                  # M = 1024 or 2048: 256-row tiles
    kind_n = int(rng.integers(0, 3))
    if kind_n == 0:      # 256 x 256, more tiles than CUs
        N = 256 * int(rng.integers(256 // mt + 1, 384 // mt + 1))
    elif kind_n == 1:    # 256 x 320 filling one or two rounds
        N = 320 * 256 * int(rng.integers(1, 3)) // mt
    else:                # fewer tiles than CUs
        N = 256 * int(rng.integers(1, 256 // mt))
    K = 128 * int(rng.integers(1, 9))
    if rng.random() < 0.75:
        G = int(rng.choice([1024, 2048, 4096, 8192]))
        br = int(rng.choice([b for b in (4, 8, 16, 32, 64) if 8 <= G // (2 * b) <= 512]))
        kind, fetch = tl.TL_LAYOUT_TILE, tl.TL_FETCH_BLOCK
    else:
        G, br, kind, fetch = 4096, 32, tl.TL_LAYOUT_NK_ROW, tl.TL_FETCH_NATIVE
    out = tl.TL_OUT_BF16 if rng.random() < 0.85 else tl.TL_OUT_F32
    pin = 256 if rng.random() < 0.2 else 0
    d = tl.layout(kind=kind, G=G, block_rows=br, out_dtype=out, tile_m=pin, tile_n=pin)
    return 256 * mt, N, K, d, fetch


def draw_w4_ragged(rng):
    """Ragged prefill shapes pinned to 256 x 256 tiles with K % 64 = 0: the
    four-wave kernel outside the persistent grid (partial tiles clamp their
    loads and guard their stores) at 1 to 40 K steps, on random memory
    tiles or a row-major weight, both output types."""
    M, N, K = int(rng.integers(65, 1500)), int(rng.integers(1, 3000)), 64 * int(rng.integers(1, 41))
    if rng.random() < 0.75:
        G = int(rng.choice([1024, 2048, 4096, 8192]))
        br = int(rng.choice([b for b in (4, 8, 16, 32, 64) if 8 <= G // (2 * b) <= 512]))
        kind, fetch = tl.TL_LAYOUT_TILE, tl.TL_FETCH_BLOCK
    else:
        G, br, kind, fetch = 4096, 32, tl.TL_LAYOUT_NK_ROW, tl.TL_FETCH_NATIVE
    out = tl.TL_OUT_BF16 if rng.random() < 0.5 else tl.TL_OUT_F32
    d = tl.layout(kind=kind, G=G, block_rows=br, out_dtype=out, tile_m=256, tile_n=256)
    return M, N, K, d, fetch


@pytest.mark.parametrize("case", range(10 * SCALE))
def test_random_w4_ragged_prefill_cases(case):
    rng = np.random.default_rng(5000 + case)
    M, N, K, d, fetch = draw_w4_ragged(rng)
    p = tl.tl_gemm_plan(M, N, K, d, fetch)
    banner(f"random ragged 256x256 prefill case {case}: M={M} N={N} K={K} G={d.G} br={d.block_rows} "
           f"kind={d.kind} out={d.out_dtype} plan={p}")
    assert p["kernel"] == 2 and (p["tile_m"], p["tile_n"], p["split_k"]) == (256, 256, 1)
    run_case(M, N, K, d, fetch, seed=11000 + case)


def draw_medium_m(rng):
    """Small and medium-M prefill with the library's plan (no tile
    requested): M 65 to 1023 (ragged), N a multiple of 256, K 1024 to 6080, so
    the plan takes 256 x 256 tiles, with K split over all the columns when
    they are fewer than the CUs, or 128 x 128 tiles; random memory tiles or a
    row-major weight, both output types."""
    M, N, K = int(rng.integers(65, 1024)), 256 * int(rng.integers(1, 49)), 64 * int(rng.integers(16, 96))
    if rng.random() < 0.75:
        G = int(rng.choice([1024, 2048, 4096, 8192]))
        br = int(rng.choice([b for b in (4, 8, 16, 32, 64) if 8 <= G // (2 * b) <= 512]))
        kind, fetch = tl.TL_LAYOUT_TILE, tl.TL_FETCH_BLOCK
    else:
        G, br, kind, fetch = 4096, 32, tl.TL_LAYOUT_NK_ROW, tl.TL_FETCH_NATIVE
    out = tl.TL_OUT_BF16 if rng.random() < 0.5 else tl.TL_OUT_F32
    d = tl.layout(kind=kind, G=G, block_rows=br, out_dtype=out)
    return M, N, K, d, fetch


@pytest.mark.parametrize("case", range(10 * SCALE))
def test_random_medium_m_prefill_cases(case):
    rng = np.random.default_rng(6000 + case)
    M, N, K, d, fetch = draw_medium_m(rng)
    p = tl.tl_gemm_plan(M, N, K, d, fetch)
    banner(f"random medium-M prefill case {case}: M={M} N={N} K={K} G={d.G} br={d.block_rows} "
           f"kind={d.kind} out={d.out_dtype} plan={p}")
    assert p["kernel"] == 2
    run_case(M, N, K, d, fetch, seed=13000 + case)


@pytest.mark.parametrize("case", range(8 * SCALE))
def test_random_whole_tile_prefill_cases(case):
    rng = np.random.default_rng(4000 + case)
    M, N, K, d, fetch = draw_whole_tiles(rng)
    p = tl.tl_gemm_plan(M, N, K, d, fetch)
    banner(f"random whole-tile prefill case {case}: M={M} N={N} K={K} G={d.G} br={d.block_rows} "
           f"kind={d.kind} out={d.out_dtype} plan={p}")
    assert p["kernel"] == 2 and p["tile_m"] == 256
    run_case(M, N, K, d, fetch, seed=9000 + case)


@pytest.mark.parametrize("case", range(6 * SCALE))
def test_random_lds_staged_cases(case):
    """17 <= M <= 32 on weights whose 32-row tiles fill the CUs in whole rounds
    (the LDS-staged kernel), random M, memory tile and output type."""
    rng = np.random.default_rng(3000 + case)
    M = int(rng.integers(17, 33))
    N, K = [(32768, 2048), (8192, 16384), (10240, 8192), (8192, 4096 * 7)][case % 4]
    G = int(rng.choice([1024, 4096, 16384]))
    br = int(rng.choice([b for b in (8, 16, 32) if G // (2 * b) <= 512]))
    d = tl.layout(G=G, block_rows=br, out_dtype=tl.TL_OUT_BF16 if case % 3 == 2 else tl.TL_OUT_F32)
    p = tl.tl_gemm_plan(M, N, K, d)
    assert p["waves"] == 8 and p["tile_n"] == 32, p
    banner(f"random lds case {case}: M={M} N={N} K={K} G={G} br={br} plan={p}")
    run_case(M, N, K, d, tl.TL_FETCH_BLOCK, seed=8000 + case)


@pytest.mark.parametrize("case", range(4 * SCALE))
def test_random_lds_staged_four_m_tile_cases(case):
    """33 <= M <= 64 on weights whose groups of four 32-row tiles and K ranges
    fill at least 7/8 of the CUs (the LDS-staged kernel with four M tiles),
    random M, memory tile and output type."""
    rng = np.random.default_rng(3100 + case)
    M = int(rng.integers(33, 65))
    N, K = [(8192, 16384), (10240, 8192), (8192, 4096 * 7), (16384, 4096)][case % 4]
    G = int(rng.choice([1024, 4096, 16384]))
    br = int(rng.choice([b for b in (8, 16, 32) if G // (2 * b) <= 512]))
    d = tl.layout(G=G, block_rows=br, out_dtype=tl.TL_OUT_BF16 if case % 3 == 2 else tl.TL_OUT_F32)
    p = tl.tl_gemm_plan(M, N, K, d)
    assert p["waves"] == 8 and p["tile_n"] == 32 and p["tile_m"] == 64, p
    banner(f"random lds four-M-tile case {case}: M={M} N={N} K={K} G={G} br={br} plan={p}")
    run_case(M, N, K, d, tl.TL_FETCH_BLOCK, seed=8100 + case)


def dev_i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


@pytest.mark.parametrize("swiglu", [False, True])
def test_random_grouped_cases(swiglu):
    """Random group tables (empty groups, groups larger than the M tile), ids,
    weight shapes, memory tiles and output types for tl_gemm_grouped and
    tl_gemm_grouped_swiglu."""
    import torch
    rng = np.random.default_rng(4000 + swiglu)
    for case in range(12 * SCALE):
        E = int(rng.integers(1, 10))
        counts = [int(rng.choice([0, 1, 3, 9, 17, 40])) for _ in range(E)]
        offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
        T = int(offsets[-1])
        if T == 0:
            continue
        a_rows = int(rng.integers(1, 50))
        ids = rng.integers(0, a_rows, size=T).astype(np.int32)
        G = int(rng.choice([1024, 4096]))
        br = int(rng.choice([8, 16, 32]))
        K = 8 * int(rng.integers(1, 300))
        N = 32 * int(rng.integers(1, 20)) if swiglu else int(rng.integers(1, 700))
        rows_w = 2 * N if swiglu else N
        bf16 = rng.random() < 0.4
        d = tl.layout(G=G, block_rows=br, out_dtype=tl.TL_OUT_BF16 if bf16 else tl.TL_OUT_F32)
        max_rows = max(counts) + int(rng.integers(0, 5))
        A = synth.normal_bf16((a_rows, K), seed=9000 + case)
        Ws = [synth.normal_bf16((rows_w, K), seed=9100 + 10 * case + e, sigma=synth.W_SIGMA) for e in range(E)]
        stride = tl.tl_tile_bytes(rows_w, K, 2, G, br)
        stride = (stride + 15) // 16 * 16
        stack = torch.zeros(E * stride // 2, dtype=torch.bfloat16, device="cuda")
        for e, W in enumerate(Ws):
            part = stack[e * stride // 2:(e + 1) * stride // 2]
            tl.tl_repack(dev_bf16(W), part, rows_w, K, 2, G, br)
        C = torch.full((T, N), float("nan"), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
        banner(f"random grouped swiglu={swiglu} case {case}: E={E} counts={counts} N={N} K={K} G={G} br={br}")
        fn = tl.tl_gemm_grouped_swiglu if swiglu else tl.tl_gemm_grouped
        fn(dev_bf16(A), a_rows, dev_i32(ids), dev_i32(offsets), E, T, max_rows, stack, stride, C, N, K, d,
           tl.TL_FETCH_BLOCK)
        torch.cuda.synchronize()
        ref = (oracle.grouped_swiglu_f64 if swiglu else oracle.grouped_gemm_f64)(A, ids, offsets, Ws)
        what = f"grouped swiglu={swiglu} case {case}"
        if bf16:
            parity_bf16_out(host_bits(C), ref, what)
        else:
            parity(host_f32(C), ref, what)


def test_random_fp8_cases():
    """Random weight-only FP8 (OCP E4M3) decode through tl_gemm_w8: ragged M,
    N and K (K a multiple of 16; padded tile-major copies), memory tiles,
    layouts, split counts, per-channel scales or none, both output types."""
    import torch
    rng = np.random.default_rng(5000)
    ran = skipped = 0
    for case in range(24 * SCALE):
        G = int(rng.choice([1024, 4096, 16384]))
        br = int(rng.choice([b for b in (16, 32, 64, 128) if G // b >= 16]))
        M, N, K = int(rng.integers(1, 65)), int(rng.integers(1, 2000)), 16 * int(rng.integers(1, 400))
        kind = tl.TL_LAYOUT_TILE if rng.random() < 0.85 else tl.TL_LAYOUT_NK_ROW
        bf16 = rng.random() < 0.3
        split_k = int(rng.choice([0, 0, 0, 1, 2, 3]))
        scaled = rng.random() < 0.5
        d = tl.layout(kind=kind, elem_bytes=1, G=G, block_rows=br, split_k=split_k,
                      out_dtype=tl.TL_OUT_BF16 if bf16 else tl.TL_OUT_F32)
        fetch = tl.TL_FETCH_BLOCK if kind == tl.TL_LAYOUT_TILE else tl.TL_FETCH_NATIVE
        try:
            p = tl.tl_gemm_plan(M, N, K, d, fetch)
        except tl.TLError as e:
            assert e.status == tl.TL_EUNSUPPORTED, (M, N, K, e)
            skipped += 1
            continue
        banner(f"random fp8 case {case}: M={M} N={N} K={K} G={G} br={br} kind={kind} scaled={scaled} plan={p}")
        W8, sc = synth.fp8_weights((N, K), seed=5100 + case)
        A = synth.normal_bf16((M, K), seed=5200 + case)
        W = torch.from_numpy(np.ascontiguousarray(W8)).cuda()
        if kind == tl.TL_LAYOUT_TILE:
            Wt = torch.zeros(tl.tl_tile_bytes(N, K, 1, G, br), dtype=torch.uint8, device="cuda")
            tl.tl_repack(W, Wt, N, K, 1, G, br)
            W = Wt
        sc_dev = torch.from_numpy(np.ascontiguousarray(sc, dtype=np.float32)).cuda() if scaled else None
        C = torch.full((M, N), float("nan"), dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
        tl.tl_gemm_w8(dev_bf16(A), W, sc_dev, C, M, N, K, d, fetch)
        torch.cuda.synchronize()
        ref = oracle.gemm_w8_f64(A, W8, sc if scaled else None)
        what = f"fp8 case {case}: M={M} N={N} K={K} G={G} br={br} kind={kind} S={split_k} scaled={scaled} bf16={bf16}"
        if bf16:
            parity_bf16_out(host_bits(C), ref, what)
        else:
            parity(host_f32(C), ref, what)
        ran += 1
    assert ran >= 12 * SCALE, (ran, skipped)
