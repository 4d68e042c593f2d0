"""Host-side tests of libtl (no GPU): the library loads and exports every
symbol include/tl.h declares; tl_read_amp equals the brute-force oracle;
tl_gemm_plan; argument validation returns the documented status before any
device work."""
import os
import re

import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KIND = {oracle.NK_ROW: tl.TL_LAYOUT_NK_ROW, oracle.KN_ROW: tl.TL_LAYOUT_KN_ROW,
        oracle.TILE: tl.TL_LAYOUT_TILE}


def header_symbols():
    text = open(os.path.join(ROOT, "include", "tl.h")).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(tl_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    lib = tl.load_library()
    syms = header_symbols()
    assert set(syms) == set(tl.EXPORTED)
    for s in syms:
        assert hasattr(lib, s), s
    # and the binding exposes the same names
    for s in syms:
        assert callable(getattr(tl, s))


def test_strerror_strings():
    for st in (tl.TL_OK, tl.TL_EINVAL, tl.TL_EUNSUPPORTED, tl.TL_EHIP, tl.TL_ENOMEM, tl.TL_ESCRATCH):
        assert tl.tl_strerror(st).startswith("TL_")
    assert "unknown" in tl.tl_strerror(12345)


def _lib_amp(M, N, K, tm, tn, tk, kind, G, layout_G=4096, br=32):
    d = tl.layout(kind=KIND[kind], G=layout_G, block_rows=br)
    return tl.tl_read_amp(M, N, K, tm, tn, tk, d, G)


def test_read_amp_matches_oracle_random_shapes():
    """Random shapes including ragged tiles, G != memory-tile size, all layouts."""
    rng = np.random.default_rng(11)
    for _ in range(120):
        kind = int(rng.choice([oracle.NK_ROW, oracle.KN_ROW, oracle.TILE]))
        s = 2
        layout_G = int(rng.choice([256, 512, 1024, 4096]))
        br = int(rng.choice([1, 2, 4, 8, 16, 32]))
        if s * br > layout_G:
            continue
        bc = layout_G // (s * br)
        if kind == oracle.TILE and rng.random() < 0.5:
            N = br * int(rng.integers(1, 5)) * (1 if br > 8 else 4)
            K = bc * int(rng.integers(1, 5))
        elif kind == oracle.TILE:                 # padded to whole memory tiles
            N = int(rng.integers(1, 70))
            K = int(rng.integers(1, 300))
        else:
            N = int(rng.integers(1, 70))
            K = int(rng.integers(1, 300))
        G = int(rng.choice([64, 256, 512, 1024, 4096])) if rng.random() < 0.5 else layout_G
        M = int(rng.integers(1, 40))
        tm = int(rng.integers(1, 20))
        tn = int(rng.choice([1, 3, 8, 16, 32, 64]))
        tk = int(rng.choice([1, 5, 16, 64, 128, 256]))
        want = oracle.read_amp(M, N, K, tm, tn, tk, kind, G, s=s, layout_G=layout_G, block_rows=br)
        got = _lib_amp(M, N, K, tm, tn, tk, kind, G, layout_G, br)
        for key in want:
            if key == "amp":
                assert got[key] == pytest.approx(want[key], rel=1e-15)
            else:
                assert got[key] == want[key], (key, kind, M, N, K, tm, tn, tk, G, layout_G, br)


@pytest.mark.parametrize("G", [512, 1024, 4096, 16384])
@pytest.mark.parametrize("br", [4, 8, 16, 32, 64])
def test_read_amp_granularity_sweep_slice_matches_oracle(G, br):
    """Down-projection [8192, 28672] (256-row slice), tiles 64..256: the
    library's closed forms equal the oracle's enumeration exactly."""
    N, K, s = 256, 28672, 2
    for tn in (64, 128, 256):
        for tk in (64, 128, 256):
            for kind in (oracle.NK_ROW, oracle.TILE):
                want = oracle.read_amp(32, N, K, 32, tn, tk, kind, G, s=s, layout_G=G, block_rows=br)
                got = _lib_amp(32, N, K, 32, tn, tk, kind, G, G, br)
                assert got == {k: (pytest.approx(v) if k == "amp" else v) for k, v in want.items()}


def test_read_amp_tiny_config():
    assert _lib_amp(16, 1024, 1024, 64, 64, 64, oracle.NK_ROW, 4096)["amp"] == 16.0
    assert _lib_amp(16, 1024, 1024, 64, 64, 64, oracle.KN_ROW, 4096)["amp"] == 16.0
    assert _lib_amp(16, 1024, 1024, 64, 64, 64, oracle.TILE, 4096)["amp"] == 1.0


def test_read_amp_rejects_bad_arguments():
    d = tl.layout()
    for args in [(0, 8, 8, 1, 1, 1), (1, 8, 8, 0, 1, 1), (1, 8, 8, 1, 1, -1)]:
        with pytest.raises(tl.TLError) as e:
            tl.tl_read_amp(*args, d, 4096)
        assert e.value.status == tl.TL_EINVAL
    with pytest.raises(tl.TLError):
        tl.tl_read_amp(1, 8, 8, 1, 1, 1, d, 0)
    bad = tl.layout(G=3000)
    with pytest.raises(tl.TLError):
        tl.tl_read_amp(1, 64, 64, 1, 1, 1, bad, 4096)
    # a tile-major weight the memory tile does not divide is the padded copy
    got = tl.tl_read_amp(1, 48, 100, 1, 16, 64, tl.layout(block_rows=32), 4096)
    want = oracle.read_amp(1, 48, 100, 1, 16, 64, oracle.TILE, 4096, s=2, layout_G=4096, block_rows=32)
    assert got == {k: (pytest.approx(v) if k == "amp" else v) for k, v in want.items()}


def test_tile_bytes_matches_oracle():
    rng = np.random.default_rng(5)
    for _ in range(300):
        s = int(rng.choice([1, 2, 4, 8]))
        G = int(rng.choice([64, 512, 4096, 16384]))
        br = int(rng.choice([1, 2, 8, 32, 64]))
        if s * br > G:
            continue
        rows, cols = int(rng.integers(1, 3000)), int(rng.integers(1, 3000))
        assert tl.tl_tile_bytes(rows, cols, s, G, br) == oracle.packed_bytes(rows, cols, s, G, br)
    assert tl.tl_tile_bytes(8192, 28672, 2, 4096, 32) == 8192 * 28672 * 2     # divisible: no padding
    assert tl.tl_tile_bytes(0, 100, 2, 4096, 32) == 0
    for args in [(-1, 8, 2, 4096, 32), (8, 8, 3, 4096, 32), (8, 8, 2, 3000, 32), (8, 8, 2, 4096, 4096),
                 (1 << 21, 1 << 21, 2, 4096, 32)]:
        with pytest.raises(tl.TLError) as e:
            tl.tl_tile_bytes(*args)
        assert e.value.status == tl.TL_EINVAL


def test_gemm_plan_decode_and_prefill_shapes():
    d = tl.layout()
    # Llama-70B-shaped decode at M = 8: whole memory tiles per compute tile
    for N, K, S, waves in [(10240, 8192, 4, 4), (8192, 8192, 1, 16), (57344, 8192, 1, 4),
                           (8192, 28672, 4, 4)]:
        p = tl.tl_gemm_plan(8, N, K, d)
        assert p["kernel"] == 1 and p["tile_n"] == 32 and p["tile_k"] == 64
        assert p["split_k"] == S and p["waves"] == waves
        assert p["workgroups"] % 256 == 0
        amp = tl.tl_read_amp(8, N, K, p["tile_m"], p["tile_n"], p["tile_k"], d, 4096)
        assert amp["amp"] == 1.0
    # 512 tiles -> 8 waves; registers cap waves as M and tile_n grow
    assert tl.tl_gemm_plan(8, 16384, 1024, d)["waves"] == 8
    assert tl.tl_gemm_plan(32, 8192, 4096, d)["tile_n"] == 64      # M > 16: 64-row tiles
    # a weight under 32 MB is latency-bound: 32-row tiles, splits down to 512 K
    for M in (8, 32, 64):
        p = tl.tl_gemm_plan(M, 512, 2048, d)                        # Qwen k/v projection
        assert (p["tile_n"], p["split_k"], p["workgroups"]) == (32, 4, 64)
        p = tl.tl_gemm_plan(M, 2048, 768, d)                        # one Qwen expert's down projection
        assert (p["tile_n"], p["split_k"], p["workgroups"]) == (32, 1, 64)
        p = tl.tl_gemm_plan(M, 4096, 2048, d)                       # Qwen q projection
        assert (p["tile_n"], p["split_k"], p["workgroups"]) == (32, 2, 256)
    # 17 <= M <= 32 on the Llama shapes: activations staged in LDS, one 8-wave
    # workgroup per CU taking T 32-row tiles (whole strips) x one of S K ranges
    for N, K, S in [(10240, 8192, 4), (57344, 8192, 1), (8192, 28672, 4), (8192, 16384, 4)]:
        for M in (17, 32):
            p = tl.tl_gemm_plan(M, N, K, d)
            assert (p["tile_n"], p["split_k"], p["waves"], p["workgroups"]) == (32, S, 8, 256)
            amp = tl.tl_read_amp(M, N, K, p["tile_m"], p["tile_n"], p["tile_k"], d, 4096)
            assert amp["amp"] == 1.0
    # ... but not when its K ranges are short (4 chunks of 512) and the
    # streaming plan already fills the CUs once: Llama O
    for M in (17, 32):
        p = tl.tl_gemm_plan(M, 8192, 8192, d)
        assert (p["tile_n"], p["split_k"], p["waves"], p["workgroups"]) == (64, 2, 8, 256)
    # tiles that neither fill two rounds of the CUs nor divide them (one
    # GPU's share of the Llama shapes under tensor parallelism): the 32- or
    # 64-row tile and K split that fill one round to >= 7/8, one workgroup per
    # CU; full QKV (320 or 160 tiles, under 7/8) keeps about 1024 workgroups
    for M, N, K, tn, S, wgs in [(8, 2560, 8192, 32, 3, 240), (32, 2560, 8192, 64, 6, 240),
                                (1, 1280, 8192, 32, 6, 240), (32, 1280, 8192, 64, 12, 240),
                                (8, 14336, 8192, 64, 1, 224), (32, 14336, 8192, 64, 1, 224),
                                (8, 7168, 8192, 32, 1, 224), (32, 7168, 8192, 64, 2, 224),
                                (8, 5120, 8192, 64, 3, 240), (64, 5120, 2048, 64, 3, 240)]:
        p = tl.tl_gemm_plan(M, N, K, d)
        assert (p["tile_n"], p["split_k"], p["workgroups"]) == (tn, S, wgs), (M, N, K, p)
    assert tl.tl_gemm_plan(8, 10240, 8192, d)["workgroups"] == 1280
    # a fixed tile or split keeps the streaming kernel: 128 tiles of 64 rows,
    # K split in two, one 8-wave workgroup per CU
    p = tl.tl_gemm_plan(32, 8192, 8192, tl.layout(tile_n=64))
    assert (p["tile_n"], p["split_k"], p["waves"], p["workgroups"]) == (64, 2, 8, 256)
    assert tl.tl_gemm_plan(32, 57344, 8192, tl.layout(tile_n=64))["split_k"] == 1   # >= 2 tiles per CU
    p = tl.tl_gemm_plan(32, 8192, 8192, tl.layout(split_k=2))
    assert (p["tile_n"], p["split_k"], p["workgroups"]) == (64, 2, 256)
    # no whole-round (T, S) grid (257 strips), or K / 512 < 4: streaming kernel
    p = tl.tl_gemm_plan(32, 8192 + 32, 8192, d)
    assert (p["tile_n"], p["split_k"], p["waves"], p["workgroups"]) == (32, 4, 4, 1028)
    assert tl.tl_gemm_plan(32, 8192, 1024, d)["tile_n"] == 32          # 16 MB: small
    assert tl.tl_gemm_plan(32, 8192, 1024, tl.layout(tile_n=32))["waves"] == 8
    assert tl.tl_gemm_plan(64, 8192, 1024, tl.layout(tile_n=32))["waves"] == 8
    # four 16-row M tiles on 64-row tiles keep one K step in flight per wave,
    # which fits two waves per SIMD: 8 waves (bf16, read natively)
    assert tl.tl_gemm_plan(64, 8192, 1024, tl.layout(tile_n=64))["waves"] == 8
    assert tl.tl_gemm_plan(64, 8192, 1024, tl.layout(tile_n=64, elem_bytes=1))["waves"] == 4
    # 33 <= M <= 64: Llama QKV, O and down stay on the decode kernel, with the
    # activations staged in LDS for T = 4 tiles per workgroup and the largest
    # S whose grid fits one round of the CUs, filling >= 7/8 of it (QKV: 80
    # groups x 3); a weight whose 128 x 128 tiles fill the CUs (N >= 32768,
    # gate+up) takes the prefill kernel's, unless a tile or split is
    # requested, the weight is FP8, or the fetch emulates whole blocks
    for M in (33, 48, 64):
        for N, K, S, wgs in [(10240, 8192, 3, 240), (8192, 8192, 4, 256), (8192, 28672, 4, 256)]:
            p = tl.tl_gemm_plan(M, N, K, d)
            assert (p["kernel"], p["tile_n"], p["split_k"], p["waves"], p["workgroups"]) == (1, 32, S, 8, wgs), p
        # too few groups x K ranges to fill 7/8 of the CUs: 64-row streaming tiles
        p = tl.tl_gemm_plan(M, 8192, 2048, d)
        assert (p["kernel"], p["tile_n"], p["split_k"], p["waves"]) == (1, 64, 2, 8), (M, p)
        assert tl.tl_gemm_plan(M, 8192, 8192, tl.layout(tile_n=64))["tile_n"] == 64
        p = tl.tl_gemm_plan(M, 57344, 8192, d)
        assert (p["kernel"], p["tile_m"], p["tile_n"], p["split_k"], p["workgroups"]) == (2, 128, 128, 1, 448)
        assert tl.tl_gemm_plan(M, 32768, 8192, d)["kernel"] == 2
        assert tl.tl_gemm_plan(M, 32768 - 128, 8192, d)["kernel"] == 1
        assert tl.tl_gemm_plan(M, 57344, 8192, tl.layout(tile_n=64))["kernel"] == 1
        assert tl.tl_gemm_plan(M, 57344, 8192, tl.layout(split_k=1))["kernel"] == 1
        assert tl.tl_gemm_plan(M, 57344, 8192, tl.layout(elem_bytes=1))["kernel"] == 1
        rm = tl.layout(kind=tl.TL_LAYOUT_NK_ROW)
        assert tl.tl_gemm_plan(M, 57344, 8192, rm, tl.TL_FETCH_BLOCK)["kernel"] == 1
        assert tl.tl_gemm_plan(M, 57344, 8192, rm, tl.TL_FETCH_NATIVE)["kernel"] == 2
    assert tl.tl_gemm_plan(32, 57344, 8192, d)["kernel"] == 1
    p = tl.tl_gemm_plan(2048, 57344, 8192, d)
    assert p["kernel"] == 2 and p["tile_m"] == 256 and p["tile_n"] == 256
    assert tl.tl_gemm_plan(2048, 57344 + 128, 8192, d)["tile_n"] == 128
    p = tl.tl_gemm_plan(2048, 57344, 8192, tl.layout(tile_m=128))
    assert p["tile_m"] == 128


def test_fp8_plans():
    """FP8 (elem_bytes 1) weights: decode kernel only; 64 x 64 memory tiles
    (G = 4096, block_rows = 64) give 64-row compute tiles; 16-byte lane loads
    need block_cols >= 16; no prefill, grouped or emulated-latency path."""
    fp8 = tl.layout(elem_bytes=1, G=4096, block_rows=64)
    p = tl.tl_gemm_plan(8, 8192, 8192, fp8)
    assert p["kernel"] == 1 and p["tile_n"] == 64 and p["tile_k"] == 64
    assert tl.tl_read_amp(8, 8192, 8192, p["tile_m"], p["tile_n"], p["tile_k"], fp8, 4096)["amp"] == 1.0
    # tiles that neither fill two rounds nor divide the CUs (Llama QKV, 160
    # tiles): at most two rounds of 8-wave workgroups, not ~1024 short splits
    p = tl.tl_gemm_plan(8, 10240, 8192, fp8)
    assert (p["tile_n"], p["split_k"], p["waves"], p["workgroups"]) == (64, 3, 8, 480), p
    for args, status in (((128, 8192, 8192, fp8), tl.TL_EUNSUPPORTED),
                         ((8, 8192, 8192, tl.layout(elem_bytes=1, G=512, block_rows=64)), tl.TL_EUNSUPPORTED),
                         ((8, 8192, 8192, tl.layout(elem_bytes=3)), tl.TL_EUNSUPPORTED),
                         ((8, 8192, 8192, tl.layout(elem_bytes=0)), tl.TL_EINVAL)):
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_plan(*args)
        assert e.value.status == status, args
    with pytest.raises(tl.TLError) as e:       # the W8 entry point needs an FP8 descriptor
        tl.tl_gemm_w8(4096, 8192, None, 1 << 20, 8, 512, 512, tl.layout(), tl.TL_FETCH_BLOCK, stream=0)
    assert e.value.status == tl.TL_EINVAL
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_lgms(4096, 8192, 1 << 20, 8, 512, 512, fp8, 1000, 2, stream=0)
    assert e.value.status == tl.TL_EUNSUPPORTED


def test_prefill_plan_column_split():
    """256 x 256 tiles whose count leaves the last round part-empty are kept on
    the widest column range with a whole number of rounds; the rest of the
    columns take 256 x 256 tiles with K split S ways when those tiles times S
    fill the CUs (fp32 partials: split_k and workspace_bytes report them),
    else 128 x 128 tiles when those fit in one round."""
    bf = tl.layout(out_dtype=tl.TL_OUT_BF16)
    # QKV, bf16 out: 256 x 320 tiles fill one round exactly (256 tiles)
    qkv = tl.tl_gemm_plan(2048, 10240, 8192, bf)
    assert (qkv["tile_n"], qkv["workgroups"], qkv["split_k"], qkv["workspace_bytes"]) == (320, 256, 1, 0)
    # QKV, fp32 out (no 256 x 320 tiles): 256 x 256 on 8192 columns, the
    # rest with K split 4 ways
    qkv = tl.tl_gemm_plan(2048, 10240, 8192, tl.layout())
    assert qkv["tile_n"] == 256 and qkv["workgroups"] == 256 + 64 * 4
    assert qkv["split_k"] == 4 and qkv["workspace_bytes"] == 4 * 2048 * 2048 * 4
    o = tl.tl_gemm_plan(2048, 8192, 8192, bf)                                      # O: no split
    assert o["workgroups"] == 256 and o["split_k"] == 1 and o["workspace_bytes"] == 0
    # gate+up: 1792 tiles, 7 rounds -> a persistent grid of one workgroup per CU
    assert tl.tl_gemm_plan(2048, 57344, 8192, bf)["workgroups"] == 256
    # fp32 output, or a ragged M: one workgroup per tile
    assert tl.tl_gemm_plan(2048, 57344, 8192, tl.layout())["workgroups"] == 1792
    assert tl.tl_gemm_plan(2000, 57344, 8192, bf)["workgroups"] == 1792
    q4 = tl.tl_gemm_plan(4096, 10240, 8192, bf)                                    # 512 tiles of 256 x 320
    assert q4["tile_n"] == 320 and q4["workgroups"] == 256 and q4["split_k"] == 1
    q4 = tl.tl_gemm_plan(4096, 10240, 8192, tl.layout())
    assert q4["workgroups"] == 512 + 128 * 2 and q4["split_k"] == 2
    # K too short for the split (8 K steps per split at least): 128 x 128 rest
    short = tl.tl_gemm_plan(2048, 10240, 1024, tl.layout())
    assert short["workgroups"] == 256 + 256 and short["split_k"] == 1
    # a memory tile of 128 rows does not divide 320: 256 x 256 and the split
    tall128 = tl.tl_gemm_plan(2048, 10240, 8192, tl.layout(G=16384, block_rows=128, out_dtype=tl.TL_OUT_BF16))
    assert tall128["tile_n"] == 256 and tall128["split_k"] == 4
    # pinned tiles are never split: the 320 tiles go to a persistent grid
    # (fp32 output: one workgroup per tile)
    pinned = tl.layout(tile_m=256, tile_n=256, out_dtype=tl.TL_OUT_BF16)
    assert tl.tl_gemm_plan(2048, 10240, 8192, pinned)["workgroups"] == 256
    assert tl.tl_gemm_plan(2048, 10240, 8192, tl.layout(tile_m=256, tile_n=256))["workgroups"] == 320
    # a memory tile taller than the 128-row remainder tiles keeps one launch
    tall = tl.layout(G=65536, block_rows=256, out_dtype=tl.TL_OUT_BF16)
    assert tl.tl_gemm_plan(2048, 10240, 8192, tall)["workgroups"] == 256
    # small and medium M: K split over all the columns where the tiles are
    # fewer than the CUs -- 128 x 128 tiles at M <= 128, 256 x 256 above
    for M in (65, 96, 128):
        for N, K, S in [(10240, 8192, 3), (8192, 8192, 4), (8192, 28672, 4)]:
            p = tl.tl_gemm_plan(M, N, K, bf)
            assert (p["tile_m"], p["tile_n"], p["split_k"]) == (128, 128, S), (M, N, K, p)
            assert p["workgroups"] == N // 128 * S and p["workspace_bytes"] == S * M * N * 4
        g = tl.tl_gemm_plan(M, 57344, 8192, bf)                 # 448 tiles: no split
        assert (g["tile_m"], g["tile_n"], g["split_k"], g["workgroups"]) == (128, 128, 1, 448)
    p = tl.tl_gemm_plan(129, 10240, 8192, bf)
    assert (p["tile_m"], p["tile_n"], p["split_k"], p["workgroups"]) == (256, 256, 6, 240)
    # a K of 1000: 16 K steps (the last partial) split in two
    p = tl.tl_gemm_plan(100, 1024, 1000, tl.layout(kind=tl.TL_LAYOUT_NK_ROW), tl.TL_FETCH_NATIVE)
    assert (p["tile_m"], p["split_k"], p["workgroups"]) == (128, 2, 16)
    # pinned tiles: no K split
    assert tl.tl_gemm_plan(96, 10240, 8192, tl.layout(tile_m=128, tile_n=128))["split_k"] == 1
    tall = tl.layout(G=65536, block_rows=256, tile_m=256, tile_n=256, out_dtype=tl.TL_OUT_BF16)
    assert tl.tl_gemm_plan(96, 10240, 8192, tall)["split_k"] == 1


def test_gemm_plan_error_codes():
    d = tl.layout()
    cases = [
        ((0, 64, 64, d), tl.TL_EINVAL),
        ((8, 64, 64, tl.layout(G=1000)), tl.TL_EINVAL),
        ((8, 64, 100, d), tl.TL_EUNSUPPORTED),               # K % 8: rows of A not 16-byte aligned
        ((2048, 64, 100, d), tl.TL_EUNSUPPORTED),
        ((8, 64, 72, tl.layout(elem_bytes=1, block_rows=64)), tl.TL_EUNSUPPORTED),   # FP8: K % 16
        ((8, 64, 64, tl.layout(elem_bytes=4)), tl.TL_EUNSUPPORTED),    # only bf16 and FP8 weights
        ((256, 64, 64, tl.layout(kind=tl.TL_LAYOUT_KN_ROW)), tl.TL_EUNSUPPORTED),   # [K][N]: decode only
        ((8, 64, 64, tl.layout(G=512, block_rows=64)), tl.TL_EUNSUPPORTED),   # bc = 4
        ((8, 64, 64, tl.layout(out_dtype=7)), tl.TL_EINVAL),
        ((8, 64, 64, tl.layout(tile_n=48)), tl.TL_EUNSUPPORTED),
    ]
    for (M, N, K, desc), want in cases:
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_plan(M, N, K, desc)
        assert e.value.status == want, (M, N, K)
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_plan(8, 64, 64, d, fetch_mode=0x8)
    assert e.value.status == tl.TL_EINVAL
    # block-granular fetch on a row-major weight: G a power of two >= 128,
    # decode kernel only
    rm = tl.layout(kind=tl.TL_LAYOUT_NK_ROW, G=4096)
    assert tl.tl_gemm_plan(8, 64, 64, rm, tl.TL_FETCH_BLOCK)["kernel"] == 1
    for bad_G in (64, 100, 0):
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_plan(8, 64, 64, tl.layout(kind=tl.TL_LAYOUT_NK_ROW, G=bad_G), tl.TL_FETCH_BLOCK)
        assert e.value.status == tl.TL_EINVAL
    # above 64 rows the prefill kernel emulates it too, with one tile shape
    # (no column split) so tl_read_amp follows its count
    pp = tl.tl_gemm_plan(2048, 10240, 8192, rm, tl.TL_FETCH_BLOCK)
    assert pp["kernel"] == 2 and pp["workgroups"] == (2048 // pp["tile_m"]) * (10240 // pp["tile_n"])
    for N, K in ((64, 96), (40, 64)):          # the block emulation needs whole 64-wide steps and 32-row tiles
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_plan(8, N, K, rm, tl.TL_FETCH_BLOCK)
        assert e.value.status == tl.TL_EUNSUPPORTED


def test_kn_row_plans():
    """A weight stored [K][N] (the paper's row-major layout) runs the decode
    kernel with 64-column tiles and 64-row K steps; its plan rules."""
    kn = tl.layout(kind=tl.TL_LAYOUT_KN_ROW)
    for M, N, K in ((1, 1024, 4096), (8, 57344, 8192), (32, 8192, 28672), (64, 8, 64)):
        p = tl.tl_gemm_plan(M, N, K, kn, tl.TL_FETCH_NATIVE)
        assert p["kernel"] == 1 and p["tile_n"] == 64 and p["tile_k"] == 64
        assert p["tile_m"] == 16 * {1: 1, 2: 2, 3: 4, 4: 4}[-(-M // 16)]
        assert p["workgroups"] == -(-N // 64) * p["split_k"]
        assert K // 64 >= p["split_k"] >= 1 and p["waves"] in (4, 8)
    assert tl.tl_gemm_plan(8, 57344, 8192, kn)["split_k"] == 1          # 896 tiles: no K split
    assert tl.tl_gemm_plan(8, 4096, 8192, kn, tl.TL_FETCH_NATIVE)["split_k"] == 8
    blk = tl.layout(kind=tl.TL_LAYOUT_KN_ROW, G=4096)
    assert tl.tl_gemm_plan(8, 1024, 2048, blk, tl.TL_FETCH_BLOCK)["tile_n"] == 64
    rejected = [
        ((65, 1024, 1024, kn, 0), tl.TL_EUNSUPPORTED),       # decode kernel only
        ((8, 1024, 1000, kn, 0), tl.TL_EUNSUPPORTED),        # whole 64-row K steps
        ((8, 1020, 1024, kn, 0), tl.TL_EUNSUPPORTED),        # 16-byte row pieces
        ((8, 1024, 1024, tl.layout(kind=tl.TL_LAYOUT_KN_ROW, tile_n=32), 0), tl.TL_EUNSUPPORTED),
        ((8, 1024, 1024, tl.layout(kind=tl.TL_LAYOUT_KN_ROW, elem_bytes=1), 0), tl.TL_EUNSUPPORTED),
        ((8, 1000, 1024, blk, tl.TL_FETCH_BLOCK), tl.TL_EUNSUPPORTED),   # block: 128-byte row segments
        ((8, 1024, 1024, tl.layout(kind=tl.TL_LAYOUT_KN_ROW, G=100), tl.TL_FETCH_BLOCK), tl.TL_EINVAL),
        ((8, 1 << 27, 64, kn, 0), tl.TL_EUNSUPPORTED),       # one lane's eight rows span < 2^31 bytes
    ]
    for (M, N, K, d, f), want in rejected:
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_plan(M, N, K, d, f)
        assert e.value.status == want, (M, N, K)


def test_noalloc_rejects_before_device_work():
    """tl_gemm_noalloc: partials beyond the static scratch -> TL_ESCRATCH and
    the per-stream tally -> TL_EUNSUPPORTED, before any HIP call; its
    arguments are otherwise checked as tl_gemm's."""
    d = tl.layout(split_k=16)
    assert tl.tl_gemm_plan(64, 32768, 65536, d)["workspace_bytes"] > tl.TL_NOALLOC_SCRATCH_BYTES
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_noalloc(4096, 8192, 16384, 64, 32768, 65536, d, tl.TL_FETCH_BLOCK, stream=0)
    assert e.value.status == tl.TL_ESCRATCH
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_noalloc(4096, 8192, 16384, 8, 64, 64, tl.layout(), tl.TL_FETCH_BLOCK | tl.TL_FETCH_COUNT,
                           stream=0)
    assert e.value.status == tl.TL_EUNSUPPORTED
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_noalloc(0, 0, 0, 8, 64, 64, tl.layout(), tl.TL_FETCH_BLOCK, stream=0)
    assert e.value.status == tl.TL_EINVAL


def test_gemm_plan_maximum_sizes():
    """The prefill kernel addresses A and W with 32-bit byte offsets: a weight
    just below 4 GB is planned, one of 4 GB is rejected; the decode kernel has
    64-bit weight offsets and takes larger weights; sizes are int32."""
    d = tl.layout()
    assert tl.tl_gemm_plan(256, 131072, 16320, d)["kernel"] == 2          # 4,278,190,080 bytes
    for N, K in ((131072, 16384), (131072, 16328)):                        # 2^32 bytes; padded copy of 2^32
        with pytest.raises(tl.TLError) as e:
            tl.tl_gemm_plan(256, N, K, d)
        assert e.value.status == tl.TL_EUNSUPPORTED
    assert tl.tl_gemm_plan(8, 131072, 32768, d)["kernel"] == 1            # 8 GiB weight, decode
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm_plan(8, (1 << 31) + 1, 64, d)
    assert e.value.status == tl.TL_EINVAL


def test_gemm_plan_padded_weights():
    """N and K that the memory tile does not divide (padded copies, Section
    3.3): ceil-sized grids, same kernels."""
    d = tl.layout()
    p = tl.tl_gemm_plan(8, 100, 200, d)
    assert p["kernel"] == 1 and p["tile_n"] == 32 and p["workgroups"] == 4 * p["split_k"]
    p = tl.tl_gemm_plan(8, 8200, 28680, d)
    assert p["kernel"] == 1 and p["workgroups"] == 257 * p["split_k"]
    p = tl.tl_gemm_plan(2048, 1000, 1000, d)
    assert p["kernel"] == 2 and p["workgroups"] == 8 * 8
    fp8 = tl.layout(elem_bytes=1, block_rows=64)
    assert tl.tl_gemm_plan(8, 100, 208, fp8)["tile_n"] == 64
    assert tl.tl_gemm_plan(8, 100, 200, tl.layout(kind=tl.TL_LAYOUT_NK_ROW), tl.TL_FETCH_NATIVE)["kernel"] == 1


def test_entry_points_reject_before_device_work():
    """NULL / misaligned pointers and bad descriptors return an error status
    and enqueue nothing; these paths make no HIP call."""
    d = tl.layout()
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm(0, 0, 0, 8, 64, 64, d, tl.TL_FETCH_BLOCK, stream=0)
    assert e.value.status == tl.TL_EINVAL
    with pytest.raises(tl.TLError) as e:
        tl.tl_gemm(16, 32, 8, 8, 64, 64, d, tl.TL_FETCH_BLOCK, stream=0)   # C misaligned
    assert e.value.status == tl.TL_EINVAL
    with pytest.raises(tl.TLError) as e:
        tl.tl_repack(0, 0, 64, 64, 2, 4096, 32, stream=0)
    assert e.value.status == tl.TL_EINVAL
    with pytest.raises(tl.TLError) as e:
        tl.tl_repack(4096, 8192, 64, 64, 3, 4096, 32, stream=0)          # elem_bytes
    assert e.value.status == tl.TL_EINVAL
    with pytest.raises(tl.TLError) as e:        # overlaps only the padding of the 64 x 64 tile-major copy
        tl.tl_repack(11264, 4096, 48, 64, 2, 4096, 32, stream=0)
    assert e.value.status == tl.TL_EINVAL
    with pytest.raises(tl.TLError) as e:
        tl.tl_unpack(4096, 11264, 48, 64, 2, 4096, 32, stream=0)
    assert e.value.status == tl.TL_EINVAL
    # a 6144-byte row-major source directly followed by its 8192-byte copy is
    # not an overlap (validation passes; the launch then fails without a GPU)
    for fn, a, b in ((tl.tl_repack, 4096, 4096 + 6144), (tl.tl_unpack, 4096 + 6144, 4096)):
        with pytest.raises(tl.TLError) as e:
            fn(a, b, 48, 64, 2, 4096, 32, stream=0)
        assert e.value.status == tl.TL_EHIP
    with pytest.raises(tl.TLError) as e:                                  # overlap
        tl.tl_repack(4096, 4096 + 1024, 64, 64, 2, 4096, 32, stream=0)
    assert e.value.status == tl.TL_EINVAL
    # empty matrices are a no-op
    tl.tl_repack(0, 0, 0, 64, 2, 4096, 32, stream=0)


def test_gemm_grouped_rejects_before_device_work():
    """tl_gemm_grouped validates every argument on the host; each case below
    fails before any HIP call (fake, aligned addresses), and total_rows == 0
    is a no-op."""
    N, K = 64, 128
    good = dict(A=1 << 12, a_rows=64, token_ids=1 << 20, group_offsets=1 << 21, num_groups=4,
                total_rows=32, max_group_rows=16, W=1 << 24, group_stride=N * K * 2, C=1 << 30,
                N=N, K=K, layout=tl.layout(), fetch_mode=tl.TL_FETCH_BLOCK)

    def call(**kw):
        a = dict(good, **kw)
        tl.tl_gemm_grouped(a["A"], a["a_rows"], a["token_ids"], a["group_offsets"], a["num_groups"],
                           a["total_rows"], a["max_group_rows"], a["W"], a["group_stride"], a["C"],
                           a["N"], a["K"], a["layout"], a["fetch_mode"], stream=0)

    cases = [
        (dict(num_groups=0), tl.TL_EINVAL),
        (dict(total_rows=-1), tl.TL_EINVAL),
        (dict(a_rows=0), tl.TL_EINVAL),
        (dict(max_group_rows=0), tl.TL_EINVAL),
        (dict(token_ids=None, a_rows=16), tl.TL_EINVAL),         # identity rows past A
        (dict(group_stride=N * K * 2 - 16), tl.TL_EINVAL),
        (dict(group_stride=N * K * 2 + 8), tl.TL_EINVAL),
        (dict(group_offsets=None), tl.TL_EINVAL),
        (dict(group_offsets=(1 << 21) + 2), tl.TL_EINVAL),
        (dict(token_ids=(1 << 20) + 1), tl.TL_EINVAL),
        (dict(A=(1 << 12) + 8), tl.TL_EINVAL),
        (dict(C=(1 << 12) + 64), tl.TL_EINVAL),                   # C overlaps A
        (dict(C=(1 << 24) + 4096), tl.TL_EINVAL),                 # C overlaps W
        (dict(N=48, K=136), tl.TL_EINVAL),                        # group_stride < the padded copy
        (dict(layout=tl.layout(split_k=2)), tl.TL_EUNSUPPORTED),
        (dict(layout=tl.layout(tile_m=128)), tl.TL_EUNSUPPORTED),
        (dict(layout=tl.layout(kind=tl.TL_LAYOUT_NK_ROW)), None),  # valid: checked by its own case below
        (dict(layout=tl.layout(kind=tl.TL_LAYOUT_NK_ROW), fetch_mode=tl.TL_FETCH_BLOCK), None),
        (dict(layout=tl.layout(kind=tl.TL_LAYOUT_KN_ROW)), tl.TL_EUNSUPPORTED),
        (dict(num_groups=1 << 30, N=4096, group_stride=4096 * K * 2), tl.TL_EUNSUPPORTED),  # grid >= 2^31
    ]
    for kw, status in cases:
        if status is None:
            continue
        with pytest.raises(tl.TLError) as e:
            call(**kw)
        assert e.value.status == status, kw
    # row-major weights read in whole blocks are a decode-only (ungrouped) mode
    with pytest.raises(tl.TLError) as e:
        call(layout=tl.layout(kind=tl.TL_LAYOUT_NK_ROW, G=4096), fetch_mode=tl.TL_FETCH_BLOCK)
    assert e.value.status == tl.TL_EUNSUPPORTED
    call(total_rows=0)                                            # enqueues nothing
