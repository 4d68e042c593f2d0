"""Pins for the CPU oracle: each test checks the oracle against something other
than itself -- a value the paper prints, a numpy library routine, a closed form,
or an invariant -- so that a dropped term, a wrong sign or index, or a transposed
operand in the oracle fails at least one of them.  CPU only."""
import itertools
import os
import math

import numpy as np
import pytest

import oracle
from oracle import NK_ROW, KN_ROW, TILE
from paper_2607_04031_amd import synth
from tests._golden import load


# ---------------------------------------------------------------------------
# Repack / Eq. 2
# ---------------------------------------------------------------------------

REPACK_CASES = [
    # rows, cols, elem_bytes, G, block_rows
    (64, 128, 2, 4096, 32),      # the evaluated (64, 32) BF16 tile
    (128, 256, 2, 4096, 8),
    (128, 64, 2, 4096, 32),      # one block column
    (256, 512, 1, 4096, 64),     # FP8 64 x 64
    (96, 320, 2, 512, 16),       # non power-of-two block counts
    (64, 512, 4, 1024, 4),       # 4-byte elements
    (32, 4096, 2, 16384, 4),
]


@pytest.mark.parametrize("rows,cols,s,G,br", REPACK_CASES)
def test_repack_equals_numpy_reshape_transpose(rows, cols, s, G, br):
    """Eq. 2 == the block reshape: [R/br, br, C/bc, bc] -> swap axes 1 and 2."""
    bc = G // (s * br)
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[s]
    src = synth.random_bytes(rows * cols * s, seed=rows + cols + G).view(dt).reshape(rows, cols)
    got = oracle.repack(src, G, br).reshape(-1)
    want = src.reshape(rows // br, br, cols // bc, bc).transpose(0, 2, 1, 3).reshape(-1)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("rows,cols,s,G,br", REPACK_CASES)
def test_repack_roundtrip_and_bijection(rows, cols, s, G, br):
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[s]
    src = synth.random_bytes(rows * cols * s, seed=7).view(dt).reshape(rows, cols)
    tm = oracle.repack(src, G, br)
    assert np.array_equal(oracle.unpack(tm, G, br), src)
    # every destination element slot is hit exactly once
    offs = np.array([oracle.tm_offset(r, c, cols, s, G, br)
                     for r in range(0, rows, max(1, rows // 16))
                     for c in range(cols)])
    assert len(set(offs.tolist())) == offs.size
    assert offs.min() >= 0 and offs.max() < rows * cols * s
    assert np.all(offs % s == 0)


# Section 3.3: a dimension that is not a multiple of the memory tile's side
# is padded to whole memory tiles.
PADDED_CASES = [
    # rows, cols, elem_bytes, G, block_rows
    (40, 100, 2, 4096, 32),      # both dimensions ragged, (64, 32) BF16 tile
    (33, 64, 2, 4096, 32),       # one row past a strip
    (32, 72, 2, 4096, 32),       # cols ragged only
    (7, 24, 2, 4096, 32),        # smaller than one memory tile
    (100, 200, 1, 4096, 64),     # FP8 64 x 64
    (50, 136, 2, 512, 8),        # bc = 32
    (65, 264, 2, 16384, 16),     # bc = 512
    (3, 5, 4, 1024, 4),          # 4-byte elements, bc = 64
]


@pytest.mark.parametrize("rows,cols,s,G,br", PADDED_CASES)
def test_padded_repack_equals_numpy_pad_then_block_reshape(rows, cols, s, G, br):
    """Zero-pad to whole memory tiles with numpy, then the block reshape: the
    padded tile-major copy, pads included, without the oracle's offsets."""
    bc = G // (s * br)
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[s]
    src = synth.random_bytes(rows * cols * s, seed=rows * cols + G).view(dt).reshape(rows, cols)
    R, C = -(-rows // br) * br, -(-cols // bc) * bc
    padded = np.pad(src, ((0, R - rows), (0, C - cols)))
    want = padded.reshape(R // br, br, C // bc, bc).transpose(0, 2, 1, 3).reshape(-1)
    got = oracle.repack(src, G, br)
    assert got.shape == (R, C)
    assert np.array_equal(got.reshape(-1), want)
    assert oracle.packed_bytes(rows, cols, s, G, br) == R * C * s == (R // br) * (C // bc) * G


@pytest.mark.parametrize("rows,cols,s,G,br", PADDED_CASES)
def test_padded_roundtrip_and_offsets_inside_copy(rows, cols, s, G, br):
    dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[s]
    src = synth.random_bytes(rows * cols * s, seed=11).view(dt).reshape(rows, cols)
    tm = oracle.repack(src, G, br)
    assert np.array_equal(oracle.unpack(tm, G, br, rows, cols), src)
    offs = np.array([oracle.tm_offset(r, c, cols, s, G, br) for r in range(rows) for c in range(cols)])
    assert len(set(offs.tolist())) == offs.size
    assert offs.min() >= 0 and offs.max() + s <= oracle.packed_bytes(rows, cols, s, G, br)
    # every memory tile of the copy holds at least one element of the matrix
    assert len(set((offs // G).tolist())) == oracle.packed_bytes(rows, cols, s, G, br) // G


def test_padding_is_invisible_when_the_tile_divides():
    """Divisible shapes: the padded definition is the paper's Eq. 2 exactly."""
    for (rows, cols, s, G, br) in REPACK_CASES:
        assert oracle.packed_bytes(rows, cols, s, G, br) == rows * cols * s
        assert oracle.repack(np.zeros((rows, cols), {1: np.uint8, 2: np.uint16, 4: np.uint32}[s]), G, br).shape \
            == (rows, cols)


def test_eq3_four_d_strides_view():
    """Eq. 3: the tile-major buffer viewed with shape (a, b, K/a, N/b) and
    element strides (1, a, ab, Kb) returns element (i, j) of the K x N matrix
    at coordinates (i mod a, j mod b, i / a, j / b).  Built with numpy's
    stride machinery, not with the oracle's offset function."""
    K, N, s, G, b = 512, 128, 2, 4096, 32
    a = G // (s * b)
    W = synth.random_bytes(N * K * s, seed=3).view(np.uint16).reshape(N, K)   # W[j][i]
    tm = oracle.repack(W, G, b).reshape(-1)
    view = np.lib.stride_tricks.as_strided(
        tm, shape=(a, b, K // a, N // b),
        strides=(1 * s, a * s, a * b * s, K * b * s))
    for i, j in itertools.product(range(0, K, 37), range(0, N, 11)):
        assert view[i % a, j % b, i // a, j // b] == W[j, i]


def test_eq4_tilebase_at_aligned_points():
    """Eq. 4: at memory-tile-aligned (i, j), offset = (K j + i b) s."""
    for (K, N, s, G, b) in [(512, 128, 2, 4096, 32), (1024, 256, 1, 4096, 64),
                            (256, 64, 2, 1024, 8)]:
        a = G // (s * b)
        for i in range(0, K, a):
            for j in range(0, N, b):
                assert oracle.tm_offset(j, i, K, s, G, b) == (K * j + i * b) * s


def test_case2_bit_permutation_example():
    """Section 4.3 Case 2: FP8 128 x 32 memory tile, 32 x 32 TMA tile.  The
    actual intra-tile offset has fields (col | sub | row); the sub-tile view
    assumed (sub | col | row)."""
    g = load("paper_case2_bitperm.txt")
    a, b, u = g["memory_tile_a"], g["memory_tile_b"], g["tma_tile_u"]
    s, G = g["elem_bytes"], g["granularity"]
    assert a * b * s == G

    def pack(fields, vals):
        out = 0
        for name_w in fields.split():
            name, w = name_w.split(":")
            w = int(w)
            assert 0 <= vals[name] < (1 << w)
            out = (out << w) | vals[name]
        return out

    K = 4 * a  # four memory tiles along the contiguous dim, one strip of b
    for sub, col, row in itertools.product(range(a // u), range(b), range(u)):
        i = sub * u + row       # contiguous index inside the memory tile
        j = col
        off = oracle.tm_offset(j, i, K, s, G, b) % G
        vals = {"sub": sub, "col": col, "row": row}
        assert off == pack(g["actual_fields"], vals)
        # the assumed sub-tile offset differs exactly by the field permutation
        assumed = pack(g["assumed_fields"], vals)
        assert assumed == sub * (u * b) + col * u + row


def test_view_example_addresses_same_elements():
    """Section 4.3: the 2-D, 3-D and 4-D descriptors of one FP8 384 x 128
    column-major matrix address the same 128 x 64 tile.  The leading-stride
    rule (strides below K feed the contiguous index i, the rest feed K*j)
    recovers (i, j), and the tile-major offsets of the three views agree."""
    g = load("paper_view_example.txt")
    K, N = g["K"], g["N"]

    def parse(v):
        return [list(map(int, p.split(","))) for p in v.split(";")]

    views = {name: parse(g[name]) for name in ("view2d", "view3d", "view4d")}
    # element strides of each view: the first dimension is contiguous; the
    # others follow from how each view tiles the K x N column-major matrix
    strides = {
        "view2d": [1, K],
        "view3d": [1, K, 128],
        "view4d": [1, K, 128, 64 * K],
    }
    sets = {}
    for name, (dims, coords, tile) in views.items():
        st = strides[name]
        offs = set()
        for idx in itertools.product(*[range(t) for t in tile]):
            lin = sum((c + x) * s_ for c, x, s_ in zip(coords, idx, st))
            i = sum((c + x) * s_ for c, x, s_ in zip(coords, idx, st) if s_ < K)
            kj = sum((c + x) * s_ for c, x, s_ in zip(coords, idx, st) if s_ >= K)
            assert kj % K == 0 and i + kj == lin
            j = kj // K
            assert 0 <= i < K and 0 <= j < N
            offs.add(oracle.tm_offset(j, i, K, 1, 4096, 64))
        sets[name] = offs
    logical = {oracle.tm_offset(j, i, K, 1, 4096, 64)
               for i in range(256, 384) for j in range(64, 128)}
    assert sets["view2d"] == sets["view3d"] == sets["view4d"] == logical
    assert len(logical) == 128 * 64


def _numpy_tile_positions(K, N, a, b):
    """Position of every element of a K x N column-major matrix (element
    (i, j) has id j * K + i) in the tile-major order, built with numpy's
    reshape and transpose alone: pos[j * K + i] = element index in the copy."""
    ids = np.arange(N * K, dtype=np.int64).reshape(N, K)          # [j][i]
    order = ids.reshape(N // b, b, K // a, a).transpose(0, 2, 1, 3).ravel()
    pos = np.empty(N * K, dtype=np.int64)
    pos[order] = np.arange(N * K, dtype=np.int64)
    return pos


def test_view_offsets_paper_example_order():
    """orc_view_offsets on the Section 4.3 example (FP8 384 x 128 column-major
    matrix, 128 x 64 box at (256, 64), 64 x 64 memory tiles): the 2-D, 3-D and
    4-D descriptors give the same offsets in the same order -- the contiguous
    index i = 256 + x0 fastest, then j = 64 + x1 -- and every offset is the
    element's place in a tile-major copy built by numpy's reshape/transpose."""
    g = load("paper_view_example.txt")
    K, N, s = g["K"], g["N"], g["elem_bytes"]
    G, b = 4096, 64
    a = G // (s * b)
    pos = _numpy_tile_positions(K, N, a, b)
    want = np.array([pos[(64 + x1) * K + 256 + x0] * s for x1 in range(64) for x0 in range(128)])

    def parse(v):
        return [list(map(int, p.split(","))) for p in v.split(";")]

    strides = {"view2d": [1, K], "view3d": [1, K, 128], "view4d": [1, K, 128, 64 * K]}
    for name in ("view2d", "view3d", "view4d"):
        _, coords, box = parse(g[name])
        got = oracle.view_offsets(strides[name], coords, box, K, s, G, b)
        assert np.array_equal(got, want), name


def test_view_offsets_identity_extreme():
    """block_rows = 1 with K * s = G: a memory tile is one whole column of
    the column-major matrix, so the tile-major copy is the matrix itself and
    every view's offsets are its linear element indices times s (dimension 0
    fastest), for 2-D, 3-D and 4-D views of bf16 and FP8 matrices."""
    for s, K, N in ((2, 2048, 48), (1, 4096, 24)):
        G = K * s
        cases = [([1, K], [5, 3], [40, 7]),
                 ([1, K, 256], [16, 2, 1], [64, 5, 3]),
                 ([1, 512, K, 4 * K], [8, 1, 1, 2], [32, 2, 3, 4])]
        for strides, coords, box in cases:
            got = oracle.view_offsets(strides, coords, box, K, s, G, 1)
            want = []
            for idx in itertools.product(*[range(n) for n in reversed(box)]):
                x = idx[::-1]                                   # dimension 0 fastest
                want.append(sum((c + xi) * st for c, xi, st in zip(coords, x, strides)) * s)
            assert np.array_equal(got, np.array(want)), (s, strides)


def test_view_offsets_case2_field_layout():
    """Section 4.3 Case 2: an FP8 128 x 32 memory tile read by a 32-wide box
    (u = 32 along the contiguous dimension, all b = 32 columns).  The box of
    sub-tile t, element (row r along the contiguous dimension, column c), sits
    at intra-tile offset c * a + t * u + r (fields col | sub | row); boxes in
    the second memory tile of the strip add G."""
    g = load("paper_case2_bitperm.txt")
    a, b, u, s, G = g["memory_tile_a"], g["memory_tile_b"], g["tma_tile_u"], g["elem_bytes"], g["granularity"]
    K = 2 * a
    for tile in range(2):
        for t in range(a // u):
            got = oracle.view_offsets([1, K], [tile * a + t * u, 0], [u, b], K, s, G, b)
            want = np.array([tile * G + (c * a + t * u + r) * s for c in range(b) for r in range(u)])
            assert np.array_equal(got, want), (tile, t)


def test_memory_tile_shapes_and_identity_extremes():
    """Section 3.1: shapes multiply to G; the (contiguous = G/s, other = 1)
    extreme is the plain row-major order, so the repack is the identity;
    a block as wide as the whole row is also the identity."""
    g = load("paper_memory_tiles.txt")
    for key in ("fp8_square_tile", "fp8_row_major_extreme", "bf16_eval_tile"):
        a, b, s, G = map(int, g[key].split(","))
        assert a * b * s == G
    a, b, s, G = map(int, g["fp8_row_major_extreme"].split(","))
    src = synth.random_bytes(8 * 8192, seed=1).reshape(8, 8192)
    assert np.array_equal(oracle.repack(src, G, b), src)
    # bc == cols: one block column per strip
    src16 = synth.random_bytes(64 * 64 * 2, seed=2).view(np.uint16).reshape(64, 64)
    assert np.array_equal(oracle.repack(src16, 4096, 32), src16)


# ---------------------------------------------------------------------------
# GEMM
# ---------------------------------------------------------------------------

def test_gemm_matches_numpy_float64():
    A = synth.normal_bf16((7, 96), seed=1)
    W = synth.normal_bf16((40, 96), seed=2, sigma=0.02)
    Af, Wf = synth.bf16_bits_to_f32(A).astype(np.float64), synth.bf16_bits_to_f32(W).astype(np.float64)
    want = Af @ Wf.T
    got = oracle.gemm_f64(A, W)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-14)


def test_gemm_orientation_not_transposed():
    """A non-square, asymmetric case where A W^T and A W (or W A^T) differ."""
    A = synth.small_int_bf16((3, 5), seed=4)
    W = synth.small_int_bf16((2, 5), seed=5)
    Af, Wf = synth.bf16_bits_to_f32(A), synth.bf16_bits_to_f32(W)
    got = oracle.gemm_f64(A, W)
    assert got.shape == (3, 2)
    for m in range(3):
        for n in range(2):
            assert got[m, n] == sum(float(Af[m, k]) * float(Wf[n, k]) for k in range(5))


def test_gemm_one_hot_selects_weight_column():
    K = 256
    A, ks = synth.one_hot_bf16(9, K, seed=3)
    W = synth.normal_bf16((33, K), seed=4, sigma=0.02)
    got = oracle.gemm_f64(A, W)
    Wf = synth.bf16_bits_to_f32(W).astype(np.float64)
    assert np.array_equal(got, Wf[:, ks].T)


def test_gemm_small_integers_exact_and_zero_weight():
    A = synth.small_int_bf16((5, 300), seed=8)
    W = synth.small_int_bf16((17, 300), seed=9)
    Ai = synth.bf16_bits_to_f32(A).astype(np.int64)
    Wi = synth.bf16_bits_to_f32(W).astype(np.int64)
    assert np.array_equal(oracle.gemm_f64(A, W), (Ai @ Wi.T).astype(np.float64))
    Z = np.zeros_like(W)
    assert np.all(oracle.gemm_f64(A, Z) == 0.0)


def test_gemm_points_equal_full():
    A = synth.normal_bf16((4, 64), seed=1)
    W = synth.normal_bf16((20, 64), seed=2, sigma=0.02)
    full = oracle.gemm_f64(A, W)
    ms = np.array([0, 3, 2, 1]); ns = np.array([19, 0, 7, 7])
    assert np.array_equal(oracle.gemm_f64_points(A, W, ms, ns), full[ms, ns])


def _group_of_row(offsets, r):
    """Group of output row r by a linear scan (the grouped oracle loops over groups instead)."""
    for e in range(len(offsets) - 1):
        if offsets[e] <= r < offsets[e + 1]:
            return e
    raise AssertionError(r)


@pytest.mark.parametrize("with_ids", [True, False])
def test_grouped_gemm_brute_force_rows(with_ids):
    """Row-wise brute force with exact integers: row r takes the weight of the
    group whose offset range holds r and the A row its token id names.  Empty
    groups (first, middle, last) and a token used by several groups included."""
    K, N = 24, 5
    offsets = [0, 0, 3, 3, 7, 8, 8]
    A = synth.small_int_bf16((6 if with_ids else 8, K), seed=21)
    Ws = [synth.small_int_bf16((N, K), seed=30 + e) for e in range(len(offsets) - 1)]
    ids = np.array([5, 0, 2, 2, 1, 4, 0, 3]) if with_ids else None
    got = oracle.grouped_gemm_f64(A, ids, offsets, Ws)
    Ai = synth.bf16_bits_to_f32(A).astype(np.int64)
    assert got.shape == (offsets[-1], N)
    for r in range(offsets[-1]):
        e = _group_of_row(offsets, r)
        t = ids[r] if with_ids else r
        Wi = synth.bf16_bits_to_f32(Ws[e]).astype(np.int64)
        for n in range(N):
            assert got[r, n] == float(sum(int(Ai[t, k]) * int(Wi[n, k]) for k in range(K)))


def test_grouped_gemm_equals_stacked_weights_einsum():
    """The same rows through a per-row weight stack and numpy einsum in float64."""
    K, N = 64, 12
    routing = synth.moe_routing(M=10, E=6, topk=2, seed=5)
    offsets, ids = synth.moe_tables(routing, E=6)
    A = synth.normal_bf16((10, K), seed=6)
    Ws = [synth.normal_bf16((N, K), seed=40 + e, sigma=0.02) for e in range(6)]
    got = oracle.grouped_gemm_f64(A, ids, offsets, Ws)
    Af = synth.bf16_bits_to_f32(A).astype(np.float64)
    Wf = np.stack([synth.bf16_bits_to_f32(W).astype(np.float64) for W in Ws])
    groups = np.searchsorted(offsets, np.arange(offsets[-1]), side="right") - 1
    want = np.einsum("rnk,rk->rn", Wf[groups], Af[ids])
    assert np.allclose(got, want, rtol=1e-12, atol=1e-14)


def test_moe_routing_tables():
    """Top-8 of 128 distinct experts per token: every token appears in exactly
    8 groups, once per group, and group rows list tokens in ascending order."""
    routing = synth.moe_routing()
    assert routing.shape == (synth.QWEN_TOKENS, synth.QWEN_TOPK)
    assert all(len(set(r)) == synth.QWEN_TOPK for r in routing.tolist())
    offsets, ids = synth.moe_tables(routing)
    assert offsets[0] == 0 and offsets[-1] == synth.QWEN_TOKENS * synth.QWEN_TOPK
    assert np.all(np.diff(offsets) >= 0)
    assert np.array_equal(np.bincount(ids, minlength=synth.QWEN_TOKENS),
                          np.full(synth.QWEN_TOKENS, synth.QWEN_TOPK))
    for e in range(synth.QWEN_EXPERTS):
        g = ids[offsets[e]:offsets[e + 1]]
        assert np.all(np.diff(g) > 0)
        assert all(e in routing[t] for t in g.tolist())


def test_silu_values():
    """silu(x) = x * sigmoid(x): closed-form points and limits."""
    assert oracle.silu(0.0) == 0.0
    assert oracle.silu(1.0) == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)
    assert oracle.silu(-1.0) == pytest.approx(-1.0 / (1.0 + math.e), rel=1e-15)
    assert oracle.silu(40.0) == pytest.approx(40.0, rel=1e-15)      # sigmoid -> 1
    assert abs(oracle.silu(-40.0)) < 1e-15                            # sigmoid -> 0
    for x in np.linspace(-6, 6, 25):                                  # silu(x) - silu(-x) = x
        assert oracle.silu(x) - oracle.silu(-x) == pytest.approx(x, abs=1e-14)


def test_swiglu_equals_gemm_halves_through_numpy():
    """The gated activation against the plain GEMM on the stacked weight, split
    into its gate and up halves and combined with numpy's exp: pins which half
    is the gate and that rows are not shifted or swapped."""
    M, I, K = 7, 48, 160
    A = synth.normal_bf16((M, K), seed=401)
    W = synth.normal_bf16((2 * I, K), seed=402, sigma=synth.W_SIGMA * 20)
    Y = oracle.gemm_f64(A, W)
    g, u = Y[:, :I], Y[:, I:]
    want = g / (1.0 + np.exp(-g)) * u
    got = oracle.swiglu_f64(A, W)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-14)
    assert not np.allclose(got, u / (1.0 + np.exp(-u)) * g)          # gate/up not interchangeable
    # grouped: each group's rows use its own weight
    Ws = [W, synth.normal_bf16((2 * I, K), seed=403, sigma=synth.W_SIGMA * 20)]
    offs = [0, 3, 3, 7]
    Ws3 = [Ws[0], Ws[1], Ws[1]]
    ids = np.array([6, 0, 2, 1, 1, 5, 4])
    Hg = oracle.grouped_swiglu_f64(A, ids, offs, Ws3)
    assert np.allclose(Hg[0:3], oracle.swiglu_f64(A[ids[0:3]], Ws[0]), rtol=1e-15)
    assert np.allclose(Hg[3:7], oracle.swiglu_f64(A[ids[3:7]], Ws[1]), rtol=1e-15)


def test_fp8_e4m3_decode_against_torch_and_special_values():
    """The oracle's E4M3 decode (written from the format) equals torch's
    float8_e4m3fn for all 256 bytes; spot values of the format."""
    import torch
    vals = np.array([oracle.fp8_e4m3(v) for v in range(256)])
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(vals), np.isnan(ref))
    assert np.array_equal(vals[~np.isnan(vals)], ref[~np.isnan(ref)])
    assert oracle.fp8_e4m3(0x7E) == 448.0 and oracle.fp8_e4m3(0xFE) == -448.0      # largest
    assert oracle.fp8_e4m3(0x08) == 2.0 ** -6 and oracle.fp8_e4m3(0x01) == 2.0 ** -9  # min normal, min subnormal
    assert oracle.fp8_e4m3(0x38) == 1.0 and oracle.fp8_e4m3(0xC0) == -2.0
    assert math.isnan(oracle.fp8_e4m3(0x7F)) and math.isnan(oracle.fp8_e4m3(0xFF))
    assert oracle.fp8_e4m3(0x80) == 0.0 and math.copysign(1.0, oracle.fp8_e4m3(0x80)) == -1.0


def test_gemm_w8_small_integers_equal_bf16_gemm():
    """Integers in [-8, 8] are exact in E4M3 and bf16: the W8 GEMM of their
    E4M3 bytes equals the bf16 GEMM of the same values, and scales multiply."""
    import torch
    A = synth.small_int_bf16((6, 200), seed=31)
    Wi = np.random.default_rng(32).integers(-8, 9, size=(13, 200)).astype(np.float32)
    W8 = torch.from_numpy(Wi).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    Wb = synth.f32_to_bf16_bits(Wi)
    assert np.array_equal(oracle.gemm_w8_f64(A, W8), oracle.gemm_f64(A, Wb))
    sc = np.linspace(0.5, 2.0, 13)
    assert np.allclose(oracle.gemm_w8_f64(A, W8, sc), oracle.gemm_f64(A, Wb) * sc[None, :], rtol=1e-15, atol=0)


def test_round_bf16_against_float32_bit_rounding():
    """The oracle's bf16 rounding of doubles equals numpy float32 -> bf16 RNE
    on values that are exactly float32, and breaks ties to even."""
    rng = np.random.default_rng(0)
    x = rng.standard_normal(4096).astype(np.float32) * np.float32(3.0)
    assert np.array_equal(oracle.round_bf16(x.astype(np.float64)), synth.f32_to_bf16_bits(x))
    one = 1.0
    ties = np.array([one + 2.0 ** -8, one + 3 * 2.0 ** -8, -(one + 2.0 ** -8), 0.0])
    got = synth.bf16_bits_to_f32(oracle.round_bf16(ties))
    assert got[0] == 1.0 and got[1] == 1.0 + 2.0 ** -6 and got[2] == -1.0 and got[3] == 0.0


# ---------------------------------------------------------------------------
# Read amplification
# ---------------------------------------------------------------------------

def test_requests_per_tile_section_6_4():
    """128 (row-major, 512 B strips) vs 16 (tile-major (64, 32)) 4 KB requests
    per 128 x 256 BF16 compute tile; the contiguous side is 256 wide."""
    g = load("paper_requests_per_tile.txt")
    G, s = g["granularity"], g["elem_bytes"]
    N = K = 2048
    # paper "row-major": N contiguous (KN_ROW); 256 along N, 128 along K
    r = oracle.read_amp(1, N, K, 1, g["tile_contiguous_elems"], g["tile_other_elems"],
                        KN_ROW, G, s=s)
    assert r["min_blocks_per_tile"] == r["max_blocks_per_tile"] == g["requests_row_major"]
    assert g["tile_contiguous_elems"] * s == g["strip_bytes"]
    # tile-major: memory tile (a, b) = (64, 32), a along the contiguous dim
    t = oracle.read_amp(1, N, K, 1, 256, 128, TILE, G, s=s,
                        layout_G=G, block_rows=g["memory_tile_b"])
    assert G // (s * g["memory_tile_b"]) == g["memory_tile_a"]
    assert t["min_blocks_per_tile"] == t["max_blocks_per_tile"] == g["requests_tile_major"]
    extra = g["requests_row_major"] - g["requests_tile_major"]
    assert extra == g["extra_requests"] and extra * G == g["extra_bytes"]


def test_amp_32x_for_128B_wide_tile():
    g = load("paper_memory_tiles.txt")
    r = oracle.read_amp(4, 256, 4096, 4, 64, 64, NK_ROW, 4096)
    assert r["amp"] == g["amp_128B_wide_tile"]


def _closed_form_amp(kind, N, K, tn, tk, s, G, layout_G, br):
    """Closed forms for power-of-two tiles/blocks with no tile row segment
    straddling a block boundary (derived by hand, independent of the
    enumeration)."""
    if kind == TILE:
        bc = layout_G // (s * br)
        assert layout_G == G
        return max(1, br // tn) * max(1, bc // tk)
    if kind == KN_ROW:
        N, K, tn, tk = K, N, tk, tn     # same formula with roles swapped
    if K * s >= G:
        return max(1, G // (tk * s))
    R = G // (K * s)                    # whole rows per block
    return math.ceil(tn / R) * G / (tn * tk * s)


@pytest.mark.parametrize("kind", [NK_ROW, KN_ROW, TILE])
@pytest.mark.parametrize("G", [512, 1024, 4096, 16384])
def test_read_amp_closed_forms(kind, G):
    N, K, s = 256, 2048, 2
    for tn, tk in itertools.product([16, 64, 128], [32, 64, 256]):
        for br in ([8, 32, 64] if kind == TILE else [32]):
            if kind == TILE and (G // (s * br)) < 1:
                continue
            if kind == TILE and (N % br or K % (G // (s * br))):
                continue
            r = oracle.read_amp(3, N, K, 2, tn, tk, kind, G, s=s, layout_G=G, block_rows=br)
            want = _closed_form_amp(kind, N, K, tn, tk, s, G, G, br)
            assert r["amp"] == pytest.approx(want, rel=0, abs=1e-12), (kind, G, tn, tk, br)
            assert r["useful_bytes"] == 2 * N * K * s      # two m-tiles of M = 3, tm = 2
            assert r["fetched_bytes"] == r["requests"] * G


def test_fit_rule_gives_no_amplification():
    """Sections 1 and 3.1: compute tile dims that are multiples of the memory
    tile dims eliminate amplification."""
    rng = np.random.default_rng(5)
    for _ in range(40):
        s = int(rng.choice([1, 2]))
        G = int(rng.choice([512, 1024, 4096]))
        br = int(rng.choice([1, 2, 4, 8, 16, 32]))
        bc = G // (s * br)
        if bc < 1:
            continue
        tn, tk = br * int(rng.integers(1, 4)), bc * int(rng.integers(1, 3))
        N, K = tn * int(rng.integers(1, 4)), tk * int(rng.integers(1, 4))
        r = oracle.read_amp(5, N, K, 5, tn, tk, TILE, G, s=s, layout_G=G, block_rows=br)
        assert r["amp"] == 1.0 and r["unique_blocks"] * G == N * K * s


def test_tiny_config_amplification():
    """W[1024, 1024] bf16, 64 x 64 compute tile, 4 KB: the K-contiguous and
    N-contiguous layouts both fetch 16x; tile-major (32 x 64) fetches 1x."""
    assert oracle.read_amp(16, 1024, 1024, 64, 64, 64, NK_ROW, 4096)["amp"] == 16.0
    assert oracle.read_amp(16, 1024, 1024, 64, 64, 64, KN_ROW, 4096)["amp"] == 16.0
    assert oracle.read_amp(16, 1024, 1024, 64, 64, 64, TILE, 4096,
                           layout_G=4096, block_rows=32)["amp"] == 1.0


def test_hand_counted_small_case():
    """W[4, 8] bf16 row-major, G = 8 B (4 elements per block), 2 x 2 tiles:
    each tile row segment sits in one block, two rows -> 2 blocks per tile,
    8 tiles -> 16 requests, 128 B fetched for 64 useful bytes."""
    r = oracle.read_amp(1, 4, 8, 1, 2, 2, NK_ROW, 8)
    assert (r["compute_tiles"], r["requests"], r["fetched_bytes"], r["useful_bytes"]) == (8, 16, 128, 64)
    assert r["unique_blocks"] == 8 and r["amp"] == 2.0
    # KN_ROW: stored [8][4]; 4 elements per block = one stored row;
    # a 2 x 2 tile covers 2 stored rows -> 2 blocks
    r = oracle.read_amp(1, 4, 8, 1, 2, 2, KN_ROW, 8)
    assert r["requests"] == 16


def test_brute_force_over_m_tiles_matches_multiplied_count():
    for kind in (NK_ROW, KN_ROW, TILE):
        a = oracle.read_amp(37, 96, 320, 8, 32, 64, kind, 1024, layout_G=1024, block_rows=8)
        b = oracle.read_amp(37, 96, 320, 8, 32, 64, kind, 1024, layout_G=1024, block_rows=8,
                            brute_m=True)
        assert a == b


def test_ragged_tiles_against_python_sets():
    """Ragged edges: tiles are clipped, useful bytes count in-matrix elements
    only, a partial block still costs G.  Cross-check with Python sets on
    tiny shapes."""
    for (N, K, tn, tk, G, kind) in [(10, 24, 4, 7, 16, NK_ROW), (9, 13, 5, 4, 8, KN_ROW),
                                    (12, 40, 8, 16, 16, NK_ROW)]:
        s = 2
        req = useful = 0
        for n0 in range(0, N, tn):
            for k0 in range(0, K, tk):
                blocks = set()
                for n in range(n0, min(n0 + tn, N)):
                    for k in range(k0, min(k0 + tk, K)):
                        off = (n * K + k) * s if kind == NK_ROW else (k * N + n) * s
                        blocks.add(off // G)
                req += len(blocks)
                useful += (min(n0 + tn, N) - n0) * (min(k0 + tk, K) - k0) * s
        r = oracle.read_amp(1, N, K, 1, tn, tk, kind, G)
        assert r["requests"] == req and r["useful_bytes"] == useful == N * K * s


@pytest.mark.parametrize("N,K,br,G", [(40, 100, 32, 4096), (100, 72, 32, 4096), (33, 200, 16, 4096),
                                      (70, 24, 8, 1024)])
def test_padded_tile_major_amp_is_the_padding_ratio(N, K, br, G):
    """Compute tile = memory tile on a padded weight: every (n-tile, k-step)
    fetches exactly one block, so fetched / useful is the ratio of the padded
    to the true matrix size -- a closed form independent of the enumeration."""
    s = 2
    bc = G // (s * br)
    r = oracle.read_amp(3, N, K, 2, br, bc, TILE, G, s=s, layout_G=G, block_rows=br)
    tiles = -(-N // br) * -(-K // bc)
    assert r["min_blocks_per_tile"] == r["max_blocks_per_tile"] == 1
    assert r["requests"] == 2 * tiles                      # ceil(3 / 2) m-tiles
    assert r["unique_blocks"] == tiles
    assert r["useful_bytes"] == 2 * N * K * s
    assert r["amp"] == pytest.approx(tiles * G / (N * K * s))


def test_padded_amp_hand_counted():
    """N = 40, K = 100, (64, 32) BF16 memory tiles -> 2 x 2 tiles of 4 KB.
    Compute tile 16 x 128: n-tiles [0,16) [16,32) [32,40) each span one strip
    and the single K step [0,100) spans both tile columns: 3 tiles x 2 blocks."""
    r = oracle.read_amp(1, 40, 100, 1, 16, 128, TILE, 4096, s=2, layout_G=4096, block_rows=32)
    assert r["requests"] == 6 and r["fetched_bytes"] == 6 * 4096
    assert r["useful_bytes"] == 40 * 100 * 2
    assert r["unique_blocks"] == 4


def test_granularity_sweep_expectations_on_slice():
    """Down-projection [8192, 28672] on a 256-row slice (the slice does not
    change per-tile counts: every tile row is the same distance from block
    boundaries).  NK_ROW: tk = 64 gives 4/8/32/128x for G = 512 B .. 16 KB."""
    N, K = 256, 28672
    for G, want in [(512, 4), (1024, 8), (4096, 32), (16384, 128)]:
        assert oracle.read_amp(32, N, K, 32, 64, 64, NK_ROW, G)["amp"] == want
    # tile-major (G = 4 KB, br = 8 -> bc = 256): 4x at tk = 64
    assert oracle.read_amp(32, N, K, 32, 64, 64, TILE, 4096, layout_G=4096, block_rows=8)["amp"] == 4.0


def test_stacked_strips_are_contiguous():
    """Eq. 2 orders memory tiles along K within a strip of block_rows rows, so
    a strip is one contiguous run of bytes: the tile-major copy of matrices
    stacked along N (each a whole number of strips) is the concatenation of
    their copies, checked against numpy's reshape of the stacked matrix."""
    rng = np.random.default_rng(21)
    for G, br in ((4096, 32), (512, 8), (16384, 64)):
        bc = G // (2 * br)
        parts = [rng.integers(0, 1 << 16, size=(br * r, bc * 3), dtype=np.uint16) for r in (1, 3, 2)]
        stacked = np.vstack(parts)
        want = stacked.reshape(stacked.shape[0] // br, br, 3, bc).transpose(0, 2, 1, 3).reshape(-1)
        got = np.concatenate([oracle.repack(x, G, br).reshape(-1) for x in parts])
        assert np.array_equal(got, want)
        assert np.array_equal(oracle.repack(stacked, G, br).reshape(-1), want)


def test_oracle_thread_count_does_not_change_results():
    """Each output element is summed by one thread in ascending k, so the
    oracle's fp64 results are bit-identical for any OpenMP thread count."""
    A = synth.normal_bf16((5, 777), seed=91)
    W = synth.normal_bf16((301, 777), seed=92, sigma=synth.W_SIGMA)
    try:
        oracle.set_threads(1)
        one = oracle.gemm_f64(A, W)
        oracle.set_threads(4)
        four = oracle.gemm_f64(A, W)
    finally:
        oracle.set_threads(os.cpu_count() or 1)
    assert np.array_equal(one, four)
