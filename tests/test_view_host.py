"""TileLens-HW address generation emulated on the host (tl_view_offsets,
Section 4.3): the offsets the split-and-sum tile base, the nested counters
of Eq. 5 and the Case-2 bit permutation produce must equal, element for
element, the oracle's plain definition (linear index -> (i, j) -> Eq. 2) for
the paper's view example, the Case-2 example and random views of random
memory-tile layouts.  CPU only."""
import numpy as np
import pytest

import oracle
import paper_2607_04031_amd as tl
from tests._golden import load


def _check(strides, coords, box, K, N, s, G, br):
    got = tl.tl_view_offsets(tl.view(strides, coords, box), K, N, s, G, br)
    want = oracle.view_offsets(strides, coords, box, K, s, G, br)
    assert np.array_equal(got, want), (strides, coords, box, K, N, s, G, br)
    return got


def test_paper_view_example_three_descriptors():
    """Section 4.3: one FP8 384 x 128 matrix, one 128 x 64 box at (256, 64)
    through 2-D, 3-D and 4-D descriptors; same offsets in the same order."""
    g = load("paper_view_example.txt")
    K, N = g["K"], g["N"]

    def parse(v):
        return [list(map(int, p.split(","))) for p in v.split(";")]
    strides = {"view2d": [1, K], "view3d": [1, K, 128], "view4d": [1, K, 128, 64 * K]}
    seqs = []
    for name in ("view2d", "view3d", "view4d"):
        _, coords, box = parse(g[name])
        seqs.append(_check(strides[name], coords, box, K, N, 1, 4096, 64))
    assert all(np.array_equal(seqs[0], x) for x in seqs[1:])


def test_paper_case2_fields():
    """Case 2: a 32 x 32 FP8 box on 128 x 32 memory tiles; the intra-tile
    offset of element (row r, col c) of the box starting at sub-tile t is
    (col | sub | row) = c * 128 + t * 32 + r."""
    g = load("paper_case2_bitperm.txt")
    a, b, u = g["memory_tile_a"], g["memory_tile_b"], g["tma_tile_u"]
    K, N = 4 * a, 2 * b
    for t in range(a // u):
        offs = _check([1, K], [t * u, 0], [u, b], K, N, 1, 4096, b)
        for c in range(b):
            for r in range(u):
                assert offs[c * u + r] % 4096 == c * a + t * u + r


def _random_view(rng, K, N, a, b):
    """A random aligned view: dimension 0 contiguous (u a power of two), then
    a shuffled mix of: one-column dimension (stride K), whole-strip column
    dimensions (stride a multiple of b K), row-index dimensions (stride a
    multiple of the assumed memory-tile width)."""
    u = int(rng.choice([x for x in (a // 4, a // 2, a, 2 * a) if x >= 1 and x <= K]))
    ap = min(u, a)
    dims = []
    # column side: j = j0 + x1 * 1 + x2 * m2 ...
    v = int(rng.choice([x for x in (b // 2, b, 2 * b, 4 * b) if 1 <= x <= N]))
    dims.append(("col", K, v))
    if rng.random() < 0.5 and N >= 2 * v:
        strips = int(rng.integers(1, max(2, N // (2 * v) + 1)))
        m = -(-v // b) * b * strips                 # whole strips past the first box
        if m + v <= N:
            dims.append(("col", m * K, 2))
    # row side: i = i0 + x0 + x3 * c3
    if rng.random() < 0.6 and K >= 2 * u:
        c = -(-u // ap) * ap * int(rng.integers(1, 3))
        n = int(rng.integers(1, 4))
        if u + (n - 1) * c <= K:
            dims.append(("row", c, n))
    rng.shuffle(dims)
    strides = [1] + [d[1] for d in dims]
    box = [u] + [d[2] for d in dims]
    # coordinates: aligned starts that keep the box inside the matrix
    i_span = (u - 1) + sum((d[2] - 1) * d[1] for d in dims if d[0] == "row")
    j_span = sum((d[2] - 1) * (d[1] // K) for d in dims if d[0] == "col")
    i0 = int(rng.integers(0, (K - 1 - i_span) // ap + 1)) * ap
    j0 = int(rng.integers(0, (N - 1 - j_span) // b + 1)) * b
    coords = [i0] + [0] * len(dims)
    # put j0 on the one-column dimension
    coords[1 + [d[1] for d in dims].index(K)] = j0
    return strides, coords, box


@pytest.mark.parametrize("s,G,br", [(1, 4096, 64), (1, 4096, 32), (2, 4096, 32), (2, 4096, 8), (2, 1024, 16),
                                    (2, 16384, 64), (4, 4096, 16), (2, 512, 8), (1, 16384, 128)])
def test_random_views_match_oracle(s, G, br):
    rng = np.random.default_rng(s * 100000 + G + br)
    a = G // (s * br)
    K, N = a * int(rng.integers(2, 9)), br * int(rng.integers(2, 9))
    for _ in range(60):
        strides, coords, box = _random_view(rng, K, N, a, br)
        _check(strides, coords, box, K, N, s, G, br)


def test_identity_extreme_is_column_major():
    """block_rows = 1 with K * s = G: tile-major is the column-major layout, so
    every offset is the linear index times s."""
    K, N, s = 2048, 16, 2
    strides, coords, box = [1, K], [0, 3], [2048, 5]
    got = _check(strides, coords, box, K, N, s, K * s, 1)
    lin = np.array([(3 + c) * K + r for c in range(5) for r in range(2048)]) * s
    assert np.array_equal(got, lin)


def test_view_errors():
    K, N = 256, 64
    bad = [
        (([2, K], [0, 0], [64, 32]), tl.TL_EINVAL),          # strides[0] != 1
        (([1, K], [0, 0], [64, 65]), tl.TL_EINVAL),          # past column N - 1
        (([1, K], [224, 0], [64, 32]), tl.TL_EINVAL),        # past row K - 1
        (([1, K + 5], [0, 0], [64, 2]), tl.TL_EINVAL),       # a column stride that is not whole columns
        (([1, K], [-64, 0], [64, 32]), tl.TL_EINVAL),
        (([1, K], [0, 0], [48, 32]), tl.TL_EUNSUPPORTED),    # box[0] not a power of two
        (([1, K], [32, 0], [64, 32]), tl.TL_EUNSUPPORTED),   # not on a memory-tile boundary (a = 64)
        (([1, K], [0, 8], [64, 32]), tl.TL_EUNSUPPORTED),    # nor along N (b = 32)
        (([1, K], [0, 0], [64, 48]), tl.TL_EUNSUPPORTED),    # one-column dimension splitting a memory tile
        (([1, K, 2 * K], [0, 0, 0], [64, 2, 2]), tl.TL_EUNSUPPORTED),   # column stride inside a strip
        (([1, K, 96], [0, 0, 0], [64, 32, 2]), tl.TL_EUNSUPPORTED),     # row stride not whole memory tiles
    ]
    for (strides, coords, box), status in bad:
        with pytest.raises(tl.TLError) as e:
            tl.tl_view_offsets(tl.view(strides, coords, box), K, N, 2, 4096, 32)
        assert e.value.status == status, (strides, coords, box)
    with pytest.raises(tl.TLError) as e:                      # rank 6
        v = tl.view([1, K], [0, 0], [64, 32])
        v.rank = 6
        tl.tl_view_offsets(v, K, N, 2, 4096, 32)
    assert e.value.status == tl.TL_EINVAL
