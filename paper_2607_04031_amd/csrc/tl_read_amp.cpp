// tl_read_amp: exact count of the G-byte blocks a tiled GEMM fetches from a
// large-granularity memory (TileLens Sections 1 and 2.5; the per-tile request
// counts of Section 6.5).  Host-only integer arithmetic.
//
// Two routes, both exact:
//  * closed forms for the aligned power-of-two cases every evaluated shape
//    falls in (a tile row segment never straddles a block boundary), and
//  * an enumerator over contiguous byte runs ("pieces") of each weight
//    sub-tile, unioned per tile with a stamp array, for everything else.
#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "tl_internal.h"

namespace {

// Largest block table the enumerator allocates (8 bytes per block: 2 GB).
constexpr int64_t kMaxEnumBlocks = int64_t(1) << 28;

struct Geometry {
    int kind;
    int64_t N, K, s;
    tl::Layout L;
};

// Byte offset of logical element (n, k).
inline int64_t elem_off(const Geometry& g, int64_t n, int64_t k) {
    switch (g.kind) {
        case TL_LAYOUT_NK_ROW: return (n * g.K + k) * g.s;
        case TL_LAYOUT_KN_ROW: return (k * g.N + n) * g.s;
        default: {
            const tl::Layout& L = g.L;
            // strips of ceil(K / bc) memory tiles (padded, Section 3.3)
            int64_t strip = n >> L.log2_br, r = n & (L.br - 1);
            int64_t kb = k >> L.log2_bc, c = k & (L.bc - 1);
            return ((strip * ((g.K + L.bc - 1) >> L.log2_bc) + kb) << L.log2_G) + ((r << L.log2_bc) + c) * g.s;
        }
    }
}

// Blocks per tile from a closed form, or -1 if the case is not covered.
// Requires full tiles (N % tn == 0, K % tk == 0) and power-of-two G, tn, tk.
// A padded tile-major weight is covered too: tiles narrower than a memory
// tile stay inside one, and wider ones (power-of-two multiples of its sides)
// dividing N or K leave nothing to pad along that dimension.
int64_t closed_form_blocks(const Geometry& g, int64_t tn, int64_t tk, int64_t G) {
    if (!tl::is_pow2(G) || !tl::is_pow2(tn) || !tl::is_pow2(tk)) return -1;
    if (g.N % tn || g.K % tk) return -1;
    if (g.kind == TL_LAYOUT_TILE) {
        if (G != g.L.G) return -1;
        return std::max<int64_t>(1, tn / g.L.br) * std::max<int64_t>(1, tk / g.L.bc);
    }
    // Linear layouts: 'len' contiguous elements per stored row, 'w' of them
    // per tile row segment, 'h' segments (stored rows) per tile.
    int64_t len = g.kind == TL_LAYOUT_NK_ROW ? g.K : g.N;
    int64_t w = g.kind == TL_LAYOUT_NK_ROW ? tk : tn;
    int64_t h = g.kind == TL_LAYOUT_NK_ROW ? tn : tk;
    int64_t row_bytes = len * g.s, seg_bytes = w * g.s;
    if (row_bytes % G == 0) {
        if (seg_bytes % G == 0) return h * (seg_bytes / G);
        if (G % seg_bytes == 0) return h;
        return -1;
    }
    if (G % row_bytes == 0) {
        int64_t R = G / row_bytes;             // whole stored rows per block
        if (h % R == 0) return h / R;
        if (R % h == 0) return 1;
    }
    return -1;
}

}  // namespace

extern "C" int tl_read_amp(int64_t M, int64_t N, int64_t K, int32_t tile_m, int32_t tile_n,
                           int32_t tile_k, const tl_layout_desc* layout, int64_t G, tl_amp* out) {
    if (!layout || !out) return TL_EINVAL;
    if (M < 1 || N < 1 || K < 1 || tile_m < 1 || tile_n < 1 || tile_k < 1 || G < 1 || G > (int64_t(1) << 40))
        return TL_EINVAL;
    Geometry g;
    g.kind = layout->kind;
    g.N = N;
    g.K = K;
    g.s = layout->elem_bytes;
    if (g.s < 1 || g.s > 16) return TL_EINVAL;
    if (g.kind != TL_LAYOUT_NK_ROW && g.kind != TL_LAYOUT_KN_ROW && g.kind != TL_LAYOUT_TILE)
        return TL_EINVAL;
    if (g.kind == TL_LAYOUT_TILE) {
        if (tl::make_tile_layout(g.s, layout->G, layout->block_rows, &g.L) != TL_OK) return TL_EINVAL;
    }
    if (N > (int64_t(1) << 40) / K) return TL_EINVAL;
    const int64_t tm = tile_m, tn = tile_n, tk = tile_k;
    const int64_t m_tiles = (M + tm - 1) / tm;
    const int64_t n_tiles = (N + tn - 1) / tn;
    const int64_t k_steps = (K + tk - 1) / tk;
    const int64_t total_bytes = N * K * g.s;   // the matrix's own bytes
    // bytes the stored weight spans: the padded copy for tile-major
    const int64_t span = g.kind == TL_LAYOUT_TILE ? tl::packed_bytes(g.L, N, K) : total_bytes;
    const int64_t nblocks = (span + G - 1) / G;

    // every count below must fit in int64
    auto mul = [](int64_t a, int64_t b, int64_t* out) { return !__builtin_mul_overflow(a, b, out); };
    tl_amp r;
    std::memset(&r, 0, sizeof r);
    int64_t nk = 0;
    if (!mul(n_tiles, k_steps, &nk) || !mul(m_tiles, nk, &r.compute_tiles) ||
        !mul(m_tiles, total_bytes, &r.useful_bytes))
        return TL_EINVAL;

    int64_t per_tile = closed_form_blocks(g, tn, tk, G);
    if (per_tile > 0) {
        if (!mul(r.compute_tiles, per_tile, &r.requests)) return TL_EINVAL;
        r.min_blocks_per_tile = r.max_blocks_per_tile = per_tile;
        r.unique_blocks = nblocks;   // every element is touched by some tile
    } else {
        // stamp[b]: last (n-tile, k-step) that touched block b, -1 if none yet
        if (nblocks > kMaxEnumBlocks) return TL_EUNSUPPORTED;
        std::vector<int64_t> stamp;
        try {
            stamp.assign(size_t(nblocks), -1);
        } catch (const std::bad_alloc&) {
            return TL_ENOMEM;
        }
        int64_t requests = 0, unique = 0, bmin = -1, bmax = 0, tile_id = 0;
        auto visit = [&](int64_t begin_byte, int64_t end_byte, int64_t& count) {
            for (int64_t b = begin_byte / G; b <= (end_byte - 1) / G; ++b) {
                if (stamp[size_t(b)] != tile_id) {
                    if (stamp[size_t(b)] < 0) ++unique;
                    stamp[size_t(b)] = tile_id;
                    ++count;
                }
            }
        };
        for (int64_t ti = 0; ti < n_tiles; ++ti) {
            const int64_t n0 = ti * tn, n1 = std::min(N, n0 + tn);
            for (int64_t kj = 0; kj < k_steps; ++kj, ++tile_id) {
                const int64_t k0 = kj * tk, k1 = std::min(K, k0 + tk);
                int64_t count = 0;
                if (g.kind == TL_LAYOUT_NK_ROW) {
                    for (int64_t n = n0; n < n1; ++n)
                        visit(elem_off(g, n, k0), elem_off(g, n, k1 - 1) + g.s, count);
                } else if (g.kind == TL_LAYOUT_KN_ROW) {
                    for (int64_t k = k0; k < k1; ++k)
                        visit(elem_off(g, n0, k), elem_off(g, n1 - 1, k) + g.s, count);
                } else {
                    // inside a memory tile a row's run along K is contiguous
                    for (int64_t n = n0; n < n1; ++n) {
                        for (int64_t ks = k0; ks < k1;) {
                            int64_t ke = std::min(k1, ((ks >> g.L.log2_bc) + 1) << g.L.log2_bc);
                            visit(elem_off(g, n, ks), elem_off(g, n, ke - 1) + g.s, count);
                            ks = ke;
                        }
                    }
                }
                requests += count;
                if (bmin < 0 || count < bmin) bmin = count;
                bmax = std::max(bmax, count);
            }
        }
        if (!mul(requests, m_tiles, &r.requests)) return TL_EINVAL;
        r.unique_blocks = unique;
        r.min_blocks_per_tile = bmin;
        r.max_blocks_per_tile = bmax;
    }
    if (!mul(r.requests, G, &r.fetched_bytes)) return TL_EINVAL;
    r.amp = double(r.fetched_bytes) / double(r.useful_bytes);
    *out = r;
    return TL_OK;
}
