// TileLens-HW address generation (Section 4.3), emulated: a multi-dimensional
// view of a tile-major weight is turned into a "counter program" -- a tile
// base address plus nested counters with byte strides, and for a memory tile
// wider than the box's contiguous extent a bit permutation of the intra-tile
// offset -- that tl_view_offsets runs on the host and tl_view_load runs on
// the GPU.  The program is built exactly as the paper's two phases describe:
//   phase 1, tileBase: the split-and-sum unit routes coordinate x stride
//     products with stride below the leading stride K to the row index i and
//     the rest to K j; tileBase = (K j + i b) s for memory-tile-aligned (i, j);
//   phase 2, counters: every dimension keeps its counter, but the dimension
//     that steps one column (stride K) becomes two nested counters, b steps of
//     a and v / b steps of b K (Eq. 5); other row-index dimensions scale by b.
// Case 2 (box narrower than the memory tile, u < a): phase 1 and 2 run as if
// the memory tile were u x b, then (sub | col | row) -> (col | sub | row)
// inside each G-byte block.  A box wider than the memory tile (u > a, a case
// the paper's kernels avoid) splits the contiguous counter the same way.
#include <cstring>

#include "tl_internal.h"

namespace tl {

constexpr int64_t kMaxView = int64_t(1) << 40;

int make_view_program(const tl_view* v, int64_t K, int64_t N, int32_t s, int64_t G, int32_t block_rows,
                      ViewProgram* out) {
    if (!v || !out) return TL_EINVAL;
    Layout L;
    if (make_tile_layout(s, G, block_rows, &L) != TL_OK) return TL_EINVAL;
    const int64_t a = L.bc, b = L.br;
    if (K < 1 || N < 1 || K % a || N % b) return TL_EINVAL;
    if (K > kMaxView || N > kMaxView || K > kMaxView / N) return TL_EINVAL;   // K N <= 2^40
    if (v->rank < 1 || v->rank > TL_VIEW_MAX_RANK) return TL_EINVAL;
    if (v->strides[0] != 1) return TL_EINVAL;
    int64_t elements = 1;
    int64_t i_max = 0, j_max = 0, i0 = 0, kj0 = 0;
    for (int d = 0; d < v->rank; ++d) {
        const int64_t st = v->strides[d], c = v->coords[d], n = v->box[d];
        // coordinates, extents and strides inside the matrix (no 64-bit overflow below)
        if (st < 1 || c < 0 || n < 1 || c >= kMaxView || n > kMaxView || st > K * N) return TL_EINVAL;
        if (st >= K && st % K) return TL_EINVAL;          // a column step is a whole number of columns
        elements *= n;
        if (elements > (int64_t(1) << 40)) return TL_EINVAL;
        if (st < K) { i_max += (c + n - 1) * st; i0 += c * st; }
        else { j_max += (c + n - 1) * (st / K); kj0 += c * st; }
    }
    if (i_max >= K || j_max >= N) return TL_EINVAL;        // the box lies inside the K x N matrix
    const int64_t j0 = kj0 / K;
    const int64_t u = v->box[0];
    if (!is_pow2(u)) return TL_EUNSUPPORTED;               // TMA boxes: power-of-two contiguous extent
    const int64_t ap = u < a ? u : a;                      // memory-tile width the counters assume
    if (i0 % ap || j0 % b) return TL_EUNSUPPORTED;         // the box starts on a memory-tile boundary

    ViewProgram P;
    std::memset(&P, 0, sizeof P);
    P.elements = elements;
    P.elem_bytes = s;
    P.tile_base = (K * j0 + i0 * b) * s;                   // Eq. 4
    int nc = 0;
    auto add = [&](int64_t count, int64_t stride_bytes) {
        P.count[nc] = count;
        P.stride[nc] = stride_bytes;
        ++nc;
    };
    for (int d = 0; d < v->rank; ++d) {
        const int64_t st = v->strides[d], n = v->box[d];
        if (d == 0) {
            if (u <= a) add(u, s);
            else { add(a, s); add(u / a, a * b * s); }    // across memory tiles along i
        } else if (st < K) {
            if (st % ap) return TL_EUNSUPPORTED;           // steps whole (assumed) memory tiles along i
            add(n, st * b * s);
        } else if (st == K) {
            if (n <= b) add(n, ap * s);                    // Eq. 5: b rows of a ...
            else {
                if (n % b) return TL_EUNSUPPORTED;
                add(b, ap * s);
                add(n / b, b * K * s);                     // ... then the next memory tile, b K away
            }
        } else {
            if ((st / K) % b) return TL_EUNSUPPORTED;      // whole strips of b columns
            add(n, st * s);
        }
    }
    P.n_counters = nc;
    // every index below 2^32 (so every count too, the counts multiplying to
    // the element count): divisions by multiplication
    P.fast32 = elements < (int64_t(1) << 32);
    if (P.fast32) {
        for (int c = 0; c < nc; ++c) {
            const uint64_t d = uint64_t(P.count[c]);
            int l = 0;
            while ((uint64_t(1) << l) < d) ++l;
            P.shift[c] = l;
            P.magic[c] = uint32_t(((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1);
        }
    }
    if (u < a) {                                           // Case 2 bit permutation
        P.permute = 1;
        P.row_bits = ilog2(u * s);
        P.col_bits = ilog2(b);
        P.sub_bits = ilog2(a / u);
        P.log2_G = L.log2_G;
    }
    *out = P;
    return TL_OK;
}

}  // namespace tl
