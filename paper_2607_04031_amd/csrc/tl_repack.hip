// Row-major <-> tile-major repack (TileLens Eq. 2, Section 3.2).
//
// The kernel walks the TILE-MAJOR buffer in order, CH bytes per lane
// (CH = min(16, bytes per memory-tile row), reduced until it divides a
// row-major row's bytes), so the tile-major side is always read or written
// with fully coalesced accesses; the row-major side is accessed in runs of
// block_cols * s bytes (128 B for the (64, 32) BF16 memory tile: one cache
// line per run).  Byte-exact and dtype-agnostic.
//
// Padding (Section 3.3): the tile-major copy holds whole memory tiles,
// ceil(rows / br) strips of ceil(cols / bc) tiles.  A chunk whose element
// lies outside the rows x cols matrix is padding: the forward repack writes
// zeros there and the inverse does not read it.  Because CH divides both a
// memory-tile row and a row-major row, a chunk is entirely inside or entirely
// outside the matrix.
#include <hip/hip_runtime.h>

#include "tl_internal.h"

namespace tl {
namespace {

struct RepackParams {
    const uint8_t* src;
    uint8_t* dst;
    int64_t total_chunks;   // tile-major bytes / CH
    int64_t cols_bytes;     // bytes per row-major row
    int64_t rows;           // rows of the matrix (rows past it are padding)
    uint32_t kblocks;       // memory tiles per strip = ceil(cols / bc)
    int log2_G;
    int log2_rowbytes;      // log2(bc * s): bytes per memory-tile row
    int log2_br;
    int inverse;            // 0: row-major -> tile-major, 1: back
};

// Native vector types (not HIP's uint4/uint2 structs) so the per-thread
// staging arrays stay in registers.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

template <int CH> struct Chunk;
template <> struct Chunk<16> { using T = u32x4; };
template <> struct Chunk<8> { using T = u32x2; };
template <> struct Chunk<4> { using T = uint32_t; };
template <> struct Chunk<2> { using T = uint16_t; };
template <> struct Chunk<1> { using T = uint8_t; };

template <int CH, int UNROLL>
__global__ __launch_bounds__(256) void repack_kernel(RepackParams p) {
    using T = typename Chunk<CH>::T;
    const int64_t G_mask = (int64_t(1) << p.log2_G) - 1;
    const int64_t row_mask = (int64_t(1) << p.log2_rowbytes) - 1;
    const int64_t stride = int64_t(gridDim.x) * 256;
    for (int64_t base = int64_t(blockIdx.x) * 256 * UNROLL + threadIdx.x; base < p.total_chunks;
         base += stride * UNROLL) {
        T v[UNROLL];
        int64_t dst_off[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int64_t i = base + int64_t(u) * 256;
            if (i >= p.total_chunks) { dst_off[u] = -1; continue; }
            const int64_t tm = i * CH;                       // tile-major byte
            const uint32_t block = uint32_t(tm >> p.log2_G);
            const int64_t in_blk = tm & G_mask;
            const int64_t r_in = in_blk >> p.log2_rowbytes;  // row inside the memory tile
            const int64_t c_byte = in_blk & row_mask;        // byte inside that row
            const uint32_t strip = block / p.kblocks;
            const uint32_t kb = block - strip * p.kblocks;
            const int64_t r = (int64_t(strip) << p.log2_br) + r_in;
            const int64_t cb = (int64_t(kb) << p.log2_rowbytes) + c_byte;   // byte along the row
            const bool inside = r < p.rows && cb < p.cols_bytes;
            const int64_t rm = r * p.cols_bytes + cb;
            if (p.inverse) {
                dst_off[u] = inside ? rm : -1;
                if (inside) v[u] = *reinterpret_cast<const T*>(p.src + tm);
            } else {
                dst_off[u] = tm;
                if (inside) v[u] = *reinterpret_cast<const T*>(p.src + rm);
                else v[u] = T(0);
            }
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
            if (dst_off[u] >= 0) *reinterpret_cast<T*>(p.dst + dst_off[u]) = v[u];
    }
}

template <int CH>
hipError_t launch_ch(const RepackParams& p, hipStream_t stream) {
    constexpr int kUnroll = 4;
    int64_t want = (p.total_chunks + 256 * kUnroll - 1) / (256 * kUnroll);
    int grid = int(want < 8192 ? want : 8192);
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL((repack_kernel<CH, kUnroll>), dim3(grid), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_repack(const void* src, void* dst, int64_t rows, int64_t cols, const Layout& L,
                         bool inverse, hipStream_t stream) {
    RepackParams p;
    p.src = static_cast<const uint8_t*>(src);
    p.dst = static_cast<uint8_t*>(dst);
    const int64_t row_bytes = L.bc * L.s;                 // power of two
    int64_t ch = row_bytes < 16 ? row_bytes : 16;
    while ((cols * L.s) % ch) ch >>= 1;                   // aligned row-major chunks
    const int64_t kblocks = (cols + L.bc - 1) / L.bc;
    const int64_t strips = (rows + L.br - 1) / L.br;
    p.total_chunks = strips * kblocks * L.G / ch;
    p.cols_bytes = cols * L.s;
    p.rows = rows;
    p.kblocks = uint32_t(kblocks);
    p.log2_G = L.log2_G;
    p.log2_rowbytes = ilog2(row_bytes);
    p.log2_br = L.log2_br;
    p.inverse = inverse ? 1 : 0;
    switch (ch) {
        case 16: return launch_ch<16>(p, stream);
        case 8: return launch_ch<8>(p, stream);
        case 4: return launch_ch<4>(p, stream);
        case 2: return launch_ch<2>(p, stream);
        default: return launch_ch<1>(p, stream);
    }
}

}  // namespace tl
