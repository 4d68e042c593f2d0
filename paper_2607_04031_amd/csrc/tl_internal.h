// Internal declarations shared by the libtl translation units (host side).
#pragma once

#include <algorithm>
#include <cstdint>

#include <hip/hip_runtime.h>

#include "../../include/tl.h"

namespace tl {

inline bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

inline int ilog2(int64_t x) {
    int r = 0;
    while ((int64_t(1) << r) < x) ++r;
    return r;
}

// A validated tile-major (or linear) weight layout with the shift amounts the
// kernels use in place of Eq. 1's divisions (Section 3.2: a and b are powers
// of two, so the tile indices are shifts and masks).
struct Layout {
    int kind = TL_LAYOUT_TILE;
    int64_t s = 2;        // element bytes
    int64_t G = 4096;     // memory-tile bytes
    int64_t br = 32;      // paper b (rows along N)
    int64_t bc = 64;      // paper a (elements along K)
    int log2_br = 5, log2_bc = 6, log2_G = 12;
};

// Checks a tile-major description; fills 'out' on success.
int make_tile_layout(int64_t s, int64_t G, int64_t br, Layout* out);

// Section 3.3: a weight whose dimensions are not multiples of the memory
// tile's sides is padded to whole memory tiles.  Columns (along K) of the
// padded copy, and its bytes: ceil(rows / br) strips of ceil(cols / bc) tiles.
inline int64_t padded_cols(const Layout& L, int64_t cols) { return (cols + L.bc - 1) / L.bc * L.bc; }
inline int64_t packed_bytes(const Layout& L, int64_t rows, int64_t cols) {
    return (rows + L.br - 1) / L.br * ((cols + L.bc - 1) / L.bc) * L.G;
}

// ---------------------------------------------------------------------------
// Kernel launchers (defined in the .hip files).  Arguments are validated by
// the callers; these only enqueue.
// ---------------------------------------------------------------------------

hipError_t launch_repack(const void* src, void* dst, int64_t rows, int64_t cols,
                         const Layout& L, bool inverse, hipStream_t stream);

struct DecodeLaunch {
    const uint16_t* A;
    const uint8_t* W;
    void* C;
    float* ws;                  // [split_k][M * N rounded up to 4] partials (split_k > 1)
    unsigned long long* fetch;  // fetch tally (TL_FETCH_COUNT) or nullptr
    int64_t M, N, K;
    Layout L;
    int tile_n;                 // 32 or 64
    int m_tiles16;              // ceil(M / 16): 1, 2 or 4
    int waves;                  // wavefronts per workgroup: 4, 8 or 16 (K split inside)
    int split_k;
    int64_t k_unit;             // K granularity of a split, in elements
    bool out_bf16;
    bool block_fetch;           // row-major weight read in whole fetch_G-byte blocks
    int64_t fetch_G;
    // grouped launch (num_groups > 0; split_k 1, waves 4): group e has weight
    // W + e * group_stride and output rows [group_offsets[e], group_offsets[e+1])
    int num_groups = 0;
    const int32_t* group_offsets = nullptr;
    const int32_t* token_ids = nullptr;
    int64_t group_stride = 0;
    int64_t a_rows = 0;
    int64_t total_rows = 0;
    // gated expert activation (grouped only): W_e stacks gate rows [0, N) and
    // up rows [N, 2N); C[r][n] = silu(gate) * up, N columns; tile_n = 64
    bool swiglu = false;
    // FP8 (E4M3) weight, bf16 activations; optional per-output-channel scales [N]
    bool fp8 = false;
    const float* scales = nullptr;
    // > 0: the LDS-staged activation kernel with this many 32-row tiles per
    // workgroup (17 <= M <= 64, tile-major, N % (32 lds_tiles) == 0, K % 512 == 0)
    int lds_tiles = 0;
};

hipError_t launch_decode(const DecodeLaunch& d, hipStream_t stream);
// *p = 0, enqueued on 'stream' as a one-thread kernel (not a memset node, so
// the clear behaves like any kernel inside a captured graph)
hipError_t launch_zero_u64(unsigned long long* p, hipStream_t stream);
// the fixed-order split-K reduce that follows a decode launch with split_k > 1
// (passes 'e' through when it is an error or split_k is 1)
hipError_t launch_splitk_reduce(const DecodeLaunch& d, hipError_t e, hipStream_t stream);
// large-granularity-memory emulation (decode, M <= 16, tile_n 32, 4 waves):
// every read completes no earlier than latency_ticks wall-clock ticks after
// issue; each wave keeps steps_in_flight (1, 2, 4 or 8) K steps in flight
hipError_t launch_lgms(const DecodeLaunch& d, int64_t latency_ticks, int steps_in_flight, hipStream_t stream);
int lgms_ctas_per_cu(int steps_in_flight);   // resident workgroups per CU, -1 on a HIP error

struct PrefillLaunch {
    const uint16_t* A;
    const uint8_t* W;
    void* C;
    unsigned long long* fetch;
    int64_t M, N, K;
    Layout L;
    int tile_m;                 // 128 or 256
    int tile_n;                 // 128, 256 or 320 (256 and 320 only with tile_m 256; 320 persistent)
    bool out_bf16;
    // columns [0, n_main) use tile_m x tile_n tiles; columns [n_main, N), if
    // any, a second launch of 128 x 128 tiles (n_main is a multiple of tile_n)
    int64_t n_main;
    bool block_fetch = false;   // row-major weight read in whole fetch_G-byte blocks
    int64_t fetch_G = 0;
    // > 1: columns [n_main, N) run as 256 x 256 tiles with K split this many
    // ways (fp32 partials in ws, M * (N - n_main) floats per split) instead
    // of 128 x 128 tiles
    int split_rest = 0;
    float* ws = nullptr;
    // columns [0, n_main) with 256 x 256 tiles, bf16 out, M and n_main
    // multiples of 256, K of 128: a persistent grid of at most one
    // workgroup per CU walks the tiles
    bool persist = false;
};

hipError_t launch_prefill(const PrefillLaunch& p, hipStream_t stream);

// tl_gemm_noalloc's split-K scratch (tl_scratch.hip): a static device array
// of kScratchBytes per GPU.  *out = its device address on the current device
// (looked up with hipGetSymbolAddress on the first call per device; no
// allocation).
constexpr int64_t kScratchBytes = TL_NOALLOC_SCRATCH_BYTES;
hipError_t scratch_address(float** out);

// Counter program of a view load (TileLens-HW emulation, tl_view.cpp):
// element e, decoded in mixed radix over count[] (counter 0 fastest), sits at
//   off = tile_base + sum_c digit_c * stride[c]
// and, if permute, the low log2_G bits of off hold (sub | col | row) with
// widths (sub_bits | col_bits | row_bits) and are rewritten as
// (col | sub | row).  Offsets are bytes from the weight's base.
constexpr int kViewMaxCounters = 2 * TL_VIEW_MAX_RANK;
struct ViewProgram {
    int n_counters;
    int64_t count[kViewMaxCounters];
    int64_t stride[kViewMaxCounters];
    int64_t tile_base;
    int64_t elements;
    int32_t elem_bytes;
    int32_t permute, row_bits, col_bits, sub_bits, log2_G;
    // Element indices below 2^32 (fast32): the division of an index by
    // count[c] as a multiplication (Granlund and Montgomery, "Division by
    // invariant integers using multiplication", 1994, Section 4): for every
    // 32-bit x, x / count[c] = (umulhi(x, magic[c]) + x) >> shift[c], with
    // shift = ceil(log2 count) and magic = floor(2^32 (2^shift - count) / count) + 1.
    int32_t fast32;
    uint32_t magic[kViewMaxCounters];
    int32_t shift[kViewMaxCounters];
};

int make_view_program(const tl_view* v, int64_t K, int64_t N, int32_t elem_bytes, int64_t G,
                      int32_t block_rows, ViewProgram* out);

// Host and device: byte offset of element e under the program.
__host__ __device__ inline int64_t view_offset(const ViewProgram& P, int64_t e) {
    int64_t off = P.tile_base;
    if (P.fast32) {
        uint32_t x = uint32_t(e);
        for (int c = 0; c < P.n_counters; ++c) {
            const uint32_t hi = uint32_t((uint64_t(x) * P.magic[c]) >> 32);
            const uint32_t q = uint32_t((uint64_t(hi) + x) >> P.shift[c]);
            off += int64_t(x - q * uint32_t(P.count[c])) * P.stride[c];
            x = q;
        }
    } else {
        for (int c = 0; c < P.n_counters; ++c) {
            const int64_t n = P.count[c];
            off += (e % n) * P.stride[c];
            e /= n;
        }
    }
    if (P.permute) {
        const int64_t G = int64_t(1) << P.log2_G;
        const int64_t low = off & (G - 1);
        const int64_t row = low & ((int64_t(1) << P.row_bits) - 1);
        const int64_t col = (low >> P.row_bits) & ((int64_t(1) << P.col_bits) - 1);
        const int64_t sub = low >> (P.row_bits + P.col_bits);
        off = (off - low) | (col << (P.sub_bits + P.row_bits)) | (sub << P.row_bits) | row;
    }
    return off;
}

// reads bytes (a multiple of 16) of src once and XORs its 32-bit words
// into *checksum (one kernel; nothing for bytes = 0)
hipError_t launch_stream_read(const uint8_t* src, int64_t bytes, unsigned* checksum, hipStream_t stream);
hipError_t launch_view_load(const uint8_t* src, int64_t src_bytes, const ViewProgram& P, uint8_t* dst,
                            hipStream_t stream);

}  // namespace tl
