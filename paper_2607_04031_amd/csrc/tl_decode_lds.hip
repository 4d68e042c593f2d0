// Decode GEMM for 17 <= M <= 64 with the activations staged in LDS.
//
// At M = 32 every workgroup of the streaming decode kernel (tl_decode.hip)
// reloads the activations of its K range from L2, as many bytes again as
// half of the weight bytes it streams (at M = 64 on 64-row tiles, as many as
// the weight bytes); those extra L2 -> CU requests, not HBM, limit it.  Here
// one workgroup (8 waves, one per CU) takes T consecutive 32-row tiles of W
// -- whole strips of memory tiles -- and one K range, and walks the range in
// chunks of 512 columns:
//   * the chunk of A (16 MT rows x 512 columns: 32 KB for MT = 2 M tiles,
//     64 KB for MT = 4) is staged once in LDS (double buffered: the next
//     chunk's loads are in flight while the current one is used), so A
//     crosses L2 -> CU once per T tiles;
//   * wave w owns the 64-wide K step w of the chunk and streams it for the T
//     tiles one after another, so the workgroup reads one strip at a time
//     (Section 2.3: tiles iterate along K; one DRAM stream per workgroup),
//     the weight loads of the next steps in flight while a step computes;
//   * the wave's A operands of that step are read from LDS once per chunk
//     and serve all T tiles (MT = 2), or once per tile (MT = 4, where
//     holding them across the tiles would leave one wave per SIMD).
// Weight loads, the lane exchange and the MFMA 16x16x32 operand layout are
// those of the streaming kernel; each wave keeps T tiles x 16 MT x 32 fp32
// partial sums, summed over the 8 waves through LDS in a fixed order at the
// end, then stored (one K range) or written as a split-K partial for the
// fixed-order reduce kernel.  The planner uses this kernel only when the
// tiles and K ranges fill the CUs (whole rounds for MT = 2, at least 7/8 of
// one round for MT = 4, T = 4), with N a multiple of 32 T, K of 512 and
// block_rows dividing 32 (tiles are whole memory-tile strips).
#include <hip/hip_runtime.h>

#include "tl_decode_common.h"

namespace tl {
namespace {

constexpr int kLdsWaves = 8;
constexpr int kLdsThreads = 64 * kLdsWaves;
constexpr int kChunkK = 512;                          // K columns per staged chunk: one 64-step per wave

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// LDS byte offset of 16-byte column c (0..63) of row r of a staged chunk:
// 1 KB rows with the columns XOR-swizzled by the row's low four bits, so the
// 16 rows one operand read touches (same column) hit 16 different groups of
// banks, and 16 consecutive columns of one row (a staging write) do too.
__device__ inline int a_lds(int r, int c) { return r * (kChunkK * 2) + ((c ^ (r & 15)) << 4); }

template <int T, int P, int MT>
__global__ __launch_bounds__(kLdsThreads) void decode_lds_kernel(DecodeParams p) {
    constexpr int NS = 2;
    constexpr int kARows = 16 * MT;                       // rows of A staged (rows past M are zero)
    constexpr int kAChunkBytes = kARows * kChunkK * 2;    // 32 or 64 KB
    constexpr int kRowsPerWave = kARows / kLdsWaves;      // staging rows per wave: 4 or 8
    // four M tiles: the A operands are read from LDS for every tile (not held
    // across the T tiles) and the next chunk is staged in two halves, to fit
    // two waves per SIMD
    constexpr bool kAPerTile = MT == 4;
    constexpr int kStageParts = kRowsPerWave / 4;
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * kAChunkBytes];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int group = blockIdx.x / p.split_k;
    const int split = blockIdx.x - group * p.split_k;
    const int c0 = int((int64_t(p.units) * split) / p.split_k);     // chunks of 512 columns
    const int c1 = int((int64_t(p.units) * (split + 1)) / p.split_k);
    const int g = lane >> 4, q = lane & 15;
    const bool lo = q < 8;
    const int kc = (((q >> 3) << 2) + g) << 3;   // k offset of this lane's weight chunk in a step

    // Tile t of the group starts t * tile_bytes after tile 0 (its rows are
    // 32 / block_rows whole strips), and a lane's offset inside a tile is
    // the same for every tile of the group.
    const int n_base0 = group * T * 32;
    const int64_t tile_bytes = int64_t(32 >> p.log2_br) * p.strip_bytes;
    const uint8_t* w0 = p.W + int64_t(n_base0 >> p.log2_br) * p.strip_bytes;
    uint32_t woff[NS][2];
#pragma unroll
    for (int j = 0; j < NS; ++j)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            const int r = j * 16 + hf * 8 + (q & 7);
            woff[j][hf] = uint32_t(int64_t(r >> p.log2_br) * p.strip_bytes +
                                   (int64_t(r & ((1 << p.log2_br) - 1)) << (p.log2_bc + 1)));
        }
    auto w_load = [&](bf16x8 (&x)[NS][2], int t, int c) {
        const uint8_t* wt = w0 + t * tile_bytes;
        const uint32_t ko = uint32_t(w_koff<true>(p, c * kChunkK + wave * 64 + kc));
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) x[j][hf] = load_stream(wt + (woff[j][hf] + ko));
    };

    // Staging of A: thread (wave, lane) moves 16-byte column 'lane' of rows
    // wave + 8 u (u < 4 in part 0, 4 <= u < 8 in part 1 for four M tiles) --
    // one contiguous 1 KB row segment per wave instruction; rows past M load
    // row M - 1 and store zeros.  Part 0 of the next chunk is loaded at the
    // top of a chunk; with two parts it is stored halfway through the tiles
    // (the other buffer is free once every wave has passed the previous
    // chunk's barrier) and part 1 loaded then, so only four registers of
    // staging are live at a time.  Every load
    // of the loop is issued unconditionally (a step or chunk past the range
    // reloads one just read, from cache), so the compiler can count the
    // loads in flight exactly and never has to drain them.
    const uint8_t* Ab = reinterpret_cast<const uint8_t*>(p.A);
    u32x4 ra[4];
    auto a_load = [&](int c, int part) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int r = wave + 8 * (u + 4 * part);
            const u32x4 z = {0u, 0u, 0u, 0u};
            const u32x4 v = *reinterpret_cast<const u32x4*>(
                Ab + (int64_t(min(r, p.M - 1)) * p.K + int64_t(c) * kChunkK + lane * 8) * 2);
            ra[u] = r < p.M ? v : z;
        }
    };
    auto a_store = [&](int buf, int part) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            *reinterpret_cast<u32x4*>(smem + buf * kAChunkBytes + a_lds(wave + 8 * (u + 4 * part), lane)) = ra[u];
    };

    f32x4 acc[T][MT][NS];
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int j = 0; j < NS; ++j) acc[t][mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Weight ring: xr[0] holds the step computed next, xr[1..P] the steps
    // after it in (chunk, tile) order.
    bf16x8 xr[P + 1][NS][2];
    // step s of the wave's sequence: tile s % T of chunk c0 + s / T; past the
    // range, the last step again
    auto w_step = [&](bf16x8 (&x)[NS][2], int t, int c) {
        const bool in = c < c1;
        w_load(x, in ? t : T - 1, in ? c : c1 - 1);
    };
    a_load(c0, 0);
#pragma unroll
    for (int s = 0; s < P; ++s) w_step(xr[s], s % T, c0 + s / T);
    a_store(0, 0);
    if constexpr (kStageParts == 2) {
        a_load(c0, 1);
        a_store(0, 1);
    }
    __syncthreads();

    for (int c = c0; c < c1; ++c) {
        const int buf = (c - c0) & 1;
        a_load(min(c + 1, c1 - 1), 0);
        __builtin_amdgcn_sched_barrier(0);
        // this wave's A operands for step 'wave' of the chunk: columns
        // 8 wave + g (k 0..31 of the step) and 8 wave + 4 + g (k 32..63)
        const uint8_t* As = smem + buf * kAChunkBytes;
        bf16x8 a0[MT], a1[MT];
        auto a_read = [&]() {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                a0[mt] = *reinterpret_cast<const bf16x8*>(As + a_lds(mt * 16 + q, wave * 8 + g));
                a1[mt] = *reinterpret_cast<const bf16x8*>(As + a_lds(mt * 16 + q, wave * 8 + 4 + g));
            }
        };
        if constexpr (!kAPerTile) a_read();
#pragma unroll
        for (int t = 0; t < T; ++t) {
            w_step(xr[P], (t + P) % T, c + (t + P) / T);   // the step P ahead
            if constexpr (kAPerTile) a_read();
            if constexpr (kStageParts == 2) {
                if (t == T / 2) {   // the first half of the next chunk, then load the second
                    a_store(buf ^ 1, 0);
                    a_load(min(c + 1, c1 - 1), 1);
                }
            }
#pragma unroll
            for (int j = 0; j < NS; ++j) {
                const bf16x8 x0 = xr[0][j][0], x1 = xr[0][j][1];
                const bf16x8 tsw = lo ? x1 : x0;
                const bf16x8 sw = swap8(tsw);
                const bf16x8 b0 = lo ? x0 : sw;
                const bf16x8 b1 = lo ? sw : x1;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    acc[t][mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[mt], b0, acc[t][mt][j], 0, 0, 0);
                    acc[t][mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[mt], b1, acc[t][mt][j], 0, 0, 0);
                }
            }
#pragma unroll
            for (int s = 0; s < P; ++s)
#pragma unroll
                for (int j = 0; j < NS; ++j)
#pragma unroll
                    for (int hf = 0; hf < 2; ++hf) xr[s][j][hf] = xr[s + 1][j][hf];
            // keep the steps in order: loads then complete in the order they
            // are consumed, so each step waits only for its own
            __builtin_amdgcn_sched_barrier(0);
        }
        a_store(buf ^ 1, kStageParts - 1);   // the next chunk (after the last, unused)
        __syncthreads();
    }

    if (p.fetch && lane == 0 && c1 > c0)   // each step: NS subtiles x 2 loads of 64 lanes x 16 B
        atomicAdd(p.fetch, (unsigned long long)(c1 - c0) * T * 2ull * NS * 1024ull);

    // ---- sum the 8 waves in a fixed order, TP tiles per pass (32 or 64 KB each) ----
    constexpr int kTileRed = kLdsWaves * MT * NS * 64;   // f32x4 entries per tile
    constexpr int TP = kLdsThreads / (MT * NS * 64);     // tiles per pass: 2 or 1
    static_assert(TP * kTileRed * 16 <= 2 * kAChunkBytes, "reduction exceeds the staging buffers");
    static_assert(TP * MT * NS * 64 == kLdsThreads, "one entry per thread per pass");
    f32x4* red = reinterpret_cast<f32x4*>(smem);
    const bool final_out = p.split_k == 1;
    float* part = p.ws + int64_t(split) * p.ws_stride;
#pragma unroll
    for (int t0 = 0; t0 < T; t0 += TP) {
#pragma unroll
        for (int tt = 0; tt < TP; ++tt)
            if (t0 + tt < T)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int j = 0; j < NS; ++j)
                        red[tt * kTileRed + ((wave * MT + mt) * NS + j) * 64 + lane] = acc[t0 + tt][mt][j];
        __syncthreads();
        const int e = threadIdx.x;
        const int tt = e / (MT * NS * 64), mt = (e / (NS * 64)) % MT, j = (e / 64) % NS, l = e % 64;
        if (t0 + tt < T) {
            f32x4 v = red[tt * kTileRed + (mt * NS + j) * 64 + l];
#pragma unroll
            for (int w = 1; w < kLdsWaves; ++w) v += red[tt * kTileRed + ((w * MT + mt) * NS + j) * 64 + l];
            const int n = n_base0 + (t0 + tt) * 32 + j * 16 + (l & 15);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = mt * 16 + (l >> 4) * 4 + r;
                if (m < p.M) {
                    if (final_out) store_out(p.C, int64_t(m) * p.N + n, v[r], p.out_bf16);
                    else part[int64_t(m) * p.N + n] = v[r];
                }
            }
        }
        __syncthreads();
    }
}

template <int T>
hipError_t launch_t(const DecodeParams& p, int grid, hipStream_t stream) {
    if (p.M > 32) {   // four M tiles: T = 4 (at T = 5 the registers spill)
        if constexpr (T == 4) {
            hipLaunchKernelGGL((decode_lds_kernel<T, 1, 4>), dim3(grid), dim3(kLdsThreads), 0, stream, p);
            return hipGetLastError();
        }
        return hipErrorInvalidValue;
    }
    hipLaunchKernelGGL((decode_lds_kernel<T, 2, 2>), dim3(grid), dim3(kLdsThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_lds_decode(const DecodeParams& p, int tiles_per_wg, int grid, hipStream_t stream) {
    switch (tiles_per_wg) {
        case 4: return launch_t<4>(p, grid, stream);
        case 5: return launch_t<5>(p, grid, stream);
        case 6: return launch_t<6>(p, grid, stream);
        case 7: return launch_t<7>(p, grid, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace tl
