// Decode GEMM, M <= 64: C[M][N] = A[M][K] * W^T with W tile-major (or plain
// row-major [N][K] for the NATIVE baseline).  HBM-bound: every weight byte is
// read exactly once per call (TileLens Section 2.1: decode reads the weights
// once per token).
//
// Work decomposition
//   workgroup = one compute tile of tile_n rows of W (a whole number of memory
//   tiles) x one K-split; 4 wavefronts interleave along K in 64-element steps,
//   so at any moment the workgroup streams consecutive memory tiles of a strip
//   (Section 2.3: tiles iterate along K).
//   Each 64-step is two bf16 MFMA 16x16x32 K-halves per 16-row n-subtile:
//     A operand = activations (rows m = lane % 16), zero-padded to 16 rows,
//     B operand = weights     (cols n = lane % 16),
//   lane l supplies 8 consecutive k (16 bytes) at k-slot group l / 16.
//   The per-lane weight address is Eq. 2 evaluated with shifts and masks
//   (Section 3.2, Eq. 1): strip = n >> log2(br), row-in-tile = n & (br - 1),
//   memory tile along K = k >> log2(bc), column-in-tile = k & (bc - 1).
//   With bc >= 8 each 16-byte load stays inside one memory-tile row.
//   Padded weights (Section 3.3: N or K not a multiple of the memory tile's
//   sides, strips of ceil(K / bc) tiles): rows past N load row N - 1 and are
//   never stored; a last 64-wide K step that is partly past K (K % 8 == 0)
//   runs once, after the streaming loops, with the lanes past K reading
//   zeros.
//   Weight loads are non-temporal (read once) and each load instruction reads
//   whole 128-byte lines (see decode_kernel).
// Reduction
//   waves -> LDS -> fixed-order sum; K-splits -> fp32 partials in a workspace,
//   summed in split order by a second small kernel.  No float atomics, so
//   results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "tl_decode_common.h"

namespace tl {
namespace {

// Weight loads.  Lane l = 16 g + q needs, per 16-row n-subtile and 64-wide K
// step, the MFMA B operands  B0 = W[row q][k-chunk g], B1 = W[row q][chunk 4+g]
// (chunks of 8 elements).  Fetching those directly touches 16 rows x 64 B per
// instruction.  Instead every lane loads
//     x0 = W[row (q & 7)    ][chunk 4 (q >> 3) + g]
//     x1 = W[row 8 + (q & 7)][chunk 4 (q >> 3) + g]
// so each instruction reads 8 rows x 128 B -- whole 128 B lines for every
// memory-tile shape with block_cols >= 8 -- and the operands are rebuilt with
// one exchange between lanes l and l ^ 8:
//     t = q < 8 ? x1 : x0,  s = t from lane l ^ 8,
//     B0 = q < 8 ? x0 : s,  B1 = q < 8 ? s : x1.
//
// Grouped launch (GROUPED): workgroup b serves group e = b / tiles_per_group
// (one weight of a stack, e.g. one MoE expert) and its tile b % tiles_per_group
// (split_k is 1).  The group's output rows [offsets[e], offsets[e+1]) are
// clamped to [0, total_rows]; row r reads A row token_ids[r] (or r), and an
// id outside [0, a_rows) reads zeros.  Rows are processed in chunks of
// 16 MT, each chunk streaming the tile's weights again.
//
// Gated expert activation (SWIGLU, grouped, NS = 4): each group's weight
// stacks its gate projection (rows [0, I)) and up projection (rows [I, 2I)),
// the fused_moe convention.  Workgroup tile t takes gate rows [32 t, 32 t + 32)
// as subtiles 0-1 and the up rows I + [32 t, 32 t + 32) as subtiles 2-3 --
// two whole 32-row strips -- and writes C[r][32 t + c] = silu(g) * u for its
// 32 columns (C has I columns).
template <int MT, int NS, int U, int WAVES, bool TILE, bool BLOCKROW, bool GROUPED, bool SWIGLU = false>
__global__ __launch_bounds__(64 * WAVES) void decode_kernel(DecodeParams p) {
    static_assert(!SWIGLU || (GROUPED && NS == 4), "gated launches are grouped, 32 gate + 32 up rows");
    constexpr int kWaves = WAVES;
    constexpr int kThreads = 64 * WAVES;
    constexpr int TN = 16 * NS;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    int tile, split, row0 = 0, rows = p.M;
    const uint8_t* W = p.W;
    if constexpr (GROUPED) {
        const int e = blockIdx.x / p.tiles_per_group;
        tile = blockIdx.x - e * p.tiles_per_group;
        split = 0;
        const int r0 = min(max(p.offsets[e], 0), p.total_rows);
        const int r1 = min(max(p.offsets[e + 1], r0), p.total_rows);
        if (r1 <= r0) return;                       // uniform over the workgroup
        row0 = r0;
        rows = r1 - r0;
        W += int64_t(e) * p.group_stride;
    } else {
        tile = blockIdx.x / p.split_k;
        split = blockIdx.x - tile * p.split_k;
    }

    // K range of this split in 64-element steps; steps from kfull on are
    // partly past K (only the last one, when K % 64 != 0)
    const int u0 = int((int64_t(p.units) * split) / p.split_k);
    const int u1 = int((int64_t(p.units) * (split + 1)) / p.split_k);
    const int st0 = u0 * p.steps_per_unit;
    const int st1 = min(u1 * p.steps_per_unit, p.ksteps);
    const int st1f = min(st1, p.kfull);

    const int n_base = SWIGLU ? tile * 32 : tile * TN;   // first output column of the tile
    const int g = lane >> 4, q = lane & 15;
    const bool lo = q < 8;
    const int kc = (((q >> 3) << 2) + g) << 3;   // k offset of this lane's weight chunk in a step

    // Weight addresses: the tile's first row as a uniform 64-bit base (scalar
    // registers) plus a per-lane 32-bit byte offset -- the rows of one tile
    // span less than 2^31 bytes (the planner checks it) -- so a load is a
    // scalar base + 32-bit vector offset and needs no 64-bit vector pointers
    // (fewer registers: more resident waves).
    const int64_t tile_off = TILE ? int64_t(n_base >> p.log2_br) * p.strip_bytes : int64_t(n_base) * p.K * 2;
    const uint8_t* wtile = W + tile_off;
    uint32_t woff[NS][2];
#pragma unroll
    for (int j = 0; j < NS; ++j)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            int n;
            if constexpr (SWIGLU) n = (j < 2 ? n_base + j * 16 : p.swiglu_up + n_base + (j - 2) * 16) + hf * 8 + (q & 7);
            else n = min(n_base + j * 16 + hf * 8 + (q & 7), p.N - 1);
            int64_t off;
            if (TILE) off = int64_t(n >> p.log2_br) * p.strip_bytes + (int64_t(n & ((1 << p.log2_br) - 1)) << (p.log2_bc + 1));
            else off = int64_t(n) * p.K * 2;
            woff[j][hf] = uint32_t(off - tile_off);
        }
    for (int mc = 0;;) {   // row chunks: one pass unless GROUPED
    const int crows = rows - mc;
    // Activations are loaded like the weights (8 rows x 128 B per
    // instruction, then the lane exchange): lane (g, q) reads row
    // 16 mt + 8 hf + (q & 7) at this lane's chunk kc.  Rows past M read zeros;
    // a half-tile that is entirely past M is not loaded at all.
    // activation rows: byte offsets from A (A spans less than 2^31 bytes)
    const uint8_t* Ab = reinterpret_cast<const uint8_t*>(p.A);
    uint32_t aoff[MT][2];
    bool aok[MT][2], aany[MT][2];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            const int m = mt * 16 + hf * 8 + (q & 7);
            aok[mt][hf] = m < crows;
            aany[mt][hf] = mt * 16 + hf * 8 < crows;
            int arow_idx = m;
            if constexpr (GROUPED) {
                arow_idx = row0 + mc + m;
                if (aok[mt][hf] && p.token_ids) arow_idx = p.token_ids[arow_idx];
                aok[mt][hf] = aok[mt][hf] && arow_idx >= 0 && arow_idx < p.a_rows;
            }
            aoff[mt][hf] = uint32_t((aok[mt][hf] ? arow_idx : 0) * p.K + kc) * 2u;
        }

    f32x4 acc[MT][NS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NS; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const bf16x8 zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
    // steps of this wave: st0 + wave + 4 * i
    const int nsteps = st1f - st0 - wave > 0 ? (st1f - st0 - wave + kWaves - 1) / kWaves : 0;
    int st = st0 + wave;
    int i = 0;
    auto exchange = [&](const bf16x8& x0, const bf16x8& x1, bf16x8& o0, bf16x8& o1) {
        const bf16x8 t = lo ? x1 : x0;
        const bf16x8 s = swap8(t);
        o0 = lo ? x0 : s;
        o1 = lo ? s : x1;
    };
    auto compute = [&](const bf16x8 (&x)[NS][2], const bf16x8 (&xa)[MT][2]) {
        bf16x8 a0[MT], a1[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) exchange(xa[mt][0], xa[mt][1], a0[mt], a1[mt]);
#pragma unroll
        for (int j = 0; j < NS; ++j) {
            bf16x8 b0, b1;
            exchange(x[j][0], x[j][1], b0, b1);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[mt], b0, acc[mt][j], 0, 0, 0);
                acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[mt], b1, acc[mt][j], 0, 0, 0);
            }
        }
    };
    auto load_a = [&](int k, bf16x8 (&xa)[MT][2]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf)
                if (aany[mt][hf])   // uniform: skips the load when the half-tile is past M
                    xa[mt][hf] = aok[mt][hf] ? *reinterpret_cast<const bf16x8*>(Ab + (aoff[mt][hf] + uint32_t(k) * 2u)) : zero8;
                else
                    xa[mt][hf] = zero8;
    };
    // Block-granular fetch on a row-major weight (emulating a memory that only
    // returns whole G-byte blocks, aligned to the weight's base): at each K
    // step every block holding one of the tile's row segments is loaded whole
    // and folded into a live sink, so a large-granularity memory's read
    // amplification is paid as real loads; the operand loads above then hit
    // in cache.  Rows are visited in address order, so a block shared by
    // consecutive rows (K * 2 < G) is fetched once per step.
    i32x4 sink = {0, 0, 0, 0};
    uint64_t fetched = 0;
    auto fetch_blocks = [&](int k0) {
        if constexpr (BLOCKROW) {
            int64_t prev = -1;
            const int64_t G = int64_t(1) << p.log2_fetch;
            for (int r = 0; r < TN; ++r) {
                const int64_t b = ((int64_t(n_base + r) * p.K + k0) * 2) >> p.log2_fetch;
                if (b == prev) continue;
                prev = b;
                const uint8_t* base = p.W + (b << p.log2_fetch);
                for (int64_t c = int64_t(lane) * 16; c < G; c += 1024)
                    if ((b << p.log2_fetch) + c < p.w_bytes)
                        sink ^= __builtin_bit_cast(i32x4, load_stream(base + c));
                fetched += uint64_t(G);
            }
        }
    };
    for (; i + U <= nsteps; i += U) {
        bf16x8 x[U][NS][2];
        bf16x8 a[U][MT][2];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = (st + u * kWaves) * 64;
            const int64_t ko = w_koff<TILE>(p, k + kc);
#pragma unroll
            for (int j = 0; j < NS; ++j)
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) x[u][j][hf] = load_stream(wtile + (woff[j][hf] + uint32_t(ko)));
            load_a(k, a[u]);
            fetch_blocks(k);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) compute(x[u], a[u]);
        st += U * kWaves;
    }
    for (; i < nsteps; ++i) {
        const int k = st * 64;
        const int64_t ko = w_koff<TILE>(p, k + kc);
        bf16x8 x[NS][2], a[MT][2];
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) x[j][hf] = load_stream(wtile + (woff[j][hf] + uint32_t(ko)));
        load_a(k, a);
        fetch_blocks(k);
        compute(x, a);
        st += kWaves;
    }
    // the last step, partly past K: its owner wave (in the K interleave)
    // loads the lanes inside K and zeros the rest (addresses of lanes past K
    // are clamped to column 0, so every access stays inside the buffers)
    const bool own_partial = p.kfull < st1 && p.kfull >= st0 && (p.kfull - st0) % kWaves == wave;
    if (own_partial) {
        const int k = p.kfull * 64;
        const bool kin = k + kc < p.K;
        const int64_t ko = w_koff<TILE>(p, kin ? k + kc : 0);
        bf16x8 x[NS][2], a[MT][2];
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                const bf16x8 v = load_stream(wtile + (woff[j][hf] + uint32_t(ko)));
                x[j][hf] = kin ? v : zero8;
            }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                const bf16x8 v = *reinterpret_cast<const bf16x8*>(Ab + (kin ? aoff[mt][hf] + uint32_t(k) * 2u
                                                                             : aoff[mt][hf] - uint32_t(kc) * 2u));
                a[mt][hf] = kin && aok[mt][hf] ? v : zero8;
            }
        compute(x, a);
    }

    const int issued = nsteps + (own_partial ? 1 : 0);
    if (p.fetch && lane == 0 && issued > 0) {
        // tile-major / native: each step issues NS subtiles x 2 loads of 64
        // lanes x 16 B; block emulation: whole blocks fetched
        atomicAdd(p.fetch, BLOCKROW ? (unsigned long long)fetched
                                    : (unsigned long long)issued * 2ull * NS * 1024ull);
    }
    if constexpr (BLOCKROW) {
        // keeps the block loads live; M >= 1 always, so this never stores
        if ((sink[0] ^ sink[1] ^ sink[2] ^ sink[3]) == 0x6c8e9cf5 && p.M < 0) static_cast<float*>(p.C)[0] = 0.f;
    }

    // ---- reduce the waves (an in-workgroup K split) in a fixed order ----
    static_assert(WAVES * MT * NS <= 128, "reduction buffer exceeds 128 KB");
    __shared__ f32x4 red[kWaves][MT][NS][64];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NS; ++j) red[wave][mt][j][lane] = acc[mt][j];
    __syncthreads();

    // split_k == 1: final output; otherwise this split's fp32 partial, summed
    // in split order by splitk_reduce_kernel.
    constexpr int kEntries = MT * NS * 64;   // f32x4 entries per wave
    const bool final_out = p.split_k == 1;
    float* part = p.ws + int64_t(split) * p.ws_stride;
    if constexpr (SWIGLU) {
        // subtile j (gate) pairs with subtile j + 2 (up) of the same columns
        for (int e = threadIdx.x; e < MT * 2 * 64; e += kThreads) {
            const int mt = e / 128;
            const int j = (e / 64) % 2;
            const int l = e % 64;
            f32x4 vg = red[0][mt][j][l], vu = red[0][mt][j + 2][l];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) {
                vg += red[w][mt][j][l];
                vu += red[w][mt][j + 2][l];
            }
            const int n = n_base + j * 16 + (l & 15);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = mt * 16 + (l >> 4) * 4 + r;
                if (m < crows) {
                    const float h = vg[r] / (1.0f + expf(-vg[r])) * vu[r];
                    store_out(p.C, int64_t(row0 + mc + m) * p.N + n, h, p.out_bf16);
                }
            }
        }
    } else
    for (int e = threadIdx.x; e < kEntries; e += kThreads) {
        const int mt = e / (NS * 64);
        const int j = (e / 64) % NS;
        const int l = e % 64;
        f32x4 v = red[0][mt][j][l];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) v += red[w][mt][j][l];
        const int n = n_base + j * 16 + (l & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + (l >> 4) * 4 + r;
            if (m < crows && n < p.N) {
                const int64_t row = GROUPED ? int64_t(row0 + mc + m) : int64_t(m);
                if (final_out) store_out(p.C, row * p.N + n, v[r], p.out_bf16);
                else part[row * p.N + n] = v[r];
            }
        }
    }
    if constexpr (!GROUPED) break;
    mc += 16 * MT;
    if (mc >= rows) break;
    __syncthreads();   // the next chunk rewrites red[]
    }
}

// C[e] = sum over s = 0..S-1 (ascending) of ws[s * stride + e] for the mn
// elements of C, four per thread (stride: mn rounded up to 4, so every
// split's partials start 16-byte aligned; the last thread's group may be
// short).  All S partial loads are issued before the in-order sum
// (latency-bound kernel); S <= kMaxSplitReduce.
constexpr int kMaxSplitReduce = 16;
template <bool OUT_BF16>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* ws, void* C, int64_t mn, int64_t stride,
                                                            int S) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i * 4 >= mn) return;
    f32x4 part[kMaxSplitReduce];
#pragma unroll
    for (int s = 0; s < kMaxSplitReduce; ++s)
        if (s < S) part[s] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(ws + int64_t(s) * stride) + i);
    f32x4 acc = part[0];
#pragma unroll
    for (int s = 1; s < kMaxSplitReduce; ++s)
        if (s < S) acc += part[s];
    if (i * 4 + 4 > mn) {   // short last group: element stores
        for (int r = 0; i * 4 + r < mn; ++r) store_out(C, i * 4 + r, acc[r], OUT_BF16);
        return;
    }
    if (OUT_BF16) {
        uint2 o;
        o.x = uint32_t(f32_to_bf16_rne(acc[0])) | (uint32_t(f32_to_bf16_rne(acc[1])) << 16);
        o.y = uint32_t(f32_to_bf16_rne(acc[2])) | (uint32_t(f32_to_bf16_rne(acc[3])) << 16);
        reinterpret_cast<uint2*>(C)[i] = o;
    } else {
        reinterpret_cast<f32x4*>(C)[i] = acc;
    }
}

__global__ void zero_u64_kernel(unsigned long long* p) { *p = 0ull; }

template <int MT, int NS, int WAVES, bool TILE, bool GROUPED, bool SWIGLU = false>
hipError_t launch_t(const DecodeParams& p, int grid, hipStream_t stream) {
    // steps in flight per wave: fewer for larger M, and for the grouped
    // 64-row tile (4 steps there take all 256 VGPRs: one wave per SIMD; with
    // 2 the kernel fits three -- Qwen expert down projection 66.5 -> 61.3 us).
    // Four 16-row M tiles on a 64-row tile take one step: with two its ~290
    // registers leave one wave per SIMD, with one two (this kernel on the
    // Llama shapes, bf16 out, one box, M = 33 / 48 / 64: QKV 66 / 70 / 77 ->
    // 50 / 53 / 58 us; with 8 waves, O 38 / 38 / 41 -> 33 / 35 / 39, down
    // 103 / 100 / 112 -> 91 / 100 / 111; the planner now gives those three
    // shapes to the LDS-staged kernel).
    constexpr int U = (MT >= 4 && NS == 4 && !GROUPED) ? 1 : (MT >= 2 || (GROUPED && NS == 4 && !SWIGLU)) ? 2 : 4;
    if constexpr (!TILE && !GROUPED) {
        if (p.log2_fetch > 0) {   // block emulation: fewer steps in flight leave room for the block loop
            hipLaunchKernelGGL((decode_kernel<MT, NS, 2, WAVES, false, true, false>), dim3(grid), dim3(64 * WAVES), 0,
                               stream, p);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((decode_kernel<MT, NS, U, WAVES, TILE, false, GROUPED, SWIGLU>), dim3(grid), dim3(64 * WAVES), 0,
                       stream, p);
    return hipGetLastError();
}

// Instantiated (MT, NS, waves) combinations -- those whose registers fit
// the waves per SIMD they need; the planner only asks for these.  Grouped
// launches use 4 waves.
template <int MT, int NS, bool TILE>
hipError_t launch_w(const DecodeParams& p, int grid, int waves, bool grouped, hipStream_t stream) {
    if constexpr (NS == 4) {
        if (grouped && p.swiglu_up > 0) return launch_t<MT, 4, 4, TILE, true, true>(p, grid, stream);
    }
    if (grouped) return launch_t<MT, NS, 4, TILE, true>(p, grid, stream);
    if constexpr (MT * NS <= 2) {
        if (waves == 16) return launch_t<MT, NS, 16, TILE, false>(p, grid, stream);
    }
    if constexpr (MT * NS <= 16) {   // 4 x 4: one step in flight, 128 KB of LDS for the wave sums
        if (waves == 8) return launch_t<MT, NS, 8, TILE, false>(p, grid, stream);
    }
    return launch_t<MT, NS, 4, TILE, false>(p, grid, stream);
}

template <int MT>
hipError_t launch_m(const DecodeParams& p, int grid, int ns, int waves, bool tile, bool grouped, hipStream_t stream) {
    if (ns == 2) return tile ? launch_w<MT, 2, true>(p, grid, waves, grouped, stream)
                             : launch_w<MT, 2, false>(p, grid, waves, grouped, stream);
    return tile ? launch_w<MT, 4, true>(p, grid, waves, grouped, stream)
                : launch_w<MT, 4, false>(p, grid, waves, grouped, stream);
}

}  // namespace

hipError_t launch_zero_u64(unsigned long long* p, hipStream_t stream) {
    hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(1), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_decode(const DecodeLaunch& d, hipStream_t stream) {
    DecodeParams p;
    p.A = d.A;
    p.W = d.W;
    p.C = d.C;
    p.ws = d.ws;
    p.fetch = d.fetch;
    p.M = int(d.M);
    p.N = int(d.N);
    p.K = int(d.K);
    p.split_k = d.split_k;
    p.steps_per_unit = int(d.k_unit / 64);
    p.units = int((d.K + d.k_unit - 1) / d.k_unit);
    p.ksteps = int((d.K + 63) / 64);
    p.kfull = int(d.K / 64);
    p.ws_stride = (d.M * d.N + 3) / 4 * 4;
    const bool tile = d.L.kind == TL_LAYOUT_TILE;
    const int64_t elem = d.fp8 ? 1 : 2;          // bytes per weight element
    p.strip_bytes = tile ? d.L.br * padded_cols(d.L, d.K) * elem : 0;
    p.log2_br = tile ? d.L.log2_br : 0;
    p.log2_bc = tile ? d.L.log2_bc : 0;
    p.log2_G = tile ? d.L.log2_G : 0;
    p.bc_mask = tile ? int(d.L.bc - 1) : 0;
    p.out_bf16 = d.out_bf16;
    p.log2_fetch = (!tile && d.block_fetch) ? ilog2(d.fetch_G) : 0;
    p.w_bytes = d.N * d.K * elem;
    p.offsets = d.group_offsets;
    p.token_ids = d.token_ids;
    p.tiles_per_group = d.swiglu ? int(d.N / 32) : int((d.N + d.tile_n - 1) / d.tile_n);
    p.swiglu_up = d.swiglu ? int(d.N) : 0;
    p.group_stride = d.group_stride;
    p.a_rows = int(d.a_rows);
    p.total_rows = int(d.total_rows);
    p.scales = d.scales;
    if (d.lds_tiles > 0) {   // chunks of 512 columns; workgroup = lds_tiles tiles x one K range
        p.units = int(d.K / 512);
        p.steps_per_unit = 8;
        const int grid = int(d.N / 32 / d.lds_tiles) * d.split_k;
        return launch_splitk_reduce(d, launch_lds_decode(p, d.lds_tiles, grid, stream), stream);
    }
    const bool grouped = d.num_groups > 0;
    const int grid = grouped ? d.num_groups * p.tiles_per_group : p.tiles_per_group * d.split_k;
    const int ns = d.tile_n / 16;
    hipError_t e;
    if (d.L.kind == TL_LAYOUT_KN_ROW)
        return launch_splitk_reduce(d, launch_kn_decode(p, grid, d.m_tiles16, d.waves, stream), stream);
    if (d.fp8) return launch_splitk_reduce(d, launch_fp8_decode(p, grid, d.m_tiles16, ns, d.waves, tile, stream), stream);
    switch (d.m_tiles16) {
        case 1: e = launch_m<1>(p, grid, ns, d.waves, tile, grouped, stream); break;
        case 2: e = launch_m<2>(p, grid, ns, d.waves, tile, grouped, stream); break;
        default: e = launch_m<4>(p, grid, ns, d.waves, tile, grouped, stream); break;
    }
    return launch_splitk_reduce(d, e, stream);
}

hipError_t launch_splitk_reduce(const DecodeLaunch& d, hipError_t e, hipStream_t stream) {
    if (e != hipSuccess || d.split_k == 1) return e;
    const int64_t mn = d.M * d.N, stride = (mn + 3) / 4 * 4;
    const int rgrid = int((stride / 4 + 255) / 256);
    if (d.out_bf16)
        hipLaunchKernelGGL((splitk_reduce_kernel<true>), dim3(rgrid), dim3(256), 0, stream, d.ws, d.C, mn, stride,
                           d.split_k);
    else
        hipLaunchKernelGGL((splitk_reduce_kernel<false>), dim3(rgrid), dim3(256), 0, stream, d.ws, d.C, mn, stride,
                           d.split_k);
    return hipGetLastError();
}

}  // namespace tl
