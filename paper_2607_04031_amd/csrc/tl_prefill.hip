// Prefill GEMM (large M): C[M][N] = A[M][K] * W^T with bf16 MFMA 32x32x16 and
// fp32 accumulation; W tile-major (or row-major [N][K]).  MFMA-bound at large
// batch (TileLens Section 6.2: the dense FFN becomes compute-bound as the batch
// grows).
//
// Workgroup tile BM x BN x 64: 128x128 and 256x128 with 4 wavefronts in a
// 2 x 2 grid, 256x256 with 8 wavefronts in a 2 x 4 grid (two per SIMD, so one
// wave's MFMAs cover the other's LDS and barrier waits); each wave owns a block
// of C as MFMA 32x32 tiles.
// Per 64-wide K step the workgroup stages its A tile and its weight tile in
// LDS; the weight tile of a (64, 32) BF16 memory tile layout is exactly four
// whole 4 KB memory tiles, so each wavefront load instruction reads 1 KB of
// one contiguous memory tile.  Per-lane weight addresses are Eq. 2 with shifts
// and masks (Section 3.2).  The next K step's global loads are issued before
// the current step's MFMAs (register double buffering; LDS is double buffered
// so one barrier per step suffices); LDS operand fragments for the next
// 16-wide sub-step are read while the current sub-step's MFMAs run.  LDS rows
// are 128 B with 16-byte chunks XOR-swizzled (see swz) so operand reads are
// free of bank conflicts.
// Padded weights (Section 3.3; strips of ceil(K / bc) memory tiles): rows
// past M or N are clamped and never stored; a last K step partly past K
// (K % 8 == 0) stages zeros for the chunks past K.
#include <hip/hip_runtime.h>

#include "tl_internal.h"

namespace tl {
namespace {

typedef short bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

struct PrefillParams {
    const uint16_t* A;
    const uint8_t* W;
    void* C;
    unsigned long long* fetch;
    int M, N, K;
    int64_t ldc;             // row stride of C in elements (N of the whole GEMM)
    int m_tiles;
    int64_t strip_bytes;
    int log2_br, log2_bc, log2_G;
    int br_mask, bc_mask;
    bool out_bf16;
    int log2_fetch;          // block-granular emulation on a row-major weight: log2(G), else 0
    int64_t w_bytes;         // bytes of the weight (the block loads stay below it)
};

__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// LDS byte offset of 16-byte chunk 'chunk' (0..7) of 128-byte row 'row'.
// gfx950 serves a 16-byte-per-lane LDS read 16 lanes at a time across 64
// four-byte banks (256 B): rows r and r + 1 fall in different halves, so the
// chunk is XORed with (r / 2) mod 8 to give the 16 rows an MFMA operand read
// touches 16 distinct 16-byte bank groups.
__device__ inline int swz(int row, int chunk) { return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4); }

typedef int i32x4p __attribute__((ext_vector_type(4)));

// BLOCKROW (row-major weight, TL_FETCH_BLOCK): before the weight loads of a K
// step, the workgroup loads whole every G-byte block (aligned to the weight's
// base) that holds one of its BN row segments -- rows in address order, so a
// block shared by consecutive rows is loaded once per step -- into a live
// sink and counts it: a large-granularity memory's amplification (Section
// 2.5) paid as real HBM traffic; the operand loads then hit in cache.
template <int BM, int BN, int WGM, int WGN, bool TILE, bool BLOCKROW = false>
__global__ __launch_bounds__(64 * WGM * WGN) void prefill_kernel(PrefillParams p) {
    static_assert(!(TILE && BLOCKROW), "block emulation is for row-major weights");
    constexpr int NT = 64 * WGM * WGN;   // threads; waves form a WGM x WGN grid
    constexpr int BK = 64;
    constexpr int A_BYTES = BM * BK * 2, W_BYTES = BN * BK * 2;
    constexpr int STAGE = A_BYTES + W_BYTES;
    constexpr int A_CH = BM * 8 / NT;    // 16-byte chunks per thread per K step
    constexpr int W_CH = BN * 8 / NT;
    constexpr int ROWS = NT / 8;         // rows one pass of the workgroup stages
    constexpr int WM = BM / WGM, WN = BN / WGN;   // wave tile
    constexpr int FM = WM / 32;          // 32-row MFMA tiles per wave
    constexpr int FN = WN / 32;          // 32-col MFMA tiles per wave
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];

    // XCD-aware order: workgroup b runs on XCD (b mod 8); give each XCD a
    // contiguous range of tiles so neighbouring tiles share that XCD's L2.
    const int T = gridDim.x, b = blockIdx.x;
    const int lb = (T % 8 == 0) ? (b % 8) * (T / 8) + b / 8 : b;
    const int tm = lb % p.m_tiles, tn = lb / p.m_tiles;
    const int m0 = tm * BM, n0 = tn * BN;

    // Thread t stages 16-byte chunk c = t % 8 of rows r = t / 8 + ROWS i of
    // both tiles (i < A_CH, i < W_CH).  Row addresses are rebuilt per step from
    // one base so they cost no registers; rows past M or N are clamped (their
    // results are never stored).
    const int t = threadIdx.x;
    const int r0 = t >> 3, c0 = t & 7;
    const int a_lds0 = swz(r0, c0);      // row r0 + ROWS i sits ROWS * 128 * i bytes further
    const int w_k = c0 * 8;

    const int lane = t & 63, wave = t >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // prefetch registers for the next K step (native vectors indexed only by
    // unrolled constants, so they stay in VGPRs)
    u32x4 ra[A_CH], rw[W_CH];
    // 32-bit byte offsets from the (uniform) base pointers: A and W are
    // below 4 GB (checked on the host), and 32-bit offsets halve the
    // registers the hoisted row addresses take.
    const uint8_t* Ab = reinterpret_cast<const uint8_t*>(p.A);
    auto a_addr = [&](int i, int k0) {
        const uint32_t m = uint32_t(min(m0 + r0 + ROWS * i, p.M - 1));
        return reinterpret_cast<const u32x4*>(Ab + (m * uint32_t(p.K) + uint32_t(k0 + w_k)) * 2u);
    };
    auto w_addr = [&](int i, uint32_t ko) {
        const uint32_t n = uint32_t(min(n0 + r0 + ROWS * i, p.N - 1));
        uint32_t off;
        if (TILE) off = (n >> p.log2_br) * uint32_t(p.strip_bytes) + ((n & uint32_t(p.br_mask)) << (p.log2_bc + 1));
        else off = n * uint32_t(p.K) * 2u;
        return reinterpret_cast<const u32x4*>(p.W + (off + ko));
    };
    auto w_koff = [&](int k) -> uint32_t {
        if (TILE) return (uint32_t(k >> p.log2_bc) << p.log2_G) + uint32_t((k & p.bc_mask) << 1);
        return uint32_t(k) << 1;
    };
    const int KT = (p.K + BK - 1) / BK;
    i32x4p sink = {0, 0, 0, 0};
    uint64_t fetched = 0;
    auto fetch_blocks = [&](int k0) {
        if constexpr (BLOCKROW) {
            const int64_t Gb = int64_t(1) << p.log2_fetch;
            int64_t prev = -1;
            for (int r = 0; r < BN; ++r) {
                const int64_t n = min(n0 + r, p.N - 1);
                const int64_t blk = ((n * p.K + k0) * 2) >> p.log2_fetch;
                if (blk == prev) continue;
                prev = blk;
                const uint8_t* base = p.W + (blk << p.log2_fetch);
                for (int64_t c = int64_t(t) * 16; c < Gb; c += int64_t(NT) * 16)
                    if ((blk << p.log2_fetch) + c < p.w_bytes)
                        sink ^= __builtin_nontemporal_load(reinterpret_cast<const i32x4p*>(base + c));
                fetched += uint64_t(Gb);
            }
        }
    };
    auto gload = [&](int kstep) {
        const int k0 = kstep * BK;
        fetch_blocks(k0);
        if (k0 + BK <= p.K) {   // uniform: every step but a partial last one
#pragma unroll
            for (int i = 0; i < A_CH; ++i) ra[i] = *a_addr(i, k0);
            const uint32_t ko = w_koff(k0 + w_k);
#pragma unroll
            for (int i = 0; i < W_CH; ++i) rw[i] = *w_addr(i, ko);
        } else {
            // chunks past K: load column 0 (in bounds), stage zeros
            const bool kin = k0 + w_k < p.K;
            const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int i = 0; i < A_CH; ++i) {
                const u32x4 v = *a_addr(i, kin ? k0 : -w_k);
                ra[i] = kin ? v : z;
            }
            const uint32_t ko = w_koff(kin ? k0 + w_k : 0);
#pragma unroll
            for (int i = 0; i < W_CH; ++i) {
                const u32x4 v = *w_addr(i, ko);
                rw[i] = kin ? v : z;
            }
        }
    };
    auto sstore = [&](int buf) {
        uint8_t* As = smem + buf * STAGE;
#pragma unroll
        for (int i = 0; i < A_CH; ++i) *reinterpret_cast<u32x4*>(As + a_lds0 + ROWS * 128 * i) = ra[i];
#pragma unroll
        for (int i = 0; i < W_CH; ++i) *reinterpret_cast<u32x4*>(As + A_BYTES + a_lds0 + ROWS * 128 * i) = rw[i];
    };
    // Pipeline: LDS buffer kt % 2 holds K step kt; the registers hold step
    // kt + 1, loaded one iteration earlier.  Each iteration first writes them
    // to the other buffer (free: every wave passed the previous barrier), then
    // issues the loads of step kt + 2, then runs step kt's MFMAs -- so the LDS
    // writes overlap the MFMAs and each global load has a full iteration to
    // arrive.
    gload(0);
    sstore(0);
    if (KT > 1) gload(1);
    __syncthreads();

    // LDS read offsets of this lane's operand rows (chunk added per sub-step)
    int a_row[FM], w_row[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) a_row[i] = wm * WM + i * 32 + (lane & 31);
#pragma unroll
    for (int j = 0; j < FN; ++j) w_row[j] = wn * WN + j * 32 + (lane & 31);
    const int khalf = lane >> 5;

    for (int kt = 0; kt < KT; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < KT) sstore(buf ^ 1);
        if (kt + 2 < KT) gload(kt + 2);
        const uint8_t* As = smem + buf * STAGE;
        const uint8_t* Ws = As + A_BYTES;
        // Operand fragments of the next 16-wide sub-step are read while the
        // current one's MFMAs run (double-buffered) unless the 128x128 wave
        // tile leaves no registers for it.
        constexpr bool kDoubleFrag = FM * FN <= 8;
        bf16x8 af[2][FM], bfr[2][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) af[0][i] = *reinterpret_cast<const bf16x8*>(As + swz(a_row[i], khalf));
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[0][j] = *reinterpret_cast<const bf16x8*>(Ws + swz(w_row[j], khalf));
        // let the scheduler interleave the LDS operand reads with the MFMAs
        __builtin_amdgcn_iglp_opt(1);
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            const int cur = kDoubleFrag ? (s & 1) : 0, nxt = kDoubleFrag ? (cur ^ 1) : 0;
            if (kDoubleFrag && s + 1 < BK / 16) {
                const int chunk = (s + 1) * 2 + khalf;
#pragma unroll
                for (int i = 0; i < FM; ++i) af[nxt][i] = *reinterpret_cast<const bf16x8*>(As + swz(a_row[i], chunk));
#pragma unroll
                for (int j = 0; j < FN; ++j) bfr[nxt][j] = *reinterpret_cast<const bf16x8*>(Ws + swz(w_row[j], chunk));
            }
            if (!kDoubleFrag && s > 0) {
                const int chunk = s * 2 + khalf;
#pragma unroll
                for (int i = 0; i < FM; ++i) af[0][i] = *reinterpret_cast<const bf16x8*>(As + swz(a_row[i], chunk));
#pragma unroll
                for (int j = 0; j < FN; ++j) bfr[0][j] = *reinterpret_cast<const bf16x8*>(Ws + swz(w_row[j], chunk));
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

    if (p.fetch && t == 0)
        atomicAdd(p.fetch, BLOCKROW ? (unsigned long long)fetched : (unsigned long long)KT * (unsigned long long)W_BYTES);
    if constexpr (BLOCKROW) {
        // keeps the block loads live; M >= 1 always, so this never stores
        if ((sink[0] ^ sink[1] ^ sink[2] ^ sink[3]) == 0x6c8e9cf5 && p.M < 0) static_cast<float*>(p.C)[0] = 0.f;
    }

    // D layout of a 32x32 MFMA tile: lane l, register v holds
    // row 8*(v/4) + 4*(l/32) + v%4, column l%32.
    const bool full = m0 + BM <= p.M && n0 + BN <= p.N;
    const int row_base = m0 + wm * WM + 4 * (lane >> 5);
    const int col_base = n0 + wn * WN + (lane & 31);
    if (p.out_bf16) {
        uint16_t* C = static_cast<uint16_t*>(p.C);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = row_base + i * 32 + 8 * (v >> 2) + (v & 3);
                    const int col = col_base + j * 32;
                    if (full || (row < p.M && col < p.N))
                        C[int64_t(row) * p.ldc + col] = f32_to_bf16_rne(acc[i][j][v]);
                }
    } else {
        float* C = static_cast<float*>(p.C);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = row_base + i * 32 + 8 * (v >> 2) + (v & 3);
                    const int col = col_base + j * 32;
                    if (full || (row < p.M && col < p.N)) C[int64_t(row) * p.ldc + col] = acc[i][j][v];
                }
    }
}

template <int BM, int BN, int WGM, int WGN>
hipError_t launch_t(const PrefillParams& p, int grid, bool tile, hipStream_t s) {
    if (tile) hipLaunchKernelGGL((prefill_kernel<BM, BN, WGM, WGN, true>), dim3(grid), dim3(64 * WGM * WGN), 0, s, p);
    else if (p.log2_fetch > 0)
        hipLaunchKernelGGL((prefill_kernel<BM, BN, WGM, WGN, false, true>), dim3(grid), dim3(64 * WGM * WGN), 0, s, p);
    else hipLaunchKernelGGL((prefill_kernel<BM, BN, WGM, WGN, false>), dim3(grid), dim3(64 * WGM * WGN), 0, s, p);
    return hipGetLastError();
}

// One launch over columns [n_begin, n_begin + n_cols) of the GEMM with
// tile_m x tile_n tiles.  The weight rows of that range start n_begin * Kp * 2
// bytes into W (Kp: K padded to whole memory tiles for tile-major, K for
// row-major; tile-major strips of block_rows rows are contiguous, and
// n_begin is a multiple of block_rows).
hipError_t launch_range(const PrefillLaunch& q, int64_t n_begin, int64_t n_cols, int tile_m, int tile_n,
                        hipStream_t stream) {
    PrefillParams p;
    const int64_t c_elem = q.out_bf16 ? 2 : 4;
    const bool tile = q.L.kind == TL_LAYOUT_TILE;
    const int64_t kp = tile ? padded_cols(q.L, q.K) : q.K;   // K of the stored weight
    p.A = q.A;
    p.W = q.W + n_begin * kp * 2;
    p.C = static_cast<uint8_t*>(q.C) + n_begin * c_elem;
    p.fetch = q.fetch;
    p.M = int(q.M);
    p.N = int(n_cols);
    p.K = int(q.K);
    p.ldc = q.N;
    p.m_tiles = int((q.M + tile_m - 1) / tile_m);
    p.strip_bytes = tile ? q.L.br * kp * 2 : 0;
    p.log2_br = tile ? q.L.log2_br : 0;
    p.log2_bc = tile ? q.L.log2_bc : 0;
    p.log2_G = tile ? q.L.log2_G : 0;
    p.br_mask = tile ? int(q.L.br - 1) : 0;
    p.bc_mask = tile ? int(q.L.bc - 1) : 0;
    p.out_bf16 = q.out_bf16;
    p.log2_fetch = (!tile && q.block_fetch) ? ilog2(q.fetch_G) : 0;
    p.w_bytes = n_cols * kp * 2;
    const int64_t n_tiles = (n_cols + tile_n - 1) / tile_n;
    const int grid = int(p.m_tiles * n_tiles);
    // 256x256: 8 waves (2 per SIMD) of 128x64; smaller tiles: 4 waves in 2 x 2
    if (tile_m == 256 && tile_n == 256) return launch_t<256, 256, 2, 4>(p, grid, tile, stream);
    if (tile_m == 256) return launch_t<256, 128, 2, 2>(p, grid, tile, stream);
    return launch_t<128, 128, 2, 2>(p, grid, tile, stream);
}

}  // namespace

hipError_t launch_prefill(const PrefillLaunch& q, hipStream_t stream) {
    hipError_t e = launch_range(q, 0, q.n_main, q.tile_m, q.tile_n, stream);
    if (e != hipSuccess || q.n_main == q.N) return e;
    return launch_range(q, q.n_main, q.N - q.n_main, 128, 128, stream);
}

}  // namespace tl
