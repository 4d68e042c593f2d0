// Prefill GEMM (large M): C[M][N] = A[M][K] * W^T with bf16 MFMA 32x32x16 and
// fp32 accumulation; W tile-major (or row-major [N][K]).  MFMA-bound at large
// batch (TileLens Section 6.2: the dense FFN becomes compute-bound as the batch
// grows).  Per-lane weight addresses are Eq. 2 with shifts and masks (Section
// 3.2); for the (64, 32) BF16 memory tile a 64-wide K step of a weight tile is
// a whole number of 4 KB memory tiles.
//
// Two kernels:
//  - prefill_w4_kernel (256 x 256 tiles, K % 64 == 0): four waves of
//    128 x 128, operands written to LDS straight from global memory (see the
//    comment above it).  The library's plan for large M.
//  - prefill_kernel (128 x 128, 256 x 128, and 256 x 256 when K % 64 != 0 or
//    with the row-major block emulation): each K step stages the A tile and
//    the weight tile through registers into LDS (double buffered, one barrier
//    per step); 4 waves in a 2 x 2 grid, or 8 in 2 x 4 for 256 x 256.  LDS
//    rows are 128 B with 16-byte chunks XOR-swizzled (see swz) so operand
//    reads are free of bank conflicts.  With 128 x 128 tiles it also takes
//    a K range per workgroup (the plan for 65 <= M <= 128 when the tiles are
//    fewer than the CUs) and writes fp32 partials for prefill_splitk_reduce.
// Padded weights (Section 3.3; strips of ceil(K / bc) memory tiles): rows
// past M or N are clamped and never stored; in prefill_kernel a last K step
// partly past K (K % 8 == 0) stages zeros for the chunks past K.
#include <hip/hip_runtime.h>

#include <type_traits>

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
    // K split across workgroups (1 = none; prefill_w4_kernel, and
    // prefill_kernel with 128 x 128 tiles): split s writes its fp32 partial
    // of the M x N range to ws + s * ws_stride (row stride N), summed by
    // prefill_splitk_reduce
    int split_k = 1;
    float* ws = nullptr;
    int64_t ws_stride = 0;
    // prefill_w4_kernel with PERSIST: the number of tiles the grid deals out
    int units = 0;
};

// fp32 -> bf16, round to nearest even; a NaN stays a (quiet) NaN.  One
// comparison and a select, so unrolled epilogues stay branch-free.
__device__ inline uint16_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    const uint32_t quiet = (u >> 16) | 0x0040u;
    return uint16_t((u & 0x7fffffffu) > 0x7f800000u ? quiet : rounded);
}

// two fp32 -> packed bf16 (lo in bits 0-15), round to nearest even: gfx950's
// v_cvt_pk_bf16_f32, one instruction where the bit arithmetic above takes
// about seven per value
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ inline uint32_t bf16x2_rne(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
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
    // K split (split_k > 1): workgroup lb takes K range lb / tiles of tile
    // lb % tiles, so the workgroups of one XCD share a K range of A
    const int tiles = T / p.split_k;
    const int split = lb / tiles, tix = lb - split * tiles;
    const int tm = tix % p.m_tiles, tn = tix / p.m_tiles;
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
    // this workgroup's 64-wide K steps: [kt0, kt0 + KT)
    const int kt_all = (p.K + BK - 1) / BK;
    const int kt0 = int(int64_t(kt_all) * split / p.split_k);
    const int KT = int(int64_t(kt_all) * (split + 1) / p.split_k) - kt0;
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
    gload(kt0);
    sstore(0);
    if (KT > 1) gload(kt0 + 1);
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
        if (kt + 2 < KT) gload(kt0 + kt + 2);
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
    if (p.split_k > 1) {   // this K range's fp32 partial (row stride N), for prefill_splitk_reduce
        float* P = p.ws + int64_t(split) * p.ws_stride;
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = row_base + i * 32 + 8 * (v >> 2) + (v & 3);
                    const int col = col_base + j * 32;
                    if (full || (row < p.M && col < p.N)) P[int64_t(row) * p.N + col] = acc[i][j][v];
                }
        return;
    }
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

// One 16-byte-per-lane load from global memory straight into LDS
// (global_load_lds_dwordx4): lane l's 16 bytes at base + voff land at LDS
// address lds + 16 l (lds is the same for every lane of the wave; M0 carries
// it).  Written as inline assembly so the compiler does not see an LDS write
// it cannot place -- it would otherwise wait for every load in flight before
// any later LDS read; the kernel waits for these loads itself (vmcnt).  A
// device function, so the LDS address-space cast stays out of code the host
// compilation pass instantiates.  Nothing else in the kernels that call it
// uses M0.
__device__ inline void load_lds16(const uint8_t* base, uint32_t voff, uint8_t* lds) {
    const uint32_t la = uint32_t(uintptr_t((__attribute__((address_space(3))) void*)lds));
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "s"(la)
                 : "memory", "m0");
#pragma clang diagnostic pop
}

// s_waitcnt vmcnt(n) alone (expcnt and lgkmcnt left free), n < 64
#define TL_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x0F70)

// PERSIST (bf16 output, no K split, whole 256 x 256 tiles, an even number of
// K steps): a grid of at most one workgroup per CU walks p.units tiles.  The
// next tile's first K step (with three weight stages, also its second step's
// weight tile) is loaded during this tile's last two steps, and
// this tile's C is stored straight from registers (bf16, quad-transposed: 8
// bytes of one row per lane), so no workgroup ends and starts between tiles
// and the next tile's first loads are not waited for.  (With one tile per
// workgroup only the direct stores remain: no LDS round trip and barrier.)
//
// NJ: 32-column MFMA tiles per wave along N -- 4 (256 x 256 tiles) or 5
// (256 x 320 tiles, each wave 128 x 160 of C: 320 sums per lane, AGPRs and
// VGPRs; persistent bf16 only, whose epilogue needs no LDS).  A 256 x 320
// tile fills the CUs in whole rounds where 256 x 256 does not (QKV at
// M = 2048: 256 tiles instead of 320).
template <bool TILE, bool OUT_BF16, bool PERSIST = false, int NJ = 4>
__global__ __launch_bounds__(256) void prefill_w4_kernel(PrefillParams p) {
    static_assert(!PERSIST || OUT_BF16, "the persistent grid writes bf16");
    static_assert(NJ == 4 || (NJ == 5 && PERSIST), "256 x 320 tiles: persistent bf16 only");
    constexpr int BM = 256, BN = 64 * NJ, BK = 64;
    constexpr int HALF = BM * BK * 2;            // A tile of a step: 32 KB
    constexpr int WHALF = BN * BK * 2;           // W tile of a step: 32 or 40 KB
    // LDS: two A stages, then WST weight stages -- three for 256 x 256 tiles
    // (step s + 2's weight tile loads during step s, so its latency has two
    // steps to hide in), two for 256 x 320 (the LDS budget)
    constexpr int WST = NJ == 4 ? 3 : 2;
    constexpr int LDS_OPS = 2 * HALF + WST * WHALF;
    constexpr int WROWS = BN / 4;                // W rows each wave loads per step
    constexpr int NWL = WROWS / 8;               // ... in loads of 8 rows: 8 or 10
    constexpr int NLOAD = 8 + NWL;               // loads per step and wave
    constexpr int NREAD = 4 + NJ;                // fragment reads per sub-step
    constexpr int C_STAGE = BM * 576;            // bf16 epilogue: the C tile with 576-byte rows
    constexpr int LDS_BYTES = (OUT_BF16 && !PERSIST && C_STAGE > LDS_OPS) ? C_STAGE : LDS_OPS;
    static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
    __shared__ __attribute__((aligned(16))) uint8_t smem[LDS_BYTES];

    // work units (tile x K split) in XCD-aware order: unit u runs on XCD
    // u mod 8 and each XCD takes a contiguous range of units.  A persistent
    // grid takes units blockIdx.x + i * gridDim.x (gridDim.x a multiple of
    // 8, so they stay on the workgroup's XCD).
    const int T = PERSIST ? p.units : int(gridDim.x);
    const int tiles = T / p.split_k;
    int v = blockIdx.x;
    auto unit_of = [&](int u, int& um0, int& un0, int& us) {
        const int lb = (T % 8 == 0) ? (u % 8) * (T / 8) + u / 8 : u;
        us = lb / tiles;
        const int tile = lb - us * tiles;
        um0 = (tile % p.m_tiles) * BM;
        un0 = (tile / p.m_tiles) * BN;
    };
    if (v >= T) return;
    int m0, n0, split;
    unit_of(v, m0, n0, split);
    // this workgroup's 64-wide K steps: [kt0, kt0 + KT) (every unit of a
    // persistent grid: split 0, all of K)
    const int KT_all = p.K / BK;
    const int kt0 = int((int64_t(KT_all) * split) / p.split_k);
    const int KT = int((int64_t(KT_all) * (split + 1)) / p.split_k) - kt0;

    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int wm = wave >> 1, wn = wave & 1;

    // loads: wave w writes rows 64 w .. 64 w + 63 of the A tile and rows
    // WROWS w .. WROWS (w + 1) - 1 of the W tile, in instructions of 8 rows;
    // lane l: row + l / 8, LDS position l % 8
    const int lrow = lane >> 3, lpos = lane & 7;
    const uint8_t* Ab = reinterpret_cast<const uint8_t*>(p.A);
    uint32_t a_off[8], w_row[NWL];
    // Eq. 1's byte offset of column k inside a strip (row-major: 2 k).  For a
    // step start k0 (a multiple of 64) and a chunk start 8 c < 64 it splits,
    // w_koff(k0 + 8 c) = w_koff(k0) + w_koff(8 c): a memory tile at least 64
    // columns wide holds the whole step (the chunk only moves inside it), and
    // a narrower one divides 64 (the step starts on a memory-tile boundary).
    auto w_koff = [&](int k) -> uint32_t {
        if (TILE) return (uint32_t(k >> p.log2_bc) << p.log2_G) + uint32_t((k & p.bc_mask) << 1);
        return uint32_t(k) << 1;
    };
    // per-lane load offsets, fixed over the K loop: the A row and chunk; the
    // weight row and Eq. 1's offset of the chunk (the step's share is a
    // uniform base, so a load needs no vector arithmetic)
    auto set_a_rows = [&](int um0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = 64 * wave + 8 * i + lrow;
            const int c = lpos ^ ((r >> 1) & 7);
            const uint32_t m = uint32_t(min(um0 + r, p.M - 1));
            a_off[i] = (m * uint32_t(p.K) + uint32_t(c * 8)) * 2u;
        }
    };
    auto set_w_rows = [&](int un0) {
#pragma unroll
        for (int i = 0; i < NWL; ++i) {
            const int r = WROWS * wave + 8 * i + lrow;
            const int c = lpos ^ ((r >> 1) & 7);
            const uint32_t n = uint32_t(min(un0 + r, p.N - 1));
            if (TILE) w_row[i] = (n >> p.log2_br) * uint32_t(p.strip_bytes) + ((n & uint32_t(p.br_mask)) << (p.log2_bc + 1));
            else w_row[i] = n * uint32_t(p.K) * 2u;
            w_row[i] += w_koff(c * 8);
        }
    };
    set_a_rows(m0);
    set_w_rows(n0);
    // step s's A stage is s mod 2 and its weight stage (g + s) mod WST, g
    // the K steps of the workgroup's earlier units (a multiple of KT, even
    // in a persistent grid, so the A stages alternate across units too);
    // g_ld is the g of the weight loads in flight, which run ahead into the
    // next unit during a unit's last two steps
    int g_rd = 0, g_ld = 0;
    auto w_stage = [&](int g, int s) -> uint8_t* {
        return smem + 2 * HALF + (WST == 3 ? (g + s) % 3 : (s & 1)) * WHALF;
    };
    // load q (0 .. NLOAD - 1) of step s: q < 8 the A rows 8 q .. of this
    // wave's 64-row share, q >= 8 the W rows 8 (q - 8) .. of its WROWS-row share
    auto issue_one = [&](int s, int q) {
        const int k0 = (kt0 + s) * BK;
        if (q < 8) load_lds16(Ab + size_t(k0) * 2, a_off[q], smem + (s & 1) * HALF + wave * 8192 + q * 1024);
        else load_lds16(p.W + w_koff(k0), w_row[q - 8], w_stage(g_ld, s) + wave * (WROWS * 128) + (q - 8) * 1024);
    };
    // fragments: lane reads row lane % 32 of its 32-row tile at K chunk
    // 2 * sub-step + lane / 32; offsets of sub-step 0 (a sub-step adds 2
    // chunks, XORed into the position)
    int fa_row[4], fb_row[NJ];
    int fa_sw[4], fb_sw[NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int ra = wm * 128 + i * 32 + (lane & 31);
        fa_row[i] = ra * 128;
        fa_sw[i] = (ra >> 1) & 7;
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int rb = wn * (32 * NJ) + j * 32 + (lane & 31);
        fb_row[j] = rb * 128;
        fb_sw[j] = (rb >> 1) & 7;
    }
    const int khalf = lane >> 5;
    // fragment q (0 .. NREAD - 1) of sub-step ss of step s: q < NJ W tile q,
    // else A tile q - NJ (the next sub-step's first MFMAs take A tile 0 with
    // every W tile, so the W tiles are read first)
    auto fread_one = [&](int s, int ss, int q, bf16x8 (&fa)[4], bf16x8 (&fb)[NJ]) {
        const int c = 2 * ss + khalf;
        if (q < NJ) fb[q] = *reinterpret_cast<const bf16x8*>(w_stage(g_rd, s) + fb_row[q] + ((c ^ fb_sw[q]) << 4));
        else fa[q - NJ] = *reinterpret_cast<const bf16x8*>(smem + (s & 1) * HALF + fa_row[q - NJ] + ((c ^ fa_sw[q - NJ]) << 4));
    };
    f32x16 acc[4][NJ];
    auto zero_acc = [&]() {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    };
    zero_acc();
    // every wave meets the others; an LDS-only fence, so loads stay in flight
    auto lds_barrier = [&]() {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    };
    bf16x8 fa0[4], fb0[NJ], fa1[4], fb1[NJ];
    // one sub-step: 4 NJ MFMAs on (fa, fb); after MFMA q, fragment q / 2 of
    // sub-step rss of step rs into (ga, gb) when q is even (READ, the first
    // NREAD) and load q / 2 + lq0 of step ls when q is odd (LOAD: the eight
    // A loads from lq0 = 0 or the NWL W loads from lq0 = 8).  READ, LOAD and
    // lq0 are compile-time at every call, so the loop holds no branch
    // between its MFMAs.
    auto substep = [&](auto read_c, auto load_c, const bf16x8 (&fa)[4], const bf16x8 (&fb)[NJ], int rs, int rss,
                       bf16x8 (&ga)[4], bf16x8 (&gb)[NJ], int ls, int lq0) {
        constexpr bool READ = decltype(read_c)::value, LOAD = decltype(load_c)::value;
#pragma unroll
        for (int q = 0; q < 4 * NJ; ++q) {
            if (q % NJ < 4) {
                acc[q / NJ][q % NJ] =
                    __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[q / NJ], fb[q % NJ], acc[q / NJ][q % NJ], 0, 0, 0);
            } else {
                // the fifth column of tiles keeps its sums in VGPRs (the
                // first four fill the 256 AGPRs; the compiler does not split
                // the accumulators between the two files by itself).  Its
                // previous MFMA on the same sums is 4 NJ - 1 MFMAs back, far
                // beyond any dependency wait.
                asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0"
                             : "+v"(acc[q / NJ][4])
                             : "v"(fa[q / NJ]), "v"(fb[4]));
            }
            if ((q & 1) == 0) {
                if constexpr (READ) {
                    if ((q >> 1) < NREAD) fread_one(rs, rss, q >> 1, ga, gb);
                }
            } else {
                if constexpr (LOAD) {
                    if ((q >> 1) < (lq0 == 0 ? 8 : NWL)) issue_one(ls, lq0 + (q >> 1));
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    const std::true_type Y{};
    const std::false_type N{};

    // quad transpose of the bf16 C: a lane holds four consecutive rows of one
    // column per MFMA row group; the four lanes of a quad (four consecutive
    // columns) swap 2 x 2 blocks with lane ^ 1 and then with lane ^ 2, so each
    // lane ends with one row's four columns (8 bytes) -- row
    // 8 g + 4 (l / 32) + qrow of MFMA tile (i, j), columns 4 (l % 32 / 4) ..
    const int qd = lane & 3;
    const int qrow = ((qd & 1) << 1) | ((qd & 2) >> 1);
    const int cquad = (lane & 31) & ~3;
    // lane selects (odd lanes / lanes 2 and 3 of a quad): per-lane
    // conditions fixed for the kernel, so each pick below is one v_cndmask
    // on a lane mask and the unrolled code has no branches
    const bool odd = (qd & 1) != 0, hi2 = (qd & 2) != 0;
    auto pick = [](bool c, uint32_t a, uint32_t b) { return c ? a : b; };
    // v_perm_b32 byte selectors (bytes 0-3: the kept pair, 4-7: the received
    // one) that merge the first swap's halves into two rows of two columns:
    // an even lane's own column comes first, an odd lane's second
    const uint32_t sel_first = (qd & 1) ? 0x01000504u : 0x05040100u;
    const uint32_t sel_second = (qd & 1) ? 0x03020706u : 0x07060302u;
    // before the first quad_pack after the MFMAs: 24 wait states, more than
    // any MFMA-result read hazard needs (the reads below are inline assembly,
    // which the compiler's hazard check does not see into; the other tiles'
    // reads come hundreds of instructions after their MFMAs)
    auto mfma_settle = []() { asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"); };
    auto quad_pack = [&](int i, int j, int g) -> uint2 {
        // the four sums, read out of their AGPRs here (an asm the compiler
        // cannot move, so the reads of one MFMA tile happen where it is used);
        // the fifth column's sums are VGPRs already
        float f0, f1, f2, f3;
        if (j < 4) {
            asm volatile("v_accvgpr_read_b32 %0, %4\n\tv_accvgpr_read_b32 %1, %5\n\t"
                         "v_accvgpr_read_b32 %2, %6\n\tv_accvgpr_read_b32 %3, %7"
                         : "=v"(f0), "=v"(f1), "=v"(f2), "=v"(f3)
                         : "a"(acc[i][j][4 * g + 0]), "a"(acc[i][j][4 * g + 1]), "a"(acc[i][j][4 * g + 2]),
                           "a"(acc[i][j][4 * g + 3]));
        } else {
            f0 = acc[i][j][4 * g + 0];
            f1 = acc[i][j][4 * g + 1];
            f2 = acc[i][j][4 * g + 2];
            f3 = acc[i][j][4 * g + 3];
        }
        const uint32_t h01 = bf16x2_rne(f0, f1), h23 = bf16x2_rne(f2, f3);
        // swap with lane ^ 1: even lanes keep rows 0-1, odd lanes rows 2-3;
        // x_first / x_second: rows 0 and 1 (even) or 2 and 3 (odd) of the
        // two columns
        const uint32_t send1 = pick(odd, h01, h23), keep1 = pick(odd, h23, h01);
        const uint32_t recv1 = uint32_t(__builtin_amdgcn_mov_dpp(int(send1), 0xB1, 0xf, 0xf, true));
        const uint32_t x_first = __builtin_amdgcn_perm(recv1, keep1, sel_first);
        const uint32_t x_second = __builtin_amdgcn_perm(recv1, keep1, sel_second);
        // swap with lane ^ 2: one row's four columns per lane
        const uint32_t send2 = pick(hi2, x_first, x_second);
        const uint32_t recv2 = uint32_t(__builtin_amdgcn_mov_dpp(int(send2), 0x4E, 0xf, 0xf, true));
        uint2 r;
        r.x = pick(hi2, recv2, x_first);
        r.y = pick(hi2, x_second, recv2);
        return r;
    };

    // first step of the first unit in flight (three weight stages: step 1's
    // weight tile too)
#pragma unroll
    for (int q = 0; q < NLOAD; ++q) issue_one(0, q);
    if (WST == 3 && KT > 1)
#pragma unroll
        for (int q = 8; q < NLOAD; ++q) issue_one(1, q);
    for (;;) {
        // step 0 loaded and visible (three weight stages: step 1's weight
        // tile, issued after it, may stay in flight), its first fragments
        // read, the A half of step 1 in flight
        if (WST == 3 && KT > 1) TL_WAIT_VMCNT(NWL);
        else TL_WAIT_VMCNT(0);
        lds_barrier();
#pragma unroll
        for (int q = 0; q < NREAD; ++q) fread_one(0, 0, q, fa0, fb0);
        if (KT > 1)
#pragma unroll
            for (int q = 0; q < 8; ++q) issue_one(1, q);
        int s = 0;
        for (; s + 2 < KT; ++s) {            // steady state: every load present
            // the weight tile of step s + WST - 1 (two stages: the rest of
            // step s + 1; three: step s + 2, into the stage step s - 1 read)
            substep(Y, Y, fa0, fb0, s, 1, fa1, fb1, s + WST - 1, 8);
            substep(Y, N, fa1, fb1, s, 2, fa0, fb0, 0, 0);
            substep(Y, N, fa0, fb0, s, 3, fa1, fb1, 0, 0);
            // step s + 1 landed (three stages: step s + 2's weight tile,
            // issued last, stays in flight)
            if constexpr (WST == 3) TL_WAIT_VMCNT(NWL);
            else TL_WAIT_VMCNT(0);
            lds_barrier();
            // first fragments of step s + 1, first half of step s + 2's loads
            // (into the stage step s has finished reading)
            substep(Y, Y, fa1, fb1, s + 1, 0, fa0, fb0, s + 2, 0);
        }
        // PERSIST: the next unit (or, after the last one, this unit again:
        // loads nothing reads) and its tile origin
        int nv = v, nm0 = m0, nn0 = n0;
        if (s + 1 < KT) {                    // step KT - 2: no step KT to load
            if constexpr (PERSIST) {
                nv = v + int(gridDim.x);
                int ns;
                if (nv < T) unit_of(nv, nm0, nn0, ns);
            }
            if constexpr (PERSIST && WST == 3) {
                // the next unit's step 0 weight tile, into the stage step
                // KT - 3 read (g_ld: the next unit's g)
                set_w_rows(nn0);
                g_ld = g_rd + KT;
                substep(Y, Y, fa0, fb0, s, 1, fa1, fb1, 0, 8);
            } else if constexpr (WST == 3) {
                substep(Y, N, fa0, fb0, s, 1, fa1, fb1, 0, 0);   // step KT - 1's weight is in flight already
            } else {
                substep(Y, Y, fa0, fb0, s, 1, fa1, fb1, s + 1, 8);
            }
            substep(Y, N, fa1, fb1, s, 2, fa0, fb0, 0, 0);
            substep(Y, N, fa0, fb0, s, 3, fa1, fb1, 0, 0);
            if constexpr (PERSIST && WST == 3) TL_WAIT_VMCNT(NWL);
            else TL_WAIT_VMCNT(0);
            lds_barrier();
            if constexpr (PERSIST) {
                // the next unit's step 0 A tile goes into the stage step
                // KT - 2 has just finished reading (stage 0: KT is even),
                // and (two weight stages) its weight tile during the last
                // step, so they land under this tile's last MFMAs
                set_a_rows(nm0);
                if constexpr (WST == 2) set_w_rows(nn0);
                substep(Y, Y, fa1, fb1, s + 1, 0, fa0, fb0, 0, 0);
            } else {
                substep(Y, N, fa1, fb1, s + 1, 0, fa0, fb0, 0, 0);
            }
            ++s;
        }
        // the last step (PERSIST: the next unit's weight tile of step 1 with
        // three stages, of step 0 with two; a persistent unit has at least
        // two K steps, so step KT - 2 above ran)
        if constexpr (PERSIST) substep(Y, Y, fa0, fb0, s, 1, fa1, fb1, WST == 3 ? 1 : 0, 8);
        else substep(Y, N, fa0, fb0, s, 1, fa1, fb1, 0, 0);
        substep(Y, N, fa1, fb1, s, 2, fa0, fb0, 0, 0);
        substep(Y, N, fa0, fb0, s, 3, fa1, fb1, 0, 0);
        substep(N, N, fa1, fb1, 0, 0, fa0, fb0, 0, 0);

        if (p.fetch && t == 0) atomicAdd(p.fetch, (unsigned long long)KT * (unsigned long long)WHALF);

        if constexpr (PERSIST) {
            // whole tiles only (the launcher's condition; a uniform test, so
            // the stores need no per-lane bounds)
            mfma_settle();
            if (m0 + BM <= p.M && n0 + BN <= p.N) {
                uint16_t* Cw = static_cast<uint16_t*>(p.C) + int64_t(m0 + wm * 128 + 4 * (lane >> 5) + qrow) * p.ldc +
                               (n0 + wn * (32 * NJ) + cquad);
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < NJ; ++j) {
#pragma unroll
                        for (int g = 0; g < 4; ++g)
                            *reinterpret_cast<uint2*>(Cw + int64_t(i * 32 + 8 * g) * p.ldc + j * 32) = quad_pack(i, j, g);
                        // one MFMA tile at a time: keeps the accumulator reads
                        // from being hoisted into 256 VGPRs at once
                        __builtin_amdgcn_sched_barrier(0);
                    }
            }
            // every accumulator is read before it is cleared (else the two
            // sets of sums overlap and spill)
            __builtin_amdgcn_sched_barrier(0);
            zero_acc();
            if (nv >= T) {
                TL_WAIT_VMCNT(0);        // the reloads land before the workgroup's LDS is released
                break;
            }
            g_rd += KT;
            g_ld = g_rd;
            v = nv;
            m0 = nm0;
            n0 = nn0;
        } else {
            // D layout of a 32x32 MFMA tile: lane l, register v holds
            // row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32
            if constexpr (OUT_BF16) {
                // through LDS (the operand stages are free once every wave is
                // past its last MFMA): the 256 x 256 bf16 tile with 576-byte
                // rows, each lane writing its quad-transposed 8 bytes (the
                // stride puts a quad's four rows in four distinct 64-byte bank
                // ranges), then 16-byte stores of eight consecutive columns
                constexpr int CS = C_STAGE / BM;
                TL_WAIT_VMCNT(0);
                __syncthreads();
                mfma_settle();
                uint8_t* Cs = smem;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int r = wm * 128 + i * 32 + 8 * g + 4 * (lane >> 5) + qrow;
                            const int c = wn * 128 + j * 32 + cquad;
                            *reinterpret_cast<uint2*>(Cs + r * CS + c * 2) = quad_pack(i, j, g);
                            __builtin_amdgcn_sched_barrier(0);
                        }
                __syncthreads();
                uint16_t* C = static_cast<uint16_t*>(p.C);
                for (int e = t; e < 256 * 32; e += 256) {
                    const int r = e >> 5, c = (e & 31) * 8;
                    const int row = m0 + r, col = n0 + c;
                    if (row >= p.M) continue;
                    const u32x4 cv = *reinterpret_cast<const u32x4*>(Cs + r * CS + c * 2);
                    uint16_t* dst = C + int64_t(row) * p.ldc + col;
                    if (col + 8 <= p.N && ((reinterpret_cast<uintptr_t>(dst) & 15) == 0)) {
                        *reinterpret_cast<u32x4*>(dst) = cv;
                    } else {
#pragma unroll
                        for (int q = 0; q < 8; ++q)
                            if (col + q < p.N) dst[q] = uint16_t(cv[q >> 1] >> (16 * (q & 1)));
                    }
                }
            } else {
                // fp32 output, or this split's fp32 partial (row stride N)
                const bool full = m0 + BM <= p.M && n0 + BN <= p.N;
                const int row_base = m0 + wm * 128 + 4 * (lane >> 5);
                const int col_base = n0 + wn * 128 + (lane & 31);
                const bool part = p.split_k > 1;
                float* C = part ? p.ws + int64_t(split) * p.ws_stride : static_cast<float*>(p.C);
                const int64_t ldc = part ? int64_t(p.N) : p.ldc;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        float* Cij = C + int64_t(row_base + i * 32) * ldc + col_base + j * 32;
#pragma unroll
                        for (int e = 0; e < 16; ++e) {
                            const int dr = 8 * (e >> 2) + (e & 3);
                            if (full || (row_base + i * 32 + dr < p.M && col_base + j * 32 < p.N)) Cij[int64_t(dr) * ldc] = acc[i][j][e];
                        }
                    }
            }
            break;
        }
    }
}

// C[m][n] (row stride ldc) = sum over s = 0..S-1, in that order, of
// ws[s * stride + m * N + n]: the K-split partials of prefill_w4_kernel,
// four consecutive columns per thread (N % 4 == 0).  No float atomics, so
// results are bitwise reproducible.
template <bool OUT_BF16>
__global__ __launch_bounds__(256) void prefill_splitk_reduce(const float* ws, int S, int64_t stride, int M, int N,
                                                             void* C, int64_t ldc) {
    typedef float f32x4p __attribute__((ext_vector_type(4)));
    const int64_t e = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 4;
    if (e >= int64_t(M) * N) return;
    const int64_t m = e / N, n = e - m * N;
    f32x4p acc = *reinterpret_cast<const f32x4p*>(ws + e);
    for (int s = 1; s < S; ++s) acc += *reinterpret_cast<const f32x4p*>(ws + int64_t(s) * stride + e);
    if (OUT_BF16) {
        uint16_t* c = static_cast<uint16_t*>(C) + m * ldc + n;
#pragma unroll
        for (int q = 0; q < 4; ++q) c[q] = f32_to_bf16_rne(acc[q]);
    } else {
        float* c = static_cast<float*>(C) + m * ldc + n;
#pragma unroll
        for (int q = 0; q < 4; ++q) c[q] = acc[q];
    }
}

// workgroups of a persistent prefill grid with more tiles than CUs: one per
// CU (a multiple of 8, so each keeps to its XCD's range of tiles)
constexpr int kPersistGrid = 256;

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
                        hipStream_t stream, int split = 1) {
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
    // 256x320: the four-wave kernel with five MFMA tiles per wave along N
    // (persistent, bf16 out, whole tiles -- the planner's conditions)
    if (tile_m == 256 && tile_n == 320) {
        if (!(q.persist && p.out_bf16 && q.M % 256 == 0 && n_cols % 320 == 0 && q.K % 128 == 0))
            return hipErrorInvalidValue;
        p.units = grid;
        const int pgrid = grid < kPersistGrid ? grid : kPersistGrid;
        if (tile)
            hipLaunchKernelGGL((prefill_w4_kernel<true, true, true, 5>), dim3(pgrid), dim3(256), 0, stream, p);
        else
            hipLaunchKernelGGL((prefill_w4_kernel<false, true, true, 5>), dim3(pgrid), dim3(256), 0, stream, p);
        return hipGetLastError();
    }
    // 256x256: 8 waves (2 per SIMD) of 128x64; smaller tiles: 4 waves in 2 x 2
    if (tile_m == 256 && tile_n == 256) {
        if (q.K % 64 == 0 && p.log2_fetch == 0) {
            // whole tiles, bf16 out: at most one workgroup per CU walks them
            if (q.persist && p.out_bf16 && q.M % 256 == 0 && n_cols % 256 == 0 && q.K % 128 == 0) {
                p.units = grid;
                const int pgrid = grid < kPersistGrid ? grid : kPersistGrid;
                if (tile)
                    hipLaunchKernelGGL((prefill_w4_kernel<true, true, true>), dim3(pgrid), dim3(256), 0, stream, p);
                else
                    hipLaunchKernelGGL((prefill_w4_kernel<false, true, true>), dim3(pgrid), dim3(256), 0, stream, p);
                return hipGetLastError();
            }
            if (tile) {
                if (p.out_bf16) hipLaunchKernelGGL((prefill_w4_kernel<true, true>), dim3(grid), dim3(256), 0, stream, p);
                else hipLaunchKernelGGL((prefill_w4_kernel<true, false>), dim3(grid), dim3(256), 0, stream, p);
            } else {
                if (p.out_bf16) hipLaunchKernelGGL((prefill_w4_kernel<false, true>), dim3(grid), dim3(256), 0, stream, p);
                else hipLaunchKernelGGL((prefill_w4_kernel<false, false>), dim3(grid), dim3(256), 0, stream, p);
            }
            return hipGetLastError();
        }
        return launch_t<256, 256, 2, 4>(p, grid, tile, stream);
    }
    if (tile_m == 256) return launch_t<256, 128, 2, 2>(p, grid, tile, stream);
    // 128 x 128 tiles, optionally with K split 'split' ways (fp32 partials
    // in ws, M * n_cols floats per split)
    p.split_k = split;
    p.ws = q.ws;
    p.ws_stride = q.M * n_cols;
    return launch_t<128, 128, 2, 2>(p, grid * split, tile, stream);
}

}  // namespace

hipError_t launch_prefill(const PrefillLaunch& q, hipStream_t stream) {
    // (n_main == 0: every column takes the K-split launch below)
    hipError_t e = q.n_main > 0 ? launch_range(q, 0, q.n_main, q.tile_m, q.tile_n, stream) : hipSuccess;
    if (e != hipSuccess || q.n_main == q.N) return e;
    if (q.split_rest <= 1) return launch_range(q, q.n_main, q.N - q.n_main, 128, 128, stream);
    if (q.n_main == 0 && q.tile_m == 128) {
        // every column: 128 x 128 tiles with K split split_rest ways, then the
        // fixed-order reduce
        e = launch_range(q, 0, q.N, 128, 128, stream, q.split_rest);
        if (e != hipSuccess) return e;
        const int rgrid = int((q.M * q.N / 4 + 255) / 256);
        if (q.out_bf16)
            hipLaunchKernelGGL((prefill_splitk_reduce<true>), dim3(rgrid), dim3(256), 0, stream, q.ws, q.split_rest,
                               q.M * q.N, int(q.M), int(q.N), q.C, int64_t(q.N));
        else
            hipLaunchKernelGGL((prefill_splitk_reduce<false>), dim3(rgrid), dim3(256), 0, stream, q.ws, q.split_rest,
                               q.M * q.N, int(q.M), int(q.N), q.C, int64_t(q.N));
        return hipGetLastError();
    }
    // the remaining columns: 256 x 256 tiles of prefill_w4_kernel, K split
    // split_rest ways (fp32 partials in ws), then the fixed-order reduce
    const bool tile = q.L.kind == TL_LAYOUT_TILE;
    const int64_t kp = tile ? padded_cols(q.L, q.K) : q.K;
    const int64_t n_cols = q.N - q.n_main;
    PrefillParams p;
    p.A = q.A;
    p.W = q.W + q.n_main * kp * 2;
    p.C = nullptr;
    p.fetch = q.fetch;
    p.M = int(q.M);
    p.N = int(n_cols);
    p.K = int(q.K);
    p.ldc = q.N;
    p.m_tiles = int((q.M + 255) / 256);
    p.strip_bytes = tile ? q.L.br * kp * 2 : 0;
    p.log2_br = tile ? q.L.log2_br : 0;
    p.log2_bc = tile ? q.L.log2_bc : 0;
    p.log2_G = tile ? q.L.log2_G : 0;
    p.br_mask = tile ? int(q.L.br - 1) : 0;
    p.bc_mask = tile ? int(q.L.bc - 1) : 0;
    p.out_bf16 = false;
    p.log2_fetch = 0;
    p.w_bytes = n_cols * kp * 2;
    p.split_k = q.split_rest;
    p.ws = q.ws;
    p.ws_stride = q.M * n_cols;
    const int grid = int(p.m_tiles * ((n_cols + 255) / 256) * q.split_rest);
    if (tile) hipLaunchKernelGGL((prefill_w4_kernel<true, false>), dim3(grid), dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((prefill_w4_kernel<false, false>), dim3(grid), dim3(256), 0, stream, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    uint8_t* c0 = static_cast<uint8_t*>(q.C) + q.n_main * (q.out_bf16 ? 2 : 4);
    const int rgrid = int((q.M * n_cols / 4 + 255) / 256);
    if (q.out_bf16)
        hipLaunchKernelGGL((prefill_splitk_reduce<true>), dim3(rgrid), dim3(256), 0, stream, q.ws, q.split_rest,
                           p.ws_stride, p.M, p.N, (void*)c0, int64_t(q.N));
    else
        hipLaunchKernelGGL((prefill_splitk_reduce<false>), dim3(rgrid), dim3(256), 0, stream, q.ws, q.split_rest,
                           p.ws_stride, p.M, p.N, (void*)c0, int64_t(q.N));
    return hipGetLastError();
}

}  // namespace tl
