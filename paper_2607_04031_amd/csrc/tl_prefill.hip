// Prefill GEMM (large M): C[M][N] = A[M][K] * W^T with bf16 MFMA 32x32x16 and
// fp32 accumulation; W tile-major (or row-major [N][K]).  MFMA-bound at large
// batch (TileLens Section 6.2: the dense FFN becomes compute-bound as the batch
// grows).
//
// Workgroup tile BM x 128 x 64 (BM = 128 or 256), 4 wavefronts in a 2 x 2
// grid, each owning a (BM/2) x 64 block of C as (BM/64) x 2 MFMA 32x32 tiles.
// Per 64-wide K step the workgroup stages its A tile and its weight tile in
// LDS; the weight tile of a (64, 32) BF16 memory tile layout is exactly four
// whole 4 KB memory tiles, so each wavefront load instruction reads 1 KB of
// one contiguous memory tile.  Per-lane weight addresses are Eq. 2 with shifts
// and masks (Section 3.2).  The next K step's global loads are issued before
// the current step's MFMAs (register double buffering; LDS is double buffered
// so one barrier per step suffices).  LDS rows are 128 B; 16-byte chunks are
// XOR-swizzled by (row mod 8) so the MFMA operand reads of 8 consecutive rows
// hit 8 different bank groups.
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
    int m_tiles;
    int64_t strip_bytes;
    int log2_br, log2_bc, log2_G;
    int br_mask, bc_mask;
};

__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

__device__ inline int swz(int row, int chunk) { return row * 128 + ((chunk ^ (row & 7)) << 4); }

template <int BM, bool TILE, bool OUT_BF16, bool COUNT>
__global__ __launch_bounds__(256) void prefill_kernel(PrefillParams p) {
    constexpr int BN = 128, BK = 64;
    constexpr int A_BYTES = BM * BK * 2, W_BYTES = BN * BK * 2;
    constexpr int A_CH = BM * 8 / 256;   // 16-byte chunks per thread per K step
    constexpr int W_CH = BN * 8 / 256;
    constexpr int FM = BM / 64;          // 32-row MFMA tiles per wave
    constexpr int FN = 2;                // 32-col MFMA tiles per wave
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * (A_BYTES + W_BYTES)];

    // XCD-aware order: workgroup b runs on XCD (b mod 8); give each XCD a
    // contiguous range of tiles so neighbouring tiles share that XCD's L2.
    const int T = gridDim.x, b = blockIdx.x;
    const int lb = (T % 8 == 0) ? (b % 8) * (T / 8) + b / 8 : b;
    const int tm = lb % p.m_tiles, tn = lb / p.m_tiles;
    const int m0 = tm * BM, n0 = tn * BN;

    const int t = threadIdx.x;
    const uint16_t* a_src[A_CH];
    int a_lds[A_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
        const int q = t + 256 * i, row = q >> 3, c = q & 7;
        const int m = min(m0 + row, p.M - 1);
        a_src[i] = p.A + int64_t(m) * p.K + c * 8;
        a_lds[i] = swz(row, c);
    }
    const uint8_t* w_src[W_CH];
    int w_k[W_CH], w_lds[W_CH];
#pragma unroll
    for (int i = 0; i < W_CH; ++i) {
        const int q = t + 256 * i, row = q >> 3, c = q & 7;
        const int n = min(n0 + row, p.N - 1);
        int64_t off;
        if (TILE) off = int64_t(n >> p.log2_br) * p.strip_bytes + (int64_t(n & p.br_mask) << (p.log2_bc + 1));
        else off = int64_t(n) * p.K * 2;
        w_src[i] = p.W + off;
        w_k[i] = c * 8;
        w_lds[i] = swz(row, c);
    }

    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // prefetch registers for the next K step (kept in VGPRs: plain scalars
    // indexed only by unrolled constants)
    u32x4 ra[A_CH], rw[W_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) ra[i] = *reinterpret_cast<const u32x4*>(a_src[i]);
#pragma unroll
    for (int i = 0; i < W_CH; ++i) {
        const int k = w_k[i];
        int64_t ko;
        if (TILE) ko = (int64_t(k >> p.log2_bc) << p.log2_G) + int64_t((k & p.bc_mask) << 1);
        else ko = int64_t(k) << 1;
        rw[i] = *reinterpret_cast<const u32x4*>(w_src[i] + ko);
    }
#pragma unroll
    for (int i = 0; i < A_CH; ++i) *reinterpret_cast<u32x4*>(smem + a_lds[i]) = ra[i];
#pragma unroll
    for (int i = 0; i < W_CH; ++i) *reinterpret_cast<u32x4*>(smem + A_BYTES + w_lds[i]) = rw[i];
    __syncthreads();

    const int KT = p.K / BK;
    for (int kt = 0; kt < KT; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < KT;
        if (more) {
            const int k0 = (kt + 1) * BK;
#pragma unroll
            for (int i = 0; i < A_CH; ++i) ra[i] = *reinterpret_cast<const u32x4*>(a_src[i] + k0);
#pragma unroll
            for (int i = 0; i < W_CH; ++i) {
                const int k = k0 + w_k[i];
                int64_t ko;
                if (TILE) ko = (int64_t(k >> p.log2_bc) << p.log2_G) + int64_t((k & p.bc_mask) << 1);
                else ko = int64_t(k) << 1;
                rw[i] = *reinterpret_cast<const u32x4*>(w_src[i] + ko);
            }
        }
        const uint8_t* As = smem + buf * (A_BYTES + W_BYTES);
        const uint8_t* Ws = As + A_BYTES;
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            const int chunk = s * 2 + (lane >> 5);
            bf16x8 af[FM], bfr[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int row = wm * (BM / 2) + i * 32 + (lane & 31);
                af[i] = *reinterpret_cast<const bf16x8*>(As + swz(row, chunk));
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int row = wn * 64 + j * 32 + (lane & 31);
                bfr[j] = *reinterpret_cast<const bf16x8*>(Ws + swz(row, chunk));
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (more) {
            uint8_t* An = smem + (buf ^ 1) * (A_BYTES + W_BYTES);
#pragma unroll
            for (int i = 0; i < A_CH; ++i) *reinterpret_cast<u32x4*>(An + a_lds[i]) = ra[i];
#pragma unroll
            for (int i = 0; i < W_CH; ++i) *reinterpret_cast<u32x4*>(An + A_BYTES + w_lds[i]) = rw[i];
        }
        __syncthreads();
    }

    if (COUNT && t == 0) atomicAdd(p.fetch, (unsigned long long)KT * (unsigned long long)W_BYTES);

    // D layout of a 32x32 MFMA tile: lane l, register v holds
    // row 8*(v/4) + 4*(l/32) + v%4, column l%32.
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = m0 + wm * (BM / 2) + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                const int col = n0 + wn * 64 + j * 32 + (lane & 31);
                if (row < p.M && col < p.N) {
                    const int64_t idx = int64_t(row) * p.N + col;
                    if (OUT_BF16) static_cast<uint16_t*>(p.C)[idx] = f32_to_bf16_rne(acc[i][j][v]);
                    else static_cast<float*>(p.C)[idx] = acc[i][j][v];
                }
            }
}

template <int BM, bool TILE>
hipError_t launch_t(const PrefillParams& p, int grid, bool out_bf16, bool count, hipStream_t s) {
    if (out_bf16) {
        if (count) hipLaunchKernelGGL((prefill_kernel<BM, TILE, true, true>), dim3(grid), dim3(256), 0, s, p);
        else hipLaunchKernelGGL((prefill_kernel<BM, TILE, true, false>), dim3(grid), dim3(256), 0, s, p);
    } else {
        if (count) hipLaunchKernelGGL((prefill_kernel<BM, TILE, false, true>), dim3(grid), dim3(256), 0, s, p);
        else hipLaunchKernelGGL((prefill_kernel<BM, TILE, false, false>), dim3(grid), dim3(256), 0, s, p);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_prefill(const PrefillLaunch& q, hipStream_t stream) {
    PrefillParams p;
    p.A = q.A;
    p.W = q.W;
    p.C = q.C;
    p.fetch = q.fetch;
    p.M = int(q.M);
    p.N = int(q.N);
    p.K = int(q.K);
    p.m_tiles = int((q.M + q.tile_m - 1) / q.tile_m);
    const bool tile = q.L.kind == TL_LAYOUT_TILE;
    p.strip_bytes = tile ? q.L.br * q.K * 2 : 0;
    p.log2_br = tile ? q.L.log2_br : 0;
    p.log2_bc = tile ? q.L.log2_bc : 0;
    p.log2_G = tile ? q.L.log2_G : 0;
    p.br_mask = tile ? int(q.L.br - 1) : 0;
    p.bc_mask = tile ? int(q.L.bc - 1) : 0;
    const int64_t n_tiles = (q.N + 127) / 128;
    const int grid = int(p.m_tiles * n_tiles);
    if (q.tile_m == 256) return tile ? launch_t<256, true>(p, grid, q.out_bf16, q.fetch, stream)
                                     : launch_t<256, false>(p, grid, q.out_bf16, q.fetch, stream);
    return tile ? launch_t<128, true>(p, grid, q.out_bf16, q.fetch, stream)
                : launch_t<128, false>(p, grid, q.out_bf16, q.fetch, stream);
}

}  // namespace tl
