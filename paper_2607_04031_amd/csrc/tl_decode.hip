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
//   lane l supplies 8 consecutive k (a 16-byte load) at k-slot group l / 16.
//   The per-lane weight address is Eq. 2 evaluated with shifts and masks
//   (Section 3.2, Eq. 1): strip = n >> log2(br), row-in-tile = n & (br - 1),
//   memory tile along K = k >> log2(bc), column-in-tile = k & (bc - 1).
//   With bc >= 8 each 16-byte load stays inside one memory-tile row.
// Reduction
//   waves -> LDS -> fixed-order sum; K-splits -> fp32 partials in a workspace;
//   the last workgroup of a tile to finish (atomic ticket) sums the partials in
//   split order and writes C, then re-arms the ticket.  No float atomics, so
//   results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include "tl_internal.h"

namespace tl {
namespace {

typedef short bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

struct DecodeParams {
    const uint16_t* A;
    const uint8_t* W;
    void* C;
    float* ws;
    int* counters;
    unsigned long long* fetch;
    int M, N, K;
    int split_k;
    int steps_per_unit;      // 64-element steps per split unit
    int units;               // K / k_unit
    int64_t strip_bytes;     // br * K * 2 (TILE) -- bytes per strip of br rows
    int log2_br, log2_bc, log2_G;
    int bc_mask;
};

__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu))  // NaN stays NaN
        return uint16_t((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

template <bool OUT_BF16>
__device__ inline void store_out(void* C, int64_t idx, float v) {
    if (OUT_BF16) static_cast<uint16_t*>(C)[idx] = f32_to_bf16_rne(v);
    else static_cast<float*>(C)[idx] = v;
}

// Byte offset of the 8-element chunk starting at (row base, k) of the weight.
template <bool TILE>
__device__ inline int64_t w_koff(const DecodeParams& p, int k) {
    if (TILE) return (int64_t(k >> p.log2_bc) << p.log2_G) + int64_t((k & p.bc_mask) << 1);
    return int64_t(k) << 1;
}

template <int MT, int NS, int U, bool TILE, bool OUT_BF16, bool COUNT>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeParams p) {
    constexpr int TN = 16 * NS;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int tile = blockIdx.x / p.split_k;
    const int split = blockIdx.x - tile * p.split_k;

    // K range of this split in 64-element steps
    const int u0 = int((int64_t(p.units) * split) / p.split_k);
    const int u1 = int((int64_t(p.units) * (split + 1)) / p.split_k);
    const int st0 = u0 * p.steps_per_unit, st1 = u1 * p.steps_per_unit;

    const int n_base = tile * TN;
    const int kq = (lane >> 4) * 8;     // this lane's k-slot group inside a 32-K half

    const uint8_t* wrow[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const int n = n_base + j * 16 + (lane & 15);
        int64_t off;
        if (TILE) off = int64_t(n >> p.log2_br) * p.strip_bytes + (int64_t(n & ((1 << p.log2_br) - 1)) << (p.log2_bc + 1));
        else off = int64_t(n) * p.K * 2;
        wrow[j] = p.W + off;
    }
    const uint16_t* arow[MT];
    bool aok[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + (lane & 15);
        aok[mt] = m < p.M;
        arow[mt] = p.A + int64_t(aok[mt] ? m : 0) * p.K;
    }

    f32x4 acc[MT][NS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NS; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const bf16x8 zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
    // steps of this wave: st0 + wave + 4 * i
    const int nsteps = st1 - st0 - wave > 0 ? (st1 - st0 - wave + kWaves - 1) / kWaves : 0;
    int st = st0 + wave;
    int i = 0;
    for (; i + U <= nsteps; i += U) {
        bf16x8 w[U][2][NS];
        bf16x8 a[U][2][MT];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = (st + u * kWaves) * 64;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int kk = k + h * 32 + kq;
                const int64_t ko = w_koff<TILE>(p, kk);
#pragma unroll
                for (int j = 0; j < NS; ++j)
                    w[u][h][j] = *reinterpret_cast<const bf16x8*>(wrow[j] + ko);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    a[u][h][mt] = aok[mt] ? *reinterpret_cast<const bf16x8*>(arow[mt] + kk) : zero8;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int j = 0; j < NS; ++j)
                        acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][h][mt], w[u][h][j],
                                                                             acc[mt][j], 0, 0, 0);
        st += U * kWaves;
    }
    for (; i < nsteps; ++i) {
        const int k = st * 64;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int kk = k + h * 32 + kq;
            const int64_t ko = w_koff<TILE>(p, kk);
            bf16x8 w[NS], a[MT];
#pragma unroll
            for (int j = 0; j < NS; ++j) w[j] = *reinterpret_cast<const bf16x8*>(wrow[j] + ko);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                a[mt] = aok[mt] ? *reinterpret_cast<const bf16x8*>(arow[mt] + kk) : zero8;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int j = 0; j < NS; ++j)
                    acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], w[j], acc[mt][j], 0, 0, 0);
        }
        st += kWaves;
    }

    if (COUNT && lane == 0 && nsteps > 0) {
        // each step: 2 K-halves x NS loads of 64 lanes x 16 B
        atomicAdd(p.fetch, (unsigned long long)nsteps * 2ull * NS * 1024ull);
    }

    // ---- reduce the four waves in a fixed order ----
    __shared__ f32x4 red[kWaves][MT][NS][64];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NS; ++j) red[wave][mt][j][lane] = acc[mt][j];
    __syncthreads();

    constexpr int kEntries = MT * NS * 64;   // f32x4 entries per wave
    if (p.split_k == 1) {
        for (int e = threadIdx.x; e < kEntries; e += kThreads) {
            const int mt = e / (NS * 64);
            const int j = (e / 64) % NS;
            const int l = e % 64;
            const f32x4 v = red[0][mt][j][l] + red[1][mt][j][l] + red[2][mt][j][l] + red[3][mt][j][l];
            const int n = n_base + j * 16 + (l & 15);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = mt * 16 + (l >> 4) * 4 + r;
                if (m < p.M) store_out<OUT_BF16>(p.C, int64_t(m) * p.N + n, v[r]);
            }
        }
        return;
    }

    // ---- K-split: publish this split's partial tile, last arrival reduces ----
    float* part = p.ws + int64_t(split) * p.M * p.N;
    for (int e = threadIdx.x; e < kEntries; e += kThreads) {
        const int mt = e / (NS * 64);
        const int j = (e / 64) % NS;
        const int l = e % 64;
        const f32x4 v = red[0][mt][j][l] + red[1][mt][j][l] + red[2][mt][j][l] + red[3][mt][j][l];
        const int n = n_base + j * 16 + (l & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + (l >> 4) * 4 + r;
            if (m < p.M) part[int64_t(m) * p.N + n] = v[r];
        }
    }
    __threadfence();            // release the partial to every XCD
    __syncthreads();
    __shared__ int s_last;
    if (threadIdx.x == 0) s_last = atomicAdd(&p.counters[tile], 1) == p.split_k - 1;
    __syncthreads();
    if (!s_last) return;
    __threadfence();            // acquire the other splits' partials
    const int outs = p.M * TN;
    for (int e = threadIdx.x; e < outs; e += kThreads) {
        const int m = e / TN;
        const int n = n_base + (e - m * TN);
        const int64_t idx = int64_t(m) * p.N + n;
        float sum = 0.f;
        for (int s = 0; s < p.split_k; ++s) sum += __builtin_nontemporal_load(p.ws + int64_t(s) * p.M * p.N + idx);
        store_out<OUT_BF16>(p.C, idx, sum);
    }
    if (threadIdx.x == 0) atomicExch(&p.counters[tile], 0);   // re-arm for the next call
}

template <int MT, int NS, bool TILE, bool OUT_BF16, bool COUNT>
hipError_t launch_t(const DecodeParams& p, int grid, hipStream_t stream) {
    constexpr int U = MT >= 4 ? 2 : 4;
    hipLaunchKernelGGL((decode_kernel<MT, NS, U, TILE, OUT_BF16, COUNT>), dim3(grid), dim3(kThreads), 0,
                       stream, p);
    return hipGetLastError();
}

template <int MT, int NS, bool TILE>
hipError_t launch_b(const DecodeParams& p, int grid, bool out_bf16, bool count, hipStream_t stream) {
    if (out_bf16) return count ? launch_t<MT, NS, TILE, true, true>(p, grid, stream)
                               : launch_t<MT, NS, TILE, true, false>(p, grid, stream);
    return count ? launch_t<MT, NS, TILE, false, true>(p, grid, stream)
                 : launch_t<MT, NS, TILE, false, false>(p, grid, stream);
}

template <int MT>
hipError_t launch_m(const DecodeParams& p, int grid, int ns, bool tile, bool out_bf16, bool count,
                    hipStream_t stream) {
    if (ns == 2) return tile ? launch_b<MT, 2, true>(p, grid, out_bf16, count, stream)
                             : launch_b<MT, 2, false>(p, grid, out_bf16, count, stream);
    return tile ? launch_b<MT, 4, true>(p, grid, out_bf16, count, stream)
                : launch_b<MT, 4, false>(p, grid, out_bf16, count, stream);
}

}  // namespace

hipError_t launch_decode(const DecodeLaunch& d, hipStream_t stream) {
    DecodeParams p;
    p.A = d.A;
    p.W = d.W;
    p.C = d.C;
    p.ws = d.ws;
    p.counters = d.counters;
    p.fetch = d.fetch;
    p.M = int(d.M);
    p.N = int(d.N);
    p.K = int(d.K);
    p.split_k = d.split_k;
    p.steps_per_unit = int(d.k_unit / 64);
    p.units = int(d.K / d.k_unit);
    const bool tile = d.L.kind == TL_LAYOUT_TILE;
    p.strip_bytes = tile ? d.L.br * d.K * 2 : 0;
    p.log2_br = tile ? d.L.log2_br : 0;
    p.log2_bc = tile ? d.L.log2_bc : 0;
    p.log2_G = tile ? d.L.log2_G : 0;
    p.bc_mask = tile ? int(d.L.bc - 1) : 0;
    const int grid = int(d.N / d.tile_n) * d.split_k;
    const int ns = d.tile_n / 16;
    switch (d.m_tiles16) {
        case 1: return launch_m<1>(p, grid, ns, tile, d.out_bf16, d.fetch != nullptr, stream);
        case 2: return launch_m<2>(p, grid, ns, tile, d.out_bf16, d.fetch != nullptr, stream);
        default: return launch_m<4>(p, grid, ns, tile, d.out_bf16, d.fetch != nullptr, stream);
    }
}

}  // namespace tl
