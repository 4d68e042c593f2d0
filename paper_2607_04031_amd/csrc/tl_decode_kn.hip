// Decode GEMM, M <= 64, over a weight stored [K][N] row-major (N contiguous:
// the paper's "row-major" layout, Section 2.4): C[M][N] = A[M][K] * W^T.
//
// The MFMA operands need eight consecutive k per lane, while a [K][N] weight
// keeps consecutive n together, so every K step goes through LDS once:
//   workgroup = 64 output columns (n) x one K split; its waves interleave
//   along K in 64-row steps.  Per step a wave loads the 64 k-rows x 128 B of
//   its columns with whole-line loads (instruction i: rows 8 i .. 8 i + 7,
//   lane l reads 16 bytes of row 8 i + l / 8), writes them to its own LDS
//   region and reads them back transposed with ds_read_b64_tr_b16 (gfx950):
//   in each 16-lane group, lanes 4r .. 4r + 3 address the 32 bytes of k-row r,
//   and lane i receives column i of the four rows -- two such reads give the
//   eight k of one column that a bf16 MFMA 16x16x32 operand holds.  The
//   region's 16-byte chunks are XOR-swizzled per row so both the row writes
//   and the transposed reads are free of bank conflicts.  A wave only reads
//   what it wrote itself (LDS instructions of a wave complete in order), so
//   the loop needs no barrier.
// Block-granular fetch (BLOCK): before the operand loads of a step, every
// G-byte block (aligned to the weight's base) that holds one of the step's
// 64 row segments is loaded whole into a live sink and counted -- rows in
// address order, so a block shared by consecutive rows is fetched once per
// step -- which pays a large-granularity memory's amplification (Section 2.5)
// as real HBM traffic; the operand loads then hit in cache.
// Waves of a workgroup are summed in LDS in a fixed order; K splits write
// fp32 partials that the split-K reduce kernel sums in split order.
#include <hip/hip_runtime.h>

#include "tl_decode_common.h"

namespace tl {
namespace {

typedef short bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kStageBytes = 64 * 128;   // one wave's K step: 64 k-rows x 64 columns of bf16

// Swizzle of k-row r's 16-byte chunks: chunk pair j (columns 16 j .. 16 j + 15)
// goes to pair j ^ f(r), f(r) = bit 1 of r | bit 3 of r << 1.  A transposed
// read serves 32 lanes = eight rows {b, b+1, b+2, b+3, b+8, .., b+11}
// (b = 4 p + 32 h); rows of one parity share banks, and f separates the four
// of each parity.
__device__ inline int kn_swz(int r, int chunk) { return r * 128 + ((chunk ^ (((r >> 1) & 1) << 1) ^ (((r >> 3) & 1) << 2)) << 4); }

template <int MT, int WAVES, bool BLOCK>
__global__ __launch_bounds__(64 * WAVES) void decode_kn_kernel(DecodeParams p) {
    constexpr int kThreads = 64 * WAVES;
    constexpr int kRedBytes = WAVES * MT * 4 * 64 * 16;
    constexpr int kLds = (WAVES * kStageBytes > kRedBytes) ? WAVES * kStageBytes : kRedBytes;
    static_assert(kLds <= 64 * 1024, "LDS budget");
    __shared__ __attribute__((aligned(16))) uint8_t smem[kLds];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int tile = blockIdx.x / p.split_k;
    const int split = blockIdx.x - tile * p.split_k;
    const int u0 = int((int64_t(p.units) * split) / p.split_k);
    const int u1 = int((int64_t(p.units) * (split + 1)) / p.split_k);
    const int st0 = u0 * p.steps_per_unit;
    const int st1 = min(u1 * p.steps_per_unit, p.ksteps);
    const int n0 = tile * 64;

    // weight loads: lane (lr, lc) reads 16 bytes at column min(n0 + 8 lc, N - 8)
    // of rows k0 + 8 i + lr (N % 8 == 0; columns past N are never stored)
    const int lr = lane >> 3, lc = lane & 7;
    const int64_t row_bytes = int64_t(p.N) * 2;
    const uint32_t wlane = uint32_t(min(n0 + 8 * lc, p.N - 8)) * 2u + uint32_t(lr) * uint32_t(row_bytes);
    uint8_t* stage = smem + wave * kStageBytes;
    int wst[8];                      // LDS offset of this lane's chunk of rows 8 i + lr
#pragma unroll
    for (int i = 0; i < 8; ++i) wst[i] = kn_swz(8 * i + lr, lc);
    // transposed reads: group g, lane i16 = lane & 15 addresses k-row
    // 32 h + 8 g + 4 pt + i16 / 4, columns 16 j + 4 (i16 & 3) .. + 3
    const int g = lane >> 4, i16 = lane & 15;
    int rtr[2][2][4];                // [h][pt][j]
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int pt = 0; pt < 2; ++pt)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 32 * h + 8 * g + 4 * pt + (i16 >> 2);
                const int c = 2 * j + ((i16 & 3) >> 1);
                rtr[h][pt][j] = kn_swz(r, c) + 8 * (i16 & 1);
            }
    // activations: lane (g, q = i16) reads A[16 mt + q][k0 + 32 h + 8 g .. + 7]
    const uint8_t* Ab = reinterpret_cast<const uint8_t*>(p.A);
    uint32_t aoff[MT];
    bool aok[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + i16;
        aok[mt] = m < p.M;
        aoff[mt] = uint32_t((aok[mt] ? m : 0) * p.K + 8 * g) * 2u;
    }

    f32x4 acc[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16x8 zero8 = {0, 0, 0, 0, 0, 0, 0, 0};

    i32x4 sink = {0, 0, 0, 0};
    uint64_t fetched = 0;
    auto fetch_blocks = [&](int k0) {
        if constexpr (BLOCK) {
            const int64_t Gb = int64_t(1) << p.log2_fetch;
            int64_t prev = -1;
            for (int r = 0; r < 64; ++r) {
                const int64_t b = ((int64_t(k0 + r) * p.N + n0) * 2) >> p.log2_fetch;
                if (b == prev) continue;
                prev = b;
                const uint8_t* base = p.W + (b << p.log2_fetch);
                for (int64_t c = int64_t(lane) * 16; c < Gb; c += 1024)
                    if ((b << p.log2_fetch) + c < p.w_bytes) sink ^= __builtin_bit_cast(i32x4, load_stream(base + c));
                fetched += uint64_t(Gb);
            }
        }
    };

    const int nsteps = st1 - st0 - wave > 0 ? (st1 - st0 - wave + WAVES - 1) / WAVES : 0;
    int st = st0 + wave;
    // two steps in flight: the loads of the next step are issued before this
    // step is staged and computed (two register sets, used alternately, so
    // every register index is a compile-time constant)
    auto gload = [&](int s, bf16x8 (&xw)[8], bf16x8 (&xa)[MT][2]) {
        const int k0 = s * 64;
        fetch_blocks(k0);
        const uint8_t* wk = p.W + int64_t(k0) * row_bytes;
#pragma unroll
        for (int i = 0; i < 8; ++i) xw[i] = load_stream(wk + int64_t(8 * i) * row_bytes + wlane);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                xa[mt][h] = aok[mt] ? *reinterpret_cast<const bf16x8*>(Ab + aoff[mt] + uint32_t(k0 + 32 * h) * 2u) : zero8;
    };
    // the wave's staging region as an LDS (address space 3) pointer
    __attribute__((address_space(3))) uint8_t* stage_lds = (__attribute__((address_space(3))) uint8_t*)stage;
    auto lds_ptr = [&](int off) { return (lds_bf16x4*)(stage_lds + off); };
    auto compute = [&](const bf16x8 (&xw)[8], const bf16x8 (&xa)[MT][2]) {
#pragma unroll
        for (int r = 0; r < 8; ++r) *reinterpret_cast<bf16x8*>(stage + wst[r]) = xw[r];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(lds_ptr(rtr[h][0][j]));
                const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(lds_ptr(rtr[h][1][j]));
                const bf16x8 b = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[mt][h], b, acc[mt][j], 0, 0, 0);
            }
    };
    bf16x8 xw0[8], xw1[8], xa0[MT][2], xa1[MT][2];
    if (nsteps > 0) gload(st, xw0, xa0);
    for (int i = 0; i < nsteps; i += 2) {
        if (i + 1 < nsteps) gload(st + WAVES, xw1, xa1);
        compute(xw0, xa0);
        if (i + 1 >= nsteps) break;
        if (i + 2 < nsteps) gload(st + 2 * WAVES, xw0, xa0);
        compute(xw1, xa1);
        st += 2 * WAVES;
    }

    if (p.fetch && lane == 0 && nsteps > 0)
        atomicAdd(p.fetch, BLOCK ? (unsigned long long)fetched : (unsigned long long)nsteps * 8ull * 1024ull);
    if constexpr (BLOCK) {
        // keeps the block loads live; M >= 1 always, so this never stores
        if ((sink[0] ^ sink[1] ^ sink[2] ^ sink[3]) == 0x6c8e9cf5 && p.M < 0) static_cast<float*>(p.C)[0] = 0.f;
    }

    // ---- sum the waves in a fixed order (the staging LDS is reused) ----
    __syncthreads();
    f32x4* red = reinterpret_cast<f32x4*>(smem);   // [WAVES][MT][4][64]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) red[((wave * MT + mt) * 4 + j) * 64 + lane] = acc[mt][j];
    __syncthreads();
    const bool final_out = p.split_k == 1;
    float* part = p.ws + int64_t(split) * p.ws_stride;
    for (int e = threadIdx.x; e < MT * 4 * 64; e += kThreads) {
        const int mt = e / 256, j = (e / 64) % 4, l = e % 64;
        f32x4 v = red[(mt * 4 + j) * 64 + l];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) v += red[((w * MT + mt) * 4 + j) * 64 + l];
        const int n = n0 + j * 16 + (l & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + (l >> 4) * 4 + r;
            if (m < p.M && n < p.N) {
                if (final_out) store_out(p.C, int64_t(m) * p.N + n, v[r], p.out_bf16);
                else part[int64_t(m) * p.N + n] = v[r];
            }
        }
    }
}

template <int MT, int WAVES>
hipError_t launch_kn_w(const DecodeParams& p, int grid, hipStream_t stream) {
    if (p.log2_fetch > 0)
        hipLaunchKernelGGL((decode_kn_kernel<MT, WAVES, true>), dim3(grid), dim3(64 * WAVES), 0, stream, p);
    else
        hipLaunchKernelGGL((decode_kn_kernel<MT, WAVES, false>), dim3(grid), dim3(64 * WAVES), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_kn_decode(const DecodeParams& p, int grid, int m_tiles16, int waves, hipStream_t stream) {
    switch (m_tiles16) {
        case 1: return waves == 8 ? launch_kn_w<1, 8>(p, grid, stream) : launch_kn_w<1, 4>(p, grid, stream);
        case 2: return waves == 8 ? launch_kn_w<2, 8>(p, grid, stream) : launch_kn_w<2, 4>(p, grid, stream);
        default: return launch_kn_w<4, 4>(p, grid, stream);
    }
}

}  // namespace tl
