// Weight-only 8-bit decode: FP8 (OCP E4M3) weights, bf16 activations.
#include <hip/hip_runtime.h>

#include "tl_decode_common.h"

namespace tl {
namespace {

// FP8 (OCP E4M3) weights, bf16 activations (weight-only 8-bit decode).  A
// 64-element K step of one weight row is 64 bytes; lane l = 16 g + q loads the
// 16 bytes k0 + 16 g .. + 15 of row q of each 16-row subtile, so with the
// (64, 64) FP8 memory tile one instruction reads 16 consecutive memory-tile
// rows = 1 KB contiguous, with no lane exchange.  The two 8-byte halves are
// converted exactly to bf16 (every E4M3 value is a bf16 value) and feed two
// MFMA 16x16x32: the first sums k0 + 16 g + 0..7 over the four lane groups,
// the second k0 + 16 g + 8..15, with the activations loaded in the same
// grouping.  Per-output-channel scales multiply the fp32 sums.
// Padded weights (Section 3.3) as in the bf16 decode kernel: rows past N load
// row N - 1 and are not stored; a last K step partly past K (K % 16 == 0)
// runs once after the streaming loops with the lanes past K reading zeros.
__device__ inline bf16x8 fp8x8_to_bf16(uint32_t lo, uint32_t hi) {
    typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
    u32x4v r;
    r[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, false));
    r[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, true));
    r[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, false));
    r[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, true));
    return __builtin_bit_cast(bf16x8, r);
}

template <int MT, int NS, int U, int WAVES, bool TILE>
__global__ __launch_bounds__(64 * WAVES) void decode_fp8_kernel(DecodeParams p) {
    typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
    constexpr int kWaves = WAVES;
    constexpr int kThreads = 64 * WAVES;
    constexpr int TN = 16 * NS;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int tile = blockIdx.x / p.split_k;
    const int split = blockIdx.x - tile * p.split_k;
    const int u0 = int((int64_t(p.units) * split) / p.split_k);
    const int u1 = int((int64_t(p.units) * (split + 1)) / p.split_k);
    const int st0 = u0 * p.steps_per_unit;
    const int st1 = min(u1 * p.steps_per_unit, p.ksteps);
    const int st1f = min(st1, p.kfull);
    const int n_base = tile * TN;
    const int g = lane >> 4, q = lane & 15;
    const int kg = g * 16;                     // this lane's 16 K values of a step
    const uint8_t* wrow[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const int n = min(n_base + j * 16 + q, p.N - 1);
        wrow[j] = p.W + (TILE ? int64_t(n >> p.log2_br) * p.strip_bytes + (int64_t(n & ((1 << p.log2_br) - 1)) << p.log2_bc)
                              : int64_t(n) * p.K);
    }
    const uint16_t* arow[MT];
    bool aok[MT], aany[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = mt * 16 + q;
        aok[mt] = m < p.M;
        aany[mt] = mt * 16 < p.M;
        arow[mt] = p.A + int64_t(aok[mt] ? m : 0) * p.K + kg;
    }
    f32x4 acc[MT][NS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NS; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bf16x8 zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
    const int nsteps = st1f - st0 - wave > 0 ? (st1f - st0 - wave + kWaves - 1) / kWaves : 0;
    int st = st0 + wave;
    int i = 0;
    auto koff = [&](int k) -> int64_t {
        if (TILE) return (int64_t(k >> p.log2_bc) << p.log2_G) + int64_t(k & p.bc_mask);
        return int64_t(k);
    };
    auto load = [&](int k, u32x4v (&x)[NS], bf16x8 (&a)[MT][2]) {
        const int64_t ko = koff(k + kg);
#pragma unroll
        for (int j = 0; j < NS; ++j) x[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(wrow[j] + ko));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            if (aany[mt]) {
                a[mt][0] = aok[mt] ? *reinterpret_cast<const bf16x8*>(arow[mt] + k) : zero8;
                a[mt][1] = aok[mt] ? *reinterpret_cast<const bf16x8*>(arow[mt] + k + 8) : zero8;
            } else {
                a[mt][0] = zero8;
                a[mt][1] = zero8;
            }
        }
    };
    auto compute = [&](const u32x4v (&x)[NS], const bf16x8 (&a)[MT][2]) {
#pragma unroll
        for (int j = 0; j < NS; ++j) {
            const bf16x8 w0 = fp8x8_to_bf16(x[j][0], x[j][1]);
            const bf16x8 w1 = fp8x8_to_bf16(x[j][2], x[j][3]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt][0], w0, acc[mt][j], 0, 0, 0);
                acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt][1], w1, acc[mt][j], 0, 0, 0);
            }
        }
    };
    for (; i + U <= nsteps; i += U) {
        u32x4v x[U][NS];
        bf16x8 a[U][MT][2];
#pragma unroll
        for (int u = 0; u < U; ++u) load((st + u * kWaves) * 64, x[u], a[u]);
#pragma unroll
        for (int u = 0; u < U; ++u) compute(x[u], a[u]);
        st += U * kWaves;
    }
    for (; i < nsteps; ++i) {
        u32x4v x[NS];
        bf16x8 a[MT][2];
        load(st * 64, x, a);
        compute(x, a);
        st += kWaves;
    }
    // the last step, partly past K, by its owner wave; lanes past K read
    // column 0 (in bounds) and use zeros
    const bool own_partial = p.kfull < st1 && p.kfull >= st0 && (p.kfull - st0) % kWaves == wave;
    if (own_partial) {
        const int k = p.kfull * 64;
        const bool kin = k + kg < p.K;
        u32x4v x[NS];
        bf16x8 a[MT][2];
        const int64_t ko = koff(kin ? k + kg : 0);
#pragma unroll
        for (int j = 0; j < NS; ++j) {
            const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(wrow[j] + ko));
            x[j] = kin ? v : u32x4v{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const uint16_t* pa = kin ? arow[mt] + k : arow[mt] - kg;
            const bf16x8 v0 = *reinterpret_cast<const bf16x8*>(pa);
            const bf16x8 v1 = *reinterpret_cast<const bf16x8*>(pa + 8);
            a[mt][0] = kin && aok[mt] ? v0 : zero8;
            a[mt][1] = kin && aok[mt] ? v1 : zero8;
        }
        compute(x, a);
    }
    const int issued = nsteps + (own_partial ? 1 : 0);
    if (p.fetch && lane == 0 && issued > 0) atomicAdd(p.fetch, (unsigned long long)issued * NS * 1024ull);

    static_assert(WAVES * MT * NS <= 64, "reduction buffer exceeds 64 KB");
    __shared__ f32x4 red[kWaves][MT][NS][64];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < NS; ++j) red[wave][mt][j][lane] = acc[mt][j];
    __syncthreads();
    constexpr int kEntries = MT * NS * 64;
    const bool final_out = p.split_k == 1;
    float* part = p.ws + int64_t(split) * p.ws_stride;
    for (int e = threadIdx.x; e < kEntries; e += kThreads) {
        const int mt = e / (NS * 64);
        const int j = (e / 64) % NS;
        const int l = e % 64;
        f32x4 v = red[0][mt][j][l];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) v += red[w][mt][j][l];
        const int n = n_base + j * 16 + (l & 15);
        const float sc = p.scales && n < p.N ? p.scales[n] : 1.0f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = mt * 16 + (l >> 4) * 4 + r;
            if (m < p.M && n < p.N) {
                if (final_out) store_out(p.C, int64_t(m) * p.N + n, v[r] * sc, p.out_bf16);
                else part[int64_t(m) * p.N + n] = v[r] * sc;
            }
        }
    }
}

template <int MT, int NS, int WAVES, bool TILE>
hipError_t launch_fp8_t(const DecodeParams& p, int grid, hipStream_t stream) {
    constexpr int U = MT >= 2 ? 2 : 4;
    hipLaunchKernelGGL((decode_fp8_kernel<MT, NS, U, WAVES, TILE>), dim3(grid), dim3(64 * WAVES), 0, stream, p);
    return hipGetLastError();
}

template <int MT, int NS, bool TILE>
hipError_t launch_fp8_w(const DecodeParams& p, int grid, int waves, hipStream_t stream) {
    if constexpr (MT * NS <= 2) {
        if (waves == 16) return launch_fp8_t<MT, NS, 16, TILE>(p, grid, stream);
    }
    if constexpr (MT * NS <= 8) {
        if (waves == 8) return launch_fp8_t<MT, NS, 8, TILE>(p, grid, stream);
    }
    return launch_fp8_t<MT, NS, 4, TILE>(p, grid, stream);
}

template <int MT>
hipError_t launch_fp8_m(const DecodeParams& p, int grid, int ns, int waves, bool tile, hipStream_t stream) {
    if (ns == 2) return tile ? launch_fp8_w<MT, 2, true>(p, grid, waves, stream)
                             : launch_fp8_w<MT, 2, false>(p, grid, waves, stream);
    return tile ? launch_fp8_w<MT, 4, true>(p, grid, waves, stream) : launch_fp8_w<MT, 4, false>(p, grid, waves, stream);
}

}  // namespace

hipError_t launch_fp8_decode(const DecodeParams& p, int grid, int m_tiles16, int ns, int waves, bool tile,
                             hipStream_t stream) {
    switch (m_tiles16) {
        case 1: return launch_fp8_m<1>(p, grid, ns, waves, tile, stream);
        case 2: return launch_fp8_m<2>(p, grid, ns, waves, tile, stream);
        default: return launch_fp8_m<4>(p, grid, ns, waves, tile, stream);
    }
}

}  // namespace tl
