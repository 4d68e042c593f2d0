// Decode GEMM on an emulated fixed-latency memory (prefetch-depth model).
#include <hip/hip_runtime.h>

#include <cstring>

#include "tl_decode_common.h"

namespace tl {
namespace {

// Large-granularity-memory emulation for the prefetch-depth model (Eq. 6,
// Section 5.3): the decode GEMM (M <= 16, 32-row tiles, 4 waves interleaved
// along K, tile-major weight) on a memory whose every read completes no
// earlier than 'latency' wall-clock ticks after it is issued.  Each wave keeps
// D K steps of loads in flight in a ring of registers -- the prefetch degree
// d = D - 1 of Eq. 6 -- and consumes step i only once the clock has passed
// its issue time plus the latency, then reissues the slot for step i + D.
// Every wait ends: the clock is monotonic and the target fixed.
template <int D>
__global__ __launch_bounds__(256) void lgms_kernel(DecodeParams p, long long latency) {
    constexpr int kWaves = 4, NS = 2, TN = 32;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int tile = blockIdx.x / p.split_k;
    const int split = blockIdx.x - tile * p.split_k;
    const int u0 = int((int64_t(p.units) * split) / p.split_k);
    const int u1 = int((int64_t(p.units) * (split + 1)) / p.split_k);
    const int st0 = u0 * p.steps_per_unit, st1 = u1 * p.steps_per_unit;
    const int n_base = tile * TN;
    const int g = lane >> 4, q = lane & 15;
    const bool lo = q < 8;
    const int kc = (((q >> 3) << 2) + g) << 3;
    const uint8_t* wrow[NS][2];
#pragma unroll
    for (int j = 0; j < NS; ++j)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            const int n = n_base + j * 16 + hf * 8 + (q & 7);
            wrow[j][hf] = p.W + int64_t(n >> p.log2_br) * p.strip_bytes +
                          (int64_t(n & ((1 << p.log2_br) - 1)) << (p.log2_bc + 1));
        }
    const int m = (q & 7);
    const bool aok0 = m < p.M, aok1 = m + 8 < p.M, aany1 = 8 < p.M;
    const uint16_t* arow0 = p.A + int64_t(aok0 ? m : 0) * p.K + kc;
    const uint16_t* arow1 = p.A + int64_t(aok1 ? m + 8 : 0) * p.K + kc;
    const bf16x8 zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
    f32x4 acc[NS];
#pragma unroll
    for (int j = 0; j < NS; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nsteps = st1 - st0 - wave > 0 ? (st1 - st0 - wave + kWaves - 1) / kWaves : 0;
    bf16x8 x[D][NS][2], xa[D][2];
    long long t_issue[D];
    auto issue = [&](int slot_i, int i) {   // loads of this wave's i-th step
        const int k = (st0 + wave + i * kWaves) * 64;
        const int64_t ko = (int64_t((k + kc) >> p.log2_bc) << p.log2_G) + int64_t(((k + kc) & p.bc_mask) << 1);
#pragma unroll
        for (int j = 0; j < NS; ++j)
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) x[slot_i][j][hf] = load_stream(wrow[j][hf] + ko);
        xa[slot_i][0] = aok0 ? *reinterpret_cast<const bf16x8*>(arow0 + k) : zero8;
        xa[slot_i][1] = (aany1 && aok1) ? *reinterpret_cast<const bf16x8*>(arow1 + k) : zero8;
        t_issue[slot_i] = wall_clock64();
    };
#pragma unroll
    for (int u = 0; u < D; ++u)
        if (u < nsteps) issue(u, u);
    for (int base = 0; base < nsteps; base += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
            const int i = base + u;
            if (i < nsteps) {
                while (wall_clock64() < t_issue[u] + latency) __builtin_amdgcn_s_sleep(1);
                bf16x8 a0, a1;
                {
                    const bf16x8 t = lo ? xa[u][1] : xa[u][0];
                    const bf16x8 sw = swap8(t);
                    a0 = lo ? xa[u][0] : sw;
                    a1 = lo ? sw : xa[u][1];
                }
#pragma unroll
                for (int j = 0; j < NS; ++j) {
                    const bf16x8 t = lo ? x[u][j][1] : x[u][j][0];
                    const bf16x8 sw = swap8(t);
                    const bf16x8 b0 = lo ? x[u][j][0] : sw, b1 = lo ? sw : x[u][j][1];
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b0, acc[j], 0, 0, 0);
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b1, acc[j], 0, 0, 0);
                }
                if (i + D < nsteps) issue(u, i + D);
            }
        }
    }
    __shared__ f32x4 red[kWaves][NS][64];
#pragma unroll
    for (int j = 0; j < NS; ++j) red[wave][j][lane] = acc[j];
    __syncthreads();
    const bool final_out = p.split_k == 1;
    float* part = p.ws + int64_t(split) * p.ws_stride;
    for (int e = threadIdx.x; e < NS * 64; e += 256) {
        const int j = e / 64, l = e % 64;
        f32x4 v = red[0][j][l];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) v += red[w][j][l];
        const int n = n_base + j * 16 + (l & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int mm = (l >> 4) * 4 + r;
            if (mm < p.M) {
                if (final_out) store_out(p.C, int64_t(mm) * p.N + n, v[r], p.out_bf16);
                else part[int64_t(mm) * p.N + n] = v[r];
            }
        }
    }
}

template <int D>
const void* lgms_fn() { return reinterpret_cast<const void*>(&lgms_kernel<D>); }

}  // namespace

int lgms_ctas_per_cu(int steps_in_flight) {
    int n = 0;
    const void* f = steps_in_flight == 1 ? lgms_fn<1>() : steps_in_flight == 2 ? lgms_fn<2>()
                  : steps_in_flight == 4 ? lgms_fn<4>() : lgms_fn<8>();
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, 256, 0) != hipSuccess) return -1;
    return n;
}

hipError_t launch_lgms(const DecodeLaunch& d, int64_t latency_ticks, int steps_in_flight, hipStream_t stream) {
    DecodeParams p;
    std::memset(&p, 0, sizeof p);
    p.A = d.A;
    p.W = d.W;
    p.C = d.C;
    p.ws = d.ws;
    p.M = int(d.M);
    p.N = int(d.N);
    p.K = int(d.K);
    p.split_k = d.split_k;
    p.ws_stride = (d.M * d.N + 3) / 4 * 4;
    p.steps_per_unit = int(d.k_unit / 64);
    p.units = int(d.K / d.k_unit);
    p.strip_bytes = d.L.br * d.K * 2;
    p.log2_br = d.L.log2_br;
    p.log2_bc = d.L.log2_bc;
    p.log2_G = d.L.log2_G;
    p.bc_mask = int(d.L.bc - 1);
    p.out_bf16 = d.out_bf16;
    const int grid = int(d.N / 32) * d.split_k;
    const long long lat = (long long)latency_ticks;
    switch (steps_in_flight) {
        case 1: hipLaunchKernelGGL(lgms_kernel<1>, dim3(grid), dim3(256), 0, stream, p, lat); break;
        case 2: hipLaunchKernelGGL(lgms_kernel<2>, dim3(grid), dim3(256), 0, stream, p, lat); break;
        case 4: hipLaunchKernelGGL(lgms_kernel<4>, dim3(grid), dim3(256), 0, stream, p, lat); break;
        default: hipLaunchKernelGGL(lgms_kernel<8>, dim3(grid), dim3(256), 0, stream, p, lat); break;
    }
    return launch_splitk_reduce(d, hipGetLastError(), stream);
}

}  // namespace tl
