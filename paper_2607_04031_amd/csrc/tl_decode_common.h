// Shared by the decode kernels (tl_decode.hip, tl_decode_fp8.hip, tl_lgms.hip):
// kernel parameters and small device helpers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "tl_internal.h"

namespace tl {

typedef short bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));


struct DecodeParams {
    const uint16_t* A;
    const uint8_t* W;
    void* C;
    float* ws;
    unsigned long long* fetch;
    int M, N, K;
    int split_k;
    int steps_per_unit;      // 64-element steps per split unit
    int units;               // ceil(K / k_unit)
    int ksteps;              // ceil(K / 64): 64-element K steps
    int kfull;               // K / 64: steps wholly inside K (a last partial step is masked)
    int64_t ws_stride;       // floats between two splits' partials (M * N rounded up to 4)
    int64_t strip_bytes;     // br * Kp * s (TILE) -- bytes per strip of br rows, Kp = K padded to bc
    int log2_br, log2_bc, log2_G;
    int bc_mask;
    bool out_bf16;
    int log2_fetch;          // block-granular emulation on a row-major weight: log2(G)
    int64_t w_bytes;         // N * K * 2
    // grouped (one launch over many weights, e.g. MoE experts)
    const int* offsets;      // [groups + 1] output-row offsets of the groups
    const int* token_ids;    // A row of each output row, or nullptr (identity)
    int tiles_per_group;     // N / tile_n
    int64_t group_stride;    // bytes between consecutive groups' weights
    int a_rows;              // rows of A; token ids outside [0, a_rows) read zeros
    int total_rows;          // rows of C; group offsets are clamped to [0, total_rows]
    const float* scales;     // FP8 weights: per-output-channel scale [N], or nullptr (1)
    int swiglu_up;           // gated grouped launch: row of the first up row (I); C has N = I columns
};

__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu))  // NaN stays NaN
        return uint16_t((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

__device__ inline void store_out(void* C, int64_t idx, float v, bool out_bf16) {
    if (out_bf16) static_cast<uint16_t*>(C)[idx] = f32_to_bf16_rne(v);
    else static_cast<float*>(C)[idx] = v;
}

// Byte offset of the 8-element chunk starting at (row base, k) of the weight.
template <bool TILE>
__device__ inline int64_t w_koff(const DecodeParams& p, int k) {
    if (TILE) return (int64_t(k >> p.log2_bc) << p.log2_G) + int64_t((k & p.bc_mask) << 1);
    return int64_t(k) << 1;
}

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Value of 'v' held by lane l ^ 8 (DPP row_ror:8 inside each 16-lane row).
__device__ inline bf16x8 swap8(bf16x8 v) {
    i32x4 x = __builtin_bit_cast(i32x4, v), y;
#pragma unroll
    for (int i = 0; i < 4; ++i) y[i] = __builtin_amdgcn_update_dpp(0, x[i], 0x128, 0xf, 0xf, false);
    return __builtin_bit_cast(bf16x8, y);
}

__device__ inline bf16x8 load_stream(const uint8_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(p));
}

// FP8-weight decode (tl_decode_fp8.hip): launches decode_fp8_kernel for the
// given M tiles, 16-row subtiles per tile, waves and layout.
hipError_t launch_fp8_decode(const DecodeParams& p, int grid, int m_tiles16, int ns, int waves, bool tile,
                             hipStream_t stream);

// Decode over a [K][N] row-major weight (tl_decode_kn.hip): 64-column tiles,
// p.units 64-row K steps split p.split_k ways, 4 or 8 waves; block-granular
// fetch when p.log2_fetch > 0.
hipError_t launch_kn_decode(const DecodeParams& p, int grid, int m_tiles16, int waves, hipStream_t stream);

// Decode with activations staged in LDS (tl_decode_lds.hip): 17 <= M <= 64,
// tile-major, tiles_per_wg 32-row tiles per workgroup (4..7 for M <= 32, 4
// above), p.units chunks of 512 columns split p.split_k ways.
hipError_t launch_lds_decode(const DecodeParams& p, int tiles_per_wg, int grid, hipStream_t stream);

}  // namespace tl
