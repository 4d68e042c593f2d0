// tl_stream_read: the HBM read ceiling the GEMM kernels are measured against.
// Every byte of a buffer is read once with the decode kernel's load pattern
// (64 lanes x 16 B, whole 128-byte lines, non-temporal) and folded into a
// 32-bit XOR checksum (XORed into the caller's word, one kernel per call),
// so the loads cannot be elided and the result is checkable.  Work order:
// 4 KB pieces dealt round-robin to every wave of the grid, four pieces in
// flight per wave (the fastest order measured on MI355X for 134 MB - 940 MB
// buffers).
#include <hip/hip_runtime.h>

#include "tl_internal.h"

namespace tl {
namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kStreamWaves = 4;
constexpr int kStreamU = 4;          // pieces in flight per wave
constexpr int64_t kPiece = 4096;     // bytes per wave per piece: 4 loads of 64 lanes x 16 B

__device__ inline u32x4 ld(const uint8_t* p) { return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)); }

__global__ __launch_bounds__(64 * kStreamWaves) void stream_read_kernel(const uint8_t* src, int64_t bytes,
                                                                        unsigned* checksum) {
    const int lane = threadIdx.x & 63;
    const int64_t gw = int64_t(blockIdx.x) * kStreamWaves + (threadIdx.x >> 6);
    const int64_t nw = int64_t(gridDim.x) * kStreamWaves;
    const int64_t pieces = bytes / kPiece;
    u32x4 acc = {0u, 0u, 0u, 0u};
    int64_t pc = gw;
    for (; pc + (kStreamU - 1) * nw < pieces; pc += kStreamU * nw) {
        u32x4 x[kStreamU][4];
#pragma unroll
        for (int u = 0; u < kStreamU; ++u) {
            const uint8_t* p = src + (pc + u * nw) * kPiece + lane * 16;
#pragma unroll
            for (int h = 0; h < 4; ++h) x[u][h] = ld(p + h * 1024);
        }
#pragma unroll
        for (int u = 0; u < kStreamU; ++u)
#pragma unroll
            for (int h = 0; h < 4; ++h) acc ^= x[u][h];
    }
    for (; pc < pieces; pc += nw) {
        const uint8_t* p = src + pc * kPiece + lane * 16;
#pragma unroll
        for (int h = 0; h < 4; ++h) acc ^= ld(p + h * 1024);
    }
    // the last bytes % 4096 (a multiple of 16): wave 0 of workgroup 0
    if (gw == 0) {
        for (int64_t off = pieces * kPiece + lane * 16; off < bytes; off += 1024) acc ^= ld(src + off);
    }
    // one atomic per workgroup: the lanes, then the waves, are folded first
    // (atomics on one word serialise; one per wave cost ~8 us per call)
    unsigned v = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) v ^= __shfl_xor(v, s);
    __shared__ unsigned part[kStreamWaves];
    if (lane == 0) part[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned w = part[0];
#pragma unroll
        for (int i = 1; i < kStreamWaves; ++i) w ^= part[i];
        atomicXor(checksum, w);
    }
}

}  // namespace

hipError_t launch_stream_read(const uint8_t* src, int64_t bytes, unsigned* checksum, hipStream_t stream) {
    if (bytes == 0) return hipSuccess;
    // one workgroup per CU: 256 x 4 waves (the best of 256 - 2048 measured)
    hipLaunchKernelGGL(stream_read_kernel, dim3(256), dim3(64 * kStreamWaves), 0, stream, src, bytes, checksum);
    return hipGetLastError();
}

}  // namespace tl
