// tl_view_load: the TMA-like load of a box of a multi-dimensional view from a
// tile-major weight into a dense destination (dimension 0 fastest), with the
// source addresses generated per element by the TileLens-HW counter program
// (Section 4.3; see tl_view.cpp).  HBM-bound byte copy: 16-byte chunks when
// the contiguous run (box[0] elements) is a multiple of 16 bytes, otherwise
// one element per thread.  A source address at or past src_bytes (which the
// host's checks already exclude) reads zeros instead of faulting.
#include <hip/hip_runtime.h>

#include "tl_internal.h"

namespace tl {
namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void view_load16_kernel(const uint8_t* src, int64_t src_bytes, ViewProgram P,
                                                          uint8_t* dst, int64_t chunks) {
    const int64_t per = 16 / P.elem_bytes;   // elements per 16-byte chunk
    for (int64_t q = int64_t(blockIdx.x) * 256 + threadIdx.x; q < chunks; q += int64_t(gridDim.x) * 256) {
        const int64_t off = view_offset(P, q * per);
        u32x4 v = {0u, 0u, 0u, 0u};
        if (off >= 0 && off + 16 <= src_bytes) v = *reinterpret_cast<const u32x4*>(src + off);
        *reinterpret_cast<u32x4*>(dst + q * 16) = v;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void view_load_elem_kernel(const uint8_t* src, int64_t src_bytes, ViewProgram P,
                                                             uint8_t* dst) {
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < P.elements; e += int64_t(gridDim.x) * 256) {
        const int64_t off = view_offset(P, e);
        T v = T(0);
        if (off >= 0 && off + int64_t(sizeof(T)) <= src_bytes) v = *reinterpret_cast<const T*>(src + off);
        reinterpret_cast<T*>(dst)[e] = v;
    }
}

}  // namespace

hipError_t launch_view_load(const uint8_t* src, int64_t src_bytes, const ViewProgram& P, uint8_t* dst,
                            hipStream_t stream) {
    const int64_t run = P.count[0] * P.elem_bytes;
    bool vec = run % 16 == 0 && P.tile_base % 16 == 0;
    for (int c = 1; c < P.n_counters; ++c) vec = vec && P.stride[c] % 16 == 0;
    const int64_t work = vec ? P.elements * P.elem_bytes / 16 : P.elements;
    const int grid = int(std::min<int64_t>((work + 255) / 256, 8192));
    if (vec) {
        hipLaunchKernelGGL(view_load16_kernel, dim3(grid), dim3(256), 0, stream, src, src_bytes, P, dst, work);
    } else {
        switch (P.elem_bytes) {
            case 1: hipLaunchKernelGGL(view_load_elem_kernel<uint8_t>, dim3(grid), dim3(256), 0, stream, src, src_bytes, P, dst); break;
            case 2: hipLaunchKernelGGL(view_load_elem_kernel<uint16_t>, dim3(grid), dim3(256), 0, stream, src, src_bytes, P, dst); break;
            case 4: hipLaunchKernelGGL(view_load_elem_kernel<uint32_t>, dim3(grid), dim3(256), 0, stream, src, src_bytes, P, dst); break;
            default: hipLaunchKernelGGL(view_load_elem_kernel<uint64_t>, dim3(grid), dim3(256), 0, stream, src, src_bytes, P, dst); break;
        }
    }
    return hipGetLastError();
}

}  // namespace tl
