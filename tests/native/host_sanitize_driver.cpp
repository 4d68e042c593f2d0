// Host-only driver for the sanitizer test (tests/test_host_sanitizers.py):
// calls the library's pure-host entry points -- planning, the exact
// read-amplification count, the view address generator, Eq. 6 and argument
// validation -- in a build with AddressSanitizer and UndefinedBehaviorSanitizer.
// The kernel launchers live in the .hip sources, which the sanitizer build leaves out;
// the stubs below stand in for them and abort if anything reaches them.
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "tl_internal.h"

namespace tl {
hipError_t launch_repack(const void*, void*, int64_t, int64_t, const Layout&, bool, hipStream_t) { std::abort(); }
hipError_t launch_decode(const DecodeLaunch&, hipStream_t) { std::abort(); }
hipError_t launch_splitk_reduce(const DecodeLaunch&, hipError_t, hipStream_t) { std::abort(); }
hipError_t launch_lgms(const DecodeLaunch&, int64_t, int, hipStream_t) { std::abort(); }
int lgms_ctas_per_cu(int) { std::abort(); }
hipError_t launch_prefill(const PrefillLaunch&, hipStream_t) { std::abort(); }
hipError_t launch_view_load(const uint8_t*, int64_t, const ViewProgram&, uint8_t*, hipStream_t) { std::abort(); }
hipError_t launch_zero_u64(unsigned long long*, hipStream_t) { std::abort(); }
hipError_t launch_stream_read(const uint8_t*, int64_t, unsigned*, hipStream_t) { std::abort(); }
hipError_t scratch_address(float**) { std::abort(); }
}  // namespace tl

int main() {
    int bad = 0;
    tl_layout_desc d = {};
    d.elem_bytes = 2;
    d.G = 4096;
    d.block_rows = 32;
    tl_amp a;
    // read amplification: every layout, ragged tiles and shapes (padded
    // tile-major copies), G != memory-tile size -- all valid
    for (int kind : {TL_LAYOUT_NK_ROW, TL_LAYOUT_KN_ROW, TL_LAYOUT_TILE})
        for (int64_t M : {1, 7, 64})
            for (int64_t N : {32, 96, 1024})
                for (int64_t K : {64, 192, 4096})
                    for (int tn : {16, 64, 96})
                        for (int tk : {32, 64, 160})
                            for (int64_t G : {512, 4096, 16384}) {
                                d.kind = kind;
                                if (tl_read_amp(M, N, K, 16, tn, tk, &d, G, &a) != TL_OK) ++bad;
                            }
    // counts past 2^63 - 1 and oversized enumerations are rejected, not wrapped
    d.kind = TL_LAYOUT_TILE;
    if (tl_read_amp(int64_t(1) << 40, 1 << 20, 1 << 20, 1, 32, 64, &d, 4096, &a) != TL_EINVAL) ++bad;
    if (tl_read_amp(8, 1 << 20, 1 << 20, 16, 32, 64, &d, int64_t(1) << 41, &a) != TL_EINVAL) ++bad;
    d.kind = TL_LAYOUT_NK_ROW;
    if (tl_read_amp(8, 1 << 20, 1 << 20, 16, 48, 48, &d, 16, &a) != TL_EUNSUPPORTED) ++bad;
    // views: 2-D to 4-D, Case 1, Case 2 and wider-than-tile boxes
    d.kind = TL_LAYOUT_TILE;
    std::vector<int64_t> offs(1 << 16);
    int64_t n = 0;
    for (int u : {16, 32, 64, 128}) {
        tl_view v = {};
        v.rank = 3;
        v.box[0] = u; v.box[1] = 64; v.box[2] = 2;
        v.strides[0] = 1; v.strides[1] = 1024; v.strides[2] = 128;
        v.coords[1] = 32;
        if (tl_view_offsets(&v, 1024, 256, 2, 4096, 32, offs.data(), int64_t(offs.size()), &n) != TL_OK) ++bad;
        v.coords[0] = 8;                               // not on a memory-tile boundary
        if (tl_view_offsets(&v, 1024, 256, 2, 4096, 32, offs.data(), int64_t(offs.size()), &n) != TL_EUNSUPPORTED) ++bad;
    }
    // planning and validation
    tl_plan p;
    for (int64_t M : {1, 8, 16, 17, 32, 64, 65, 1000, 2048, 4096})
        for (int64_t N : {512, 8192, 10240, 57344})
            if (tl_gemm_plan(M, N, 8192, &d, TL_FETCH_BLOCK, &p) != TL_OK) ++bad;
    tl_layout_desc bad_desc = d;
    bad_desc.G = 1000;
    if (tl_gemm_plan(8, 512, 512, &bad_desc, TL_FETCH_BLOCK, &p) != TL_EINVAL) ++bad;
    if (tl_gemm(nullptr, nullptr, nullptr, 8, 512, 512, &d, TL_FETCH_BLOCK, nullptr) != TL_EINVAL) ++bad;
    if (tl_gemm_plan(8, (int64_t(1) << 30) + 1, 64, &d, TL_FETCH_BLOCK, &p) != TL_EINVAL) ++bad;
    // a prefill grid of 2^31 workgroups or more (A and W each 2^31 bytes)
    tl_layout_desc rm = d;
    rm.kind = TL_LAYOUT_NK_ROW;
    if (tl_gemm_plan(int64_t(1) << 26, int64_t(1) << 26, 16, &rm, TL_FETCH_NATIVE, &p) != TL_EUNSUPPORTED) ++bad;
    if (tl_gemm_plan(int64_t(1) << 16, int64_t(1) << 16, 16, &rm, TL_FETCH_NATIVE, &p) != TL_OK) ++bad;
    // row-major [K][N] decode plans (native and block fetch), the prefill
    // plan's K-split remaining columns, and the allocation-free entry
    // point's rejections (before anything reaches the device)
    tl_layout_desc kn = d;
    kn.kind = TL_LAYOUT_KN_ROW;
    for (int64_t M : {1, 8, 32, 64})
        for (int64_t N : {64, 520, 8192})
            if (tl_gemm_plan(M, N, 4096, &kn, TL_FETCH_NATIVE, &p) != TL_OK) ++bad;
    if (tl_gemm_plan(8, 8192, 4096, &kn, TL_FETCH_BLOCK, &p) != TL_OK) ++bad;
    if (tl_gemm_plan(8, 520, 4096, &kn, TL_FETCH_BLOCK, &p) != TL_EUNSUPPORTED) ++bad;
    if (tl_gemm_plan(2048, 10240, 8192, &d, TL_FETCH_BLOCK, &p) != TL_OK || p.split_k != 4 ||
        p.workspace_bytes != int64_t(4) * 2048 * 2048 * 4)
        ++bad;
    tl_layout_desc bf = d;
    bf.out_dtype = TL_OUT_BF16;
    if (tl_gemm_plan(2048, 10240, 8192, &bf, TL_FETCH_BLOCK, &p) != TL_OK || p.tile_n != 320 || p.workgroups != 256)
        ++bad;
    tl_layout_desc big = d;
    big.split_k = 16;
    const void* dp = reinterpret_cast<const void*>(uintptr_t(1) << 42);
    if (tl_gemm_noalloc(dp, dp, const_cast<void*>(dp), 64, 32768, 65536, &big, TL_FETCH_BLOCK, nullptr) != TL_ESCRATCH)
        ++bad;
    if (tl_gemm_noalloc(dp, dp, const_cast<void*>(dp), 8, 64, 64, &d, TL_FETCH_BLOCK | TL_FETCH_COUNT, nullptr) !=
        TL_EUNSUPPORTED)
        ++bad;
    // tl_stream_read argument checks (no device work)
    uint32_t* ck = reinterpret_cast<uint32_t*>(uintptr_t(1) << 40);
    const void* src = reinterpret_cast<const void*>(uintptr_t(1) << 41);
    if (tl_stream_read(src, 4096, nullptr, nullptr) != TL_EINVAL) ++bad;
    if (tl_stream_read(src, 4095, ck, nullptr) != TL_EINVAL) ++bad;
    if (tl_stream_read(src, -16, ck, nullptr) != TL_EINVAL) ++bad;
    if (tl_stream_read(static_cast<const char*>(src) + 8, 4096, ck, nullptr) != TL_EINVAL) ++bad;
    if (tl_stream_read(src, 4096, reinterpret_cast<uint32_t*>(uintptr_t(src) + 64), nullptr) != TL_EINVAL) ++bad;
    int64_t deg = -1;
    if (tl_prefetch_degree(8e12, 5e-6, 16777216.0, 128, 1.0, &deg) != TL_OK || deg != 2) ++bad;
    std::printf("host sanitize driver: %d unexpected results, last view %lld elements\n", bad, (long long)n);
    return bad ? 1 : 0;
}
