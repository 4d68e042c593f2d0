// libtl C ABI: argument validation, kernel planning, per-(device, stream)
// library state, dispatch.  Nothing is enqueued unless every check passes.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <utility>
#include <vector>

#include "tl_internal.h"

namespace tl {

int make_tile_layout(int64_t s, int64_t G, int64_t br, Layout* out) {
    if (!(s == 1 || s == 2 || s == 4 || s == 8)) return TL_EINVAL;
    if (!is_pow2(G) || !is_pow2(br)) return TL_EINVAL;
    if (s * br > G) return TL_EINVAL;
    if (G > (int64_t(1) << 30)) return TL_EINVAL;
    Layout L;
    L.kind = TL_LAYOUT_TILE;
    L.s = s;
    L.G = G;
    L.br = br;
    L.bc = G / (s * br);
    L.log2_br = ilog2(br);
    L.log2_bc = ilog2(L.bc);
    L.log2_G = ilog2(G);
    *out = L;
    return TL_OK;
}

namespace {

// ---------------------------------------------------------------------------
// Library state: split-K workspace and the fetch tally, one set per
// (device, stream).  A workspace that has to grow is retired, not freed: a
// HIP graph captured earlier on the stream, or a call of another thread that
// took the old pointer, may still use it.  Retired workspaces are freed by
// tl_release.  Each call holds a shared reference to its state, so the
// buffers it enqueues on outlive a concurrent tl_release's host-side cleanup.
// ---------------------------------------------------------------------------
struct StreamState {
    int dev = 0;
    float* ws = nullptr;
    size_t ws_bytes = 0;
    unsigned long long* fetch = nullptr;
    std::vector<float*> retired;
    ~StreamState() {
        int cur = 0;
        const bool restore = hipGetDevice(&cur) == hipSuccess;
        (void)hipSetDevice(dev);
        for (float* p : retired) (void)hipFree(p);
        if (ws) (void)hipFree(ws);
        if (fetch) (void)hipFree(fetch);
        if (restore) (void)hipSetDevice(cur);
    }
};

// What one call uses: the buffers as they were when it looked them up.
struct StateRef {
    std::shared_ptr<StreamState> keep;
    float* ws = nullptr;
    unsigned long long* fetch = nullptr;
};

std::mutex g_mu;
std::map<std::pair<int, void*>, std::shared_ptr<StreamState>> g_state;

int current_device(int* dev) {
    return hipGetDevice(dev) == hipSuccess ? TL_OK : TL_EHIP;
}

// Looks up (current device, stream), creating its tally (cleared on 'stream',
// so the clear is ordered before any kernel that uses it) and growing its
// workspace to at least ws_bytes.  The lock covers the map and the
// allocations only; nothing here waits for the GPU.
int get_state(hipStream_t stream, size_t ws_bytes, StateRef* out) {
    int dev = 0;
    if (current_device(&dev) != TL_OK) return TL_EHIP;
    std::lock_guard<std::mutex> lock(g_mu);
    std::shared_ptr<StreamState>& sp = g_state[{dev, (void*)stream}];
    if (!sp) {
        sp = std::make_shared<StreamState>();
        sp->dev = dev;
    }
    StreamState& st = *sp;
    if (!st.fetch) {
        if (hipMalloc(&st.fetch, sizeof(unsigned long long)) != hipSuccess) { st.fetch = nullptr; return TL_ENOMEM; }
        if (launch_zero_u64(st.fetch, stream) != hipSuccess) {   // the next call allocates and clears again
            (void)hipFree(st.fetch);
            st.fetch = nullptr;
            return TL_EHIP;
        }
    }
    if (ws_bytes > st.ws_bytes) {
        // at least double, so the retired buffers never add up to more than
        // the current one
        const size_t bytes = std::max({ws_bytes, 2 * st.ws_bytes, size_t(1) << 20});
        float* p = nullptr;
        if (hipMalloc(&p, bytes) != hipSuccess) return TL_ENOMEM;
        if (st.ws) st.retired.push_back(st.ws);
        st.ws = p;
        st.ws_bytes = bytes;
    }
    out->keep = sp;
    out->ws = st.ws;
    out->fetch = st.fetch;
    return TL_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlap(const void* a, int64_t a_bytes, const void* b, int64_t b_bytes) {
    auto x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + uintptr_t(b_bytes) && y < x + uintptr_t(a_bytes);
}

constexpr int64_t kMaxElems = int64_t(1) << 40;   // rows * cols bound (keeps byte counts in int64)

int check_repack_args(const void* src, const void* dst, int64_t rows, int64_t cols, int32_t s,
                      int64_t G, int32_t br, bool inverse, Layout* L) {
    if (rows < 0 || cols < 0) return TL_EINVAL;
    if (make_tile_layout(s, G, br, L) != TL_OK) return TL_EINVAL;
    if (rows == 0 || cols == 0) return TL_OK;
    if (!src || !dst || !aligned16(src) || !aligned16(dst)) return TL_EINVAL;
    if (rows > kMaxElems / std::max<int64_t>(cols, 1) || cols > kMaxElems) return TL_EINVAL;
    // the row-major matrix and the padded tile-major copy (src and dst, or the reverse)
    const int64_t rm_bytes = rows * cols * s, tm_bytes = packed_bytes(*L, rows, cols);
    if (overlap(src, inverse ? tm_bytes : rm_bytes, dst, inverse ? rm_bytes : tm_bytes)) return TL_EINVAL;
    return TL_OK;
}

int do_repack(const void* src, void* dst, int64_t rows, int64_t cols, int32_t s, int64_t G,
              int32_t br, void* stream, bool inverse) {
    Layout L;
    int rc = check_repack_args(src, dst, rows, cols, s, G, br, inverse, &L);
    if (rc != TL_OK) return rc;
    if (rows == 0 || cols == 0) return TL_OK;
    if (packed_bytes(L, rows, cols) / L.G >= (int64_t(1) << 32)) return TL_EUNSUPPORTED;  // 32-bit block index
    hipError_t e = launch_repack(src, dst, rows, cols, L, inverse, (hipStream_t)stream);
    return e == hipSuccess ? TL_OK : TL_EHIP;
}

// ---------------------------------------------------------------------------
// GEMM planning
// ---------------------------------------------------------------------------
struct Plan {
    tl_plan pub;
    Layout L;
    bool out_bf16 = false;
    bool count = false;
    int m_tiles16 = 1;
    int waves = 4;
    int64_t k_unit = 64;
    bool block_row = false;      // block-granular emulation on a row-major weight
    int64_t fetch_G = 0;
    int64_t n_main = 0;          // prefill: columns covered by the main tiles (rest: 128 x 128)
    bool fp8 = false;            // 1-byte (OCP E4M3) weight, decode kernel
    int lds_tiles = 0;           // > 0: decode with activations staged in LDS, tiles per workgroup
    bool kn_row = false;         // weight stored [K][N] (N contiguous): the transposing decode kernel
    int split_rest = 0;          // prefill: K splits of the 256 x 256 tiles past n_main (0: 128 x 128 tiles)
    bool persist = false;        // prefill: one workgroup per CU walks the main launch's tiles
};

constexpr int kDecodeMaxM = 64;
constexpr int64_t kMaxDim = int64_t(1) << 30;   // largest M, N or K
constexpr int kTargetWorkgroups = 1024;   // 4 per CU on 256 CUs
constexpr int kMaxSplitK = 16;            // partials the reduce kernel sums
constexpr int kCUs = 256;                  // MI355X compute units

int plan_gemm(int64_t M, int64_t N, int64_t K, const tl_layout_desc* d, int32_t fetch_mode,
              Plan* P) {
    if (!d) return TL_EINVAL;
    if (M < 1 || N < 1 || K < 1) return TL_EINVAL;
    if (fetch_mode & ~(TL_FETCH_BLOCK | TL_FETCH_COUNT)) return TL_EINVAL;
    if (d->out_dtype != TL_OUT_F32 && d->out_dtype != TL_OUT_BF16) return TL_EINVAL;
    if (d->tile_m < 0 || d->tile_n < 0 || d->tile_k < 0 || d->split_k < 0) return TL_EINVAL;
    if (d->kind != TL_LAYOUT_NK_ROW && d->kind != TL_LAYOUT_KN_ROW && d->kind != TL_LAYOUT_TILE)
        return TL_EINVAL;
    if (d->elem_bytes != 2 && d->elem_bytes != 1) return d->elem_bytes < 1 ? TL_EINVAL : TL_EUNSUPPORTED;
    const int s = d->elem_bytes;
    // kernel-side row and column indices are 32-bit, with room for a tile past the edge
    if (M > kMaxDim || N > kMaxDim || K > kMaxDim) return TL_EINVAL;

    Plan p;
    std::memset(&p.pub, 0, sizeof p.pub);
    p.out_bf16 = d->out_dtype == TL_OUT_BF16;
    p.count = (fetch_mode & TL_FETCH_COUNT) != 0;
    p.fp8 = s == 1;
    const bool block = (fetch_mode & TL_FETCH_BLOCK) != 0;

    if (d->kind == TL_LAYOUT_TILE) {
        if (make_tile_layout(s, d->G, d->block_rows, &p.L) != TL_OK) return TL_EINVAL;
        if (p.L.bc * s < 16) return TL_EUNSUPPORTED;   // a 16-byte lane load stays in one memory-tile row
    } else if (d->kind == TL_LAYOUT_NK_ROW) {
        p.L.kind = TL_LAYOUT_NK_ROW;
        if (block && !p.fp8) {
            // whole G-byte blocks of the row-major weight; G >= 128 keeps each
            // 128-byte row segment of a K step inside one block
            if (!is_pow2(d->G) || d->G < 128 || d->G > (int64_t(1) << 30)) return TL_EINVAL;
            p.block_row = true;
            p.fetch_G = d->G;
        }
    } else {
        // [K][N] row-major (the paper's row-major layout): the decode kernel
        // that transposes each K step through LDS, bf16 only, M <= 64; whole
        // 64-row K steps, rows of 16-byte multiples, and the rows one lane's
        // eight loads span below 2^31 bytes
        p.L.kind = TL_LAYOUT_KN_ROW;
        p.kn_row = true;
        if (block) {
            if (!is_pow2(d->G) || d->G < 128 || d->G > (int64_t(1) << 30)) return TL_EINVAL;
            p.block_row = true;
            p.fetch_G = d->G;
        }
        if (p.fp8 || M > kDecodeMaxM || d->tile_m > 64) return TL_EUNSUPPORTED;
        if (K % 64 || N % 8 || N >= (int64_t(1) << 27)) return TL_EUNSUPPORTED;
    }
    // Any N; K a multiple of one 16-byte lane load, so activation (and
    // row-major weight) rows stay 16-byte aligned and a load is either wholly
    // inside K or wholly past it.  Ragged N or K (padded tile-major weights,
    // Section 3.3) is not implemented for the row-major block emulation.
    if (K % (16 / s)) return TL_EUNSUPPORTED;
    // block emulation: whole 64-wide K steps, and tiles whose row segments
    // start on 128-byte boundaries (so none straddles a block edge)
    if (p.block_row && (K % 64 || N % (p.kn_row ? 64 : 32))) return TL_EUNSUPPORTED;

    const bool tile = d->kind == TL_LAYOUT_TILE;
    p.k_unit = tile ? std::max<int64_t>(64, p.L.bc) : 64;

    if (p.fp8 && !(M <= kDecodeMaxM && d->tile_m <= 64)) return TL_EUNSUPPORTED;        // FP8: decode kernel only
    // 33 <= M <= 64 on a wide bf16 weight (128 x 128 tiles fill the CUs at
    // least once: N >= 32768), no tile or split requested, within the
    // prefill kernel's limits (whole memory-tile strips per 128-row tile,
    // weights under 4 GB): its 128 x 128 tiles stream the weight faster than
    // the decode kernel's 64-row tiles at four 16-row M tiles, whose
    // activation reloads from L2 match the weight bytes (Llama gate+up, bf16
    // out, one box, M = 33 / 48 / 64: 187 / 211 / 240 -> 169 / 171 / 172 us)
    const bool wide_mid_m = M > 32 && M <= kDecodeMaxM && !d->tile_m && !d->tile_n && !d->split_k && !p.fp8 &&
                            !p.kn_row && !p.block_row && N / 128 >= kCUs && (!tile || 128 % p.L.br == 0) &&
                            (tile ? packed_bytes(p.L, N, K) : N * K * 2) < (int64_t(1) << 32);
    if (p.kn_row) {
        // 64-column tiles (128-byte row segments), K split until there are
        // about 1024 workgroups with >= 1024 K per split; 8 waves when the
        // tiles need no more than two rounds of the CUs and their registers
        // and LDS allow it
        p.pub.kernel = 1;
        p.m_tiles16 = int((M + 15) / 16);
        if (p.m_tiles16 == 3) p.m_tiles16 = 4;
        if (d->tile_n && d->tile_n != 64) return TL_EUNSUPPORTED;
        if (d->tile_k && d->tile_k != 64) return TL_EUNSUPPORTED;
        if (M * K * 2 >= (int64_t(1) << 31)) return TL_EUNSUPPORTED;
        p.k_unit = 64;
        const int64_t n_tiles = (N + 63) / 64, units = K / 64;
        int64_t S = d->split_k;
        if (S == 0) {
            const int64_t max_s = std::max<int64_t>(1, std::min<int64_t>(units / 16, kMaxSplitK));
            S = n_tiles >= 2 * kCUs ? 1 : std::min((kTargetWorkgroups + n_tiles - 1) / n_tiles, max_s);
        }
        if (S < 1 || S > units || S > kMaxSplitK) return TL_EUNSUPPORTED;
        const int64_t wgs = n_tiles * S;
        p.waves = (wgs <= 2 * kCUs && p.m_tiles16 <= 2) ? 8 : 4;
        p.pub.tile_m = 16 * p.m_tiles16;
        p.pub.tile_n = 64;
        p.pub.tile_k = 64;
        p.pub.split_k = int(S);
        p.pub.waves = p.waves;
        p.pub.workgroups = wgs;
        p.pub.workspace_bytes = S > 1 ? S * ((M * N + 3) / 4 * 4) * 4 : 0;
    } else if (M <= kDecodeMaxM && d->tile_m <= 64 && !wide_mid_m) {
        p.pub.kernel = 1;
        p.m_tiles16 = int((M + 15) / 16);
        if (p.m_tiles16 == 3) p.m_tiles16 = 4;
        // A small weight (under 32 MB: a few microseconds of HBM time) is
        // latency-bound: 32-row tiles and K splits down to 512 columns give
        // more workgroups (shorter splits cost more in the reduce launch than
        // they gain).  Otherwise 64-row tiles halve the activation
        // reloads per weight byte, which pays off once M exceeds one 16-row
        // MFMA tile.  (Measured on the Qwen attention projections at M = 8,
        // 32 and 64 and the Llama-70B shapes.)
        const bool small = N * K * s < (int64_t(32) << 20);
        int tn_default = p.m_tiles16 >= 2 && N % 64 == 0 && !small ? 64 : 32;
        if (tile) tn_default = int(std::max<int64_t>(tn_default, p.L.br));
        int tn = d->tile_n ? d->tile_n : tn_default;
        if (tn != 32 && tn != 64) return TL_EUNSUPPORTED;
        if (tile && tn % p.L.br) return TL_EUNSUPPORTED;
        if (d->tile_k && (d->tile_k != p.k_unit)) return TL_EUNSUPPORTED;
        int64_t n_tiles = (N + tn - 1) / tn;
        const int64_t units = (K + p.k_unit - 1) / p.k_unit;
        // Balance: every CU should stream the same number of bytes.
        //  - at least two tiles per CU: one workgroup per tile, K not split
        //    -- except between two and four rounds of the CUs that do not
        //    come out even (896 tiles: 3.5 per CU), where two K splits even
        //    them out if their fp32 partials (written and read back) stay
        //    within 2 % of the weight bytes (FP8 gate+up at M = 8: -9 %);
        //  - tiles that divide the CUs or fill them a whole number of times
        //    (N = 8192: 256 tiles of 32 rows, 128 of 64): one workgroup per
        //    CU, whose 8 or 16 waves split K among themselves (reduced in
        //    LDS), or four per CU when each K split still streams >= 4096 K
        //    (the reduce launch then costs a few per cent at most);
        //  - fewer tiles than two rounds that do not divide the CUs: the
        //    32- or 64-row tile and K split that fill one round of the CUs
        //    to at least 7/8 (one workgroup per CU, its waves splitting K
        //    too), as for tiles that divide the CUs -- measured on the
        //    tensor-parallel shards of the Llama-70B shapes (40 - 448 tiles:
        //    gate+up / 4 at M = 8 43.9 -> 37.9 us, QKV / 4 at M = 32
        //    19.7 -> 14.7; equal fills take 64-row tiles above M = 16);
        //  - otherwise split K until there are about 1024 workgroups.
        // K splits write fp32 partials that a fixed-order reduce kernel sums;
        // every split covers >= 1024 K (>= 512 for a small weight).  (Chosen
        // from measurements of the Llama-70B decode shapes at M = 1, 8 and 32.)
        int64_t S = d->split_k;
        if (S == 0) {
            const int64_t min_units = std::max<int64_t>(1, (small ? 512 : 1024) / p.k_unit);
            const int64_t max_s = std::max<int64_t>(1, std::min<int64_t>(units / min_units, kMaxSplitK));
            if (n_tiles >= 2 * kCUs) {
                S = 1;
                const int64_t w_bytes = N * K * s;
                if (n_tiles < 4 * kCUs && n_tiles % kCUs != 0 && max_s >= 2 && 2 * 2 * M * N * 4 * 50 <= w_bytes)
                    S = 2;
            } else if (kCUs % n_tiles == 0 || n_tiles % kCUs == 0) {
                S = std::max<int64_t>(1, kCUs / n_tiles);
                if (K / (4 * S) >= 4096) S *= 4;
                S = std::min(S, max_s);
            } else {
                int best_tn = 0;
                int64_t best_w = 0, best_s = 0;
                const int prefer = p.m_tiles16 >= 2 ? 64 : 32;
                for (int c : {32, 64}) {
                    if (d->tile_n ? c != tn : (c == 64 && N % 64)) continue;
                    if (tile && c % p.L.br) continue;
                    const int64_t nt = (N + c - 1) / c;
                    const int64_t sc = std::min<int64_t>(kCUs / nt, max_s);
                    if (sc < 1) continue;
                    if (nt * sc > best_w || (nt * sc == best_w && c == prefer)) {
                        best_tn = c;
                        best_w = nt * sc;
                        best_s = sc;
                    }
                }
                if (8 * best_w >= 7 * kCUs) {
                    tn = best_tn;
                    n_tiles = (N + tn - 1) / tn;
                    S = best_s;
                } else if (p.fp8) {
                    // one-byte weights: splits for about 1024 workgroups are
                    // short (Llama QKV: 7 of 1170 K, 75 KB each) and pay their
                    // start and drain more than they gain; at most two
                    // rounds of 8-wave workgroups instead (QKV at M = 8,
                    // rotated weights, one box: 20.3 -> 18.8 us)
                    S = std::max<int64_t>(1, std::min(2 * kCUs / n_tiles, max_s));
                } else {
                    S = std::min((kTargetWorkgroups + n_tiles - 1) / n_tiles, max_s);
                }
            }
        }
        if (S < 1 || S > units || S > kMaxSplitK) return TL_EUNSUPPORTED;
        // the decode kernels address a tile's weight rows and the activations
        // with 32-bit byte offsets from a uniform base
        const int64_t kp = tile ? padded_cols(p.L, K) : K;
        if (int64_t(tn) * kp * s >= (int64_t(1) << 31) || M * K * 2 >= (int64_t(1) << 31)) return TL_EUNSUPPORTED;
        const int64_t wgs = n_tiles * S;
        const int ns = tn / 16;
        int waves = wgs <= kCUs ? 16 : (wgs <= 2 * kCUs ? 8 : 4);
        // registers: 16 waves (4 per SIMD, <= 128 VGPRs) only fit one 16-row
        // M tile x 32 rows of N; 8 waves (<= 256 VGPRs) fit up to 8 of those,
        // and the 64-row tile at four M tiles, which keeps one K step in
        // flight (bf16 weights read natively)
        const int mn = p.m_tiles16 * ns / 2;
        if (waves == 16 && mn > 1) waves = 8;
        if (waves == 8 && mn > 4 && !(mn == 8 && !p.fp8 && !p.block_row)) waves = 4;
        p.waves = waves;
        // 17 <= M <= 32 on whole tile-major strips: stage the activations in
        // LDS, one 8-wave workgroup per CU taking T of the 32-row tiles and
        // one of S K ranges, when the (T, S) grid covers the CUs in whole
        // rounds (A crosses L2 -> CU once per T tiles instead of once per
        // tile) -- unless its K ranges are short (under 8 chunks, so its
        // staging and wave reduction weigh more) while the streaming plan
        // already has one or two workgroups per CU (Llama O at M = 32:
        // 29.8 vs 29.0 us; QKV, whose streaming plan needs 1120 workgroups,
        // 35.6 vs 43.0; down 81.7 vs 84.1; gate+up 150.9 vs 181.4)
        if (tile && !p.fp8 && p.m_tiles16 == 2 && !d->tile_n && !d->split_k && N % 32 == 0 && K % 512 == 0 &&
            p.L.br <= 32 && 512 % p.k_unit == 0) {
            const int64_t strips = N / 32, chunks = K / 512;
            bool found = false;   // the first whole-round (T, S) decides
            for (int T = 7; T >= 4 && !found; --T) {
                if (strips % T) continue;
                for (int64_t s2 = 1; s2 <= 8 && chunks / s2 >= 4 && !found; s2 *= 2) {
                    const int64_t w = strips / T * s2;
                    if (w % kCUs == 0 && w <= 4 * kCUs) {
                        found = true;
                        if (s2 == 1 || chunks / s2 >= 8 || wgs > 2 * kCUs) {
                            p.lds_tiles = T;
                            S = s2;
                        }
                    }
                }
            }
            if (p.lds_tiles) {
                tn = 32;
                p.waves = 8;
            }
        }
        // 33 <= M <= 64 (four M tiles) on whole tile-major strips: the same
        // staging with T = 4 tiles per workgroup (64 KB chunks of A; at T = 5
        // the registers spill) and the largest S (K ranges of >= 4 chunks)
        // whose grid fits one round of the CUs, when that fills at least 7/8
        // of it (or S = 1 when the tile groups fill a round by themselves):
        // a 64-row streaming tile reloads as many activation bytes from L2 as
        // it streams weight bytes (Llama shapes, bf16 out, one box, M = 33 /
        // 48 / 64: QKV (S = 3, 240 workgroups) 50 / 54 / 58 -> 41 / 42 / 44 us,
        // O 33 / 35 / 39 -> 32 / 33 / 35, down 93 / 100 / 112 -> 88 / 90 / 92)
        if (tile && !p.fp8 && p.m_tiles16 == 4 && !d->tile_n && !d->split_k && N % 128 == 0 && K % 512 == 0 &&
            p.L.br <= 32 && 512 % p.k_unit == 0) {
            const int64_t groups = N / 128, chunks = K / 512;
            int64_t s_fit = groups >= kCUs ? 1 : 0;
            for (int64_t s2 = 1; s2 <= 8 && chunks / s2 >= 4 && groups < kCUs; ++s2)
                if (groups * s2 <= kCUs) s_fit = s2;
            if (s_fit && 8 * groups * s_fit >= 7 * kCUs) {
                p.lds_tiles = 4;
                S = s_fit;
                tn = 32;
                p.waves = 8;
            }
        }
        const int64_t wgs_final = p.lds_tiles ? N / 32 / p.lds_tiles * S : wgs;
        p.pub.tile_m = 16 * p.m_tiles16;
        p.pub.tile_n = tn;
        p.pub.tile_k = int(p.k_unit);
        p.pub.split_k = int(S);
        p.pub.waves = p.waves;
        p.pub.workgroups = wgs_final;
        p.pub.workspace_bytes = S > 1 ? S * ((M * N + 3) / 4 * 4) * 4 : 0;
    } else {
        p.pub.kernel = 2;
        int tm = d->tile_m ? d->tile_m : (M >= 1024 ? 256 : 128);
        if (tm != 128 && tm != 256) return TL_EUNSUPPORTED;
        int tn = d->tile_n ? d->tile_n : ((tm == 256 && N % 256 == 0) ? 256 : 128);
        if (tn != 128 && !(tn == 256 && tm == 256)) return TL_EUNSUPPORTED;
        if (tile && tn % p.L.br) return TL_EUNSUPPORTED;
        if (d->tile_k && d->tile_k != p.k_unit) return TL_EUNSUPPORTED;
        if (d->split_k > 1) return TL_EUNSUPPORTED;
        // the kernel addresses A and W with 32-bit byte offsets
        const int64_t wb = tile ? packed_bytes(p.L, N, K) : N * K * 2;
        if (M * K * 2 >= (int64_t(1) << 32) || wb >= (int64_t(1) << 32)) return TL_EUNSUPPORTED;
        // 256 x 320 tiles (each wave 128 x 160 of C) where they fill the CUs
        // in whole rounds and 256 x 256 tiles do not: QKV at M = 2048, 256
        // tiles instead of 320 -- one round, no second launch, no partials
        // (persistent bf16 only; no tile requested)
        if (!d->tile_m && !d->tile_n && tm == 256 && p.out_bf16 && !p.block_row && K % 128 == 0 && M % 256 == 0 &&
            N % 320 == 0 && (!tile || 320 % p.L.br == 0)) {
            const int64_t t320 = (M / 256) * (N / 320);
            const int64_t t256 = N % 256 == 0 ? (M / 256) * (N / 256) : 1;
            if (t320 % kCUs == 0 && t256 % kCUs != 0 && t320 < (int64_t(1) << 31) - kCUs) {
                p.n_main = N;
                p.persist = true;
                p.pub.tile_m = 256;
                p.pub.tile_n = 320;
                p.pub.tile_k = int(p.k_unit);
                p.pub.split_k = 1;
                p.pub.waves = 4;
                p.pub.workgroups = kCUs;
                p.pub.workspace_bytes = 0;
                *P = p;
                return TL_OK;
            }
        }
        // Small and medium M (no tile requested): when 256 x 256 tiles are
        // fewer than the CUs, the same tiles with K split S ways over all the
        // columns (S = CUs / tiles, up to 8, each split >= 8 of the 64-wide K
        // steps; fp32 partials, at most 256 tiles x 64 K elements x S <= 64
        // MiB, summed in split order by the reduce kernel); above M = 128,
        // when they fill at least half the CUs, 256 x 256 tiles rather than
        // 128 x 128 (at M <= 128 those waste half their rows: gate+up at
        // M = 128, 224 tiles, 193 us as 128 x 128, 224 as 256 x 256).
        // Llama-70B-shaped layer, bf16 out, whole layers on one box: M = 128
        // 730 -> 464 us, 256 851 -> 514, 512 1132 -> 779, 1024 1667 -> 1419
        // (down alone at M = 1024: 535 -> 388).
        // 65 <= M <= 128 (one row of 128-row tiles): 128 x 128 tiles with K
        // split over all the columns in the same way, when they are fewer
        // than the CUs -- no padded rows past 128, against half or more of a
        // 256-row tile's
        if (!d->tile_m && !d->tile_n && M > kDecodeMaxM && M <= 128 && N % 128 == 0 && !p.block_row &&
            (!tile || 128 % p.L.br == 0) && N / 128 < kCUs) {
            const int64_t t128 = N / 128;
            const int64_t S = std::min<int64_t>({kCUs / t128, 8, (K + 63) / 64 / 8});
            if (S >= 2) {
                p.n_main = 0;                // no main launch: every column splits K
                p.split_rest = int(S);
                p.persist = false;
                p.pub.tile_m = 128;
                p.pub.tile_n = 128;
                p.pub.tile_k = int(p.k_unit);
                p.pub.split_k = int(S);
                p.pub.waves = 4;
                p.pub.workgroups = t128 * S;
                p.pub.workspace_bytes = S * M * N * 4;
                *P = p;
                return TL_OK;
            }
        }
        if (!d->tile_m && !d->tile_n && M > kDecodeMaxM && K % 64 == 0 && N % 256 == 0 && !p.block_row &&
            (!tile || 256 % p.L.br == 0)) {
            const int64_t t256 = ((M + 255) / 256) * (N / 256);
            if (t256 < kCUs) {
                const int64_t S = std::min<int64_t>({kCUs / t256, 8, K / 64 / 8});
                if (S >= 2) {
                    p.n_main = 0;                // no main launch: every column splits K
                    p.split_rest = int(S);
                    p.persist = false;
                    p.pub.tile_m = 256;
                    p.pub.tile_n = 256;
                    p.pub.tile_k = int(p.k_unit);
                    p.pub.split_k = int(S);
                    p.pub.waves = 4;
                    p.pub.workgroups = t256 * S;
                    p.pub.workspace_bytes = S * M * N * 4;
                    *P = p;
                    return TL_OK;
                }
            }
            if (tm == 128 && M > 128 && 2 * t256 >= kCUs) {
                tm = 256;
                tn = 256;
            }
        }
        // Quantisation: 256 x 256 tiles that leave the last round of
        // workgroups part-empty (QKV at M = 2048: 320 tiles on 256 CUs) cover
        // the widest column range whose tile count is a multiple of the CU
        // count, and a second launch of 128 x 128 tiles covers the remaining
        // columns when they fit in one round (two 128 x 128 workgroups per CU).
        p.n_main = N;
        const int64_t mt = (M + tm - 1) / tm;
        const int64_t tiles = mt * ((N + tn - 1) / tn);
        // (not with the block emulation: its count follows one tile shape)
        if (!d->tile_m && !d->tile_n && tm == 256 && tn == 256 && N % 256 == 0 && tiles > kCUs &&
            tiles % kCUs != 0 && (!tile || 128 % p.L.br == 0) && !p.block_row) {
            for (int64_t n1 = N - 256; n1 >= 256; n1 -= 256) {
                if ((mt * (n1 / 256)) % kCUs) continue;
                const int64_t rest = ((M + 127) / 128) * ((N - n1) / 128);
                if (rest <= 2 * kCUs) p.n_main = n1;
                break;
            }
            // The remaining columns as 256 x 256 tiles of the four-wave
            // kernel with K split S ways, when those tiles times S fill the
            // CUs exactly and each split keeps >= 8 of the 64-wide K steps
            // (fp32 partials summed in a fixed order by a second kernel):
            // QKV at M = 2048, 64 tiles x 4 splits (on one box 1021 -> 1113
            // TFLOP/s against the 128 x 128 tiles).
            if (p.n_main < N && K % 64 == 0) {
                const int64_t rest256 = mt * ((N - p.n_main) / 256);
                if (rest256 > 0 && kCUs % rest256 == 0) {
                    const int64_t S = kCUs / rest256;
                    if (S >= 2 && S <= 8 && K / 64 / S >= 8) p.split_rest = int(S);
                }
            }
        }
        // Whole 256 x 256 tiles with bf16 output and an even number of
        // 64-wide K steps: a persistent grid of at most one workgroup per CU
        // walks them, loading a tile's first step under the previous tile's
        // last MFMAs and storing C straight from registers (gate+up at
        // M = 2048, 7 tiles per CU: 1476 -> 1441 us on one box; down, one
        // tile per CU: 720 -> 706 us on another).
        const int64_t main_tiles = mt * (p.n_main / tn + (p.n_main % tn ? 1 : 0));
        p.persist = tm == 256 && tn == 256 && K % 128 == 0 && !p.block_row && p.out_bf16 && M % 256 == 0 &&
                    p.n_main % 256 == 0;
        p.pub.tile_m = tm;
        p.pub.tile_n = tn;
        p.pub.tile_k = int(p.k_unit);
        p.pub.split_k = 1;
        p.pub.waves = tm == 256 && tn == 256 ? (K % 64 == 0 && !p.block_row ? 4 : 8) : 4;
        p.pub.workgroups = (p.persist ? std::min<int64_t>(main_tiles, kCUs) : main_tiles) +
                           (p.split_rest ? mt * ((N - p.n_main) / 256) * p.split_rest
                                         : ((M + 127) / 128) * ((N - p.n_main) / 128));
        // one launch's grid, and the persistent grid's tile count (an int
        // that stays below 2^31 after one more step of 256)
        if (p.pub.workgroups >= (int64_t(1) << 31) || main_tiles >= (int64_t(1) << 31) - kCUs)
            return TL_EUNSUPPORTED;
        // split_k reports the K splits of the remaining columns' tiles
        p.pub.split_k = p.split_rest ? p.split_rest : 1;
        p.pub.workspace_bytes = p.split_rest ? int64_t(p.split_rest) * M * (N - p.n_main) * 4 : 0;
    }
    *P = p;
    return TL_OK;
}

// A grouped launch runs the decode kernel over every group's weight with
// 4-wave workgroups, one per (group, tile) and no K split; the group row
// bound only chooses the 16-row M tiles per pass (larger groups take more
// passes over their weights).
int plan_grouped(int64_t max_group_rows, int64_t N, int64_t K, const tl_layout_desc* d, int32_t fetch_mode,
                 Plan* P) {
    if (!d || max_group_rows < 1) return TL_EINVAL;
    if (d->split_k < 0 || d->tile_m < 0) return TL_EINVAL;
    if (d->split_k > 1 || d->tile_m > kDecodeMaxM) return TL_EUNSUPPORTED;
    tl_layout_desc d1 = *d;
    d1.split_k = 1;
    int rc = plan_gemm(std::min<int64_t>(max_group_rows, kDecodeMaxM), N, K, &d1, fetch_mode, P);
    if (rc != TL_OK) return rc;
    if (P->pub.kernel != 1 || P->block_row || P->fp8 || P->kn_row) return TL_EUNSUPPORTED;
    // A 32-row tile of a short weight (K < 1024: under 64 KB per tile, e.g. a
    // Qwen expert's down projection, K = 768) is little work per workgroup;
    // 64-row tiles halve the workgroups and their fixed costs (down: -3 %).
    if (!d->tile_n && P->pub.tile_n == 32 && K < 1024 && N % 64 == 0 &&
        (d->kind != TL_LAYOUT_TILE || P->L.br <= 64)) {
        P->pub.tile_n = 64;
        P->pub.workgroups = (N + 63) / 64;
    }
    P->waves = 4;
    P->pub.waves = 4;
    P->pub.workspace_bytes = 0;
    return TL_OK;
}

}  // namespace
}  // namespace tl

using namespace tl;

extern "C" {

int tl_repack(const void* src, void* dst, int64_t rows, int64_t cols, int32_t elem_bytes,
              int64_t G, int32_t block_rows, void* stream) {
    return do_repack(src, dst, rows, cols, elem_bytes, G, block_rows, stream, false);
}

int tl_unpack(const void* src_tm, void* dst, int64_t rows, int64_t cols, int32_t elem_bytes,
              int64_t G, int32_t block_rows, void* stream) {
    return do_repack(src_tm, dst, rows, cols, elem_bytes, G, block_rows, stream, true);
}

int tl_tile_bytes(int64_t rows, int64_t cols, int32_t elem_bytes, int64_t G, int32_t block_rows, int64_t* bytes) {
    Layout L;
    if (!bytes || rows < 0 || cols < 0) return TL_EINVAL;
    if (make_tile_layout(elem_bytes, G, block_rows, &L) != TL_OK) return TL_EINVAL;
    if (cols > kMaxElems || (cols > 0 && rows > kMaxElems / cols)) return TL_EINVAL;
    *bytes = rows == 0 || cols == 0 ? 0 : packed_bytes(L, rows, cols);
    return TL_OK;
}

int tl_gemm_plan(int64_t M, int64_t N, int64_t K, const tl_layout_desc* layout, int32_t fetch_mode,
                 tl_plan* out) {
    if (!out) return TL_EINVAL;
    Plan p;
    int rc = plan_gemm(M, N, K, layout, fetch_mode, &p);
    if (rc != TL_OK) return rc;
    *out = p.pub;
    return TL_OK;
}

// noalloc: split-K partials in the static scratch (tl_scratch.hip), no
// library state (no workspace, no tally), nothing allocated.
static int gemm_impl(const void* A, const void* W, const float* scales, void* C, int64_t M, int64_t N, int64_t K,
                     const tl_layout_desc* layout, int32_t fetch_mode, void* stream, bool noalloc = false) {
    Plan p;
    int rc = plan_gemm(M, N, K, layout, fetch_mode, &p);
    if (rc != TL_OK) return rc;
    if (noalloc && p.count) return TL_EUNSUPPORTED;
    if (noalloc && p.pub.workspace_bytes > kScratchBytes) return TL_ESCRATCH;
    if (!A || !W || !C || !aligned16(A) || !aligned16(W) || !aligned16(C)) return TL_EINVAL;
    if (scales && (reinterpret_cast<uintptr_t>(scales) & 3u)) return TL_EINVAL;
    const int64_t c_bytes = M * N * (p.out_bf16 ? 2 : 4);
    const int64_t w_bytes = layout->kind == TL_LAYOUT_TILE ? packed_bytes(p.L, N, K) : N * K * layout->elem_bytes;
    if (overlap(C, c_bytes, A, M * K * 2) || overlap(C, c_bytes, W, w_bytes)) return TL_EINVAL;
    if (scales && overlap(C, c_bytes, scales, N * 4)) return TL_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    StateRef st;
    if (noalloc) {
        if (p.pub.workspace_bytes > 0 && scratch_address(&st.ws) != hipSuccess) return TL_EHIP;
    } else {
        rc = get_state(s, size_t(p.pub.workspace_bytes), &st);
        if (rc != TL_OK) return rc;
    }

    hipError_t e;
    if (p.pub.kernel == 1) {
        DecodeLaunch d;
        d.A = static_cast<const uint16_t*>(A);
        d.W = static_cast<const uint8_t*>(W);
        d.C = C;
        d.ws = st.ws;
        d.fetch = p.count ? st.fetch : nullptr;
        d.M = M;
        d.N = N;
        d.K = K;
        d.L = p.L;
        d.tile_n = p.pub.tile_n;
        d.m_tiles16 = p.m_tiles16;
        d.waves = p.waves;
        d.split_k = p.pub.split_k;
        d.k_unit = p.k_unit;
        d.out_bf16 = p.out_bf16;
        d.block_fetch = p.block_row;
        d.fetch_G = p.fetch_G;
        d.fp8 = p.fp8;
        d.scales = scales;
        d.lds_tiles = p.lds_tiles;
        e = launch_decode(d, s);
    } else {
        PrefillLaunch q;
        q.A = static_cast<const uint16_t*>(A);
        q.W = static_cast<const uint8_t*>(W);
        q.C = C;
        q.fetch = p.count ? st.fetch : nullptr;
        q.M = M;
        q.N = N;
        q.K = K;
        q.L = p.L;
        q.tile_m = p.pub.tile_m;
        q.tile_n = p.pub.tile_n;
        q.out_bf16 = p.out_bf16;
        q.n_main = p.n_main;
        q.block_fetch = p.block_row;
        q.fetch_G = p.fetch_G;
        q.split_rest = p.split_rest;
        q.ws = st.ws;
        q.persist = p.persist;
        e = launch_prefill(q, s);
    }
    return e == hipSuccess ? TL_OK : TL_EHIP;
}

// One grouped launch.  swiglu: every weight stacks gate rows [0, N) and up
// rows [N, 2N) and C receives silu(gate) * up, N columns.
static int grouped_impl(const void* A, int64_t a_rows, const int32_t* token_ids, const int32_t* group_offsets,
                        int32_t num_groups, int64_t total_rows, int64_t max_group_rows, const void* W,
                        int64_t group_stride, void* C, int64_t N, int64_t K, const tl_layout_desc* layout,
                        int32_t fetch_mode, void* stream, bool swiglu) {
    Plan p;
    if (swiglu && N > kMaxDim / 2) return TL_EINVAL;
    const int64_t w_rows = swiglu ? 2 * N : N;
    int rc = plan_grouped(max_group_rows, w_rows, K, layout, fetch_mode, &p);
    if (rc != TL_OK) return rc;
    if (swiglu) {
        // a tile is 32 gate rows + the 32 matching up rows: whole memory-tile
        // strips when block_rows divides 32
        if (N % 32 || (layout->kind == TL_LAYOUT_TILE && 32 % p.L.br)) return TL_EUNSUPPORTED;
        p.pub.tile_n = 64;
    }
    if (num_groups < 1 || total_rows < 0 || a_rows < 1) return TL_EINVAL;
    if (total_rows >= (int64_t(1) << 31) || a_rows >= (int64_t(1) << 31)) return TL_EINVAL;
    if (!token_ids && a_rows < total_rows) return TL_EINVAL;
    // 32-bit byte offsets inside the kernel: A, and the rows one tile reads
    // (gate and up halves together for swiglu)
    if (a_rows * K * 2 >= (int64_t(1) << 31)) return TL_EUNSUPPORTED;
    if (swiglu && 2 * N * (layout->kind == TL_LAYOUT_TILE ? padded_cols(p.L, K) : K) * 2 >= (int64_t(1) << 31))
        return TL_EUNSUPPORTED;
    const int64_t one_w = layout->kind == TL_LAYOUT_TILE ? packed_bytes(p.L, w_rows, K) : w_rows * K * 2;
    if (group_stride < one_w || group_stride % 16) return TL_EINVAL;
    if (!A || !W || !C || !group_offsets || !aligned16(A) || !aligned16(W) || !aligned16(C)) return TL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(group_offsets) & 3u) || (reinterpret_cast<uintptr_t>(token_ids) & 3u))
        return TL_EINVAL;
    const int64_t tiles = swiglu ? N / 32 : (N + p.pub.tile_n - 1) / p.pub.tile_n;
    if (int64_t(num_groups) * tiles >= (int64_t(1) << 31)) return TL_EUNSUPPORTED;
    if (total_rows == 0) return TL_OK;
    const int64_t c_bytes = total_rows * N * (p.out_bf16 ? 2 : 4);
    const int64_t w_bytes = (int64_t(num_groups) - 1) * group_stride + one_w;
    if (overlap(C, c_bytes, A, a_rows * K * 2) || overlap(C, c_bytes, W, w_bytes)) return TL_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    StateRef st;
    rc = get_state(s, 0, &st);
    if (rc != TL_OK) return rc;
    DecodeLaunch d;
    d.A = static_cast<const uint16_t*>(A);
    d.W = static_cast<const uint8_t*>(W);
    d.C = C;
    d.ws = nullptr;
    d.fetch = p.count ? st.fetch : nullptr;
    d.M = std::min<int64_t>(max_group_rows, kDecodeMaxM);
    d.N = N;
    d.K = K;
    d.L = p.L;
    d.tile_n = p.pub.tile_n;
    d.m_tiles16 = p.m_tiles16;
    d.waves = 4;
    d.split_k = 1;
    d.k_unit = p.k_unit;
    d.out_bf16 = p.out_bf16;
    d.block_fetch = false;
    d.fetch_G = 0;
    d.num_groups = num_groups;
    d.group_offsets = group_offsets;
    d.token_ids = token_ids;
    d.group_stride = group_stride;
    d.a_rows = a_rows;
    d.total_rows = total_rows;
    d.swiglu = swiglu;
    return launch_decode(d, s) == hipSuccess ? TL_OK : TL_EHIP;
}

int tl_gemm_grouped(const void* A, int64_t a_rows, const int32_t* token_ids, const int32_t* group_offsets,
                    int32_t num_groups, int64_t total_rows, int64_t max_group_rows, const void* W,
                    int64_t group_stride, void* C, int64_t N, int64_t K, const tl_layout_desc* layout,
                    int32_t fetch_mode, void* stream) {
    return grouped_impl(A, a_rows, token_ids, group_offsets, num_groups, total_rows, max_group_rows, W, group_stride,
                        C, N, K, layout, fetch_mode, stream, false);
}

int tl_gemm_grouped_swiglu(const void* A, int64_t a_rows, const int32_t* token_ids, const int32_t* group_offsets,
                           int32_t num_groups, int64_t total_rows, int64_t max_group_rows, const void* W_gate_up,
                           int64_t group_stride, void* H, int64_t I, int64_t K, const tl_layout_desc* layout,
                           int32_t fetch_mode, void* stream) {
    return grouped_impl(A, a_rows, token_ids, group_offsets, num_groups, total_rows, max_group_rows, W_gate_up,
                        group_stride, H, I, K, layout, fetch_mode, stream, true);
}

int tl_gemm(const void* A, const void* W, void* C, int64_t M, int64_t N, int64_t K,
            const tl_layout_desc* layout, int32_t fetch_mode, void* stream) {
    return gemm_impl(A, W, nullptr, C, M, N, K, layout, fetch_mode, stream);
}

int tl_gemm_noalloc(const void* A, const void* W, void* C, int64_t M, int64_t N, int64_t K,
                    const tl_layout_desc* layout, int32_t fetch_mode, void* stream) {
    return gemm_impl(A, W, nullptr, C, M, N, K, layout, fetch_mode, stream, true);
}

int tl_gemm_w8(const void* A, const void* W_fp8, const float* scales, void* C, int64_t M, int64_t N, int64_t K,
               const tl_layout_desc* layout, int32_t fetch_mode, void* stream) {
    if (!layout) return TL_EINVAL;
    if (layout->elem_bytes != 1) return TL_EINVAL;
    return gemm_impl(A, W_fp8, scales, C, M, N, K, layout, fetch_mode, stream);
}

int tl_prefetch_degree(double bandwidth, double latency, double bytes_per_iteration, int64_t k_iterations,
                       double collision_factor, int64_t* degree) {
    if (!degree || !(bandwidth > 0) || !(latency >= 0) || !(bytes_per_iteration > 0) || k_iterations < 0 ||
        !(collision_factor > 0))
        return TL_EINVAL;
    const double first = std::floor(collision_factor * bandwidth * latency / bytes_per_iteration);   // Eq. 6
    *degree = first < double(k_iterations) ? int64_t(first) : k_iterations;
    return TL_OK;
}

int tl_lgms_occupancy(int32_t steps_in_flight, int32_t* workgroups_per_cu) {
    if (!workgroups_per_cu) return TL_EINVAL;
    if (steps_in_flight != 1 && steps_in_flight != 2 && steps_in_flight != 4 && steps_in_flight != 8) return TL_EINVAL;
    const int n = lgms_ctas_per_cu(steps_in_flight);
    if (n < 0) return TL_EHIP;
    *workgroups_per_cu = n;
    return TL_OK;
}

int tl_gemm_lgms(const void* A, const void* W, void* C, int64_t M, int64_t N, int64_t K, const tl_layout_desc* layout,
                 int64_t latency_ns, int32_t steps_in_flight, void* stream) {
    if (!layout) return TL_EINVAL;
    if (steps_in_flight != 1 && steps_in_flight != 2 && steps_in_flight != 4 && steps_in_flight != 8) return TL_EINVAL;
    if (latency_ns < 0 || latency_ns > 1000000000) return TL_EINVAL;
    if (layout->kind != TL_LAYOUT_TILE || layout->elem_bytes != 2) return TL_EUNSUPPORTED;
    tl_layout_desc d1 = *layout;
    d1.tile_n = 32;
    d1.tile_m = 0;
    d1.split_k = layout->split_k;
    Plan p;
    int rc = plan_gemm(M, N, K, &d1, TL_FETCH_BLOCK, &p);
    if (rc != TL_OK) return rc;
    if (M > 16 || p.pub.kernel != 1) return TL_EUNSUPPORTED;
    if (N % 32 || K % 64 || N % p.L.br || K % p.L.bc) return TL_EUNSUPPORTED;   // no padded weights here
    if (!A || !W || !C || !aligned16(A) || !aligned16(W) || !aligned16(C)) return TL_EINVAL;
    const int64_t c_bytes = M * N * (p.out_bf16 ? 2 : 4);
    if (overlap(C, c_bytes, A, M * K * 2) || overlap(C, c_bytes, W, N * K * 2)) return TL_EINVAL;
    // 4-wave workgroups: split K until there are about 1024 of them
    const int64_t n_tiles = N / 32, units = K / p.k_unit;
    int64_t S = layout->split_k;
    if (S == 0) {
        S = (kTargetWorkgroups + n_tiles - 1) / n_tiles;
        S = std::max<int64_t>(1, std::min<int64_t>({S, units / std::max<int64_t>(1, 1024 / p.k_unit), kMaxSplitK}));
    }
    if (S < 1 || S > units || S > kMaxSplitK) return TL_EUNSUPPORTED;
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess) return TL_EHIP;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || khz <= 0) return TL_EHIP;
    const int64_t ticks = (latency_ns * int64_t(khz) + 999999) / 1000000;
    hipStream_t s = (hipStream_t)stream;
    StateRef st;
    rc = get_state(s, size_t(S > 1 ? S * ((M * N + 3) / 4 * 4) * 4 : 0), &st);
    if (rc != TL_OK) return rc;
    DecodeLaunch dl;
    dl.A = static_cast<const uint16_t*>(A);
    dl.W = static_cast<const uint8_t*>(W);
    dl.C = C;
    dl.ws = st.ws;
    dl.fetch = nullptr;
    dl.M = M;
    dl.N = N;
    dl.K = K;
    dl.L = p.L;
    dl.tile_n = 32;
    dl.m_tiles16 = 1;
    dl.waves = 4;
    dl.split_k = int(S);
    dl.k_unit = p.k_unit;
    dl.out_bf16 = p.out_bf16;
    dl.block_fetch = false;
    dl.fetch_G = 0;
    return launch_lgms(dl, ticks, steps_in_flight, s) == hipSuccess ? TL_OK : TL_EHIP;
}

int tl_view_offsets(const tl_view* view, int64_t K, int64_t N, int32_t elem_bytes, int64_t G, int32_t block_rows,
                    int64_t* offsets, int64_t capacity, int64_t* count) {
    ViewProgram P;
    int rc = make_view_program(view, K, N, elem_bytes, G, block_rows, &P);
    if (rc != TL_OK) return rc;
    if (count) *count = P.elements;
    if (!offsets) return TL_OK;
    if (capacity < P.elements) return TL_EINVAL;
    for (int64_t e = 0; e < P.elements; ++e) offsets[e] = view_offset(P, e);
    return TL_OK;
}

int tl_view_load(const void* src_tm, const tl_view* view, int64_t K, int64_t N, int32_t elem_bytes, int64_t G,
                 int32_t block_rows, void* dst, void* stream) {
    ViewProgram P;
    int rc = make_view_program(view, K, N, elem_bytes, G, block_rows, &P);
    if (rc != TL_OK) return rc;
    if (!src_tm || !dst || !aligned16(src_tm) || !aligned16(dst)) return TL_EINVAL;
    const int64_t src_bytes = N * K * elem_bytes, dst_bytes = P.elements * elem_bytes;
    if (overlap(src_tm, src_bytes, dst, dst_bytes)) return TL_EINVAL;
    hipError_t e = launch_view_load(static_cast<const uint8_t*>(src_tm), src_bytes, P, static_cast<uint8_t*>(dst),
                                    (hipStream_t)stream);
    return e == hipSuccess ? TL_OK : TL_EHIP;
}

int tl_stream_read(const void* src, int64_t bytes, uint32_t* checksum, void* stream) {
    if (!checksum || (reinterpret_cast<uintptr_t>(checksum) & 3u)) return TL_EINVAL;
    if (bytes < 0 || bytes % 16 || bytes >= (int64_t(1) << 48)) return TL_EINVAL;
    if (bytes > 0 && (!src || !aligned16(src) || overlap(src, bytes, checksum, 4))) return TL_EINVAL;
    hipError_t e = launch_stream_read(static_cast<const uint8_t*>(src), bytes, checksum, (hipStream_t)stream);
    return e == hipSuccess ? TL_OK : TL_EHIP;
}

int tl_fetch_counter_read(void* stream, int64_t* bytes) {
    if (!bytes) return TL_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    StateRef st;   // holds the tally's buffer for the rest of this call
    int rc = get_state(s, 0, &st);
    if (rc != TL_OK) return rc;
    unsigned long long v = 0;
    if (hipStreamSynchronize(s) != hipSuccess) return TL_EHIP;
    if (hipMemcpy(&v, st.fetch, sizeof v, hipMemcpyDeviceToHost) != hipSuccess) return TL_EHIP;
    if (launch_zero_u64(st.fetch, s) != hipSuccess) return TL_EHIP;
    if (hipStreamSynchronize(s) != hipSuccess) return TL_EHIP;
    *bytes = int64_t(v);
    return TL_OK;
}

int tl_release(void) {
    // the states leave the map under the lock; their buffers are freed when
    // the last call still holding one returns (here, when none does)
    std::map<std::pair<int, void*>, std::shared_ptr<StreamState>> old;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        old.swap(g_state);
    }
    old.clear();
    return TL_OK;
}

const char* tl_strerror(int status) {
    switch (status) {
        case TL_OK: return "TL_OK: success";
        case TL_EINVAL: return "TL_EINVAL: invalid argument";
        case TL_EUNSUPPORTED: return "TL_EUNSUPPORTED: no kernel implements this combination";
        case TL_EHIP: return "TL_EHIP: HIP runtime or launch failure";
        case TL_ENOMEM: return "TL_ENOMEM: workspace allocation failed";
        case TL_ESCRATCH: return "TL_ESCRATCH: the split-K partials exceed the static scratch (TL_NOALLOC_SCRATCH_BYTES)";
        default: return "unknown tl_status";
    }
}

}  // extern "C"
