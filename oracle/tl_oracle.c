/*
 * CPU oracle for the tile-major GEMM path (TileLens, arxiv 2607.04031).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is built into liboracle.so and is
 * loaded by the tests, by the smoke check and by the benchmark's CPU-baseline
 * leg.  The product library never includes, links or calls anything here, and
 * this file includes nothing from the product library.
 *
 * Everything is written to be checked by eye against the paper:
 *   - integer work uses plain '/' and '%' (no shifts, no masks);
 *   - the GEMM is the textbook triple loop, summed in fp64, k ascending;
 *   - read amplification is a brute-force enumeration of the distinct
 *     G-byte blocks touched by every compute tile.
 *
 * Coordinates.  A weight is stored as W[rows][cols] with 'cols' the
 * contiguous dimension.  For a GEMM weight rows = N (output features) and
 * cols = K (reduction).  The paper (Section 3.2) describes a K x N
 * "column-major" matrix with element (i, j), i along K (contiguous) and j
 * along N; here c = i and r = j.  The memory tile is a x b elements with
 * a along the contiguous dimension: block_cols = a, block_rows = b,
 * a * b * s = G (Section 3.1).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

/* ---------------------------------------------------------------------- */
/* Layouts                                                                 */
/* ---------------------------------------------------------------------- */

enum { ORC_NK_ROW = 0, ORC_KN_ROW = 1, ORC_TILE = 2 };

/* Eq. 1 (tile indices) and Eq. 2 (tile-major byte offset), Section 3.2.
 *   T_i = i / a, i' = i mod a, T_j = j / b, j' = j mod b
 *   offset = (T_j * K/a + T_i) * (a*b*s) + (j' * a + i') * s
 * with i = c, j = r, K = cols, a = block_cols, b = block_rows.
 * Section 3.3: when a dimension is not a multiple of the memory tile's side
 * the weight is padded to whole memory tiles, so a strip of b rows holds
 * ceil(K / a) memory tiles (K / a when a divides K, the paper's case). */
int64_t orc_tm_offset(int64_t r, int64_t c, int64_t cols, int64_t s,
                      int64_t G, int64_t block_rows) {
    int64_t b = block_rows;
    int64_t a = G / (s * b);
    int64_t tiles_per_strip = (cols + a - 1) / a;
    int64_t Ti = c / a, ip = c % a;
    int64_t Tj = r / b, jp = r % b;
    return (Tj * tiles_per_strip + Ti) * (a * b * s) + (jp * a + ip) * s;
}

/* Bytes of the tile-major copy of a rows x cols matrix: whole memory tiles,
 * ceil(rows / b) strips of ceil(cols / a) tiles of G bytes (Section 3.3). */
int64_t orc_packed_bytes(int64_t rows, int64_t cols, int64_t s, int64_t G, int64_t block_rows) {
    int64_t b = block_rows;
    int64_t a = G / (s * b);
    return ((rows + b - 1) / b) * ((cols + a - 1) / a) * G;
}

/* Byte offset of logical weight element (n, k) of a logical W[N][K], for
 * each of the three storage layouts (Section 2.4 for the two linear ones). */
int64_t orc_elem_offset(int kind, int64_t n, int64_t k, int64_t N, int64_t K,
                        int64_t s, int64_t layout_G, int64_t block_rows) {
    if (kind == ORC_NK_ROW) return (n * K + k) * s;     /* K contiguous */
    if (kind == ORC_KN_ROW) return (k * N + n) * s;     /* N contiguous */
    return orc_tm_offset(n, k, K, s, layout_G, block_rows);
}

/* Row-major -> tile-major: every element moves from its row-major byte
 * offset to its Eq. 2 offset; the padding of partial memory tiles is zero
 * (dst holds orc_packed_bytes).  Plain definition, one element at a time. */
void orc_repack(const uint8_t* src, uint8_t* dst, int64_t rows, int64_t cols,
                int64_t s, int64_t G, int64_t block_rows) {
    memset(dst, 0, (size_t)orc_packed_bytes(rows, cols, s, G, block_rows));
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t c = 0; c < cols; ++c)
            memcpy(dst + orc_tm_offset(r, c, cols, s, G, block_rows),
                   src + (r * cols + c) * s, (size_t)s);
}

/* Tile-major -> row-major, the inverse permutation (padding is not read). */
void orc_unpack(const uint8_t* src, uint8_t* dst, int64_t rows, int64_t cols,
                int64_t s, int64_t G, int64_t block_rows) {
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t c = 0; c < cols; ++c)
            memcpy(dst + (r * cols + c) * s,
                   src + orc_tm_offset(r, c, cols, s, G, block_rows), (size_t)s);
}

/* A multi-dimensional view of a K x N column-major matrix (Section 4.3,
 * "Challenges of supporting tile-major in TMA"): dimension d has extent
 * dims[d] and element stride strides[d]; the box of box[0] x ... elements
 * starts at coords.  Elements are visited with dimension 0 fastest (the
 * order in which a TMA load writes its destination).  For each one the
 * view's linear element index lin = sum_d (coords[d] + x_d) * strides[d] is
 * the column-major index j * K + i of the matrix element, so i = lin mod K and
 * j = lin / K, and its tile-major byte offset is Eq. 2.  out[] receives one
 * offset per box element.  Returns the number of elements. */
int64_t orc_view_offsets(int rank, const int64_t* strides, const int64_t* coords,
                         const int64_t* box, int64_t K, int64_t s, int64_t G,
                         int64_t block_rows, int64_t* out) {
    int64_t x[8] = {0};
    int64_t n = 1;
    for (int d = 0; d < rank; ++d) n *= box[d];
    for (int64_t e = 0; e < n; ++e) {
        int64_t lin = 0;
        for (int d = 0; d < rank; ++d) lin += (coords[d] + x[d]) * strides[d];
        int64_t i = lin % K, j = lin / K;
        out[e] = orc_tm_offset(j, i, K, s, G, block_rows);
        /* next element: dimension 0 fastest */
        for (int d = 0; d < rank; ++d) {
            x[d] += 1;
            if (x[d] < box[d]) break;
            x[d] = 0;
        }
    }
    return n;
}

/* ---------------------------------------------------------------------- */
/* GEMM                                                                    */
/* ---------------------------------------------------------------------- */

/* bf16 is the upper half of an IEEE binary32; decoding is exact. */
static double orc_bf16_to_f64(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* y[m][n] = sum_{k=0}^{K-1} A[m][k] * W[n][k]  (Section 2.3: an M x K input
 * times the K x N weight).  A is row-major [M][K]; W is the ROW-MAJOR
 * original [N][K] (never the tile-major copy), so a layout bug on the device
 * side cannot cancel against one here.  fp64, k ascending, one output at a
 * time; OpenMP only splits the independent outputs, so the result does not
 * depend on the thread count. */
void orc_gemm_f64(const uint16_t* A, const uint16_t* W, double* Y,
                  int64_t M, int64_t N, int64_t K) {
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        const uint16_t* w = W + n * K;
        for (int64_t m = 0; m < M; ++m) {
            const uint16_t* a = A + m * K;
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k)
                acc += orc_bf16_to_f64(a[k]) * orc_bf16_to_f64(w[k]);
            Y[m * N + n] = acc;
        }
    }
}

/* Same definition on a list of output coordinates only (for spot checks of
 * full-size results): y[i] = sum_k A[m_i][k] * W[n_i][k]. */
/* OCP FP8 E4M3 byte -> value: sign bit, 4 exponent bits (bias 7), 3
 * mantissa bits; exponent 0 is subnormal (m / 8 * 2^-6); exponent 15 with
 * mantissa 7 is NaN; there are no infinities. */
double orc_fp8_e4m3(uint8_t v) {
    int sign = v / 128, e = (v / 8) % 16, m = v % 8;
    double mag;
    if (e == 15 && m == 7) return NAN;
    if (e == 0) mag = ldexp((double)m / 8.0, -6);
    else mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -mag : mag;
}

/* Weight-only 8-bit GEMM: Y[m][n] = scale[n] * sum_k A[m][k] * W8[n][k],
 * A bf16 row-major [M][K], W8 FP8 E4M3 row-major [N][K], scale NULL = 1;
 * fp64, k ascending. */
void orc_gemm_w8_f64(const uint16_t* A, const uint8_t* W8, const double* scale, double* Y,
                     int64_t M, int64_t N, int64_t K) {
    #pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
        for (int64_t m = 0; m < M; ++m) {
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k)
                acc += orc_bf16_to_f64(A[m * K + k]) * orc_fp8_e4m3(W8[n * K + k]);
            Y[m * N + n] = scale ? acc * scale[n] : acc;
        }
    }
}

/* SiLU (swish with beta = 1): silu(x) = x / (1 + e^-x). */
double orc_silu(double x) { return x / (1.0 + exp(-x)); }

/* Gated expert activation of a mixture-of-experts layer (the fused_moe
 * convention of the paper's main workload, Sections 2.3 and 6.2): with the
 * expert's gate and up projections stacked as W[2I][K] (rows [0, I) gate,
 * [I, 2I) up), H[m][i] = silu(sum_k A[m][k] W[i][k]) * sum_k A[m][k] W[I+i][k];
 * each sum in fp64, k ascending. */
void orc_swiglu_f64(const uint16_t* A, const uint16_t* W, double* H, int64_t M, int64_t I, int64_t K) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < I; ++i) {
        const uint16_t* wg = W + i * K;
        const uint16_t* wu = W + (I + i) * K;
        for (int64_t m = 0; m < M; ++m) {
            const uint16_t* a = A + m * K;
            double g = 0.0, u = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                g += orc_bf16_to_f64(a[k]) * orc_bf16_to_f64(wg[k]);
                u += orc_bf16_to_f64(a[k]) * orc_bf16_to_f64(wu[k]);
            }
            H[m * I + i] = orc_silu(g) * u;
        }
    }
}

void orc_gemm_f64_points(const uint16_t* A, const uint16_t* W,
                         const int64_t* ms, const int64_t* ns, double* y,
                         int64_t count, int64_t K) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const uint16_t* a = A + ms[i] * K;
        const uint16_t* w = W + ns[i] * K;
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k)
            acc += orc_bf16_to_f64(a[k]) * orc_bf16_to_f64(w[k]);
        y[i] = acc;
    }
}

/* Round a real number to bfloat16 (8 significant bits), ties to even, and
 * return the bf16 bit pattern.  Definition: write |x| = f * 2^e with f in
 * [0.5, 1), round f * 2^8 to an integer with ties to even, scale back. */
uint16_t orc_round_bf16(double x) {
    if (x == 0.0) return signbit(x) ? 0x8000u : 0u;
    int e;
    double f = frexp(fabs(x), &e);           /* |x| = f * 2^e */
    double q = f * 256.0;                    /* in [128, 256) */
    double fl = floor(q);
    double rem = q - fl;
    double r;
    if (rem > 0.5) r = fl + 1.0;
    else if (rem < 0.5) r = fl;
    else r = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
    double y = ldexp(r, e - 8);
    float yf = (float)y;                     /* exact: y has <= 9 significant bits */
    uint32_t u;
    memcpy(&u, &yf, sizeof u);
    uint16_t h = (uint16_t)(u >> 16);
    return x < 0 ? (uint16_t)(h | 0x8000u) : h;
}

void orc_round_bf16_array(const double* x, uint16_t* out, int64_t count) {
    for (int64_t i = 0; i < count; ++i) out[i] = orc_round_bf16(x[i]);
}

/* ---------------------------------------------------------------------- */
/* Read amplification                                                      */
/* ---------------------------------------------------------------------- */

typedef struct {
    int64_t compute_tiles;        /* (m-tile, n-tile, k-step) triples */
    int64_t requests;             /* G-byte blocks fetched, summed over tiles */
    int64_t fetched_bytes;        /* requests * G */
    int64_t useful_bytes;         /* weight bytes the tiles actually need */
    int64_t unique_blocks;        /* distinct blocks touched by the whole GEMM */
    int64_t min_blocks_per_tile;
    int64_t max_blocks_per_tile;
    double amp;                   /* fetched_bytes / useful_bytes */
} orc_amp;

/* Read amplification of a tiled GEMM C[M,N] = A[M,K] W^T whose weight lives
 * in a memory that can only be read in aligned G-byte blocks (Sections 1 and
 * 2.5: every request fetches a whole block; a compute tile cannot start until
 * all of its blocks have arrived).  Model: each compute tile fetches, at each
 * K-step, every block that holds at least one element of its weight sub-tile;
 * nothing is reused across tiles, K-steps or M-tiles.  Only the weight is
 * counted: activations stay in HBM (Section 5.1).  Blocks are aligned relative
 * to the matrix base (Section 3.3 assumes an aligned base).
 *
 * Brute force: for every (n-tile, k-step), visit every element of the clipped
 * weight sub-tile, map it to its block offset / G and count distinct blocks
 * with a per-tile stamp.  If brute_m != 0 the whole enumeration is repeated
 * for every m-tile; otherwise the count of one pass is multiplied by the
 * number of m-tiles (the weight sub-tile does not depend on the m-tile).
 *
 * Returns 0 on success, -1 on bad arguments or allocation failure. */
int orc_read_amp(int64_t M, int64_t N, int64_t K, int64_t tm, int64_t tn, int64_t tk,
                 int kind, int64_t s, int64_t layout_G, int64_t block_rows,
                 int64_t G, int brute_m, orc_amp* out) {
    if (M < 1 || N < 1 || K < 1 || tm < 1 || tn < 1 || tk < 1 || s < 1 || G < 1) return -1;
    /* bytes the stored weight spans: the padded copy for tile-major */
    int64_t total_bytes = kind == ORC_TILE ? orc_packed_bytes(N, K, s, layout_G, block_rows) : N * K * s;
    int64_t nblocks = (total_bytes + G - 1) / G;
    int64_t* stamp = (int64_t*)malloc((size_t)nblocks * sizeof(int64_t));
    uint8_t* seen = (uint8_t*)calloc((size_t)nblocks, 1);
    if (!stamp || !seen) { free(stamp); free(seen); return -1; }
    for (int64_t b = 0; b < nblocks; ++b) stamp[b] = -1;

    int64_t m_tiles = (M + tm - 1) / tm;
    int64_t n_tiles = (N + tn - 1) / tn;
    int64_t k_steps = (K + tk - 1) / tk;
    int64_t passes = brute_m ? m_tiles : 1;
    int64_t mult = brute_m ? 1 : m_tiles;

    int64_t requests = 0, useful = 0, unique = 0;
    int64_t bmin = -1, bmax = 0;
    int64_t tile_id = 0;
    for (int64_t p = 0; p < passes; ++p) {
        for (int64_t tn_i = 0; tn_i < n_tiles; ++tn_i) {
            int64_t n0 = tn_i * tn, n1 = n0 + tn < N ? n0 + tn : N;
            for (int64_t tk_i = 0; tk_i < k_steps; ++tk_i) {
                int64_t k0 = tk_i * tk, k1 = k0 + tk < K ? k0 + tk : K;
                int64_t count = 0;
                for (int64_t n = n0; n < n1; ++n) {
                    for (int64_t k = k0; k < k1; ++k) {
                        int64_t off = orc_elem_offset(kind, n, k, N, K, s, layout_G, block_rows);
                        int64_t blk = off / G;
                        if (stamp[blk] != tile_id) {
                            stamp[blk] = tile_id;
                            ++count;
                            if (!seen[blk]) { seen[blk] = 1; ++unique; }
                        }
                    }
                }
                requests += count * mult;
                useful += (n1 - n0) * (k1 - k0) * s * mult;
                if (bmin < 0 || count < bmin) bmin = count;
                if (count > bmax) bmax = count;
                ++tile_id;
            }
        }
    }
    free(stamp);
    free(seen);

    out->compute_tiles = m_tiles * n_tiles * k_steps;
    out->requests = requests;
    out->fetched_bytes = requests * G;
    out->useful_bytes = useful;
    out->unique_blocks = unique;
    out->min_blocks_per_tile = bmin;
    out->max_blocks_per_tile = bmax;
    out->amp = (double)out->fetched_bytes / (double)useful;
    return 0;
}
