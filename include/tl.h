/*
 * tl.h -- C ABI of libtl: GEMMs over weights stored in a tile-major layout,
 * for AMD Instinct MI355X (gfx950).
 *
 * Method: TileLens (arxiv 2607.04031).  A large-granularity memory returns a
 * whole G-byte block (e.g. 4 KB) per request.  In a row- or column-major
 * weight each block is a 1-D strip that mostly falls outside the 2-D compute
 * tile that asked for it: read amplification (Sections 1 and 2.5).  The
 * tile-major layout reshapes every contiguous G-byte block into a 2-D
 * "memory tile" of block_rows x block_cols elements (Section 3.1) so that a
 * compute tile whose sides are multiples of the memory tile's sides uses
 * every byte it fetches.  Kernels that compute their own addresses adopt the
 * layout by replacing their address arithmetic with the shifts and masks of
 * Eq. 1 and Eq. 2 (Sections 3.2 and 4.4); the kernels behind this ABI do so.
 *
 * Conventions (every entry point):
 *  - A GEMM weight is logically W[N][K] (outputs x inputs, the orientation of
 *    a linear layer's weight).  The paper's "column-major K x N" weight is
 *    this matrix stored row-major (TL_LAYOUT_NK_ROW); its "row-major" weight
 *    is TL_LAYOUT_KN_ROW (Section 2.4).
 *  - Sizes are element counts unless the name says bytes; G is in bytes.
 *  - Device pointers are allocated and owned by the caller, must be 16-byte
 *    aligned, and must stay valid until the work enqueued on 'stream' has
 *    finished.  The library never frees caller memory.
 *  - 'stream' is a hipStream_t passed as void*; NULL is the null stream.
 *  - Every call returns a tl_status.  All arguments are checked on the host
 *    before anything is enqueued; on an error nothing is enqueued.  A fault
 *    inside a kernel surfaces at the caller's next synchronisation.
 *  - Calls are thread-safe.  The library owns, per (device, stream), a split-K
 *    workspace and a fetch counter; concurrent calls on the SAME stream from
 *    several host threads are serialised by the stream, as usual.  A
 *    workspace that must grow is replaced by a larger one and the old one is
 *    kept (not freed) until tl_release, so work already enqueued or captured
 *    with it stays valid.
 *  - HIP graphs: the GEMM and repack calls enqueue kernels only (no memset or
 *    copy nodes) and may be captured, once the stream's library state exists:
 *    the first call on a stream, and a call that needs a larger split-K
 *    workspace than any before it on that stream, allocate device memory
 *    (hipMalloc) and must be made outside capture.  A captured graph binds
 *    the capture stream's workspace as it was at capture time: replay it on
 *    that stream (or serialised with it), never concurrently with split-K
 *    calls on that stream, and not after tl_release.  tl_fetch_counter_read
 *    synchronises its stream and cannot be captured.
 */
#ifndef TL_H_
#define TL_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TL_OK = 0,
    TL_EINVAL = -1,        /* an argument violates the contract below */
    TL_EUNSUPPORTED = -2,  /* valid, but no kernel implements this combination */
    TL_EHIP = -3,          /* a HIP runtime call or a launch failed */
    TL_ENOMEM = -4,        /* the library could not allocate its workspace */
    TL_ESCRATCH = -5       /* tl_gemm_noalloc: the call needs more split-K
                              scratch than TL_NOALLOC_SCRATCH_BYTES */
} tl_status;

/* Storage layout of a weight that is logically W[N][K]. */
typedef enum {
    TL_LAYOUT_NK_ROW = 0,  /* W[N][K] row-major: K contiguous (paper: column-major) */
    TL_LAYOUT_KN_ROW = 1,  /* stored as [K][N] row-major: N contiguous (paper: row-major) */
    TL_LAYOUT_TILE = 2     /* tile-major, the output of tl_repack(W, rows=N, cols=K) */
} tl_layout_kind;

typedef enum { TL_OUT_F32 = 0, TL_OUT_BF16 = 1 } tl_out_dtype;

/* fetch_mode of tl_gemm. */
enum {
    TL_FETCH_NATIVE = 0,   /* load what the compute tile needs, 16 B per lane */
    TL_FETCH_BLOCK = 1,    /* whenever a byte of an aligned G-byte block (aligned
                              relative to the weight's base) is needed, load the
                              whole block: emulates a large-granularity memory
                              on HBM (Sections 2.2 and 2.5) */
    TL_FETCH_COUNT = 0x100 /* OR-able: tally weight bytes into this stream's
                              fetch counter.  With BLOCK on a row- or
                              column-major weight: G per whole block the
                              kernel loads (counted as it loads them).
                              Otherwise: the bytes of the weight load
                              instructions of every K step the kernel issues
                              (a construction check that each byte is loaded
                              once; HBM traffic itself is what a hardware
                              counter such as FETCH_SIZE measures) */
};

/* Layout descriptor: the memory-tile shape travels as a runtime argument, so
 * one library binary serves every memory-tile shape (Sections 1 and 4.3). */
typedef struct tl_layout_desc {
    int32_t kind;        /* tl_layout_kind */
    int32_t elem_bytes;  /* element size s in bytes; tl_gemm: 2 (bf16) or 1 (FP8 E4M3) */
    int64_t G;           /* TL_LAYOUT_TILE: memory-tile size in bytes (power of
                            two).  *_ROW with TL_FETCH_BLOCK: the emulated fetch
                            block.  Otherwise ignored. */
    int32_t block_rows;  /* TL_LAYOUT_TILE: rows of W (along N) per memory tile,
                            paper b, a power of two.  block_cols (paper a, along
                            K) = G / (elem_bytes * block_rows). */
    int32_t out_dtype;   /* tl_gemm: tl_out_dtype of C */
    int32_t tile_m;      /* tl_gemm: requested compute tile, 0 = library's */
    int32_t tile_n;      /*   choice; see tl_gemm_plan for what is accepted */
    int32_t tile_k;
    int32_t split_k;     /* tl_gemm: K-splits across workgroups (decode kernel,
                            1..16), 0 = library's choice; partial sums are
                            reduced in a fixed order, so results are bitwise
                            reproducible */
} tl_layout_desc;

/* Read-amplification report (tl_read_amp). */
typedef struct tl_amp {
    int64_t compute_tiles;        /* (m-tile, n-tile, k-step) triples */
    int64_t requests;             /* G-byte block fetches, summed over all of them */
    int64_t fetched_bytes;        /* requests * G */
    int64_t useful_bytes;         /* weight bytes the tiles need (ceil(M/tile_m) * N*K*s) */
    int64_t unique_blocks;        /* distinct blocks touched by the whole GEMM */
    int64_t min_blocks_per_tile;  /* fewest / most blocks one (n-tile, k-step) touches */
    int64_t max_blocks_per_tile;
    double amp;                   /* fetched_bytes / useful_bytes */
} tl_amp;

/* What tl_gemm will launch for given arguments (tl_gemm_plan). */
typedef struct tl_plan {
    int32_t kernel;      /* 1 = decode (skinny, M <= 64), 2 = prefill (MFMA tiles; also 33 <= M <= 64 on wide weights) */
    int32_t tile_m;      /* compute tile used by the kernel; with tile_k it is  */
    int32_t tile_n;      /* the tile to pass to tl_read_amp to account for the  */
    int32_t tile_k;      /* kernel's fetches                                     */
    int32_t split_k;     /* workgroups per output tile along K (prefill: > 1
                            when 256 x 256 tiles -- 128 x 128 at M <= 128 --
                            are fewer than the CUs and all columns run with
                            K split, or when the
                            columns past the whole rounds of 256 x 256 tiles
                            do; fp32 partials summed in a fixed order) */
    int32_t waves;       /* wavefronts per workgroup (decode: 4, 8 or 16; the
                            waves of a workgroup also split K, reduced in LDS) */
    int64_t workgroups;  /* grid size, summed over the call's launches (a
                            persistent prefill grid: at most 256) */
    int64_t workspace_bytes;  /* split-K partials the call needs from the library */
} tl_plan;

/*
 * tl_tile_bytes -- host only: *bytes = size of the tile-major copy of a
 * rows x cols matrix, ceil(rows / br) * ceil(cols / bc) memory tiles of G
 * bytes (br = block_rows, bc = G / (elem_bytes * br)).  Equals
 * rows * cols * elem_bytes when br divides rows and bc divides cols, the
 * paper's assumption (Section 3.3); otherwise the copy is padded to whole
 * memory tiles, the remedy the same section names.  0 for an empty matrix.
 * Errors: TL_EINVAL for a NULL bytes, negative sizes, rows * cols > 2^40 or
 * a bad (elem_bytes, G, block_rows) (see tl_repack).
 */
int tl_tile_bytes(int64_t rows, int64_t cols, int32_t elem_bytes, int64_t G, int32_t block_rows,
                  int64_t* bytes);

/*
 * tl_repack -- row-major -> tile-major (Eq. 2, Section 3.2).
 *
 * src: device, rows x cols elements of elem_bytes each, row-major (cols
 *      contiguous).  For a GEMM weight rows = N and cols = K.
 * dst: device, tl_tile_bytes(rows, cols, ...) bytes, written in tile-major
 *      order: element (r, c) goes to byte
 *        ((r / br) * ceil(cols / bc) + c / bc) * G + ((r % br) * bc + c % bc) * s
 *      with br = block_rows, bc = G / (s * br), s = elem_bytes.  Memory tiles
 *      follow one another along cols inside each strip of br rows.  When br
 *      does not divide rows or bc does not divide cols, the last strip and the
 *      last memory tile of every strip are padded (Section 3.3): their bytes
 *      outside the matrix are written as zeros.
 * The copy moves bytes only (dtype-agnostic); weights are repacked once, when
 * they are loaded (Section 5.1).
 * Errors: TL_EINVAL unless elem_bytes in {1,2,4,8}; G and block_rows powers of
 * two with elem_bytes * block_rows <= G <= 2^30; rows * cols <= 2^40; src,
 * dst non-NULL, 16-byte aligned, and not overlapping; TL_EUNSUPPORTED for a
 * copy of 2^32 memory tiles or more.  Empty matrices (rows == 0 or cols == 0)
 * are a no-op.
 */
int tl_repack(const void* src, void* dst, int64_t rows, int64_t cols, int32_t elem_bytes,
              int64_t G, int32_t block_rows, void* stream);

/* tl_unpack -- the inverse permutation of tl_repack, same contract: src_tm
 * holds tl_tile_bytes bytes (its padding is not read), dst rows x cols
 * elements row-major. */
int tl_unpack(const void* src_tm, void* dst, int64_t rows, int64_t cols, int32_t elem_bytes,
              int64_t G, int32_t block_rows, void* stream);

/*
 * tl_gemm -- C[M][N] = A[M][K] * W^T, fp32 accumulation (Section 2.3: a tiled
 * GEMM whose workgroups iterate along K, loading a weight tile per step).
 *
 * A:   device bf16, row-major [M][K] (lda = K).  Activations are read from HBM
 *      as usual; only the weight lives in the large-granularity layout
 *      (Section 5.1).
 * W:   device bf16 weight in the layout layout->kind describes; tile-major:
 *      the tl_tile_bytes bytes tl_repack wrote, padded when N or K is not a
 *      multiple of the memory tile's sides (Section 3.3) -- any N and K.
 * C:   device, row-major [M][N] (ldc = N), fp32 or bf16 (round to nearest
 *      even) per layout->out_dtype.  C must not overlap A or W.
 * fetch_mode: TL_FETCH_NATIVE or TL_FETCH_BLOCK, optionally | TL_FETCH_COUNT.
 *      For TL_LAYOUT_TILE both modes load whole memory tiles (the compute tile
 *      is a whole number of memory tiles).  For TL_LAYOUT_NK_ROW and
 *      TL_LAYOUT_KN_ROW, BLOCK loads every layout->G-byte block a K step
 *      touches, whole (G a power of two, 128 <= G <= 2^30; NK_ROW in both
 *      kernels, without the prefill plan's column split; KN_ROW in the
 *      decode kernel): the amplification of Section 2.5 paid as real HBM
 *      traffic, and the blocks loaded are counted by TL_FETCH_COUNT.
 * TL_LAYOUT_KN_ROW (W stored [K][N], N contiguous: the paper's row-major
 * layout) runs a decode kernel (M <= 64) that loads each 64-row K step of a
 * 64-column tile with whole 128-byte lines and transposes it through LDS
 * into MFMA operands; it needs K % 64 == 0, N % 8 == 0 (N % 64 == 0 with
 * BLOCK) and N < 2^27.
 * M <= 64 runs the decode kernel (skinny GEMM, HBM-bound; at 17 <= M <= 32
 * on tile-major weights whose 32-row tiles and 512-column K chunks fill the
 * CUs in whole rounds, and at 33 <= M <= 64 where groups of four such tiles
 * and the K ranges fill at least 7/8 of one round, a variant that stages the
 * activations in LDS and shares them across several tiles) -- except that
 * at 33 <= M <= 64 a bf16
 * weight read natively with N >= 32768 (its 128x128 tiles fill the CUs), no
 * tile or split requested and the prefill kernel's limits met, takes the
 * prefill kernel's 128x128 tiles; larger M runs the prefill kernels (bf16
 * MFMA tiles 256x256x64, 256x320x64, 256x128x64 or 128x128x64, MFMA-bound;
 * with bf16 output, whole 256x256 tiles and K % 128 == 0 a persistent grid of
 * at most 256 workgroups walks the tiles, and 256x320 tiles replace them
 * where those fill the CUs in whole rounds and 256x256 tiles do not; when
 * 256x256 tiles would leave the last round of workgroups part-empty, the
 * columns past the whole rounds take 256x256 tiles with K split across
 * workgroups, or 128x128 tiles; when 256x256 tiles are fewer than the CUs
 * (and K % 64 == 0, N % 256 == 0), every column takes them with K split, up
 * to 8 ways -- at M <= 128, 128x128 tiles with K split when those are fewer
 * than the CUs (N % 128 == 0); see tl_gemm_plan).  layout->elem_bytes = 1 means an FP8 weight (OCP E4M3, one
 * byte per element, e.g. 64 x 64 memory tiles of 4 KB, Section 3.1): decode
 * kernel only, converted exactly to bf16 in registers (see tl_gemm_w8 for
 * per-channel scales).
 * Errors: TL_EINVAL for M, N, K < 1, NULL or misaligned pointers, a bad
 * descriptor (see tl_repack), or a bad G for NK_ROW with TL_FETCH_BLOCK;
 * TL_EUNSUPPORTED for elem_bytes other than 1 or 2, K not a multiple of
 * 16 / elem_bytes (one 16-byte load: keeps rows of A 16-byte aligned),
 * block_cols * elem_bytes < 16, a combination of layout, fetch mode and tile
 * that no kernel implements (NK_ROW with BLOCK with FP8, or with K % 64 or
 * N % 32 != 0; FP8 above 64 rows; KN_ROW above 64 rows, with
 * FP8, or outside the shape rules above), or sizes
 * past the kernels' 32-bit byte offsets: for M <= 64, 2 * M * K or the bytes
 * of tile_n weight rows (tile_n * K * elem_bytes, K padded for tile-major)
 * of 2^31 or more; above 64 rows, A or W of 2^32 bytes or more, or more
 * than 2^31 - 1 workgroups.  M, N or K above 2^30: TL_EINVAL.
 * TL_ENOMEM if the split-K workspace cannot be allocated; TL_EHIP if the
 * launch fails.
 */
int tl_gemm(const void* A, const void* W, void* C, int64_t M, int64_t N, int64_t K,
            const tl_layout_desc* layout, int32_t fetch_mode, void* stream);

/*
 * tl_gemm_w8 -- weight-only 8-bit decode: C[m][n] = scales[n] *
 * sum_k A[m][k] * W[n][k], with W an FP8 weight (OCP E4M3: sign, 4 exponent
 * bits with bias 7, 3 mantissa bits, no infinities, S.1111.111 = NaN) in the
 * layout 'layout' describes (layout->elem_bytes must be 1; tile-major with
 * e.g. 64 x 64 memory tiles of 4 KB, or TL_LAYOUT_NK_ROW), A bf16.  scales:
 * device fp32 [N] or NULL (all 1).  Each weight byte is converted exactly to
 * bf16 and the products accumulate in fp32 as in tl_gemm.  M <= 64.
 * Errors: TL_EINVAL for layout->elem_bytes != 1, misaligned scales, scales
 * overlapping C, and what tl_gemm rejects with TL_EINVAL; TL_EUNSUPPORTED as
 * tl_gemm.
 */
int tl_gemm_w8(const void* A, const void* W_fp8, const float* scales, void* C, int64_t M, int64_t N,
               int64_t K, const tl_layout_desc* layout, int32_t fetch_mode, void* stream);

/* tl_gemm_plan -- host only: fill *out with what tl_gemm would launch for the
 * same arguments (no device work).  Same error rules as tl_gemm. */
int tl_gemm_plan(int64_t M, int64_t N, int64_t K, const tl_layout_desc* layout,
                 int32_t fetch_mode, tl_plan* out);

/*
 * tl_gemm_grouped -- one launch over a stack of weights that each serve their
 * own rows: the expert GEMMs of a mixture-of-experts layer, whose decode-time
 * kernel (fused_moe) is the paper's main workload (Sections 2.3 and 6.2).
 * For every group e in [0, num_groups) and every output row r in
 * [group_offsets[e], group_offsets[e+1]):
 *      C[r][n] = sum_k A[t][k] * W_e[n][k],   t = token_ids ? token_ids[r] : r
 * with W_e at W + e * group_stride bytes, each in the layout 'layout'
 * describes (TL_LAYOUT_TILE or TL_LAYOUT_NK_ROW, repacked one by one).
 *
 * A:             device bf16 [a_rows][K] row-major.
 * token_ids:     device int32 [total_rows] or NULL (row r reads A row r; then
 *                a_rows >= total_rows).  An id outside [0, a_rows) reads a
 *                row of zeros.
 * group_offsets: device int32 [num_groups + 1], nondecreasing, from 0 to
 *                total_rows; read by the kernel, clamped to [0, total_rows].
 *                Out-of-order offsets give unspecified rows of C, never an
 *                access outside A, W or C.
 * max_group_rows: host bound on the rows of one group; it picks the kernel's
 *                M tile (16, 32 or 64 rows).  A group with more rows is
 *                processed in several passes over its weight (correct, more
 *                traffic).
 * W:             device, group_stride bytes apart (a multiple of 16, at least
 *                one weight: tl_tile_bytes for tile-major, N * K * 2 else).
 * C:             device [total_rows][N] row-major, fp32 or bf16 per
 *                layout->out_dtype; rows of empty groups are not written.
 * Weights stream once per group and pass (4-wave workgroups, one per (group,
 * tile_n-row tile), K not split), so results match tl_gemm to rounding.
 * fetch_mode: as tl_gemm (TL_FETCH_BLOCK on NK_ROW is not supported here).
 * Errors: TL_EINVAL for num_groups < 1, total_rows < 0, a_rows < 1, rows
 * beyond 2^31 - 1, a short or misaligned group_stride, NULL or misaligned
 * pointers (offsets and ids 4-byte aligned), overlap of C with A or W, or a
 * descriptor tl_gemm rejects with TL_EINVAL; TL_EUNSUPPORTED for split_k > 1,
 * tile_m > 64, a_rows * K * 2 >= 2^31, and what tl_gemm rejects with
 * TL_EUNSUPPORTED.  total_rows == 0 enqueues nothing.
 */
int tl_gemm_grouped(const void* A, int64_t a_rows, const int32_t* token_ids,
                    const int32_t* group_offsets, int32_t num_groups, int64_t total_rows,
                    int64_t max_group_rows, const void* W, int64_t group_stride, void* C,
                    int64_t N, int64_t K, const tl_layout_desc* layout, int32_t fetch_mode,
                    void* stream);

/*
 * tl_gemm_grouped_swiglu -- the gated expert activation of a mixture-of-experts
 * layer fused into the grouped gate+up projection (the paper's fused_moe
 * workload, Sections 2.3 and 6.2).  Every group's weight W_e stacks its gate
 * projection (rows [0, I)) and its up projection (rows [I, 2I)) as one
 * [2I][K] matrix (tile-major: repacked as one matrix of 2I rows), and
 *      H[r][i] = silu(sum_k A[t][k] * W_e[i][k]) * sum_k A[t][k] * W_e[I + i][k]
 * for rows r of group e as in tl_gemm_grouped (t = token_ids[r] or r), with
 * silu(x) = x / (1 + e^-x) evaluated in fp32 on the fp32 sums.  H: device
 * [total_rows][I] row-major, fp32 or bf16 per layout->out_dtype.  Every
 * workgroup reads 32 gate rows and the 32 matching up rows -- whole memory
 * tiles when block_rows divides 32 -- so the [total_rows][2I] projection is
 * never written.  Arguments, ownership and errors as tl_gemm_grouped with
 * N = I for C and 2I weight rows (group_stride >= the bytes of a [2I][K]
 * weight: tl_tile_bytes(2I, K, ...) for tile-major); in addition
 * TL_EUNSUPPORTED for I % 32 != 0, a tile-major block_rows that does not
 * divide 32, or a [2I][K] weight of 2^31 bytes or more; TL_EINVAL for
 * I > 2^29 (2I weight rows).
 */
int tl_gemm_grouped_swiglu(const void* A, int64_t a_rows, const int32_t* token_ids,
                           const int32_t* group_offsets, int32_t num_groups, int64_t total_rows,
                           int64_t max_group_rows, const void* W_gate_up, int64_t group_stride, void* H,
                           int64_t I, int64_t K, const tl_layout_desc* layout, int32_t fetch_mode,
                           void* stream);

/*
 * tl_read_amp -- host only, exact integer count of the bytes a tiled GEMM
 * fetches at granularity G (Sections 1, 2.5; the per-tile request counts of
 * Section 6.5).  Model: the grid has ceil(M/tile_m) x ceil(N/tile_n) tiles,
 * each iterating ceil(K/tile_k) K-steps; at each step a tile fetches every
 * G-byte block (aligned relative to the weight's base) holding at least one
 * element of its weight sub-tile (clipped at the matrix edge); nothing is
 * reused across tiles, steps or m-tiles; only the weight is counted
 * (Section 5.1).  layout->kind, elem_bytes and, for TILE, layout->G and
 * block_rows define byte offsets (a padded tile-major copy when the memory
 * tile does not divide N or K, as tl_repack writes it; useful bytes count the
 * N x K matrix only); G here is the memory system's granularity and may
 * differ from layout->G.  Other descriptor fields are ignored.
 * Errors: TL_EINVAL for non-positive sizes or tiles, G < 1 or G > 2^40,
 * N * K > 2^40, a bad TILE descriptor, NULL pointers, or a count past
 * 2^63 - 1; TL_EUNSUPPORTED when no closed form applies (non-power-of-two
 * tiles or G, ragged tiles, segments that straddle blocks) and the weight
 * spans more than 2^28 G-byte blocks (the exact enumerator's block table);
 * TL_ENOMEM if that table cannot be allocated.
 */
int tl_read_amp(int64_t M, int64_t N, int64_t K, int32_t tile_m, int32_t tile_n,
                int32_t tile_k, const tl_layout_desc* layout, int64_t G, tl_amp* out);

/*
 * tl_prefetch_degree -- host only, Eq. 6 (Section 5.3): the prefetch degree
 * that keeps a memory of the given bandwidth busy over the given read
 * latency when every K iteration of the resident workgroups demands
 * bytes_per_iteration bytes:
 *     d = min(floor(collision_factor * bandwidth * latency / bytes_per_iteration), k_iterations)
 * (requests of equal size make the request form and this byte form equal;
 * the paper uses collision_factor 2 for NAND plane collisions, 1 is the plain
 * equation).  Units: any consistent pair, e.g. bytes/s and s.
 * Errors: TL_EINVAL for NULL degree, bandwidth <= 0, latency < 0,
 * bytes_per_iteration <= 0, k_iterations < 0 or collision_factor <= 0.
 */
int tl_prefetch_degree(double bandwidth, double latency, double bytes_per_iteration, int64_t k_iterations,
                       double collision_factor, int64_t* degree);

/*
 * tl_gemm_lgms -- the decode GEMM of tl_gemm (M <= 16, tile-major weight,
 * 32-row compute tiles, 4-wave workgroups interleaved along K, K split across
 * workgroups until there are about 1024 of them unless layout->split_k says
 * otherwise) on an emulated large-granularity memory whose every read
 * completes no earlier than latency_ns after it is issued (Section 5.3's
 * microsecond-scale reads, imposed on HBM by waiting on the GPU's constant
 * clock).  Each wave keeps steps_in_flight (1, 2, 4 or 8) K steps of 64 of its
 * weight tile's loads outstanding: the prefetch degree d = steps_in_flight - 1
 * of Eq. 6 at workgroup granularity.  Same results as tl_gemm up to fp32
 * summation order.
 * Errors: TL_EINVAL for steps_in_flight not in {1, 2, 4, 8}, latency_ns
 * outside [0, 1e9], and what tl_gemm rejects with TL_EINVAL;
 * TL_EUNSUPPORTED for M > 16, a layout other than TL_LAYOUT_TILE,
 * block_rows > 32, a padded weight (N % 32, K % 64, N % block_rows or
 * K % block_cols != 0), or what tl_gemm rejects with it; TL_EHIP, TL_ENOMEM
 * as tl_gemm.
 */
int tl_gemm_lgms(const void* A, const void* W_tm, void* C, int64_t M, int64_t N, int64_t K,
                 const tl_layout_desc* layout, int64_t latency_ns, int32_t steps_in_flight, void* stream);

/* tl_lgms_occupancy -- resident tl_gemm_lgms workgroups per CU for a given
 * steps_in_flight (registers grow with it), to size Eq. 6's per-iteration
 * demand.  Errors: TL_EINVAL for a NULL pointer or a steps_in_flight not in
 * {1, 2, 4, 8}; TL_EHIP if the occupancy query fails. */
int tl_lgms_occupancy(int32_t steps_in_flight, int32_t* workgroups_per_cu);

/* A multi-dimensional view of a weight, as a TMA descriptor would give it
 * (Section 4.3): the K x N weight (K contiguous: W[N][K] row-major, the
 * paper's column-major K x N) seen as a tensor of rank 'rank' whose
 * dimension d advances strides[d] elements (strides[0] = 1, the contiguous
 * dimension; a stride >= K is a whole number of columns, K apart), and a box
 * of box[0] x ... x box[rank-1] elements starting at coords. */
#define TL_VIEW_MAX_RANK 5
typedef struct tl_view {
    int32_t rank;                         /* 1 .. TL_VIEW_MAX_RANK */
    int32_t box[TL_VIEW_MAX_RANK];        /* elements loaded per dimension (the TMA tile) */
    int64_t strides[TL_VIEW_MAX_RANK];    /* element strides; strides[0] = 1 */
    int64_t coords[TL_VIEW_MAX_RANK];     /* first element of the box per dimension */
} tl_view;

/*
 * tl_view_offsets -- host only: the byte offsets, from the weight's base, of
 * every element of the view's box in a tile-major weight (memory tile
 * G / (elem_bytes * block_rows) x block_rows, as tl_repack writes it), in
 * the order a TMA load visits them (dimension 0 fastest).  They are generated
 * the way TileLens-HW extends the TMA engine (Section 4.3): the tile base from
 * the split-and-sum of coordinate x stride products around the leading stride
 * K (Eq. 4), nested counters with the strides of Eq. 5, and for a box
 * narrower than the memory tile (Case 2) the bit permutation of the
 * intra-tile offset.  *count (if not NULL) receives the element count; with
 * offsets == NULL nothing else is written.
 * Errors: TL_EINVAL for a bad layout (see tl_repack), K % block_cols or
 * N % block_rows != 0, K * N > 2^40, rank outside 1..5, strides[0] != 1, a
 * non-positive stride or box, a negative coordinate, a stride >= K that is
 * not a multiple of K or above K * N, a box reaching outside the K x N
 * matrix, or capacity < count;
 * TL_EUNSUPPORTED when the view breaks the invariants the hardware relies on:
 * box[0] not a power of two, a box not starting on a memory-tile boundary, a
 * row-index stride that is not a whole number of memory tiles, or a column
 * stride that splits a memory tile other than the one-column stride K.
 */
int tl_view_offsets(const tl_view* view, int64_t K, int64_t N, int32_t elem_bytes, int64_t G,
                    int32_t block_rows, int64_t* offsets, int64_t capacity, int64_t* count);

/*
 * tl_view_load -- device: the TMA-like load of the view's box from a
 * tile-major weight.  src_tm: device, the N x K weight as tl_repack wrote it.
 * dst: device, receives count * elem_bytes bytes, the box's elements densely
 * in view order (dimension 0 fastest).  Source addresses are computed on the
 * GPU by the same generator as tl_view_offsets.  Both pointers 16-byte
 * aligned, not overlapping.  Errors: those of tl_view_offsets, TL_EINVAL for
 * NULL, misaligned or overlapping pointers, TL_EHIP if the launch fails.
 */
int tl_view_load(const void* src_tm, const tl_view* view, int64_t K, int64_t N, int32_t elem_bytes,
                 int64_t G, int32_t block_rows, void* dst, void* stream);

/*
 * tl_stream_read -- the HBM read ceiling the GEMM kernels are measured
 * against (the decode path is bound by reading every weight byte once,
 * Section 2.1): reads the 'bytes' bytes at src once, with the decode kernel's
 * load pattern (64 lanes x 16 B, whole 128-byte lines, non-temporal), and
 * XORs its little-endian 32-bit words into *checksum (the caller clears it;
 * unchanged for bytes = 0), so the reads cannot be elided and the result is
 * checkable.  src: device, 16-byte aligned; bytes: a multiple of 16, < 2^48;
 * checksum: device uint32, 4-byte aligned, not inside src.  One kernel
 * enqueued on 'stream' (none for bytes = 0).
 * Errors: TL_EINVAL for NULL or misaligned pointers, bytes < 0, not a
 * multiple of 16 or too large, or checksum inside src; TL_EHIP if a launch
 * fails.
 */
int tl_stream_read(const void* src, int64_t bytes, uint32_t* checksum, void* stream);

/* Bytes of the static device scratch behind tl_gemm_noalloc, per GPU. */
#define TL_NOALLOC_SCRATCH_BYTES ((int64_t)64 << 20)

/*
 * tl_gemm_noalloc -- for callers that cannot allocate device memory: code
 * under HIP graph capture, serving loops and harnesses that forbid hipMalloc.
 * Same arguments, plan, kernels and results as tl_gemm, except that the
 * split-K partials go to a static device array of TL_NOALLOC_SCRATCH_BYTES
 * bytes (64 MiB) instead of the stream's library workspace.  The array
 * belongs to the library's code object: every GPU the library runs on holds
 * its own copy from the first use until the process ends.  This call
 * allocates and frees nothing (no hipMalloc, no library state); its first
 * call on a device looks up the array's device address
 * (hipGetSymbolAddress), so make that first call outside graph capture if
 * the capture mode forbids runtime queries.
 * Every call on a GPU shares that GPU's array, and the array keeps the last
 * call's contents (nothing in it needs to start at zero: every K split writes
 * its whole partial before the reduce kernel reads it).  Calls that overlap
 * on one GPU -- on two streams, or from two host threads -- race on the
 * array and give unspecified results: serialise them (one stream, or events).
 * A plan without K splits (split_k 1: most prefill plans, and most
 * M = 1..16 calls on large weights) does not touch the array.
 * Errors: those of tl_gemm (except TL_ENOMEM); TL_ESCRATCH when the plan's
 * split-K partials (tl_gemm_plan's workspace_bytes) exceed
 * TL_NOALLOC_SCRATCH_BYTES -- layout->split_k can ask for fewer splits;
 * TL_EUNSUPPORTED with TL_FETCH_COUNT (the tally is per-stream library
 * state); TL_EHIP if the address lookup or a launch fails.
 */
int tl_gemm_noalloc(const void* A, const void* W, void* C, int64_t M, int64_t N, int64_t K,
                    const tl_layout_desc* layout, int32_t fetch_mode, void* stream);

/* tl_fetch_counter_read -- synchronises 'stream', stores the weight bytes
 * tallied by tl_gemm calls made on it with TL_FETCH_COUNT since the last read
 * into *bytes, and resets the tally to zero.  Errors: TL_EINVAL for NULL
 * bytes; TL_EHIP if a HIP call fails. */
int tl_fetch_counter_read(void* stream, int64_t* bytes);

/* tl_release -- frees every workspace (current and retired) and counter the
 * library holds (all devices, all streams); a call still running in another
 * thread keeps its own buffers until it returns.  The caller must ensure no
 * library work is still in flight on the GPU and replays no graph captured
 * before it.  Always TL_OK. */
int tl_release(void);

/* tl_strerror -- static, NUL-terminated description of a tl_status. */
const char* tl_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* TL_H_ */
