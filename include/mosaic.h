/*
 * mosaic.h -- C ABI of the MI355X (gfx950) MosaicKV hot path.
 *
 * MosaicKV (arXiv 2607.00760) keeps a long-context KV cache compressed in two
 * dimensions.  Every K/V vector is rotated by its window's SVD rotation and
 * keeps only its top-r elements (stage 1, Sec. 4.2).  Decode scores
 * mean-of-block keys against the query and attends only the top-k blocks
 * (stage 2, Sec. 4.2).  Each 64-token segment gets its own strategy: kept
 * channels r, element group size g, token block size B (Sec. 4.3, Sec. 5.5).
 * The strategy is stored in the packed KV format: packed values plus a
 * position bitmap (Sec. 5.1).
 *
 * Conventions for every entry point:
 *  - Pointers are DEVICE pointers unless the name ends in _host.
 *  - The caller allocates and owns all device memory: inputs, the cache arena,
 *    workspaces and outputs.  It keeps them alive until the enqueued work
 *    completes.  The library never allocates device memory.  Only
 *    mosaic_cache_stats and mosaic_window_poll synchronize.
 *  - `stream` is a hipStream_t (NULL = the null stream).  All work is enqueued
 *    on it, in order.
 *  - Validation happens before anything is enqueued.  On error nothing is
 *    launched, the cache is unchanged, and mosaic_last_error() describes the
 *    cause.
 *  - head_dim is 128.  K, V and q share one element type: fp16 or bf16,
 *    little-endian 16-bit.  Outputs are fp32.
 *  - A cache holds num_seqs sequences x num_kv_heads kv heads.  Query head h
 *    of a sequence reads kv head h / group_size (GQA).
 */
#ifndef MOSAIC_H
#define MOSAIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MOSAIC_OK = 0,
    MOSAIC_ERR_INVALID = -1,     /* bad argument (NULL, shape, alignment, parameter) */
    MOSAIC_ERR_UNSUPPORTED = -2, /* valid request outside what this build implements */
    MOSAIC_ERR_CAPACITY = -3,    /* more tokens than the cache was created for */
    MOSAIC_ERR_STATE = -4,       /* call out of order (e.g. decode before compress) */
    MOSAIC_ERR_HIP = -5          /* a HIP runtime call failed */
} mosaic_status;

typedef enum { MOSAIC_FP16 = 0, MOSAIC_BF16 = 1 } mosaic_dtype;

/* Method parameters.  The strategy set is Sec. 4.3: rotation, compression
 * rate, element group size, sequence compression rate, token block size.
 * The candidates are those of Sec. 5.5 (rates 87.5/75/62.5 % -> r = 16/32/48
 * of 128 channels, g = 1/2/4, B = 4/8/16).  The defaults are those of
 * Sec. 6.1 (25 % channels, block 8, 10 % of tokens). */
typedef struct {
    int32_t head_dim;          /* D, must be 128 */
    int32_t num_kv_heads;      /* Hkv >= 1 */
    int32_t group_size;        /* G = query heads per kv head, 1..8 */
    int32_t dtype;             /* mosaic_dtype */
    int32_t seg_len;           /* S: strategy segment length, must be 64 */
    int32_t rot_window;        /* W: tokens sharing one rotation, multiple of S */
    int32_t update_buf;        /* U: update-buffer tokens (Sec. 5.3), must be 32 */
    int32_t keep_cand[3];      /* r candidates, tried in this order; multiple of g, <= 128 */
    int32_t group_cand[3];     /* g candidates in {1, 2, 4}, tried in this order per r */
    int32_t block_cand[3];     /* B candidates in {4, 8, 16}, tried in this order */
    int32_t default_keep;      /* strategy of a provisional chunk with no finalized */
    int32_t default_group;     /*   predecessor, and of every segment when */
    int32_t default_block;     /*   force_default_strategy is set */
    float tau_channel;         /* accept (r, g) if dropped energy < tau * energy, K and V */
    float tau_block;           /* accept B if intra-block key variance < tau * energy */
    int32_t select_num;        /* rho = select_num / select_den: tokens selected per */
    int32_t select_den;        /*   (sequence, kv head) >= ceil(rho * scoreable tokens) */
    int32_t force_default_strategy; /* 1: skip the search, use the default */
    int32_t trunc_channels;    /* T: channels represented in the bitmaps (Sec. 5.2 channel
                                  truncation: after the rotation the last D - T channels are
                                  never kept and get no bitmap bit: a bitmap is T / g bits);
                                  32, 64, 96 or 128, at least every kept count.  128 = no
                                  truncation */
    int32_t value_fp8;         /* 1: the kept values of the K and V token records are stored as
                                  OCP FP8 E4M3 codes (Sec. 7: the compressed elements can be
                                  quantized further), one byte each, each the nearest code to
                                  the fp32 rotated value (ties to the even code, saturating at
                                  +-448, no scale factor); every kept count must then be a
                                  multiple of 4.  Block keys, the update buffer and the staging
                                  area keep the 16-bit dtype.  0 = 16-bit values */
    int32_t dyn_windows;       /* 1: windows of decode tokens close on their accumulated
                                  compression loss (Sec. 4.3 dynamic partitioning of output
                                  tokens, Sec. 5.5 incremental strategy generation; see
                                  mosaic_window_poll); needs rotated = 1.  0: every window
                                  holds rot_window tokens */
    float tau_window;          /* summed segment loss above which a window closes */
    int32_t min_window;        /* tokens a window holds at least before it closes on its
                                  loss; a multiple of 64 in [64, rot_window] (rot_window is
                                  the maximum window length) */
} mosaic_params;

/* Fills *p with the paper's defaults (Sec. 5.5, Sec. 6.1): r in {16, 32, 48},
 * g in {4, 2, 1}, B in {16, 8, 4}, default (32, 1, 8), S = 64, U = 32,
 * W = 65536, tau = (0.30, 0.90), rho = 1/10, fp16, 8 kv heads, G = 4,
 * T = 128 (no truncation), 16-bit values, fixed windows (dyn_windows = 0;
 * tau_window = 8, min_window = 1024 when enabled). */
void mosaic_params_default(mosaic_params *p);

typedef struct mosaic_cache mosaic_cache;  /* host bookkeeping + bound arena */

/* Creates the host side of a cache for num_seqs sequences of up to max_tokens
 * tokens each.  rotated = 1 if mosaic_compress will receive rotation matrices
 * (Sec. 2.3); 0 for the identity rotation.  The handle owns host memory
 * only.  With dyn_windows the cache holds max(ceil(max_tokens / W),
 * max_tokens / min_window + 1) rotation windows per pair.  Errors: INVALID
 * (parameters; dyn_windows without rotation), UNSUPPORTED (head_dim != 128,
 * S != 64, U != 32, more than 1024 windows), CAPACITY (a per-(sequence,
 * kv head) arena would exceed 4 GiB). */
mosaic_status mosaic_cache_create(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                  int32_t rotated, mosaic_cache **out);

/* The same with a capacity per sequence (max_tokens_host[num_seqs], each >= 1):
 * the descriptor, score and token regions of each (sequence, kv head) pair are
 * sized for its own sequence, so ragged batches do not reserve the longest
 * sequence's worst case for every pair.  Rotation windows, workspaces and the
 * other regions are sized for the longest.  Compress and append check each
 * sequence against its own capacity.  The pair regions' offsets are then not a
 * multiple of a stride (mosaic_cache_pair_regions). */
mosaic_status mosaic_cache_create_ragged(const mosaic_params *params, int32_t num_seqs,
                                         const int32_t *max_tokens_host, int32_t rotated, mosaic_cache **out);

/* Bytes of device memory the cache needs (worst case over strategies).  The
 * caller allocates it, 256-byte aligned, and binds it once. */
mosaic_status mosaic_cache_arena_bytes(const mosaic_cache *cache, size_t *bytes);
mosaic_status mosaic_cache_bind(mosaic_cache *cache, void *arena, size_t bytes);
mosaic_status mosaic_cache_destroy(mosaic_cache *cache);

/* Where each region lives inside the bound arena.  Every region holds one
 * slot per (sequence, kv head) pair p = seq * num_kv_heads + kv_head, at
 * off + p * stride.  Use it for inspection (tests, stats); the layout of a
 * region's contents is the packed format of Sec. 5.1:
 *   meta     : int32 tokens, int32 finalized blocks, uint32 token-arena
 *              bytes, uint32 score-arena bytes (finalized segments); with
 *              dyn_windows also int32 windows in use, fp32 loss summed in
 *              the open window, int32 window awaiting its rotation (-1:
 *              none), and from byte 64 the window table: int32
 *              [num_windows + 1] first segment of each window in use
 *   desc     : 16-byte segment descriptors {uint32 token-arena offset,
 *              uint32 score-arena offset, uint32 first block, uint8 r,
 *              uint8 log2 g, uint8 log2 B, uint8 flags (bit 0 provisional)}
 *   score    : block-key records [bitmap T/(8g) B][r values], block order
 *   token    : per block [K bitmaps][K values][V bitmaps][V values]
 *   buffer   : update buffer [2 (K, V)][U][D] raw elements (Sec. 5.3)
 *   stage    : raw tokens of the trailing segment [2][S][D] (Sec. 5.4)
 *   rot      : per window {R_k^T, R_v^T, R_v} fp32 [3][D][D]
 *   cov      : (dyn_windows) fp64 [2][2][D][D]: in slot w % 2 the uncentered
 *              covariance X^T X of window w's K (then V) tokens, updated
 *              segment by segment as segments are finalized (Sec. 5.5
 *              incremental covariance); a closed window's stays in its slot
 *              until the window after next accumulates, so it can be read
 *              after mosaic_window_poll to compute the window's rotation.
 *              Entry (i, j) is the fp64 sum over each segment's tokens in
 *              order of x[i] x[j], added to the window's running entry.
 */
typedef struct {
    uint64_t meta_off, meta_stride;
    uint64_t desc_off, desc_stride;
    uint64_t score_off, score_stride;
    uint64_t token_off, token_stride;
    uint64_t buf_off, buf_stride;
    uint64_t stage_off, stage_stride;
    uint64_t rot_off, rot_stride;
    uint64_t total;
    int32_t num_pairs, max_desc, num_windows, reserved;
    uint64_t cov_off, cov_stride;   /* dyn_windows only (else 0) */
    uint64_t pairs_off;             /* uint64 [num_pairs][4] device copy of the pair table below
                                       (written by mosaic_compress; the kernels locate the pair
                                       regions through it) */
} mosaic_layout;
mosaic_status mosaic_cache_layout(const mosaic_cache *cache, mosaic_layout *out);

/* Per pair p: out_host[4 p + 0..2] = byte offsets of its desc, score and token
 * regions from desc_off, score_off and token_off, [4 p + 3] = its token region's
 * bytes.  For caches of one capacity these are p * stride and token_stride; for
 * ragged capacities (mosaic_cache_create_ragged) desc_stride, score_stride and
 * token_stride are 0 and only this table locates the regions.  out_host holds
 * 4 * num_pairs entries. */
mosaic_status mosaic_cache_pair_regions(const mosaic_cache *cache, uint64_t *out_host);

enum { MOSAIC_OP_COMPRESS = 0, MOSAIC_OP_APPEND = 1, MOSAIC_OP_DECODE = 2, MOSAIC_OP_WINDOW_ROTATIONS = 3 };
/* Workspace bytes an operation can use (0 if none).  Depends only on the
 * cache's shape and capacity, so one allocation serves every call.  DECODE
 * requires its workspace; COMPRESS's is optional (see mosaic_compress): a
 * worst-case slot of packed records per (pair, segment). */
mosaic_status mosaic_workspace_bytes(const mosaic_cache *cache, int32_t op, size_t *bytes);

/* Layout of the decode workspace (inspection): per pair p,
 *   qrot  + p * qrot_stride  : fp32 [windows][D][GP] rotated queries
 *   score + p * score_stride : fp32 [max_blocks] block scores
 *   sel   + p * sel_stride   : int32 [max_blocks] selected blocks, ascending
 *   wsel  + p * wsel_stride  : int32 [windows + 3]: first selected entry of
 *                              each window, then k, then the block count;
 *                              for pair 0 then the call's selected blocks
 *                              per split-K partition
 *   part  + p * part_stride  : fp32 [max_splits][GP * (D + 2)]: split-K
 *                              partials (max, sum, accumulator per head; a
 *                              window's splits hold it in the window's
 *                              rotated space, the buffer's split unrotated)
 *   tag   + p * tag_stride   : int32 [max_splits]: window of each split
 *                              (-1 the update buffer, -2 none)
 *   binfo + p * binfo_stride : uint32 [max_blocks][2]: per block, its
 *                              token-arena offset and r << 8 | log2 g << 16 |
 *                              log2 B << 20
 *   bsize + p * bsize_stride : uint8 [max_blocks]: per block, log2 B
 *   selinfo + p * selinfo_stride : uint32 [max_blocks][2]: binfo of each
 *                              entry of the selected list
 *   wres  + p * wres_stride  : fp32 [D / 16][windows + 1][GP][18]: for each
 *                              block of 16 output columns and each window
 *                              (the last slot: the update buffer), the
 *                              window's merged max and sum per head and its
 *                              back-rotated output columns
 * Calls that overlap on one workspace race; separate streams need separate
 * workspaces. */
typedef struct {
    uint64_t qrot_off, qrot_stride, score_off, score_stride, sel_off, sel_stride, wsel_off, wsel_stride;
    uint64_t part_off, part_stride, tag_off, tag_stride, binfo_off, binfo_stride, bsize_off, bsize_stride,
             selinfo_off, selinfo_stride, wres_off, wres_stride, total;
    int32_t max_blocks, max_splits, gp, reserved;
    uint64_t tkx_off, tkx_stride;   /* caches of more than 32768 blocks per pair: the
                                       selection's per-pair state (histograms of three
                                       radix passes, their states, per-chunk counts of
                                       4096 blocks); else 0 */
} mosaic_ws_layout;
mosaic_status mosaic_decode_ws_layout(const mosaic_cache *cache, mosaic_ws_layout *out);

/* Prefill compression (Sec. 5.2 compressed KV encoding; strategy Sec. 4.3).
 *   k, v      : [num_seqs][num_kv_heads][seq_stride][128], first
 *               ctx_lens_host[s] tokens of sequence s valid.
 *   rot_k/v   : [num_seqs][num_kv_heads][num_windows][128][128] fp32; row j
 *               is rotated channel j, so y = x . R^T (Sec. 2.3).  Window w
 *               covers tokens [w W, (w+1) W); num_windows = ceil(max_tokens
 *               / W).  NULL (both) iff the cache was created with rotated = 0.
 *               With dyn_windows the prefill's windows are these fixed ones;
 *               the window holding the first token after the full segments
 *               stays open for decode tokens (its rotation is the one given).
 *   Full segments get their own strategy.  The remaining ctx_len mod S tokens
 *   take the update path (buffer, provisional flush), as if appended.
 * Replaces any previous contents.
 *   ws        : NULL, or 16-byte aligned and at least
 *               mosaic_workspace_bytes(MOSAIC_OP_COMPRESS) bytes.  With it each
 *               token is rotated once: a segment is packed right after its
 *               strategy is chosen, into its slot of ws, and the records move
 *               to their offsets once all sizes are known.  With NULL the
 *               tokens are rotated twice (strategy pass, then packing pass)
 *               and nothing extra is needed.  Both give the same bytes.
 * Errors: STATE (not bound), CAPACITY (ctx_len > max_tokens),
 * INVALID (NULL, negative length, misaligned pointer, seq_stride < max ctx,
 * workspace too small). */
mosaic_status mosaic_compress(mosaic_cache *cache, const void *k, const void *v, int64_t seq_stride,
                              const int32_t *ctx_lens_host, const float *rot_k, const float *rot_v,
                              void *ws, size_t ws_bytes, void *stream);

/* Appends one token to every sequence (Sec. 5.3 update buffer; Sec. 5.4
 * heterogeneous double compression buffering).  k_new, v_new:
 * [num_seqs][num_kv_heads][128].  When a sequence's buffer reaches U tokens,
 * they are compressed with the previous finalized segment's strategy, as a
 * provisional chunk.  When its trailing segment reaches S tokens, the
 * segment gets its own strategy and is recompressed in place.
 * Errors: STATE (not compressed yet; with dyn_windows, a poll or a close is
 * due first: see mosaic_window_poll), CAPACITY (a sequence is full). */
mosaic_status mosaic_append(mosaic_cache *cache, const void *k_new, const void *v_new, void *stream);

/* Windows closed by their compression loss (Sec. 4.3: output tokens are
 * partitioned dynamically, a segment being closed once its compression loss
 * passes a threshold, with a maximum length; Sec. 5.5: the loss of each new
 * token compares its channel-compressed vectors with the original ones, and
 * the closed segment's rotation comes from its covariance).  For caches
 * created with dyn_windows = 1.  Every segment completed by mosaic_append
 * adds its loss -- the larger of K's and V's relative dropped energy under
 * the provisional strategy it was compressed with -- to the open window's
 * sum.  After that segment the window closes if it holds rot_window tokens,
 * or if the sum exceeds tau_window and it holds at least min_window tokens;
 * the next segment opens a window whose provisional rotation is the closed
 * window's.  A closed window keeps its provisional encoding until
 * mosaic_window_close gives it its own rotation.
 *
 * mosaic_window_poll synchronizes `stream`, then reports for every pair p
 * (= seq * num_kv_heads + kv_head) the window awaiting its rotation:
 *   out_host[3 p]     : its index, -1 if none
 *   out_host[3 p + 1] : its first token
 *   out_host[3 p + 2] : its token count (a multiple of 64)
 * and in *n_closed_host the number of such pairs.  Protocol: after an append
 * that completed a segment, a poll must precede the next append that
 * compresses an update buffer, and a window it reports must be closed before
 * its sequence's buffer is compressed again (at most 32 appends later);
 * mosaic_append fails with STATE, changing nothing, until then.  Decode may
 * run at any time.  Errors: INVALID (NULL; no dynamic windows), STATE (not
 * compressed). */
mosaic_status mosaic_window_poll(mosaic_cache *cache, int32_t *out_host, int32_t *n_closed_host, void *stream);

/* Rotations of the windows the last poll reported, on the GPU, from their
 * incremental covariances (Sec. 5.5: with the covariance kept up to date the
 * closed segment's rotation follows directly from it): each K and V
 * covariance is cast to fp32 and solved by the cyclic Jacobi eigensolver of
 * mosaic_compute_rotations (rows by descending eigenvalue, each signed so that
 * its largest-magnitude component is positive).
 *   rot_k, rot_v : [num_seqs][num_kv_heads][128][128] fp32 outputs, in the
 *                  layout mosaic_window_close takes; pairs with nothing to
 *                  close get the identity.
 *   ws           : at least mosaic_workspace_bytes(MOSAIC_OP_WINDOW_ROTATIONS)
 *                  bytes, 256-byte aligned.
 * Errors: INVALID (NULL, misaligned, small workspace, no dynamic windows),
 * STATE (a segment completed since the last poll). */
mosaic_status mosaic_window_rotations(mosaic_cache *cache, float *rot_k, float *rot_v, void *ws, size_t ws_bytes,
                                      void *stream);

/* Closes every window the last poll reported.
 *   rot_k, rot_v : [num_seqs][num_kv_heads][128][128] fp32: each such pair's
 *                  rotation of its closed window (row j = rotated channel j),
 *                  e.g. the eigenvectors of the window's K (V) covariance by
 *                  descending eigenvalue; other pairs' entries are not read.
 *   k, v         : [num_seqs][num_kv_heads][seq_stride][128] the closed
 *                  windows' raw tokens (cache dtype), row 0 = the window's
 *                  first token; seq_stride >= the longest closed window.
 * The rotation replaces the window's provisional one and becomes the
 * provisional rotation of the window the close opened; every segment of the
 * closed window is encoded again from its tokens with its own strategy (two
 * passes: strategy, then packing), in place (it is the last compressed
 * window).  Nothing to close: OK, nothing enqueued.  Errors: INVALID (NULL,
 * misaligned, seq_stride too small, no dynamic windows), STATE (a segment
 * completed since the last poll). */
mosaic_status mosaic_window_close(mosaic_cache *cache, const float *rot_k, const float *rot_v, const void *k,
                                  const void *v, int64_t seq_stride, void *stream);

/* One decode step of PackedAttention (Sec. 5.3) for every sequence.  Steps:
 * rotate q into each window (rotation merged into the query), score every
 * block key (max over the GQA group's heads), select per (sequence, kv head)
 * blocks in (score desc, block index asc) order while fewer than
 * ceil(rho * scoreable tokens) tokens are taken (Sec. 4.2 stage 2; Sec. 6.1
 * selects 10 % of tokens), attend the selected blocks' packed K/V plus the
 * uncompressed update-buffer tokens, and rotate each window's output back
 * with its R_v.
 *   q   : [num_seqs][num_kv_heads * group_size][128] (cache dtype)
 *   out : [num_seqs][num_kv_heads * group_size][128] fp32
 *   sm_scale: softmax scale (e.g. 1/sqrt(128)).
 *   ws  : at least mosaic_workspace_bytes(MOSAIC_OP_DECODE) bytes.
 * A sequence with no tokens gets a zero output.
 * Errors: STATE, INVALID (NULL, small workspace). */
mosaic_status mosaic_decode_attention(mosaic_cache *cache, const void *q, float *out, float sm_scale,
                                      void *ws, size_t ws_bytes, void *stream);

/* mosaic_decode_attention for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same step and output, with the decode workspace taken
 * from a fixed library-owned device buffer of MOSAIC_NOALLOC_SCRATCH_BYTES
 * per GPU instead of a caller's.  The buffer is reserved when the library's
 * code is loaded on a GPU and held until the process ends; the call itself
 * allocates nothing.  Every call on one GPU shares that GPU's buffer: calls
 * that overlap on a GPU (other streams or threads) race and must be ordered
 * by the caller.  The cache must be bound to memory of the current device.
 * Errors: as mosaic_decode_attention; UNSUPPORTED when the cache's decode
 * workspace (mosaic_workspace_bytes, MOSAIC_OP_DECODE) exceeds the buffer;
 * HIP if the buffer's address cannot be obtained. */
#define MOSAIC_NOALLOC_SCRATCH_BYTES (64u << 20)
mosaic_status mosaic_decode_attention_noalloc(mosaic_cache *cache, const void *q, float *out, float sm_scale,
                                              void *stream);

/* Rotation matrices computed from the cache on the GPU (Sec. 2.3; Sec. 5.2:
 * once the KV cache exists, the SVD rotation of each window's K matrix and of
 * its V matrix is computed; the paper does this on the host).  For every
 * (sequence, kv head) and window w, R's rows are the eigenvectors of the
 * uncentered covariance X^T X of the window's vectors X (tokens
 * [w W, min((w + 1) W, ctx_len))), by descending eigenvalue, each signed so
 * that its largest-magnitude component is positive.  A window past the last
 * token repeats the last window that has tokens; a sequence with no token
 * gets the identity.  The output is what mosaic_compress takes as rot_k/v.
 *   params        : num_kv_heads, dtype, rot_window W (a multiple of 64)
 *   k, v          : as for mosaic_compress ([num_seqs][num_kv_heads][seq_stride][128])
 *   ctx_lens_host : [num_seqs], each <= max_tokens
 *   rot_k, rot_v  : outputs [num_seqs][num_kv_heads][ceil(max_tokens / W)][128][128] fp32
 *   evals_k/v     : optional outputs (both or neither) [...][ceil(max_tokens / W)][128]
 *                   fp32, the eigenvalues in row order (descending)
 *   ws            : at least mosaic_rotation_workspace_bytes bytes, 16-byte aligned
 * Arithmetic: fp32 covariance (exact 16-bit products, one chain per element
 * in token order per 4096-token slice, slices summed in order), cyclic Jacobi
 * in fp32 until the off-diagonal energy is below 1e-14 of the diagonal's.
 * Errors: INVALID (NULL, misaligned, bad shape, small workspace), CAPACITY
 * (a context longer than max_tokens), UNSUPPORTED (head_dim != 128). */
mosaic_status mosaic_rotation_workspace_bytes(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                              size_t *bytes);
mosaic_status mosaic_compute_rotations(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                       const void *k, const void *v, int64_t seq_stride,
                                       const int32_t *ctx_lens_host, float *rot_k, float *rot_v, float *evals_k,
                                       float *evals_v, void *ws, size_t ws_bytes, void *stream);

/* Selection-pattern channel reorder (Sec. 5.5 asks for the rotated channels to be
 * reordered so that channels with similar selection patterns become neighbours,
 * without fixing a procedure; this is the one taken here).  For every rotation
 * window of every (sequence, kv head), K and V apart: each of the window's tokens
 * selects its default_keep largest magnitudes (y = x . R^T by the compressor's own
 * fp32 chain, lowest channel first on ties); n[c] counts the tokens selecting c and
 * C[i][j] those selecting both i and j.  The rows of the window's R are then
 * permuted in place, in groups of four: a group starts with the unplaced channel of
 * the largest n (lowest on ties) and three times takes the unplaced channel with the
 * largest sum of C over the group so far, then the larger n, then the lower channel.
 * A window without tokens takes the order of the last window with tokens; the
 * windows of a sequence without tokens are left alone.  Eigenvalues returned by
 * mosaic_compute_rotations keep the old row order.
 *   k, v, seq_stride, ctx_lens_host, rot_k, rot_v: as mosaic_compute_rotations
 *                   (rot_k / rot_v are read and rewritten in place)
 *   ws            : at least mosaic_reorder_workspace_bytes bytes, 256-byte aligned
 *                   (context lengths, every token's 16-byte selection mask, the
 *                   co-selection counts, transposed copies of R)
 * Errors: INVALID (NULL, misaligned, bad shape, small workspace, default_keep out
 * of 1..128), CAPACITY (a context longer than max_tokens), UNSUPPORTED
 * (head_dim != 128). */
mosaic_status mosaic_reorder_workspace_bytes(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                             size_t *bytes);
mosaic_status mosaic_reorder_rotations(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                       const void *k, const void *v, int64_t seq_stride,
                                       const int32_t *ctx_lens_host, float *rot_k, float *rot_v, void *ws,
                                       size_t ws_bytes, void *stream);

/* Uncompressed baseline: dense split-K decode attention over K/V laid out as
 * for mosaic_compress (the "Full" baseline of Sec. 6.1).
 *   ctx_lens: DEVICE int32 [num_seqs].  ws: mosaic_dense_workspace_bytes. */
mosaic_status mosaic_dense_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t group_size,
                                           int32_t max_ctx, size_t *bytes);
mosaic_status mosaic_dense_decode_attention(const void *q, const void *k, const void *v, float *out,
                                            int32_t num_seqs, int32_t num_kv_heads, int32_t group_size,
                                            int32_t head_dim, int32_t dtype, int64_t seq_stride,
                                            int32_t max_ctx, const int32_t *ctx_lens, float sm_scale,
                                            void *ws, size_t ws_bytes, void *stream);

/* Memory accounting of Sec. 6.3 (reads the device state: synchronizes the
 * given stream).  used_bytes counts packed tokens, block keys, descriptors
 * and live buffer tokens; rotation matrices are reported apart. */
typedef struct {
    int64_t tokens;            /* sum of sequence lengths */
    int64_t dense_bytes;       /* 2 * tokens * 128 * 2 * num_kv_heads */
    int64_t used_bytes;
    int64_t rotation_bytes;    /* R_k and R_v of the windows in use, fp32 */
    int64_t segments;          /* finalized segments */
    int64_t strategy_hist[3][3][3]; /* finalized segments by (r, g, B) candidate index */
} mosaic_stats;
mosaic_status mosaic_cache_stats(const mosaic_cache *cache, mosaic_stats *out, void *stream);

/* Per-kernel timing of mosaic_decode_attention (tracing aid, Sec. 6.3's
 * Score / TopK / Attn breakdown).  With enable = 1, every later decode records
 * HIP events on its stream around each of its kernels (no device memory is
 * allocated).  mosaic_decode_timing waits for the last timed decode and writes
 * its kernel times in milliseconds to ms[0..4] = q rotation, block scoring,
 * top-k, split-K attention, reduce.  Errors: STATE (timing off or no decode
 * yet), HIP. */
mosaic_status mosaic_set_timing(mosaic_cache *cache, int32_t enable);
mosaic_status mosaic_decode_timing(mosaic_cache *cache, float *ms);

/* Host view of a sequence's length (no device access). */
int32_t mosaic_seq_tokens(const mosaic_cache *cache, int32_t seq);

/* Message of the last error on this thread ("" if none). */
const char *mosaic_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* MOSAIC_H */
