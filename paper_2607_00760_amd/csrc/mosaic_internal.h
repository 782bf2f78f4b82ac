// mosaic_internal.h -- shared definitions of the gfx950 MosaicKV library
// (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mosaic {

constexpr int D = 128;        // head dim
constexpr int SEG = 64;       // strategy segment (tokens)
constexpr int UBUF = 32;      // update buffer (tokens)
constexpr int WAVE = 64;
// selected blocks per split-K partition: chosen per call between these bounds
// (the fewest sizes the per-pair partial arrays, the most the attention's
// block table)
constexpr int SPLIT_MIN = 48;
constexpr int SPLIT_MAX = 128;
constexpr int MAX_WINDOWS = 1024;  // rotation windows per sequence (the selection tracks them in LDS)
constexpr int SCORE_SEGS = 128;    // segments per block-scoring workgroup (one launch round)
constexpr int CMB_COLS = 16;                  // output columns per combine workgroup
constexpr int CMB_NCC = D / CMB_COLS;         // column blocks of an output row
constexpr int CMB_RES = 2 + CMB_COLS;         // floats per head of a window result: max, sum, columns

struct Desc {                 // 16-byte segment descriptor (layout is part of the ABI)
    uint32_t tok_off, sc_off, first_block;
    uint8_t r, log2g, log2b, flags;
};
static_assert(sizeof(Desc) == 16, "descriptor size");

struct PairMeta {             // per (sequence, kv head) device counters, 64 bytes
    int32_t L;                // tokens in the cache
    int32_t nblk_final;       // scoreable blocks of finalized segments
    uint32_t tok_tail;        // token-arena bytes of finalized segments
    uint32_t sc_tail;         // score-arena bytes of finalized segments
    // windows closed by their loss (caches with dynamic windows only; the
    // window table of int32 first segments follows this struct)
    int32_t nwin;             // windows in use; window nwin - 1 is open
    float wloss;              // accumulated loss of the open window
    int32_t pend;             // closed window awaiting its rotation, -1 none
    int32_t pad[9];
};
static_assert(sizeof(PairMeta) == 64, "meta size");

// Everything a kernel needs to find a pair's regions; passed by value.
struct Geom {
    int npairs, hkv, G, GP, dtype;
    int W, nw, cap, max_desc, rotated;
    uint8_t *meta, *desc, *sc, *tok;
    uint16_t *buf, *stg;
    float *rot;
    double *cov; uint64_t cov_stride;   // dynamic windows: [2][2][D][D] per pair
    const uint64_t *poff;               // [npairs][4]: desc, score, token offsets; token bytes
    uint64_t meta_stride, desc_stride, sc_stride, tok_stride, buf_stride, stg_stride, rot_stride;
    int keep_cand[3], group_cand[3], block_cand[3];
    int def_keep, def_group, def_block;
    float tau_ch, tau_blk;
    int sel_num, sel_den, force;
    int trunc;                        // channels represented in the bitmaps (T)
    int fp8;                          // K and V token values stored as E4M3 codes
    int dyn;                          // windows of decode tokens closed by their loss
    int min_win;                      // tokens a window holds before a loss close
    float tau_win;                    // accumulated loss that closes a window

    __host__ __device__ PairMeta *meta_of(int p) const { return (PairMeta *)(meta + (uint64_t)p * meta_stride); }
    // a pair's descriptor, score and token regions, from the pair table (one
    // read each; the table serves caches of one capacity and ragged ones alike)
    __host__ __device__ Desc *desc_of(int p) const { return (Desc *)(desc + poff[4 * p]); }
    __host__ __device__ uint8_t *sc_of(int p) const { return sc + poff[4 * p + 1]; }
    __host__ __device__ uint8_t *tok_of(int p) const { return tok + poff[4 * p + 2]; }
    __host__ __device__ uint64_t tok_size(int p) const { return poff[4 * p + 3]; }
    __host__ __device__ uint16_t *buf_of(int p) const { return (uint16_t *)((uint8_t *)buf + (uint64_t)p * buf_stride); }
    __host__ __device__ uint16_t *stg_of(int p) const { return (uint16_t *)((uint8_t *)stg + (uint64_t)p * stg_stride); }
    // slot of window w's K (which 0) or V (1) covariance, pair p
    __host__ __device__ double *cov_of(int p, int w, int which) const {
        return (double *)((uint8_t *)cov + (uint64_t)p * cov_stride) + ((uint64_t)(w & 1) * 2 + which) * D * D;
    }
    // first segment of each window of pair p (dynamic windows)
    __host__ __device__ int32_t *wtab_of(int p) const {
        return (int32_t *)(meta + (uint64_t)p * meta_stride + sizeof(PairMeta));
    }
    // rotation window w of pair p: [0] = R_k^T, [1] = R_v^T, [2] = R_v  (each D x D fp32)
    __host__ __device__ float *rot_of(int p, int w) const {
        if (w >= nw) w = nw - 1;
        return (float *)((uint8_t *)rot + (uint64_t)p * rot_stride) + (uint64_t)w * 3 * D * D;
    }
};

struct WsGeom {               // decode workspace
    float *qrot; uint64_t qrot_stride;      // [nw][D][GP]
    float *score; uint64_t score_stride;    // [max_blocks]
    int32_t *sel; uint64_t sel_stride;      // [max_blocks]
    int32_t *wsel; uint64_t wsel_stride;    // [nw + 2]
    float *part; uint64_t part_stride;      // [max_splits][GP * (D + 2)]
    int32_t *tag; uint64_t tag_stride;      // [max_splits]
    uint2 *binfo; uint64_t binfo_stride;    // [max_blocks]: per block, blk_info
    uint8_t *bsize; uint64_t bsize_stride;  // [max_blocks]: per block, log2 of its token count
    uint2 *selinfo; uint64_t selinfo_stride; // [max_blocks]: blk_info of each selected entry
    float *wres; uint64_t wres_stride;      // [CMB_NCC][nw + 1][GP][CMB_RES]: per-window merged results
    uint32_t *tkx; uint64_t tkx_stride;     // multi-workgroup top-k state, or null (pairs of <= 16 K blocks)
    int max_blocks, max_splits, max_sel;
    int split_slots;                        // attention workgroups resident at once on the device
};

// First segment of window w of pair p: every W tokens, or from the window
// table (a window not in use starts past every segment).
__device__ __forceinline__ int win_first_seg(const Geom &g, int p, int w) {
    if (!g.dyn) return w * (g.W / SEG);
    return w < g.meta_of(p)->nwin ? g.wtab_of(p)[w] : 0x7fffffff;
}
// Window of segment s of pair p: the last window starting at or before s.
__device__ __forceinline__ int win_of_seg(const Geom &g, int p, int s) {
    if (!g.dyn) return (s * SEG) / g.W;
    const int32_t *wt = g.wtab_of(p);
    int lo = 0, hi = g.meta_of(p)->nwin - 1;          // wt[0] = 0 <= s
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (wt[mid] <= s) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// a block's record: its byte offset in the pair's token arena, and
// r << 8 | log2 g << 16 | log2 B << 20
__host__ __device__ __forceinline__ uint2 blk_info(uint32_t tok_off, int r, int log2g, int log2b) {
    return make_uint2(tok_off, ((uint32_t)r << 8) | ((uint32_t)log2g << 16) | ((uint32_t)log2b << 20));
}
__host__ __device__ __forceinline__ uint32_t blk_tokens(uint32_t info) { return 1u << ((info >> 20) & 7u); }

// ---------------------------------------------------------------- elements
__device__ __forceinline__ float h2f(uint16_t h, int dtype) {
    if (dtype) return __uint_as_float((uint32_t)h << 16);
    return (float)__builtin_bit_cast(_Float16, h);
}
__device__ __forceinline__ uint16_t f2h(float f, int dtype) {
    if (dtype) {   // bf16, round to nearest even (inputs are finite)
        uint32_t u = __float_as_uint(f);
        u += 0x7fffu + ((u >> 16) & 1u);
        return (uint16_t)(u >> 16);
    }
    return __builtin_bit_cast(uint16_t, (_Float16)f);   // v_cvt_f16_f32, RNE
}

// bitmap bytes of a vector whose first T channels are represented: exactly
// T / g bits (T a multiple of 32, g <= 4: whole bytes).  A truncated bitmap of
// g = 2 or 4 is 6, 3, 4, 2 or 1 bytes, so such token bitmaps and block-key
// records can sit at any byte; a token record's values (and every run of B >=
// 4 bitmaps) stay 4-byte aligned.  And the record size:
__host__ __device__ __forceinline__ int bm_bytes(int log2g, int T) { return (T >> log2g) >> 3; }
__host__ __device__ __forceinline__ int vec_bytes(int r, int log2g, int T) { return 2 * r + bm_bytes(log2g, T); }
// a K or V token record: one byte per kept value with E4M3 values, else two
// (block keys always hold 16-bit values: vec_bytes)
__host__ __device__ __forceinline__ int tok_vec_bytes(int r, int log2g, int T, int fp8) {
    return (fp8 ? r : 2 * r) + bm_bytes(log2g, T);
}

// OCP FP8 E4M3 code (bias 7, largest finite 448, no infinities) of a finite
// fp32 value: the nearest code, ties to the even code; magnitudes of 448 and
// more saturate to 448.  Below 2^-6 the codes are the multiples of 2^-9
// (x 512 is exact, then one round-to-nearest-even to an integer); above, the
// fp32 exponent is rebiased and the mantissa rounded to 3 bits, a carry
// moving into the exponent field.
__device__ __forceinline__ uint32_t f2e4m3(float f) {
    const uint32_t u = __float_as_uint(f), s = (u >> 24) & 0x80u, a = u & 0x7fffffffu;
    uint32_t c;
    if (a >= 0x43e00000u) {
        c = 0x7eu;
    } else if (a < 0x3c800000u) {
        c = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);
    } else {
        const uint32_t m = a & 0x7fffffu, rem = m & 0xfffffu;
        c = (((a >> 23) - 120u) << 3) | (m >> 20);
        c += (rem > 0x80000u || (rem == 0x80000u && (c & 1u))) ? 1u : 0u;
        c = c > 0x7eu ? 0x7eu : c;
    }
    return s | c;
}

// ---------------------------------------------------------------- wave helpers
// Workgroup barrier for data exchanged through LDS only: it waits for the
// wave's own LDS (and scalar memory) operations, not for its outstanding
// global loads and stores, so loads issued before it stay in flight across
// it (__syncthreads also waits for those, as its fence orders global memory).
// Only for uniform control flow.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }


__device__ __forceinline__ float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, WAVE); }

// data-parallel-primitive lane move: lane i reads lane i - shift (row shifts),
// or a row reads the last lane of the row before it (row broadcasts); lanes
// outside ROWS, or without a source, read 0
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_read(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROWS, 0xf, false));
}

// pairwise adjacent tree over the 64 lanes: (x0+x1), (x2+x3), ... level by
// level.  Level L adds, in lane 2^L k + 2^L - 1, the partial sum 2^(L-1)
// lanes below (row shifts by 1, 2, 4, 8, then the broadcasts of lanes 15 and
// 31), so lane 63 ends with the tree's sum; it is returned to every lane.
// The operands of every addition are those of the butterfly form of the
// same tree.
__device__ __forceinline__ float tree64(float x) {
    x = x + dpp_read<0x111, 0xf>(x);
    x = x + dpp_read<0x112, 0xf>(x);
    x = x + dpp_read<0x114, 0xf>(x);
    x = x + dpp_read<0x118, 0xf>(x);
    x = x + dpp_read<0x142, 0xa>(x);
    x = x + dpp_read<0x143, 0xc>(x);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

// tree sum over the 128 channels held as (lane l: channel l, channel l+64):
// the adjacent tree of each half, then the two halves joined -- the pairwise
// adjacent tree of 128.
__device__ __forceinline__ float tree128(float lo, float hi) { return tree64(lo) + tree64(hi); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) v = fmaxf(v, shfl_xor_f(v, m));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) v += shfl_xor_f(v, m);
    return v;
}

// orderable key of an fp32 score (larger score -> larger key); -0 is +0
__device__ __forceinline__ uint32_t score_key(float s) {
    uint32_t b = __float_as_uint(s);
    if (b == 0x80000000u) b = 0;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------- launchers
// (implemented in the .hip files; all return hipError_t of the launch)
hipError_t launch_ctx_copy(int32_t *dst_dev, const int32_t *src_host, int n, hipStream_t s);
// the pair table of a cache with per-sequence capacities into its arena
hipError_t launch_pairs_copy(uint64_t *dst_dev, const uint64_t *src_host, int npairs, hipStream_t s);
// nw_src: windows of rk / rv per pair; slots past them repeat the last one
hipError_t launch_copy_rot(const Geom &g, const float *rk, const float *rv, int nw_src, hipStream_t s);
// rotations of the windows awaiting them, from their incremental covariances
// (dynamic windows): part = pairs * 2 * D * D floats, one_tok = pairs int32
hipError_t launch_window_rotations(const Geom &g, float *rot_k, float *rot_v, float *part, int32_t *one_tok,
                                   hipStream_t s);
// close of the windows awaiting their rotation (dynamic windows): the new
// rotations rk / rv [pairs][D][D], the windows' raw tokens k / v
// [pairs][seq_stride][D]; max_segs: segments of the longest closed window
hipError_t launch_close(const Geom &g, const float *rk, const float *rv, const uint16_t *k, const uint16_t *v,
                        int64_t seq_stride, int max_segs, hipStream_t s);
// ws: NULL (two passes, each rotating the tokens) or the single-pass
// workspace of slot_tok + slot_sc bytes per (pair, segment slot)
hipError_t launch_compress(const Geom &g, const uint16_t *k, const uint16_t *v, int64_t seq_stride,
                           const int32_t *ctx_dev, int max_full_segs, int any_tail, uint8_t *ws, uint32_t slot_tok,
                           uint32_t slot_sc, hipStream_t s);
hipError_t launch_set_meta(const Geom &g, const int32_t *ctx_dev, hipStream_t s);
hipError_t launch_append(const Geom &g, const uint16_t *k, const uint16_t *v, hipStream_t s);
// what: MAINT_FLUSH and / or MAINT_FINALIZE, the kernels to launch (each
// acts only on the pairs whose state calls for it)
hipError_t launch_maintain(const Geom &g, int mode, int what, hipStream_t s);
hipError_t launch_decode(const Geom &g, const WsGeom &w, const uint16_t *q, float *out, float scale,
                         int max_desc_used, int max_windows_used, hipStream_t s, hipEvent_t *ev);
hipError_t launch_dense(const uint16_t *q, const uint16_t *k, const uint16_t *v, float *out, int nseq,
                        int hkv, int G, int dtype, int64_t seq_stride, int max_ctx, const int32_t *ctx,
                        float scale, float *part, int max_splits, hipStream_t s);

size_t dense_part_bytes(int npairs, int G, int max_ctx);
size_t rotation_ctx_bytes(int num_seqs);
size_t rotation_ws_bytes(int num_seqs, int hkv, int nw, int W);
// wtok = min(W, max_tokens): tokens of a window at most
size_t reorder_ws_bytes(int num_seqs, int hkv, int nw, int wtok);
hipError_t launch_reorder(const uint16_t *k, const uint16_t *v, int64_t seq_stride, int num_seqs, int hkv, int dtype,
                          const int32_t *ctx_dev, int W, int nw, int wtok, int r, float *rot_k, float *rot_v,
                          uint8_t *ws, hipStream_t s);
hipError_t launch_rotations(const uint16_t *k, const uint16_t *v, int64_t seq_stride, int num_seqs, int hkv,
                            int dtype, const int32_t *ctx_dev, int W, int nw, float *rot_k, float *rot_v, float *ev_k,
                            float *ev_v, float *part, hipStream_t s);

constexpr int MAINT_APPEND = 0;        // after an append: flush or finalize where a buffer filled
constexpr int MAINT_AFTER_PREFILL = 1; // after compress: flush a >= U-token remainder
constexpr int MAINT_FLUSH = 1;
constexpr int MAINT_FINALIZE = 2;

}  // namespace mosaic
