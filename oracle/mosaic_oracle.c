/*
 * mosaic_oracle.c -- plain, slow CPU reference of the MosaicKV compressed-cache
 * hot path (arXiv 2607.00760).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls
 * this file; it is used by tests/, by __graft_entry__.smoke() and by the
 * cpu_baseline leg of bench.py.  It shares no code, header, table or constant
 * generator with the HIP library: only the dense K/V/q inputs and the
 * rotation matrices (inputs of the method) are common.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared
 * (no SIMD intrinsics; fmaf is the C library's correctly rounded fused
 * multiply-add).
 *
 * What is computed, in the paper's terms:
 *  - Stage-1 per-vector channel compression (Sec. 4.2 "Stage-1"): rotate each
 *    K/V vector by its window's SVD rotation (Sec. 2.3: K . R^T), keep the
 *    top-r elements by magnitude, discard the rest.
 *  - Element groups of 1/2/4 with one bitmap bit per group and packed
 *    values (Sec. 5.1, packed KV format and variable-granularity bitmap).
 *  - Per-segment strategy (Sec. 4.3 "Compression Strategy", Sec. 5.5):
 *    highest compression rate, then largest group size, whose loss is below a
 *    threshold; largest token block size whose intra-block key variance is
 *    below a threshold.
 *  - Stage-2 sequence compression (Sec. 4.2 "Stage-2"): block keys are the
 *    mean of the block's keys, channel-compressed like K; blocks are scored
 *    by q . block-key and the top-k blocks are kept.
 *  - PackedAttention (Sec. 5.3): attention over the selected blocks' packed
 *    K/V with the rotation merged into the single query / output vector.
 *  - KV update buffer (Sec. 5.3) and heterogeneous double compression
 *    buffering (Sec. 5.4): new tokens stay uncompressed in a 32-token buffer;
 *    a full buffer is compressed with the previous segment's strategy
 *    (provisional), and a completed segment is finalized with its own
 *    strategy and recompressed in place.
 *
 * Where the paper is silent these readings are taken (labels R-n): loss = relative dropped energy (R-3), group
 * score = L1 of the group's magnitudes (R-2), candidate order rate-first
 * (R-4), block variance relative to total energy (R-5), a global token
 * budget per (sequence, kv head): blocks taken in (score desc, index asc)
 * order while fewer than ceil(rho * scoreable tokens) tokens are taken
 * (R-7; Sec. 6.1 selects 10 % of tokens), GQA block score =
 * max over the group's query heads (R-8), buffer tokens always attended
 * dense and unrotated (R-9), provisional strategy = previous finalized
 * segment or the default (R-10), prefill remainder handled as appends
 * (R-11), y = x . R^T with row j of R the j-th rotated channel (R-12), a
 * truncated bitmap of exactly T / g bits (R-19), FP8 values as OCP
 * E4M3 without a scale factor, block keys kept 16-bit (R-20), per-vector and
 * per-segment energies as pairwise trees over the 128 channels and the 64
 * tokens (R-22); with dynamic windows, a window of decode tokens closes after
 * a segment when it holds the maximum length, or when the sum of its
 * segments' losses (larger of K's and V's relative dropped energy under the
 * provisional strategy) exceeds a threshold and it holds a minimum length;
 * its rotation then comes from the caller and its segments are encoded
 * again (R-23).
 *
 * Exactly-defined orders (so that integer and byte results are unique):
 *  chain(a, b)  : acc = 0; for i ascending: acc = fmaf(a_i, b_i, acc)
 *  tree(n)      : pairwise sum of adjacent elements, level by level
 *                 (x0+x1), (x2+x3), ... until one value; n a power of two.
 *  Every comparison that decides an index uses fp32 values and breaks ties
 *  by the lowest index.
 *
 * Parity status: see the pin list in tests/test_oracle_pins.py.  The strategy
 * thresholds' arithmetic (dropped-energy and block-variance tree sums) is
 * pinned only by closed forms and limiting cases; between those it is the
 * reading above ("parity unpinned" beyond its closed forms).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define D 128
#define MAXG 16

/* ------------------------------------------------------------------ */
/* Public structures (mirrored by oracle/oracle.py with ctypes).       */
/* ------------------------------------------------------------------ */
typedef struct {
    int32_t group;          /* G: query heads per kv head */
    int32_t dtype;          /* 0 = fp16, 1 = bf16 */
    int32_t seg_len;        /* S (64) */
    int32_t rot_window;     /* W, multiple of S */
    int32_t update_buf;     /* U (32) */
    int32_t keep_cand[3];   /* kept channels r, tried in this order */
    int32_t group_cand[3];  /* element group sizes g, tried in this order per r */
    int32_t block_cand[3];  /* token block sizes B, tried in this order */
    int32_t def_keep, def_group, def_block;
    float tau_channel, tau_block;
    int32_t select_num, select_den;  /* rho = num / den */
    int32_t force_default;           /* 1: every segment uses the default */
    int32_t trunc;                   /* channels represented (Sec. 5.2 channel truncation):
                                        channels >= trunc are never kept and have no bitmap
                                        bit; a multiple of 32 up to D (0 means D); the
                                        bitmap holds exactly trunc / g bits */
    int32_t fp8;                     /* 1: K and V token values stored as OCP FP8 E4M3
                                        (Sec. 7, quantizing the compressed elements);
                                        block keys keep the 16-bit dtype (reading R-20) */
    int32_t dyn;                     /* 1: windows of decode tokens close on their
                                        accumulated compression loss (Sec. 4.3, Sec. 5.5;
                                        reading R-23) instead of every rot_window tokens */
    float tau_window;                /* accumulated loss above which a window closes */
    int32_t min_window;              /* tokens a window holds at least before a loss close */
} orc_params;

typedef struct {
    uint32_t tok_off, sc_off, first_block;
    uint8_t r, log2g, log2b, flags; /* flags bit0: provisional */
} orc_desc;

typedef struct {
    orc_params P;
    int32_t cap;         /* capacity in tokens */
    int32_t nw;          /* rotation windows held */
    int32_t L;           /* tokens in the cache */
    int32_t nblk_final;  /* scoreable blocks in finalized segments */
    uint32_t tok_tail, sc_tail; /* bytes used by finalized segments */
    uint8_t *tok, *sc;
    size_t tok_cap, sc_cap;
    orc_desc *desc;
    int32_t desc_cap;
    uint16_t bufk[32 * D], bufv[32 * D];   /* update buffer (raw dtype bits) */
    uint16_t stgk[64 * D], stgv[64 * D];   /* raw tokens of the trailing segment */
    float *rk, *rv;      /* [nw][D][D] or NULL (identity) */
    /* windows closed by the compression loss (P.dyn; reading R-23) */
    int32_t *wseg;       /* [nw + 1]: first segment of each window */
    int32_t nwin;        /* windows in use; window nwin - 1 is open */
    float wloss;         /* accumulated loss of the open window */
    int32_t pend;        /* closed window awaiting its rotation, or -1 */
    double *cov;         /* [2][2][D][D]: window w's uncentered K and V covariance in slot w % 2 */
} orc_pair;

typedef struct {
    int32_t L, n_final, prov, n_buf, n_desc, nblk_final, nblk;
    uint32_t tok_tail, sc_tail;
    uint64_t used_bytes;
} orc_info;

/* ------------------------------------------------------------------ */
/* Element conversions (own implementations, round to nearest even).  */
/* ------------------------------------------------------------------ */
float orc_f16_to_f32(uint16_t h) {
    uint32_t s = (uint32_t)(h & 0x8000) << 16;
    uint32_t e = (h >> 10) & 0x1f, m = h & 0x3ff, u;
    if (e == 0) {
        if (m == 0) { u = s; }
        else {
            /* subnormal: m * 2^-24 is exact in fp32 */
            float f = (float)m * 0x1p-24f;
            memcpy(&u, &f, 4);
            u |= s;
        }
    } else if (e == 31) {
        u = s | 0x7f800000u | (m << 13);
    } else {
        u = s | ((e + 112) << 23) | (m << 13);
    }
    float f; memcpy(&f, &u, 4);
    return f;
}

uint16_t orc_f32_to_f16(float f) {
    uint32_t x; memcpy(&x, &f, 4);
    uint32_t sign = (x >> 16) & 0x8000u, ax = x & 0x7fffffffu;
    if (ax > 0x7f800000u) return (uint16_t)(sign | 0x7e00u);
    if (ax >= 0x477ff000u) return (uint16_t)(sign | 0x7c00u);
    if (ax < 0x38800000u) {                 /* below 2^-14: fp16 subnormal or 0 */
        if (ax < 0x33000000u) return (uint16_t)sign;   /* <= 2^-25 rounds to 0 */
        uint32_t e = ax >> 23, mant = (ax & 0x7fffffu) | 0x800000u;
        uint32_t sh = 126u - e;              /* value / 2^-24 = mant >> sh */
        uint32_t q = mant >> sh, rem = mant & ((1u << sh) - 1u), half = 1u << (sh - 1u);
        if (rem > half || (rem == half && (q & 1u))) q++;
        return (uint16_t)(sign | q);
    }
    uint32_t e = ax >> 23, m = ax & 0x7fffffu;
    uint32_t h = ((e - 112u) << 10) | (m >> 13), rem = m & 0x1fffu;
    if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) h++;
    return (uint16_t)(sign | h);
}

float orc_bf16_to_f32(uint16_t b) {
    uint32_t u = (uint32_t)b << 16; float f; memcpy(&f, &u, 4); return f;
}

uint16_t orc_f32_to_bf16(float f) {
    uint32_t u; memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* OCP 8-bit floating point E4M3 (sign, 4 exponent bits with bias 7, 3
   mantissa bits, no infinities, only S.1111.111 is NaN): the value of a code
   and the nearest code of a finite fp32 value (ties to the even code),
   saturated to +-448, the largest finite magnitude.  Written from the format's
   definition with exact double arithmetic. */
float orc_e4m3_to_f32(uint8_t c) {
    int s = c >> 7, e = (c >> 3) & 15, m = c & 7;
    if (e == 15 && m == 7) return NAN;
    double v = e == 0 ? ldexp((double)m / 8.0, -6) : ldexp(1.0 + (double)m / 8.0, e - 7);
    return (float)(s ? -v : v);
}

uint8_t orc_f32_to_e4m3(float f) {
    uint8_t sign = signbit(f) ? 0x80 : 0x00;
    double a = fabs((double)f);
    if (a >= 448.0) return (uint8_t)(sign | 0x7e);
    int e;
    if (a < ldexp(1.0, -6)) e = -6;                  /* subnormal spacing 2^-9 */
    else { (void)frexp(a, &e); e -= 1; }             /* a in [2^e, 2^(e+1)) */
    double step = ldexp(1.0, e - 3);                 /* spacing of the codes at a */
    double q = a / step, n = floor(q), fr = q - n;   /* exact: step is a power of two */
    if (fr > 0.5 || (fr == 0.5 && fmod(n, 2.0) == 1.0)) n += 1.0;
    /* n * step is the rounded magnitude: n < 8 only below 2^-6 (subnormal
       codes 0..7), else 8 <= n <= 16 with n = 16 the next binade */
    int code;
    if (n < 8.0) code = (int)n;
    else code = ((e + 7) << 3) + (int)n - 8;
    if (code > 0x7e) code = 0x7e;
    return (uint8_t)(sign | code);
}

static float to_f32(uint16_t v, int dtype) { return dtype ? orc_bf16_to_f32(v) : orc_f16_to_f32(v); }
static uint16_t from_f32(float v, int dtype) { return dtype ? orc_f32_to_bf16(v) : orc_f32_to_f16(v); }

/* ------------------------------------------------------------------ */
/* Ordered arithmetic helpers.                                         */
/* ------------------------------------------------------------------ */
/* pairwise adjacent tree sum over n (power of two) values */
float orc_tree_sum(const float *a, int n) {
    float buf[256];
    memcpy(buf, a, (size_t)n * sizeof(float));
    for (int w = n; w > 1; w >>= 1)
        for (int i = 0; i < w / 2; ++i) buf[i] = buf[2 * i] + buf[2 * i + 1];
    return buf[0];
}

/* Sec. 2.3: the cache is rotated as x . R^T; y[j] = chain_c(x[c], R[j][c]).
   R == NULL is the identity (y = x exactly). */
void orc_rotate(const float *x, const float *R, float *y) {
    if (!R) { memcpy(y, x, D * sizeof(float)); return; }
    for (int j = 0; j < D; ++j) {
        float acc = 0.0f;
        for (int c = 0; c < D; ++c) acc = fmaf(x[c], R[j * D + c], acc);
        y[j] = acc;
    }
}

/* Group importance (reading R-2): g = 1 is |y| exactly as in Sec. 4.2
   ("largest absolute values"); groups of 2 and 4 sum magnitudes pairwise. */
void orc_group_scores(const float *y, int g, float *s) {
    int n = D / g;
    for (int i = 0; i < n; ++i) {
        if (g == 1) s[i] = fabsf(y[i]);
        else if (g == 2) s[i] = fabsf(y[2 * i]) + fabsf(y[2 * i + 1]);
        else s[i] = (fabsf(y[4 * i]) + fabsf(y[4 * i + 1])) + (fabsf(y[4 * i + 2]) + fabsf(y[4 * i + 3]));
    }
}

typedef struct { float v; int32_t i; } vi_t;
static int cmp_desc(const void *pa, const void *pb) {
    const vi_t *a = (const vi_t *)pa, *b = (const vi_t *)pb;
    if (a->v > b->v) return -1;
    if (a->v < b->v) return 1;
    return (a->i > b->i) - (a->i < b->i);
}

/* Top-k of n values by (value descending, index ascending): keep[i] = 1 for
   the k selected.  A library sort is the selection step.  Returns 0, or -1
   on a non-finite input. */
int orc_topk_mask(const float *s, int n, int k, uint8_t *keep) {
    vi_t *a = (vi_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(vi_t));
    if (!a) return -2;
    for (int i = 0; i < n; ++i) {
        if (!isfinite(s[i])) { free(a); return -1; }
        a[i].v = s[i]; a[i].i = i; keep[i] = 0;
    }
    qsort(a, (size_t)n, sizeof(vi_t), cmp_desc);
    if (k > n) k = n;
    for (int j = 0; j < k; ++j) keep[a[j].i] = 1;
    free(a);
    return 0;
}

/* kept-channel mask of one rotated vector for strategy (r, g): the top r / g
   groups among the first T / g (channels >= T are truncated, never kept) */
static void keep_channels(const float *y, int r, int g, int T, uint8_t *kch) {
    float s[D]; uint8_t kg[D];
    orc_group_scores(y, g, s);
    for (int i = 0; i < D / g; ++i) kg[i] = 0;
    orc_topk_mask(s, T / g, r / g, kg);
    for (int c = 0; c < D; ++c) kch[c] = kg[c / g];
}

/* ------------------------------------------------------------------ */
/* Packed KV format (Sec. 5.1).                                        */
/* A packed vector = [bitmap: D/g bits as little-endian u32 words, bit */
/* i = group i kept][values: the r kept elements in ascending channel  */
/* order, fp32 -> dtype RNE, or -> E4M3 when fp8 is set (token records */
/* only)].                                                             */
/* ------------------------------------------------------------------ */
static int trunc_of(const orc_params *P) { return (P->trunc > 0 && P->trunc < D) ? P->trunc : D; }
/* bytes per kept value of the K and V token records */
static int tok_eb(const orc_params *P) { return P->fp8 ? 1 : 2; }
/* a bitmap of exactly T / g bits (reading R-19): T is a multiple of 32 and g
   divides 4, so T / g is a whole number of bytes */
int orc_bitmap_bytes_t(int g, int T) { return T / g / 8; }
int orc_vec_bytes_t(int r, int g, int elem_bytes, int T) { return r * elem_bytes + orc_bitmap_bytes_t(g, T); }
int orc_bitmap_bytes(int g) { return orc_bitmap_bytes_t(g, D); }
int orc_vec_bytes(int r, int g, int elem_bytes) { return orc_vec_bytes_t(r, g, elem_bytes, D); }

/* T / g bits, bit i = group i kept, least significant bit first in each
   byte (bit i is bit i % 32 of little-endian 32-bit word i / 32 wherever
   whole words exist) */
static void pack_bitmap(const uint8_t *kch, int g, int T, uint8_t *out) {
    int nbytes = orc_bitmap_bytes_t(g, T);
    for (int i = 0; i < nbytes; ++i) {
        uint8_t byte = 0;
        for (int b = 0; b < 8; ++b)
            if (kch[(i * 8 + b) * g]) byte |= (uint8_t)(1u << b);
        out[i] = byte;
    }
}

/* the kept values in ascending channel order: eb = 2 -> the 16-bit dtype
   (little-endian), eb = 1 -> E4M3 codes; one rounding from fp32 either way */
static void pack_values(const float *y, const uint8_t *kch, int dtype, int eb, uint8_t *out) {
    int slot = 0;
    for (int c = 0; c < D; ++c) {
        if (!kch[c]) continue;
        if (eb == 1) {
            out[slot] = orc_f32_to_e4m3(y[c]);
        } else {
            uint16_t h = from_f32(y[c], dtype);
            out[2 * slot] = (uint8_t)(h & 0xff);
            out[2 * slot + 1] = (uint8_t)(h >> 8);
        }
        slot++;
    }
}

/* Public: pack one rotated vector (for layout tests). */
void orc_pack_vector(const float *y, int r, int g, int dtype, uint8_t *out) {
    uint8_t kch[D];
    keep_channels(y, r, g, D, kch);
    pack_bitmap(kch, g, D, out);
    pack_values(y, kch, dtype, 2, out + orc_bitmap_bytes(g));
}

static int ilog2(int v) { int l = 0; while ((1 << l) < v) ++l; return l; }

/* ------------------------------------------------------------------ */
/* Strategy selection (Sec. 4.3, Sec. 5.5; readings R-3..R-6).         */
/* ------------------------------------------------------------------ */
/* yk, yv: [n][D] rotated vectors of one segment (n == S == 64).
   Energies (reading R-22): a vector's energy and its dropped energy are the
   pairwise tree over its 128 channels of y_c^2 (dropped channels only for
   the latter), and a segment's are the pairwise tree over its 64 tokens;
   the candidate (r, g) must pass for K and for V (R-3, R-4), the block size
   looks at the rotated keys only (R-5). */
void orc_choose_strategy(const orc_params *P, const float *yk, const float *yv, int n,
                         int *r_out, int *g_out, int *b_out) {
    if (P->force_default) { *r_out = P->def_keep; *g_out = P->def_group; *b_out = P->def_block; return; }
    const int T = trunc_of(P);
    float totk[64], totv[64], dk[9][64], dv[9][64];
    for (int t = 0; t < n; ++t) {
        float ek[D], ev[D];
        for (int c = 0; c < D; ++c) { ek[c] = yk[t * D + c] * yk[t * D + c]; ev[c] = yv[t * D + c] * yv[t * D + c]; }
        totk[t] = orc_tree_sum(ek, D); totv[t] = orc_tree_sum(ev, D);
        for (int ci = 0; ci < 9; ++ci) {
            int r = P->keep_cand[ci / 3], g = P->group_cand[ci % 3];
            uint8_t kk[D], kv[D]; float mk[D], mv[D];
            keep_channels(yk + t * D, r, g, T, kk); keep_channels(yv + t * D, r, g, T, kv);
            for (int c = 0; c < D; ++c) { mk[c] = kk[c] ? 0.0f : ek[c]; mv[c] = kv[c] ? 0.0f : ev[c]; }
            dk[ci][t] = orc_tree_sum(mk, D); dv[ci][t] = orc_tree_sum(mv, D);
        }
    }
    float TK = orc_tree_sum(totk, n), TV = orc_tree_sum(totv, n);
    int chosen = 8;
    for (int ci = 0; ci < 9; ++ci) {
        float DK = orc_tree_sum(dk[ci], n), DV = orc_tree_sum(dv[ci], n);
        float lk = P->tau_channel * TK, lv = P->tau_channel * TV;
        if (DK < lk && DV < lv) { chosen = ci; break; }
    }
    *r_out = P->keep_cand[chosen / 3]; *g_out = P->group_cand[chosen % 3];
    int bsel = P->block_cand[2];
    for (int bi = 0; bi < 3; ++bi) {
        int B = P->block_cand[bi];
        float d[64];
        for (int b0 = 0; b0 < n; b0 += B) {
            float mu[D];
            for (int c = 0; c < D; ++c) {
                float s = yk[b0 * D + c];
                for (int t = b0 + 1; t < b0 + B; ++t) s = s + yk[t * D + c];
                mu[c] = s * (1.0f / (float)B);
            }
            for (int t = b0; t < b0 + B; ++t) {
                float e[D];
                for (int c = 0; c < D; ++c) { float df = yk[t * D + c] - mu[c]; e[c] = df * df; }
                d[t] = orc_tree_sum(e, D);
            }
        }
        float VB = orc_tree_sum(d, n), lim = P->tau_block * TK;
        if (VB < lim) { bsel = B; break; }
    }
    *b_out = bsel;
}

/* Block key of tokens [b0, b0+B): mean in fp32, ascending token order. */
static void block_mean(const float *yk, int b0, int B, float *mu) {
    for (int c = 0; c < D; ++c) {
        float s = yk[b0 * D + c];
        for (int t = b0 + 1; t < b0 + B; ++t) s = s + yk[t * D + c];
        mu[c] = s * (1.0f / (float)B);
    }
}

/* Encode n tokens (n = S or U) with strategy (r, g, B) into a token-arena
   record and a score-arena record (Sec. 5.2 compressed KV encoding). */
static void encode_segment(const float *yk, const float *yv, int n, int r, int g, int B, int dtype, int T,
                           int eb, uint8_t *tok, uint8_t *sc) {
    /* token records hold eb-byte values, block keys 16-bit ones */
    int bmb = orc_bitmap_bytes_t(g, T), vb = r * eb, rec = bmb + vb, srec = bmb + 2 * r;
    uint8_t kch[D];
    for (int b0 = 0, bi = 0; b0 < n; b0 += B, ++bi) {
        uint8_t *blk = tok + (size_t)bi * B * 2 * rec;
        uint8_t *kbm = blk, *kval = blk + B * bmb, *vbm = kval + B * vb, *vval = vbm + B * bmb;
        for (int j = 0; j < B; ++j) {
            const float *k = yk + (size_t)(b0 + j) * D, *v = yv + (size_t)(b0 + j) * D;
            keep_channels(k, r, g, T, kch); pack_bitmap(kch, g, T, kbm + j * bmb); pack_values(k, kch, dtype, eb, kval + j * vb);
            keep_channels(v, r, g, T, kch); pack_bitmap(kch, g, T, vbm + j * bmb); pack_values(v, kch, dtype, eb, vval + j * vb);
        }
        float mu[D];
        block_mean(yk, b0, B, mu);
        keep_channels(mu, r, g, T, kch);
        pack_bitmap(kch, g, T, sc + (size_t)bi * srec);
        pack_values(mu, kch, dtype, 2, sc + (size_t)bi * srec + bmb);
    }
}

/* ------------------------------------------------------------------ */
/* Per-(sequence, kv head) cache state.                                */
/* ------------------------------------------------------------------ */
static int max_vec_bytes(const orc_params *P) {
    const int T = trunc_of(P);
    int m = orc_vec_bytes_t(P->def_keep, P->def_group, 2, T);
    for (int i = 0; i < 3; ++i) for (int j = 0; j < 3; ++j) {
        int v = orc_vec_bytes_t(P->keep_cand[i], P->group_cand[j], 2, T);
        if (v > m) m = v;
    }
    return m;
}
static int min_block(const orc_params *P) {
    int m = P->def_block;
    for (int i = 0; i < 3; ++i) if (P->block_cand[i] < m) m = P->block_cand[i];
    return m;
}

/* Rotation windows a cache of cap tokens can hold: every closed window has at
   least min_window tokens, so at most cap / min_window close, plus the open
   one (reading R-23). */
int orc_max_windows(const orc_params *P, int cap) {
    int nw = (cap + P->rot_window - 1) / P->rot_window;
    if (P->dyn && P->min_window > 0) {
        int m = cap / P->min_window + 1;
        if (m > nw) nw = m;
    }
    return nw > 0 ? nw : 1;
}

orc_pair *orc_pair_new(const orc_params *P, int cap, const float *rk, const float *rv, int nw_given) {
    orc_pair *p = (orc_pair *)calloc(1, sizeof(orc_pair));
    if (!p) return NULL;
    int nw = nw_given;
    if (P->dyn && rk && rv && nw_given > 0) { int m = orc_max_windows(P, cap); if (m > nw) nw = m; }
    p->P = *P; p->cap = cap; p->nw = nw;
    p->pend = -1; p->nwin = 1;
    p->wseg = (int32_t *)calloc((size_t)(nw > 0 ? nw : 1) + 1, sizeof(int32_t));
    if (P->dyn) p->cov = (double *)calloc((size_t)4 * D * D, sizeof(double));
    int mv = max_vec_bytes(P), mb = min_block(P);
    int nseg = cap / P->seg_len + 2;
    p->tok_cap = (size_t)nseg * P->seg_len * 2 * mv;
    p->sc_cap = (size_t)nseg * (P->seg_len / mb) * mv;
    p->desc_cap = nseg;
    p->tok = (uint8_t *)calloc(p->tok_cap, 1);
    p->sc = (uint8_t *)calloc(p->sc_cap, 1);
    p->desc = (orc_desc *)calloc((size_t)nseg, sizeof(orc_desc));
    if (rk && rv && nw > 0) {
        p->rk = (float *)malloc((size_t)nw * D * D * sizeof(float));
        p->rv = (float *)malloc((size_t)nw * D * D * sizeof(float));
        memcpy(p->rk, rk, (size_t)nw_given * D * D * sizeof(float));
        memcpy(p->rv, rv, (size_t)nw_given * D * D * sizeof(float));
        for (int w = nw_given; w < nw; ++w) {      /* slots of later windows: filled when they close */
            memcpy(p->rk + (size_t)w * D * D, rk + (size_t)(nw_given - 1) * D * D, D * D * sizeof(float));
            memcpy(p->rv + (size_t)w * D * D, rv + (size_t)(nw_given - 1) * D * D, D * D * sizeof(float));
        }
    }
    return p;
}

void orc_pair_free(orc_pair *p) {
    if (!p) return;
    free(p->tok); free(p->sc); free(p->desc); free(p->rk); free(p->rv); free(p->wseg); free(p->cov); free(p);
}

/* Window of segment s: every rot_window tokens, or with dynamic windows the
   last window of the table that starts at or before s. */
static int win_of_seg(const orc_pair *p, int s) {
    if (!p->P.dyn) return s * p->P.seg_len / p->P.rot_window;
    int w = 0;
    while (w + 1 < p->nwin && p->wseg[w + 1] <= s) ++w;
    return w;
}

static const float *rot_of(const orc_pair *p, const float *R, int token_pos) {
    if (!R) return NULL;
    int w = win_of_seg(p, token_pos / p->P.seg_len);
    if (w >= p->nw) w = p->nw - 1;
    return R + (size_t)w * D * D;
}

static void rotate_tokens(const orc_pair *p, const uint16_t *raw, int n, int pos0, const float *R, float *y) {
    const float *Rw = rot_of(p, R, pos0);
    for (int t = 0; t < n; ++t) {
        float x[D];
        for (int c = 0; c < D; ++c) x[c] = to_f32(raw[(size_t)t * D + c], p->P.dtype);
        orc_rotate(x, Rw, y + (size_t)t * D);
    }
}

static int state_nfinal(const orc_pair *p) { return p->L / p->P.seg_len; }
static int state_prov(const orc_pair *p) { return (p->L % p->P.seg_len) >= p->P.update_buf; }
static int state_nbuf(const orc_pair *p) { return (p->L % p->P.seg_len) - (state_prov(p) ? p->P.update_buf : 0); }

/* Compression loss of a segment under the strategy (r, g) (Sec. 4.3: the
   loss of the current strategy on new vectors; Sec. 5.5: the channel-
   compressed vectors compared with the original ones; reading R-23): the
   larger of K's and V's relative dropped energy, each the segment's dropped
   energy over its energy with the pairwise trees of the strategy search
   (R-22), 0 for a part without energy.  fp32 with correctly rounded
   divisions.  yk, yv: [n][D] rotated vectors, n == S == 64. */
float orc_segment_loss(const orc_params *P, const float *yk, const float *yv, int n, int r, int g) {
    const int T = trunc_of(P);
    float tk[64], tv[64], dk[64], dv[64];
    for (int t = 0; t < n; ++t) {
        float ek[D], ev[D], mk[D], mv[D];
        uint8_t kk[D], kv[D];
        for (int c = 0; c < D; ++c) { ek[c] = yk[t * D + c] * yk[t * D + c]; ev[c] = yv[t * D + c] * yv[t * D + c]; }
        keep_channels(yk + t * D, r, g, T, kk); keep_channels(yv + t * D, r, g, T, kv);
        for (int c = 0; c < D; ++c) { mk[c] = kk[c] ? 0.0f : ek[c]; mv[c] = kv[c] ? 0.0f : ev[c]; }
        tk[t] = orc_tree_sum(ek, D); tv[t] = orc_tree_sum(ev, D);
        dk[t] = orc_tree_sum(mk, D); dv[t] = orc_tree_sum(mv, D);
    }
    float TK = orc_tree_sum(tk, n), TV = orc_tree_sum(tv, n), DK = orc_tree_sum(dk, n), DV = orc_tree_sum(dv, n);
    float lk = TK > 0.0f ? DK / TK : 0.0f, lv = TV > 0.0f ? DV / TV : 0.0f;
    return lk > lv ? lk : lv;
}

/* Incremental covariance of a window (Sec. 5.5: the covariance is updated
   with each new token's outer product, so that the rotation of a closed
   window comes from it at once).  One segment's 64 raw tokens (k, v: [S][D])
   are added to window w's uncentered K and V covariance: per entry (i, j),
   the fp64 sum over the tokens in order of x_t[i] x_t[j] (each product exact
   in fp64), then added to the window's running entry (which the window's
   first segment replaces).  Windows alternate between two slots. */
static void cov_add_segment(orc_pair *p, int w, const uint16_t *k, const uint16_t *v, int first) {
    const int S = p->P.seg_len;
    for (int which = 0; which < 2; ++which) {
        const uint16_t *x = which ? v : k;
        double *C = p->cov + ((size_t)(w & 1) * 2 + which) * D * D;
        for (int i = 0; i < D; ++i)
            for (int j = 0; j < D; ++j) {
                double s = 0.0;
                for (int t = 0; t < S; ++t)
                    s = s + (double)to_f32(x[(size_t)t * D + i], p->P.dtype) * (double)to_f32(x[(size_t)t * D + j], p->P.dtype);
                C[i * D + j] = (first ? 0.0 : C[i * D + j]) + s;
            }
    }
}

/* Segment s, finalized by the append path, belongs to the open window: add
   its loss; the window closes after s when it holds rot_window tokens (the
   maximum length), or when the accumulated loss exceeds tau_window and it
   holds at least min_window tokens (Sec. 4.3; reading R-23).  The closed
   window then awaits its own rotation (orc_pair_close), and the next
   segment opens a new window. */
static void window_update(orc_pair *p, int s, float loss) {
    const orc_params *P = &p->P;
    int w = p->nwin - 1;
    int ntok = (s + 1 - p->wseg[w]) * P->seg_len;
    float acc = p->wloss + loss;
    int close = ntok >= P->rot_window || (acc > P->tau_window && ntok >= P->min_window);
    if (close && p->nwin < p->nw) {
        p->wseg[p->nwin] = s + 1;
        p->nwin++;
        p->pend = w;
        p->wloss = 0.0f;
    } else {
        p->wloss = acc;
    }
}

/* Segment s (S rotated tokens yk, yv) encoded with its own strategy at the
   tails of the arenas. */
static void encode_final(orc_pair *p, int s, const float *yk, const float *yv) {
    const orc_params *P = &p->P;
    int S = P->seg_len, r, g, B;
    orc_choose_strategy(P, yk, yv, S, &r, &g, &B);
    int rec = orc_vec_bytes_t(r, g, tok_eb(P), trunc_of(P)), srec = orc_vec_bytes_t(r, g, 2, trunc_of(P));
    encode_segment(yk, yv, S, r, g, B, P->dtype, trunc_of(P), tok_eb(P), p->tok + p->tok_tail, p->sc + p->sc_tail);
    orc_desc *d = &p->desc[s];
    d->tok_off = p->tok_tail; d->sc_off = p->sc_tail; d->first_block = (uint32_t)p->nblk_final;
    d->r = (uint8_t)r; d->log2g = (uint8_t)ilog2(g); d->log2b = (uint8_t)ilog2(B); d->flags = 0;
    p->tok_tail += (uint32_t)(S * 2 * rec);
    p->sc_tail += (uint32_t)((S / B) * srec);
    p->nblk_final += S / B;
}

/* finalize the trailing segment: staging holds S raw tokens.  A segment
   completed by an append also counts toward its window's loss, under the
   provisional strategy (R-10) that new tokens were compressed with. */
static void finalize_segment(orc_pair *p, int from_append) {
    const orc_params *P = &p->P;
    int S = P->seg_len, nf = p->L / S - 1;   /* index of the segment being finalized */
    float *yk = (float *)malloc((size_t)S * D * sizeof(float)), *yv = (float *)malloc((size_t)S * D * sizeof(float));
    rotate_tokens(p, p->stgk, S, nf * S, p->rk, yk);
    rotate_tokens(p, p->stgv, S, nf * S, p->rv, yv);
    float loss = 0.0f;
    const int dyn = P->dyn && from_append;
    if (dyn) {
        const int w = p->nwin - 1;
        cov_add_segment(p, w, p->stgk, p->stgv, nf == p->wseg[w]);
        int rp = P->def_keep, gp = P->def_group;
        if (nf > 0) { rp = p->desc[nf - 1].r; gp = 1 << p->desc[nf - 1].log2g; }
        loss = orc_segment_loss(P, yk, yv, S, rp, gp);
    }
    encode_final(p, nf, yk, yv);
    if (dyn) window_update(p, nf, loss);
    free(yk); free(yv);
}

/* flush: the first U tokens of the trailing segment, compressed with the
   previous finalized segment's strategy (Sec. 5.4) or the default */
static void flush_provisional(orc_pair *p) {
    const orc_params *P = &p->P;
    int S = P->seg_len, U = P->update_buf, nf = p->L / S;
    int r = P->def_keep, g = P->def_group, B = P->def_block;
    if (nf > 0) { orc_desc *pd = &p->desc[nf - 1]; r = pd->r; g = 1 << pd->log2g; B = 1 << pd->log2b; }
    float *yk = (float *)malloc((size_t)U * D * sizeof(float)), *yv = (float *)malloc((size_t)U * D * sizeof(float));
    rotate_tokens(p, p->stgk, U, nf * S, p->rk, yk);
    rotate_tokens(p, p->stgv, U, nf * S, p->rv, yv);
    encode_segment(yk, yv, U, r, g, B, P->dtype, trunc_of(P), tok_eb(P), p->tok + p->tok_tail, p->sc + p->sc_tail);
    orc_desc *d = &p->desc[nf];
    d->tok_off = p->tok_tail; d->sc_off = p->sc_tail; d->first_block = (uint32_t)p->nblk_final;
    d->r = (uint8_t)r; d->log2g = (uint8_t)ilog2(g); d->log2b = (uint8_t)ilog2(B); d->flags = 1;
    free(yk); free(yv);
}

/* Append one token (Sec. 5.3 update buffer, Sec. 5.4 double buffering).
   Returns 0, -3 when the capacity is exhausted, or -4 (nothing appended)
   when the token would compress the buffer while a closed window still
   awaits its rotation. */
int orc_pair_append(orc_pair *p, const uint16_t *k, const uint16_t *v) {
    const orc_params *P = &p->P;
    if (p->L >= p->cap) return -3;
    int S = P->seg_len, U = P->update_buf;
    int m = p->L % S, nb = state_nbuf(p);
    if (p->pend >= 0 && nb + 1 == U) return -4;    /* a closed window awaits its rotation */
    memcpy(p->bufk + (size_t)nb * D, k, D * 2); memcpy(p->bufv + (size_t)nb * D, v, D * 2);
    memcpy(p->stgk + (size_t)m * D, k, D * 2); memcpy(p->stgv + (size_t)m * D, v, D * 2);
    p->L++;
    if (nb + 1 == U) {
        if (p->L % S == 0) finalize_segment(p, 1);
        else flush_provisional(p);
    }
    return 0;
}

/* Prefill compression (Sec. 5.2): full segments encoded with their own
   strategy; the remainder of L mod S tokens goes through the append path
   (reading R-11).  k, v: [L][D] raw dtype bits. */
int orc_pair_compress(orc_pair *p, const uint16_t *k, const uint16_t *v, int L) {
    const orc_params *P = &p->P;
    if (L > p->cap || L < 0) return -3;
    p->L = 0; p->nblk_final = 0; p->tok_tail = 0; p->sc_tail = 0;
    int S = P->seg_len, nfull = L / S;
    p->wloss = 0.0f; p->pend = -1; p->nwin = 1;
    if (P->dyn) {
        /* input tokens: fixed windows of rot_window tokens (Sec. 4.3); the
           window holding the first token after the full segments stays open */
        p->nwin = nfull * S / P->rot_window + 1;
        if (p->nwin > p->nw) p->nwin = p->nw > 0 ? p->nw : 1;
        for (int w = 0; w < p->nwin; ++w) p->wseg[w] = w * (P->rot_window / S);
    }
    for (int s = 0; s < nfull; ++s) {
        memcpy(p->stgk, k + (size_t)s * S * D, (size_t)S * D * 2);
        memcpy(p->stgv, v + (size_t)s * S * D, (size_t)S * D * 2);
        p->L = (s + 1) * S;
        finalize_segment(p, 0);
    }
    if (P->dyn) {   /* the open window's covariance over its prefill segments */
        const int w = p->nwin - 1;
        for (int s = p->wseg[w]; s < nfull; ++s)
            cov_add_segment(p, w, k + (size_t)s * S * D, v + (size_t)s * S * D, s == p->wseg[w]);
    }
    p->L = nfull * S;
    for (int t = nfull * S; t < L; ++t) orc_pair_append(p, k + (size_t)t * D, v + (size_t)t * D);
    return 0;
}

/* Close of the window awaiting its rotation (Sec. 4.3, Sec. 5.5): rk_new /
   rv_new ([D][D], row j = rotated channel j), computed by the caller from the
   window's raw tokens, replace its provisional rotation and become the
   provisional rotation of the window the close opened; every segment of the
   closed window is encoded again, with its own strategy, from its raw tokens
   k, v ([n][D], the window's tokens from its first one).  The closed window
   is the last compressed one (a buffer flush waits for the close), so the
   new records start where its old ones did.  Returns 0, or -4 when no window
   awaits a rotation. */
int orc_pair_close(orc_pair *p, const float *rk_new, const float *rv_new, const uint16_t *k, const uint16_t *v) {
    if (p->pend < 0 || !p->rk || !p->rv) return -4;
    const orc_params *P = &p->P;
    int w = p->pend, s0 = p->wseg[w], s1 = p->wseg[w + 1], S = P->seg_len;
    for (int i = w; i <= w + 1 && i < p->nw; ++i) {
        memcpy(p->rk + (size_t)i * D * D, rk_new, D * D * sizeof(float));
        memcpy(p->rv + (size_t)i * D * D, rv_new, D * D * sizeof(float));
    }
    p->tok_tail = p->desc[s0].tok_off; p->sc_tail = p->desc[s0].sc_off;
    p->nblk_final = (int32_t)p->desc[s0].first_block;
    float *yk = (float *)malloc((size_t)S * D * sizeof(float)), *yv = (float *)malloc((size_t)S * D * sizeof(float));
    for (int s = s0; s < s1; ++s) {
        rotate_tokens(p, k + (size_t)(s - s0) * S * D, S, s * S, p->rk, yk);
        rotate_tokens(p, v + (size_t)(s - s0) * S * D, S, s * S, p->rv, yv);
        encode_final(p, s, yk, yv);
    }
    free(yk); free(yv);
    p->pend = -1;
    return 0;
}

/* Window state: windows in use, the window awaiting its rotation (-1: none),
   the open window's accumulated loss, and the first segment of each window
   (wseg, capacity nwin, may be NULL). */
void orc_pair_windows(const orc_pair *p, int32_t *nwin, int32_t *pend, float *wloss, int32_t *wseg) {
    *nwin = p->nwin; *pend = p->pend; *wloss = p->wloss;
    if (wseg) for (int w = 0; w < p->nwin; ++w) wseg[w] = p->wseg[w];
}

/* Window w's incremental covariance (which: 0 K, 1 V) into out [D][D]; it
   stays readable until the window two after it first accumulates. */
void orc_pair_cov(const orc_pair *p, int w, int which, double *out) {
    if (!p->cov) { memset(out, 0, (size_t)D * D * sizeof(double)); return; }
    memcpy(out, p->cov + ((size_t)(w & 1) * 2 + which) * D * D, (size_t)D * D * sizeof(double));
}

void orc_pair_info(const orc_pair *p, orc_info *o) {
    const orc_params *P = &p->P;
    o->L = p->L; o->n_final = state_nfinal(p); o->prov = state_prov(p); o->n_buf = state_nbuf(p);
    o->n_desc = o->n_final + o->prov; o->nblk_final = p->nblk_final;
    o->nblk = p->nblk_final;
    uint64_t used = (uint64_t)p->tok_tail + p->sc_tail + 16ull * (uint64_t)o->n_desc
                  + (uint64_t)o->n_buf * 2 * D * 2;
    if (o->prov) {
        const orc_desc *d = &p->desc[o->n_final];
        int B = 1 << d->log2b, rec = orc_vec_bytes_t(d->r, 1 << d->log2g, tok_eb(P), trunc_of(P)),
            srec = orc_vec_bytes_t(d->r, 1 << d->log2g, 2, trunc_of(P));
        o->nblk += P->update_buf / B;
        used += (uint64_t)P->update_buf * 2 * rec + (uint64_t)(P->update_buf / B) * srec;
    }
    o->tok_tail = p->tok_tail; o->sc_tail = p->sc_tail; o->used_bytes = used;
}

const uint8_t *orc_pair_tok(const orc_pair *p) { return p->tok; }
const uint8_t *orc_pair_sc(const orc_pair *p) { return p->sc; }
const orc_desc *orc_pair_desc(const orc_pair *p) { return p->desc; }
const uint16_t *orc_pair_bufk(const orc_pair *p) { return p->bufk; }
const uint16_t *orc_pair_bufv(const orc_pair *p) { return p->bufv; }
const uint16_t *orc_pair_stgk(const orc_pair *p) { return p->stgk; }
const uint16_t *orc_pair_stgv(const orc_pair *p) { return p->stgv; }

/* ------------------------------------------------------------------ */
/* Decode (Sec. 4.2 stage-2, Sec. 5.3 PackedAttention).                */
/* ------------------------------------------------------------------ */
static int desc_ntok(const orc_pair *p, const orc_desc *d) {
    return (d->flags & 1) ? p->P.update_buf : p->P.seg_len;
}

/* q rotation merged into the single query vector (Sec. 5.3): fp32 chain,
   used for block scores. */
static void qrot32(const orc_pair *p, const uint16_t *qh, int pos, float *out) {
    float x[D];
    for (int c = 0; c < D; ++c) x[c] = to_f32(qh[c], p->P.dtype);
    orc_rotate(x, rot_of(p, p->rk, pos), out);
}

/* Block scores s_b = max over the G heads of chain over kept slots of
   (q_rot[c], value).  Returns the number of scoreable blocks. */
int orc_pair_scores(const orc_pair *p, const uint16_t *q, float *scores, int cap) {
    const orc_params *P = &p->P;
    orc_info inf; orc_pair_info(p, &inf);
    int G = P->group, nb = 0;
    float qr[MAXG][D];
    int cur_w = -1;
    for (int di = 0; di < inf.n_desc; ++di) {
        const orc_desc *d = &p->desc[di];
        int pos = di * P->seg_len, w = win_of_seg(p, di);
        if (w != cur_w) { for (int h = 0; h < G; ++h) qrot32(p, q + (size_t)h * D, pos, qr[h]); cur_w = w; }
        const int T = trunc_of(P);
        int g = 1 << d->log2g, B = 1 << d->log2b, r = d->r, rec = orc_vec_bytes_t(r, g, 2, T), bmb = orc_bitmap_bytes_t(g, T);
        int nblk = desc_ntok(p, d) / B;
        for (int j = 0; j < nblk; ++j) {
            const uint8_t *rp = p->sc + d->sc_off + (size_t)j * rec;
            float best = 0.0f;
            for (int h = 0; h < G; ++h) {
                float acc = 0.0f; int slot = 0;
                for (int gi = 0; gi < T / g; ++gi) {
                    if (!((rp[gi >> 3] >> (gi & 7)) & 1)) continue;
                    for (int e = 0; e < g; ++e) {
                        int c = gi * g + e;
                        uint16_t hv = (uint16_t)(rp[bmb + 2 * slot] | (rp[bmb + 2 * slot + 1] << 8));
                        acc = fmaf(qr[h][c], to_f32(hv, P->dtype), acc);
                        slot++;
                    }
                }
                best = (h == 0) ? acc : fmaxf(best, acc);
            }
            if (best == 0.0f) best = 0.0f;   /* -0 -> +0 */
            if (nb < cap) scores[nb] = best;
            nb++;
        }
    }
    return nb;
}

int orc_select_count(int nblk, int num, int den) {
    if (nblk <= 0) return 0;
    long long k = ((long long)nblk * num + den - 1) / den;
    if (k < 1) k = 1;
    if (k > nblk) k = nblk;
    return (int)k;
}

/* Token budget of the selection (reading R-7 of Sec. 4.2 stage 2 and Sec.
   6.1, which selects 10 % of tokens): ceil(rho * ntok) tokens, rho = num /
   den, in integers; at least one token when any is scoreable. */
int orc_select_budget(int ntok, int num, int den) { return orc_select_count(ntok, num, den); }

/* Blocks by (score desc, index asc), taken while the tokens of the blocks
   already taken are fewer than the budget: the shortest prefix of that order
   whose tokens reach the budget (the last block may pass it).  sizes[b] is
   block b's token count.  A library sort is the ordering step.  Returns the
   number of blocks taken, or -1 on a non-finite score. */
int orc_select_blocks(const float *s, const int32_t *sizes, int n, int budget, uint8_t *keep) {
    vi_t *a = (vi_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(vi_t));
    if (!a) return -2;
    for (int i = 0; i < n; ++i) {
        if (!isfinite(s[i])) { free(a); return -1; }
        a[i].v = s[i]; a[i].i = i; keep[i] = 0;
    }
    qsort(a, (size_t)n, sizeof(vi_t), cmp_desc);
    long long taken = 0;
    int nsel = 0;
    for (int j = 0; j < n && taken < budget; ++j) {
        keep[a[j].i] = 1;
        taken += sizes[a[j].i];
        nsel++;
    }
    free(a);
    return nsel;
}

/* unpack one packed vector into dense fp64 (0 at dropped channels) */
static void unpack64(const uint8_t *bm, const uint8_t *vals, int g, int T, int dtype, int eb, double *out) {
    int slot = 0;
    for (int gi = 0; gi < D / g; ++gi) {
        int kept = gi < T / g ? (bm[gi >> 3] >> (gi & 7)) & 1 : 0;
        for (int e = 0; e < g; ++e) {
            int c = gi * g + e;
            if (kept) {
                if (eb == 1) out[c] = (double)orc_e4m3_to_f32(vals[slot]);
                else out[c] = (double)to_f32((uint16_t)(vals[2 * slot] | (vals[2 * slot + 1] << 8)), dtype);
                slot++;
            } else out[c] = 0.0;
        }
    }
}

/* Full decode step for one (sequence, kv head): block scores, top-k,
   attention over the selected blocks and the update buffer, back-rotation.
   q: [G][D] raw; out: [G][D] fp64.  sel (optional, capacity cap): selected
   block indices ascending.  Returns the number selected, or < 0 on error. */
int orc_pair_decode(const orc_pair *p, const uint16_t *q, float scale, double *out, int32_t *sel, int cap) {
    const orc_params *P = &p->P;
    orc_info inf; orc_pair_info(p, &inf);
    int G = P->group, nb = inf.nblk;
    float *scores = (float *)malloc((size_t)(nb > 0 ? nb : 1) * sizeof(float));
    uint8_t *keep = (uint8_t *)malloc((size_t)(nb > 0 ? nb : 1));
    int32_t *bsz = (int32_t *)malloc((size_t)(nb > 0 ? nb : 1) * sizeof(int32_t));
    orc_pair_scores(p, q, scores, nb);
    int ntok = 0;                             /* tokens of the scoreable blocks */
    for (int di = 0, b = 0; di < inf.n_desc; ++di) {
        const orc_desc *d = &p->desc[di];
        for (int j = 0; j < desc_ntok(p, d) >> d->log2b; ++j) bsz[b++] = 1 << d->log2b;
        ntok += desc_ntok(p, d);
    }
    int budget = orc_select_budget(ntok, P->select_num, P->select_den);
    if (nb > 0 && orc_select_blocks(scores, bsz, nb, budget, keep) < 0) {
        free(scores); free(keep); free(bsz); return -1;
    }
    free(bsz);
    int ns = 0;
    for (int b = 0; b < nb; ++b) if (keep[b]) { if (sel && ns < cap) sel[ns] = b; ns++; }

    /* collect logits; tokens of selected blocks grouped by window */
    int ntok_max = nb * 16 + P->update_buf + 1;
    double *z = (double *)malloc((size_t)ntok_max * G * sizeof(double));
    int *tw = (int *)malloc((size_t)ntok_max * sizeof(int));       /* window, -1 = buffer */
    double *vv = (double *)malloc((size_t)ntok_max * D * sizeof(double));
    int nt = 0;
    double qd[MAXG][D];
    for (int h = 0; h < G; ++h) for (int c = 0; c < D; ++c) qd[h][c] = (double)to_f32(q[h * D + c], P->dtype);
    int bglob = 0, cur_w = -1;
    double qr[MAXG][D];
    for (int di = 0; di < inf.n_desc; ++di) {
        const orc_desc *d = &p->desc[di];
        int pos = di * P->seg_len, w = win_of_seg(p, di);
        if (w != cur_w) {   /* q . R_k^T in fp64 for this window */
            const float *Rk = rot_of(p, p->rk, pos);
            for (int h = 0; h < G; ++h) for (int j = 0; j < D; ++j) {
                if (!Rk) { qr[h][j] = qd[h][j]; continue; }
                double a = 0.0;
                for (int c = 0; c < D; ++c) a += qd[h][c] * (double)Rk[j * D + c];
                qr[h][j] = a;
            }
            cur_w = w;
        }
        int g = 1 << d->log2g, B = 1 << d->log2b, r = d->r, bmb = orc_bitmap_bytes_t(g, trunc_of(P)), eb = tok_eb(P),
            vb = eb * r, rec = bmb + vb;
        int nblk = desc_ntok(p, d) / B;
        for (int j = 0; j < nblk; ++j, ++bglob) {
            if (!keep[bglob]) continue;
            const uint8_t *blk = p->tok + d->tok_off + (size_t)j * B * 2 * rec;
            const uint8_t *kbm = blk, *kval = blk + B * bmb, *vbm = kval + B * vb, *vval = vbm + B * bmb;
            for (int t = 0; t < B; ++t) {
                double kd[D];
                unpack64(kbm + t * bmb, kval + t * vb, g, trunc_of(P), P->dtype, eb, kd);
                unpack64(vbm + t * bmb, vval + t * vb, g, trunc_of(P), P->dtype, eb, vv + (size_t)nt * D);
                for (int h = 0; h < G; ++h) {
                    double a = 0.0;
                    for (int c = 0; c < D; ++c) a += qr[h][c] * kd[c];
                    z[(size_t)nt * G + h] = (double)scale * a;
                }
                tw[nt] = w; nt++;
            }
        }
    }
    for (int i = 0; i < inf.n_buf; ++i) {
        for (int h = 0; h < G; ++h) {
            double a = 0.0;
            for (int c = 0; c < D; ++c) a += qd[h][c] * (double)to_f32(p->bufk[i * D + c], P->dtype);
            z[(size_t)nt * G + h] = (double)scale * a;
        }
        for (int c = 0; c < D; ++c) vv[(size_t)nt * D + c] = (double)to_f32(p->bufv[i * D + c], P->dtype);
        tw[nt] = -1; nt++;
    }
    int nwin = p->nw > 0 ? p->nw : 1;
    if (!p->rv) nwin = 1;
    for (int h = 0; h < G; ++h) {
        double *o = out + (size_t)h * D;
        for (int j = 0; j < D; ++j) o[j] = 0.0;
        if (nt == 0) continue;
        double m = -INFINITY;
        for (int t = 0; t < nt; ++t) if (z[(size_t)t * G + h] > m) m = z[(size_t)t * G + h];
        double l = 0.0;
        double *acc = (double *)calloc((size_t)(nwin + 1) * D, sizeof(double));
        for (int t = 0; t < nt; ++t) {
            double e = exp(z[(size_t)t * G + h] - m);
            l += e;
            int slotw = (tw[t] < 0) ? nwin : (p->rv ? (tw[t] < p->nw ? tw[t] : p->nw - 1) : 0);
            for (int c = 0; c < D; ++c) acc[(size_t)slotw * D + c] += e * vv[(size_t)t * D + c];
        }
        for (int w = 0; w < nwin; ++w) {
            const double *a = acc + (size_t)w * D;
            if (!p->rv) { for (int j = 0; j < D; ++j) o[j] += a[j]; continue; }
            const float *Rv = p->rv + (size_t)w * D * D;
            for (int j = 0; j < D; ++j) {
                double s = 0.0;
                for (int c = 0; c < D; ++c) s += a[c] * (double)Rv[c * D + j];   /* x = y . R */
                o[j] += s;
            }
        }
        for (int j = 0; j < D; ++j) o[j] = (o[j] + acc[(size_t)nwin * D + j]) / l;
        free(acc);
    }
    free(scores); free(keep); free(z); free(tw); free(vv);
    return ns;
}

/* Dense attention of one GQA group (the uncompressed reference). */
void orc_dense_attention(const uint16_t *q, const uint16_t *k, const uint16_t *v, int L, int G, int dtype,
                         float scale, double *out) {
    double *z = (double *)malloc((size_t)(L > 0 ? L : 1) * sizeof(double));
    for (int h = 0; h < G; ++h) {
        double qd[D];
        for (int c = 0; c < D; ++c) qd[c] = (double)to_f32(q[h * D + c], dtype);
        double m = -INFINITY;
        for (int t = 0; t < L; ++t) {
            double a = 0.0;
            for (int c = 0; c < D; ++c) a += qd[c] * (double)to_f32(k[(size_t)t * D + c], dtype);
            z[t] = (double)scale * a;
            if (z[t] > m) m = z[t];
        }
        double l = 0.0, o[D];
        for (int j = 0; j < D; ++j) o[j] = 0.0;
        for (int t = 0; t < L; ++t) {
            double e = exp(z[t] - m); l += e;
            for (int j = 0; j < D; ++j) o[j] += e * (double)to_f32(v[(size_t)t * D + j], dtype);
        }
        for (int j = 0; j < D; ++j) out[h * D + j] = L > 0 ? o[j] / l : 0.0;
    }
    free(z);
}

/* Byte accounting per token of a full segment (for the ratio closed form):
   2 packed vectors per token with elem_bytes-byte values, plus one block key
   (16-bit values) per B tokens. */
double orc_bytes_per_token_t(int r, int g, int B, int elem_bytes, int T) {
    return 2.0 * (double)orc_vec_bytes_t(r, g, elem_bytes, T) + (double)orc_vec_bytes_t(r, g, 2, T) / (double)B;
}
double orc_bytes_per_token(int r, int g, int B, int elem_bytes) { return orc_bytes_per_token_t(r, g, B, elem_bytes, D); }
