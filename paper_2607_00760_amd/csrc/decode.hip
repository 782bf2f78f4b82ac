// decode.hip -- gfx950 kernels of MosaicKV's decode step (PackedAttention,
// Sec. 5.3; stage-2 dynamic sequence compression, Sec. 4.2).
//
//   qrot   : q . R_k^T once per (pair, window) -- the rotation is merged into
//            the single query vector instead of un-rotating the cache.  R_k^T
//            is staged in LDS; each output channel is an fp32 fused chain.
//   score  : every block key of a pair streamed once (a workgroup stages a
//            contiguous run of segments' records in LDS with 16-byte loads);
//            lane per block key: a packed vector product walking the bitmap's
//            set bits in ascending order, fp32 fused chain, max over the GQA
//            group.  These scores decide the selection, so their arithmetic
//            order is fixed.
//   topk   : exact radix select (8-bit digits, LDS histograms) of the k-th
//            largest score key, then an ordered compaction breaking ties by
//            the lowest block index; scores live in LDS when they fit.
//   attn   : split-K over the selected list, one rotation window per split.
//            A wave processes chunks of whole blocks (<= 64 tokens): their
//            packed records are staged in LDS with coalesced 16-byte loads
//            (the next chunk is prefetched into registers meanwhile), the
//            packed K and V are scattered into a dense LDS tile, and both
//            contractions run on the matrix cores (16x16x32): logits as
//            K . q^T with q split into two 16-bit halves, online softmax in
//            fp32 on the accumulator layout, then P . V with P split the same
//            way.  The update buffer is one more split (dense, unrotated).
//   reduce : log-sum-exp merge of the splits per window, back-rotation of
//            each window's accumulator by R_v (staged in LDS), merge of the
//            windows and the buffer.
#include "mosaic_internal.h"

namespace mosaic {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 halfx8;
typedef __attribute__((ext_vector_type(4))) float floatx4;

template <int DT> struct Mma;
template <> struct Mma<1> {
    using v8 = bf16x8;
    static __device__ __forceinline__ floatx4 run(v8 a, v8 b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mma<0> {
    using v8 = halfx8;
    static __device__ __forceinline__ floatx4 run(v8 a, v8 b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};

__device__ __forceinline__ void wave_sync() { __builtin_amdgcn_wave_barrier(); }

__device__ __forceinline__ int pair_ndesc(const PairMeta &m, int &n_final, int &prov, int &nbuf) {
    n_final = m.L / SEG;
    const int rem = m.L % SEG;
    prov = rem >= UBUF;
    nbuf = rem - (prov ? UBUF : 0);
    return n_final + prov;
}

__device__ __forceinline__ int pair_nblocks(const Geom &g, int p, const PairMeta &m) {
    int nf, prov, nbuf;
    pair_ndesc(m, nf, prov, nbuf);
    int nb = m.nblk_final;
    if (prov) nb += UBUF >> g.desc_of(p)[nf].log2b;
    return nb;
}

// Copy nbytes (multiple of 16) from global to LDS with 16-byte loads; all of
// a thread's loads are issued before its stores.
template <int NT, int MAXPER>
__device__ __forceinline__ void stage_copy(uint4 *dst, const uint4 *src, int nbytes, int tid) {
    const int n = nbytes >> 4;
    uint4 r[MAXPER];
#pragma unroll
    for (int k = 0; k < MAXPER; ++k) {
        const int i = tid + k * NT;
        if (i < n) r[k] = src[i];
        else r[k] = make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int k = 0; k < MAXPER; ++k) {
        const int i = tid + k * NT;
        if (i < n) dst[i] = r[k];
    }
}

// packed vector product: acc[h] = chain over kept slots of (q[c][h], value)
template <int GP>
__device__ __forceinline__ void packed_dot(const uint32_t *bm, const uint16_t *vals, int log2g, int dtype,
                                           const float *qs /* [D][GP] */, float (&acc)[GP]) {
#pragma unroll
    for (int h = 0; h < GP; ++h) acc[h] = 0.0f;
    const int nwords = 4 >> log2g, gsz = 1 << log2g;
    int slot = 0;
    for (int wi = 0; wi < nwords; ++wi) {
        uint32_t bits = bm[wi];
        while (bits) {
            const int bpos = __builtin_ctz(bits);
            bits &= bits - 1u;
            const int c0 = (wi * 32 + bpos) << log2g;
            for (int e = 0; e < gsz; ++e) {
                const float v = h2f(vals[slot++], dtype);
                const float *qc = qs + (c0 + e) * GP;
#pragma unroll
                for (int h = 0; h < GP; ++h) acc[h] = fmaf(qc[h], v, acc[h]);
            }
        }
    }
}

// ------------------------------------------------------------------ qrot
__global__ void __launch_bounds__(256) k_qrot(Geom g, WsGeom ws, const uint16_t *q) {
    __shared__ __align__(16) float rt[D * D];
    __shared__ float qs[8][D];
    const int w = blockIdx.x, p = blockIdx.y, tid = threadIdx.x;
    const int G = g.G;
    for (int i = tid; i < G * D; i += 256) qs[i / D][i % D] = h2f(q[((uint64_t)p * G) * D + i], g.dtype);
    if (g.rotated) stage_copy<256, 16>((uint4 *)rt, (const uint4 *)g.rot_of(p, w), D * D * 4, tid);
    __syncthreads();
    if (tid >= D) return;
    const int j = tid;
    float acc[8];
#pragma unroll
    for (int h = 0; h < 8; ++h) acc[h] = 0.0f;
    if (g.rotated) {
        for (int c = 0; c < D; ++c) {           // R_k^T: rt[c*D + j] = R_k[j][c]
            const float r = rt[c * D + j];
#pragma unroll
            for (int h = 0; h < 8; ++h)
                if (h < G) acc[h] = fmaf(qs[h][c], r, acc[h]);
        }
    } else {
#pragma unroll
        for (int h = 0; h < 8; ++h) acc[h] = (h < G) ? qs[h][j] : 0.0f;
    }
    float *dst = ws.qrot + (uint64_t)p * (ws.qrot_stride / 4) + ((uint64_t)w * D + j) * g.GP;
#pragma unroll
    for (int h = 0; h < 8; ++h)
        if (h < g.GP) dst[h] = (h < G) ? acc[h] : 0.0f;
}

// ------------------------------------------------------------------ score
// Ascending set bits of a packed vector's bitmap (group indices), one at a time.
struct BitIter {
    uint32_t cur, w1, w2, w3;
    int base;
    __device__ __forceinline__ BitIter(uint32_t a, uint32_t b, uint32_t c, uint32_t d)
        : cur(a), w1(b), w2(c), w3(d), base(0) {}
    __device__ __forceinline__ int next() {
        while (cur == 0u) { cur = w1; w1 = w2; w2 = w3; w3 = 0u; base += 32; }
        const int b = __builtin_ctz(cur);
        cur &= cur - 1u;
        return base + b;
    }
};

// element s (static) of r packed 16-bit values held two per dword
template <int N>
__device__ __forceinline__ uint32_t half_at(const uint32_t (&v)[N], int s) {
    return (s & 1) ? (v[s >> 1] >> 16) : (v[s >> 1] & 0xffffu);
}

template <int GP, int RMAX>
__global__ void __launch_bounds__(256) k_score(Geom g, WsGeom ws, int spw, int stage_bytes) {
    extern __shared__ __align__(16) uint8_t smem[];
    float *qs = (float *)smem;                                   // [2][D][GP]
    Desc *ds = (Desc *)(smem + 2 * D * GP * 4);                   // [<= 32]
    int *bpre = (int *)(ds + 32);                                 // [<= 33]
    uint32_t *arena = (uint32_t *)(smem + 2 * D * GP * 4 + 32 * sizeof(Desc) + 48 * 4);   // 16-aligned

    const int p = blockIdx.y, tid = threadIdx.x;
    const PairMeta meta = *g.meta_of(p);
    int nf, prov, nbuf;
    const int ndesc = pair_ndesc(meta, nf, prov, nbuf);
    const int s0 = blockIdx.x * spw;
    if (s0 >= ndesc) return;
    const int ns = min(spw, ndesc - s0);
    const Desc *gd = g.desc_of(p);
    if (tid < ns) ds[tid] = gd[s0 + tid];
    __syncthreads();
    if (tid == 0) {
        int acc = 0;
        for (int i = 0; i < ns; ++i) {
            bpre[i] = acc;
            const int ntok = (ds[i].flags & 1) ? UBUF : SEG;
            acc += ntok >> ds[i].log2b;
        }
        bpre[ns] = acc;
    }
    const int w0 = (s0 * SEG) / g.W;
    const int qw0 = g.rotated ? w0 : 0;
    const int qw1 = g.rotated ? ((s0 + ns - 1) * SEG) / g.W : 0;
    {
        const float *src = ws.qrot + (uint64_t)p * (ws.qrot_stride / 4);
        for (int i = tid; i < D * GP; i += 256) {
            qs[i] = src[(uint64_t)qw0 * D * GP + i];
            qs[D * GP + i] = src[(uint64_t)qw1 * D * GP + i];
        }
    }
    const Desc dl = ds[ns - 1];
    const int ntl = (dl.flags & 1) ? UBUF : SEG;
    const uint32_t lo = ds[0].sc_off;
    const uint32_t hi = dl.sc_off + (uint32_t)(ntl >> dl.log2b) * (uint32_t)vec_bytes(dl.r, dl.log2g);
    const int nbytes = (int)((hi - lo + 15u) & ~15u);
    stage_copy<256, 12>((uint4 *)arena, (const uint4 *)(g.sc_of(p) + lo), min(nbytes, stage_bytes), tid);
    __syncthreads();
    const int nblk = bpre[ns];
    float *out = ws.score + (uint64_t)p * (ws.score_stride / 4);
    uint32_t *bseg = ws.bseg + (uint64_t)p * (ws.bseg_stride / 4);
    for (int b = tid; b < nblk; b += 256) {
        int i = 0;
        while (i + 1 < ns && bpre[i + 1] <= b) ++i;
        const Desc d = ds[i];
        const int j = b - bpre[i];
        const int r = d.r, l2g = d.log2g, nwd = 4 >> l2g, gm = (1 << l2g) - 1;
        const uint32_t *rp = arena + ((d.sc_off - lo + (uint32_t)j * vec_bytes(r, l2g)) >> 2);
        // the record: bitmap words, then r values (two per dword)
        BitIter it(rp[0], nwd > 1 ? rp[1] : 0u, nwd > 2 ? rp[2] : 0u, nwd > 3 ? rp[3] : 0u);
        uint32_t v[RMAX / 2];
#pragma unroll
        for (int k = 0; k < RMAX / 2; ++k) v[k] = (2 * k < r) ? rp[nwd + k] : 0u;
        const int w = ((s0 + i) * SEG) / g.W;
        const float *q = qs + ((g.rotated && w != w0) ? D * GP : 0);
        float acc[GP];
#pragma unroll
        for (int h = 0; h < GP; ++h) acc[h] = 0.0f;
        int cb = 0;
#pragma unroll
        for (int sl = 0; sl < RMAX; ++sl) {
            if (sl < r) {
                if ((sl & gm) == 0) cb = it.next() << l2g;
                const float *qc = q + (cb + (sl & gm)) * GP;
                const float x = h2f((uint16_t)half_at(v, sl), g.dtype);
#pragma unroll
                for (int h = 0; h < GP; ++h) acc[h] = fmaf(qc[h], x, acc[h]);
            }
        }
        float best = acc[0];
#pragma unroll
        for (int h = 1; h < GP; ++h)
            if (h < g.G) best = fmaxf(best, acc[h]);
        if (__float_as_uint(best) == 0x80000000u) best = 0.0f;
        out[d.first_block + j] = best;
        bseg[d.first_block + j] = ((uint32_t)(s0 + i) << 4) | (uint32_t)j;
    }
}

// ------------------------------------------------------------------ topk
constexpr int TOPK_LDS_KEYS = 32768;

__device__ uint32_t block_excl_scan_1024(uint32_t v, uint32_t *s) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    uint32_t x = v;                                      // inclusive wave scan
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) s[wv] = x;
    __syncthreads();
    if (tid < 16) {
        uint32_t t = s[tid];
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
            const uint32_t y = __shfl_up(t, off, 64);
            if (tid >= off) t += y;
        }
        s[16 + tid] = t;
    }
    __syncthreads();
    const uint32_t base = wv ? s[16 + wv - 1] : 0u;
    __syncthreads();
    return base + x - v;
}

__global__ void __launch_bounds__(1024) k_topk(Geom g, WsGeom ws) {
    extern __shared__ __align__(16) uint32_t keys[];            // [min(nb, TOPK_LDS_KEYS)] when staged
    __shared__ uint32_t hist[256];
    __shared__ uint32_t scan[64];
    __shared__ uint32_t s_prefix, s_rem;
    const int p = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const PairMeta meta = *g.meta_of(p);
    const int nb = pair_nblocks(g, p, meta);
    int nf, prov, nbuf;
    const int ndesc = pair_ndesc(meta, nf, prov, nbuf);
    int k = 0;
    if (nb > 0) {
        const long long kk = ((long long)nb * g.sel_num + g.sel_den - 1) / g.sel_den;
        k = (int)(kk < 1 ? 1 : (kk > nb ? nb : kk));
    }
    const float *sc = ws.score + (uint64_t)p * (ws.score_stride / 4);
    int32_t *sel = ws.sel + (uint64_t)p * (ws.sel_stride / 4);
    int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    const bool in_lds = nb <= TOPK_LDS_KEYS;
    if (in_lds) {
        for (int i0 = 0; i0 < nb; i0 += 1024 * 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) { const int i = i0 + u * 1024 + tid; v[u] = i < nb ? sc[i] : 0.0f; }
#pragma unroll
            for (int u = 0; u < 8; ++u) { const int i = i0 + u * 1024 + tid; if (i < nb) keys[i] = score_key(v[u]); }
        }
    }
    if (tid == 0) { s_prefix = 0; s_rem = (uint32_t)k; }
    __syncthreads();
    uint32_t mask = 0;
    for (int pass = 0; pass < 4 && k > 0; ++pass) {
        const int shift = 24 - 8 * pass;
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        const uint32_t prefix = s_prefix;
        for (int i = tid; i < nb; i += 1024) {
            const uint32_t key = in_lds ? keys[i] : score_key(sc[i]);
            if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (tid < 64) {
            // digit d: largest with count(digit >= d) >= rem; lane owns 4 digits, high to low
            const uint32_t rem = s_rem;
            uint32_t c4[4], own = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) { c4[u] = hist[255 - (lane * 4 + u)]; own += c4[u]; }
            uint32_t incl = own;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const uint32_t y = __shfl_up(incl, off, 64);
                if (lane >= off) incl += y;
            }
            const uint32_t excl = incl - own;
            if (excl < rem && incl >= rem) {
                uint32_t cum = excl;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (cum + c4[u] >= rem) {
                        s_prefix = prefix | ((uint32_t)(255 - (lane * 4 + u)) << shift);
                        s_rem = rem - cum;
                        break;
                    }
                    cum += c4[u];
                }
            }
        }
        mask |= 255u << shift;
        __syncthreads();
    }
    const uint32_t T = s_prefix, take_eq_total = s_rem;
    const int chunk = (nb + 1023) / 1024;
    const int i0 = min(nb, tid * chunk), i1 = min(nb, i0 + chunk);
    uint32_t gt = 0, eq = 0;
    if (k > 0)
        for (int i = i0; i < i1; ++i) {
            const uint32_t key = in_lds ? keys[i] : score_key(sc[i]);
            gt += key > T; eq += key == T;
        }
    const uint32_t eq_before = block_excl_scan_1024(eq, scan);
    uint32_t take = 0;
    if (take_eq_total > eq_before) take = min(eq, take_eq_total - eq_before);
    const uint32_t pos0 = block_excl_scan_1024(gt + take, scan);
    if (k > 0) {
        uint32_t pos = pos0, seen = 0;
        for (int i = i0; i < i1; ++i) {
            const uint32_t key = in_lds ? keys[i] : score_key(sc[i]);
            if (key > T) sel[pos++] = i;
            else if (key == T && seen < take) { sel[pos++] = i; ++seen; }
        }
    }
    __syncthreads();
    const int segs_per_win = g.W / SEG;
    const Desc *gd = g.desc_of(p);
    for (int w = tid; w < g.nw; w += 1024) {
        const int s = w * segs_per_win;
        const int fb = (s < ndesc) ? (int)gd[s].first_block : nb;
        int lo = 0, hi = k;
        while (lo < hi) { const int mid = (lo + hi) >> 1; if (sel[mid] < fb) lo = mid + 1; else hi = mid; }
        wsel[w] = lo;
    }
    if (tid == 0) { wsel[g.nw] = k; wsel[g.nw + 1] = nb; }
}

// ------------------------------------------------------------------ attention
struct BlkInfo { uint32_t goff; int16_t r, log2g, log2b, tok0; int32_t pad; };   // 16 bytes

__device__ __forceinline__ void split_of(const int32_t *wsel, int nw, int s, int &w_out, int &e0, int &e1,
                                         int &total) {
    int acc = 0;
    w_out = -2; e0 = e1 = 0;
    for (int w = 0; w < nw; ++w) {
        const int a = wsel[w], b = wsel[w + 1];
        const int nsp = (b - a + SPLIT_BLOCKS - 1) / SPLIT_BLOCKS;
        if (w_out == -2 && s < acc + nsp) {
            w_out = w;
            e0 = a + (s - acc) * SPLIT_BLOCKS;
            e1 = min(b, e0 + SPLIT_BLOCKS);
        }
        acc += nsp;
    }
    total = acc;
}

constexpr int CH_TOK = 64;           // tokens per chunk (one wave)
constexpr int KT_STRIDE = 136;       // u16 per token row of the K tile (128 + 8 pad)
constexpr int VT_STRIDE = 68;        // u16 per channel row of the V tile (64 + 4 pad)
constexpr int TILE_BYTES = 17408;    // max(64 * 272, 128 * 136)
constexpr int ATTN_NWV = 2;          // waves per attention workgroup
constexpr int MAX_CHUNKS = SPLIT_BLOCKS * 16 / CH_TOK;
// block table + chunk tables, rounded up to 16 bytes (pointer arithmetic on
// LDS stays in the LDS address space)
constexpr int ATTN_HDR_BYTES = (16 * SPLIT_BLOCKS + 4 * (2 * MAX_CHUNKS + 2) + 16 + 15) / 16 * 16;

template <int DT>
__device__ __forceinline__ typename Mma<DT>::v8 pack8(const uint16_t (&h)[8]) {
    uint4 u;
    u.x = h[0] | ((uint32_t)h[1] << 16); u.y = h[2] | ((uint32_t)h[3] << 16);
    u.z = h[4] | ((uint32_t)h[5] << 16); u.w = h[6] | ((uint32_t)h[7] << 16);
    return __builtin_bit_cast(typename Mma<DT>::v8, u);
}

// One token's packed K and V vectors, held in registers.
template <int RMAX>
struct TokRec {
    uint32_t kb[4], vb[4];          // bitmap words
    uint32_t kv[RMAX / 2], vv[RMAX / 2];   // values, two per dword
};

template <int RMAX>
__device__ __forceinline__ void load_tok(TokRec<RMAX> &t, const uint8_t *blkrec, int j, int r, int l2g, int B,
                                         bool valid) {
    const int bmb = 16 >> l2g, vb = 2 * r, nwd = 4 >> l2g;
    const uint32_t *kb = (const uint32_t *)(blkrec + j * bmb);
    const uint32_t *kv = (const uint32_t *)(blkrec + B * bmb + j * vb);
    const uint32_t *vbm = (const uint32_t *)(blkrec + B * (bmb + vb) + j * bmb);
    const uint32_t *vv = (const uint32_t *)(blkrec + B * (2 * bmb + vb) + j * vb);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        t.kb[k] = (valid && k < nwd) ? kb[k] : 0u;
        t.vb[k] = (valid && k < nwd) ? vbm[k] : 0u;
    }
#pragma unroll
    for (int k = 0; k < RMAX / 2; ++k) {
        t.kv[k] = (valid && 2 * k < r) ? kv[k] : 0u;
        t.vv[k] = (valid && 2 * k < r) ? vv[k] : 0u;
    }
}

// scatter a packed vector held in registers into a dense 16-bit tile:
// element c goes to base[c * cstride]; slots are walked in fixed order
template <int RMAX>
__device__ __forceinline__ void scatter_regs(const uint32_t (&bw)[4], const uint32_t (&vals)[RMAX / 2], int r,
                                             int l2g, uint16_t *base, int cstride) {
    BitIter it(bw[0], bw[1], bw[2], bw[3]);
    const int gm = (1 << l2g) - 1;
    int cb = 0;
#pragma unroll
    for (int sl = 0; sl < RMAX; ++sl) {
        if (sl < r) {
            if ((sl & gm) == 0) cb = it.next() << l2g;
            base[(cb + (sl & gm)) * cstride] = (uint16_t)half_at(vals, sl);
        }
    }
}

template <int DT, int GP, int RMAX, bool DBUF>
__global__ void __launch_bounds__(128) k_attn(Geom g, WsGeom ws, float scale, const uint16_t *qraw) {
    using M8 = typename Mma<DT>::v8;
    constexpr int NWV = ATTN_NWV;
    extern __shared__ __align__(16) uint8_t smem[];
    BlkInfo *blk = (BlkInfo *)smem;                         // [SPLIT_BLOCKS], sorted by block size
    int *ch_first = (int *)(blk + SPLIT_BLOCKS);            // [MAX_CHUNKS + 1]
    int *ch_ntok = ch_first + MAX_CHUNKS + 1;               // [MAX_CHUNKS]
    int *s_nch = ch_ntok + MAX_CHUNKS + 1;                  // [1]
    uint8_t *wbase = smem + ATTN_HDR_BYTES;                 // [NWV] tiles

    const int p = blockIdx.y, s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, q4 = lane >> 4;
    uint16_t *tile = (uint16_t *)(wbase + wave * TILE_BYTES);

    const PairMeta meta = *g.meta_of(p);
    int nf, prov, nbuf;
    pair_ndesc(meta, nf, prov, nbuf);
    const int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    const int32_t *sel = ws.sel + (uint64_t)p * (ws.sel_stride / 4);
    int w, e0, e1, total;
    split_of(wsel, g.nw, s, w, e0, e1, total);
    int32_t *tag = ws.tag + (uint64_t)p * (ws.tag_stride / 4);
    float *part = ws.part + (uint64_t)p * (ws.part_stride / 4) + (uint64_t)s * GP * (D + 2);
    const bool is_buf = (w == -2) && (s == total) && nbuf > 0;
    if (w == -2 && !is_buf) {
        if (tid == 0) tag[s] = -2;
        return;
    }
    const int G = g.G;

    if (is_buf) {
        // update-buffer tokens: dense and unrotated (Sec. 5.3), VALU on wave 0
        float *qsb = (float *)wbase;                        // [D][GP]
        float *psb = qsb + D * GP;                          // [64][GP]
        for (int i = tid; i < D * GP; i += NWV * 64) {
            const int c = i / GP, h = i % GP;
            qsb[i] = (h < G) ? h2f(qraw[((uint64_t)p * G + h) * D + c], g.dtype) : 0.0f;
        }
        __syncthreads();
        if (wave == 0) {
            const uint16_t *bk = g.buf_of(p), *bv = bk + UBUF * D;
            float z[GP], bm[GP], bl[GP], ba[GP][2];
#pragma unroll
            for (int h = 0; h < GP; ++h) z[h] = 0.0f;
            const bool valid = lane < nbuf;
            if (valid)
                for (int c = 0; c < D; ++c) {
                    const float kv = h2f(bk[lane * D + c], g.dtype);
#pragma unroll
                    for (int h = 0; h < GP; ++h) z[h] = fmaf(qsb[c * GP + h], kv, z[h]);
                }
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                const float zz = valid ? z[h] * scale : -INFINITY;
                const float m = wave_max(zz);
                const float pv = valid ? __expf(zz - m) : 0.0f;
                bm[h] = m;
                bl[h] = wave_sum(pv);
                psb[lane * GP + h] = pv;
                ba[h][0] = ba[h][1] = 0.0f;
            }
            wave_sync();
            for (int t = 0; t < nbuf; ++t) {
                const float vlo = h2f(bv[t * D + lane], g.dtype), vhi = h2f(bv[t * D + lane + 64], g.dtype);
#pragma unroll
                for (int h = 0; h < GP; ++h) {
                    const float pv = psb[t * GP + h];
                    ba[h][0] = fmaf(pv, vlo, ba[h][0]);
                    ba[h][1] = fmaf(pv, vhi, ba[h][1]);
                }
            }
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                part[2 * GP + h * D + lane] = ba[h][0];
                part[2 * GP + h * D + lane + 64] = ba[h][1];
                if (lane == 0) { part[h] = bm[h]; part[GP + h] = bl[h]; }
            }
            if (lane == 0) tag[s] = -1;
        }
        return;
    }

    // ---- split setup (wave 0): blocks sorted by size (16, 8, 4; stable), so
    // every block starts at a multiple of its size and no block straddles a
    // 64-token chunk; chunk c holds tokens [64c, 64c + 64) of the sorted run
    const int nbk = e1 - e0;
    if (wave == 0) {
        const bool on = lane < nbk;
        uint32_t goff = 0; int r = 0, l2g = 0, l2b = 0;
        if (on) {
            const uint32_t bs = ws.bseg[(uint64_t)p * (ws.bseg_stride / 4) + sel[e0 + lane]];
            const Desc d = g.desc_of(p)[bs >> 4];
            const int jb = (int)(bs & 15u);
            r = d.r; l2g = d.log2g; l2b = d.log2b;
            goff = d.tok_off + (uint32_t)(jb << l2b) * (uint32_t)(2 * vec_bytes(r, l2g));
        }
        const uint64_t m16 = __ballot(on && l2b == 4), m8 = __ballot(on && l2b == 3), m4 = __ballot(on && l2b == 2);
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        const int c16 = __popcll(m16), c8 = __popcll(m8), c4 = __popcll(m4);
        int pos = 0, off = 0;
        if (l2b == 4) { const int rk = __popcll(m16 & below); pos = rk; off = 16 * rk; }
        else if (l2b == 3) { const int rk = __popcll(m8 & below); pos = c16 + rk; off = 16 * c16 + 8 * rk; }
        else { const int rk = __popcll(m4 & below); pos = c16 + c8 + rk; off = 16 * c16 + 8 * c8 + 4 * rk; }
        if (on) {
            BlkInfo bi;
            bi.goff = goff; bi.r = (int16_t)r; bi.log2g = (int16_t)l2g; bi.log2b = (int16_t)l2b;
            bi.tok0 = (int16_t)(off & (CH_TOK - 1)); bi.pad = 0;
            blk[pos] = bi;
            if ((off & (CH_TOK - 1)) == 0) ch_first[off / CH_TOK] = pos;
        }
        const int T = 16 * c16 + 8 * c8 + 4 * c4;
        const int nch = (T + CH_TOK - 1) / CH_TOK;
        if (lane < nch) ch_ntok[lane] = min(CH_TOK, T - CH_TOK * lane);
        if (lane == 0) { ch_first[nch] = nbk; s_nch[0] = nch; }
    }
    // q operand: B[k = channel][n = head] of the logits K . q^T, split hi + lo
    M8 qhi[4], qlo[4];
    {
        const int qw = g.rotated ? w : 0;
        const float *src = ws.qrot + (uint64_t)p * (ws.qrot_stride / 4) + (uint64_t)qw * D * GP;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            uint16_t hh[8], ll[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = ks * 32 + q4 * 8 + i;
                const float x = (l16 < G) ? src[c * GP + (l16 < GP ? l16 : 0)] : 0.0f;
                hh[i] = f2h(x, DT);
                ll[i] = f2h(x - h2f(hh[i], DT), DT);
            }
            qhi[ks] = pack8<DT>(hh);
            qlo[ks] = pack8<DT>(ll);
        }
    }
    __syncthreads();
    const int nch = s_nch[0];
    const uint8_t *tokg = g.tok_of(p);

    float m_run = -INFINITY, l_run = 0.0f;                  // head l16
    floatx4 acc_o[8];                                       // [channel tile][head 4*q4 + r]
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) acc_o[ct] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    // this lane's token of chunk c: block info and index inside the block
    auto locate = [&](int c, BlkInfo &info, int &j, bool &valid) {
        int bi = ch_first[c];
        const int b1 = ch_first[c + 1];
        while (bi + 1 < b1 && blk[bi + 1].tok0 > 0 && blk[bi + 1].tok0 <= lane) ++bi;
        info = blk[bi];
        j = lane - info.tok0;
        valid = lane < ch_ntok[c];
    };
    auto process = [&](const TokRec<RMAX> &t, const BlkInfo &info, bool valid, int ntok) {
        // ---- K: zero the tile, scatter packed keys (token-major rows), logits on MFMA
        {
            uint4 *t4 = (uint4 *)tile;
            const uint4 zz = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int k = 0; k < TILE_BYTES / 16 / 64; ++k) t4[lane + k * 64] = zz;
        }
        wave_sync();
        if (valid) scatter_regs<RMAX>(t.kb, t.kv, info.r, info.log2g, tile + lane * KT_STRIDE, 1);
        wave_sync();
        float z[4][4];
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            floatx4 a4 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const uint4 kv = *(const uint4 *)(tile + (n * 16 + l16) * KT_STRIDE + ks * 32 + q4 * 8);
                const M8 a = __builtin_bit_cast(M8, kv);
                a4 = Mma<DT>::run(a, qhi[ks], a4);
                a4 = Mma<DT>::run(a, qlo[ks], a4);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tt = n * 16 + q4 * 4 + r;
                z[n][r] = (tt < ntok) ? a4[r] * scale : -INFINITY;
            }
        }
        // ---- online softmax for head l16 (tokens across r, n and the lane quarters)
        float cm = -INFINITY;
#pragma unroll
        for (int n = 0; n < 4; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) cm = fmaxf(cm, z[n][r]);
        cm = fmaxf(cm, __shfl_xor(cm, 16, 64));
        cm = fmaxf(cm, __shfl_xor(cm, 32, 64));
        const float mn = fmaxf(m_run, cm);
        const float alpha = (m_run == -INFINITY) ? 0.0f : __expf(m_run - mn);
        float ls = 0.0f;
#pragma unroll
        for (int n = 0; n < 4; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                z[n][r] = (z[n][r] == -INFINITY) ? 0.0f : __expf(z[n][r] - mn);
                ls += z[n][r];
            }
        ls += __shfl_xor(ls, 16, 64);
        ls += __shfl_xor(ls, 32, 64);
        l_run = l_run * alpha + ls;
        m_run = mn;
        // ---- V: zero the tile, scatter packed values (channel-major rows)
        wave_sync();
        {
            uint4 *t4 = (uint4 *)tile;
            const uint4 zz = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int k = 0; k < TILE_BYTES / 16 / 64; ++k) t4[lane + k * 64] = zz;
        }
        wave_sync();
        if (valid) scatter_regs<RMAX>(t.vb, t.vv, info.r, info.log2g, tile + lane, VT_STRIDE);
        wave_sync();
        // ---- P . V on MFMA: A = P[head l16][tokens], B = V[tokens][channel tile]
        float ar[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) ar[r] = __shfl(alpha, q4 * 4 + r, 64);
#pragma unroll
        for (int ct = 0; ct < 8; ++ct)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc_o[ct][r] *= ar[r];
#pragma unroll
        for (int kv = 0; kv < 2; ++kv) {
            uint16_t hh[8], ll[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const float x = z[2 * kv + (i >> 2)][i & 3];
                hh[i] = f2h(x, DT);
                ll[i] = f2h(x - h2f(hh[i], DT), DT);
            }
            const M8 ah = pack8<DT>(hh), al = pack8<DT>(ll);
#pragma unroll
            for (int ct = 0; ct < 8; ++ct) {
                const uint16_t *row = tile + (ct * 16 + l16) * VT_STRIDE + kv * 32 + q4 * 4;
                const uint2 v0 = *(const uint2 *)row, v1 = *(const uint2 *)(row + 16);
                const uint4 vv4 = {v0.x, v0.y, v1.x, v1.y};
                const M8 bv = __builtin_bit_cast(M8, vv4);
                acc_o[ct] = Mma<DT>::run(ah, bv, acc_o[ct]);
                acc_o[ct] = Mma<DT>::run(al, bv, acc_o[ct]);
            }
        }
        wave_sync();
    };

    if (DBUF) {
        // two register sets: the next chunk's loads are in flight while one is processed
        TokRec<RMAX> ta, tb;
        BlkInfo ia, ib;
        int ja = 0, jb = 0;
        bool va = false, vb = false;
        int c = wave;
        if (c < nch) {
            locate(c, ia, ja, va);
            load_tok<RMAX>(ta, tokg + ia.goff, ja, ia.r, ia.log2g, 1 << ia.log2b, va);
        }
        for (; c < nch; c += 2 * NWV) {
            const int cn = c + NWV;
            if (cn < nch) {
                locate(cn, ib, jb, vb);
                load_tok<RMAX>(tb, tokg + ib.goff, jb, ib.r, ib.log2g, 1 << ib.log2b, vb);
            }
            process(ta, ia, va, ch_ntok[c]);
            if (cn >= nch) break;
            const int cnn = cn + NWV;
            if (cnn < nch) {
                locate(cnn, ia, ja, va);
                load_tok<RMAX>(ta, tokg + ia.goff, ja, ia.r, ia.log2g, 1 << ia.log2b, va);
            }
            process(tb, ib, vb, ch_ntok[cn]);
        }
    } else {
        for (int c = wave; c < nch; c += NWV) {
            TokRec<RMAX> t;
            BlkInfo info;
            int j = 0;
            bool valid = false;
            locate(c, info, j, valid);
            load_tok<RMAX>(t, tokg + info.goff, j, info.r, info.log2g, 1 << info.log2b, valid);
            process(t, info, valid, ch_ntok[c]);
        }
    }
    // ---- merge the waves' (m, l, acc) and write the split's partial
    __syncthreads();
    float *mrg = (float *)(wbase + wave * TILE_BYTES);      // [16][D + 2]
    if (q4 == 0) { mrg[l16 * (D + 2)] = m_run; mrg[l16 * (D + 2) + 1] = l_run; }
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r) mrg[(q4 * 4 + r) * (D + 2) + 2 + ct * 16 + l16] = acc_o[ct][r];
    __syncthreads();
    for (int i = tid; i < GP * D; i += NWV * 64) {
        const int h = i / D, cc = i % D;
        float Mx = -INFINITY;
#pragma unroll
        for (int x = 0; x < NWV; ++x) Mx = fmaxf(Mx, ((const float *)(wbase + x * TILE_BYTES))[h * (D + 2)]);
        float A = 0.0f, Ls = 0.0f;
#pragma unroll
        for (int x = 0; x < NWV; ++x) {
            const float *mw = (const float *)(wbase + x * TILE_BYTES);
            const float f = (mw[h * (D + 2)] == -INFINITY) ? 0.0f : __expf(mw[h * (D + 2)] - Mx);
            A += mw[h * (D + 2) + 2 + cc] * f;
            Ls += mw[h * (D + 2) + 1] * f;
        }
        part[2 * GP + h * D + cc] = A;
        if (cc == 0) { part[h] = Mx; part[GP + h] = Ls; }
    }
    if (tid == 0) tag[s] = w;
}

// ------------------------------------------------------------------ reduce
constexpr int REDUCE_MAX_SPLITS = 1024;

template <int GP>
__global__ void __launch_bounds__(256) k_reduce(Geom g, WsGeom ws, float *out) {
    __shared__ __align__(16) float rv[D * D];
    __shared__ float A[GP][D];
    extern __shared__ __align__(16) float hdr[];            // [nsplit][2 GP + 1]: m, l, tag
    const int p = blockIdx.x, tid = threadIdx.x, G = g.G;
    const PairMeta meta = *g.meta_of(p);
    float *o = out + (uint64_t)p * G * D;
    const int32_t *tag = ws.tag + (uint64_t)p * (ws.tag_stride / 4);
    const float *part = ws.part + (uint64_t)p * (ws.part_stride / 4);
    const int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    int nf, prov, nbuf;
    pair_ndesc(meta, nf, prov, nbuf);
    int w_, e0_, e1_, total;
    split_of(wsel, g.nw, 0, w_, e0_, e1_, total);
    const int nsplit = min(total + (nbuf > 0 ? 1 : 0), REDUCE_MAX_SPLITS);
    constexpr int HW = 2 * GP + 1;
    for (int i = tid; i < nsplit * HW; i += 256) {
        const int s = i / HW, k = i % HW;
        hdr[i] = (k < 2 * GP) ? part[(uint64_t)s * GP * (D + 2) + k] : __int_as_float(tag[s]);
    }
    __syncthreads();
    constexpr int HPT = GP / 2;                    // heads per thread; thread (half, j)
    const int j = tid & 127, hb = (tid >> 7) * HPT;
    float Mg[HPT], Lg[HPT], Og[HPT];
#pragma unroll
    for (int u = 0; u < HPT; ++u) { Mg[u] = -INFINITY; Lg[u] = 0.0f; Og[u] = 0.0f; }
    for (int w = -1; w < g.nw; ++w) {              // -1 = update buffer
        // per head: window max and its weights (every thread computes its own heads)
        float M[HPT];
        bool any = false;
#pragma unroll
        for (int u = 0; u < HPT; ++u) M[u] = -INFINITY;
        for (int s = 0; s < nsplit; ++s) {
            if (__float_as_int(hdr[s * HW + 2 * GP]) != w) continue;
            any = true;
#pragma unroll
            for (int u = 0; u < HPT; ++u) M[u] = fmaxf(M[u], hdr[s * HW + hb + u]);
        }
        if (!any) continue;                         // uniform: the same for every thread
        const bool rot = (w >= 0) && g.rotated;
        __syncthreads();
        if (rot) stage_copy<256, 16>((uint4 *)rv, (const uint4 *)(g.rot_of(p, w) + 2 * D * D), D * D * 4, tid);
        float Lw[HPT], Aw[HPT];
#pragma unroll
        for (int u = 0; u < HPT; ++u) { Lw[u] = 0.0f; Aw[u] = 0.0f; }
        for (int s0 = 0; s0 < nsplit; s0 += 8) {
            float av[8][HPT];
#pragma unroll
            for (int x = 0; x < 8; ++x) {            // issue the loads of 8 splits together
                const int s = s0 + x;
                const bool use = s < nsplit && __float_as_int(hdr[s * HW + 2 * GP]) == w;
#pragma unroll
                for (int u = 0; u < HPT; ++u)
                    av[x][u] = use ? part[(uint64_t)s * GP * (D + 2) + 2 * GP + (hb + u) * D + j] : 0.0f;
            }
#pragma unroll
            for (int x = 0; x < 8; ++x) {
                const int s = s0 + x;
                if (s >= nsplit || __float_as_int(hdr[s * HW + 2 * GP]) != w) continue;
#pragma unroll
                for (int u = 0; u < HPT; ++u) {
                    const float m = hdr[s * HW + hb + u];
                    const float f = (m == -INFINITY) ? 0.0f : __expf(m - M[u]);
                    Aw[u] += av[x][u] * f;
                    Lw[u] += hdr[s * HW + GP + hb + u] * f;
                }
            }
        }
        float Ow[HPT];
        if (rot) {
#pragma unroll
            for (int u = 0; u < HPT; ++u) A[hb + u][j] = Aw[u];
            __syncthreads();
#pragma unroll
            for (int u = 0; u < HPT; ++u) Ow[u] = 0.0f;
            for (int c = 0; c < D; ++c) {
                const float r = rv[c * D + j];              // R_v[c][j]: x = y . R
#pragma unroll
                for (int u = 0; u < HPT; ++u) Ow[u] = fmaf(A[hb + u][c], r, Ow[u]);
            }
        } else {
#pragma unroll
            for (int u = 0; u < HPT; ++u) Ow[u] = Aw[u];
        }
#pragma unroll
        for (int u = 0; u < HPT; ++u) {
            if (M[u] == -INFINITY) continue;
            const float mn = fmaxf(Mg[u], M[u]);
            const float a = (Mg[u] == -INFINITY) ? 0.0f : __expf(Mg[u] - mn), b = __expf(M[u] - mn);
            Og[u] = Og[u] * a + Ow[u] * b;
            Lg[u] = Lg[u] * a + Lw[u] * b;
            Mg[u] = mn;
        }
    }
#pragma unroll
    for (int u = 0; u < HPT; ++u)
        if (hb + u < G) o[(hb + u) * D + j] = (Lg[u] > 0.0f) ? Og[u] / Lg[u] : 0.0f;
}

int max_record_bytes(const Geom &g) {
    int maxrec = 2 * g.def_keep + (16 >> (31 - __builtin_clz(g.def_group)));
    for (int i = 0; i < 3; ++i)
        for (int k = 0; k < 3; ++k)
            maxrec = max(maxrec, 2 * g.keep_cand[i] + (16 >> (31 - __builtin_clz(g.group_cand[k]))));
    return maxrec;
}

template <int DT, int GP>
hipError_t launch_attn(const Geom &g, const WsGeom &w, const uint16_t *q, float scale, hipStream_t s) {
    const size_t smem = ATTN_HDR_BYTES + (size_t)ATTN_NWV * TILE_BYTES;
    const dim3 grid(w.max_splits, g.npairs), block(64 * ATTN_NWV);
    if (max_record_bytes(g) <= 2 * 48 + 16)
        hipLaunchKernelGGL((k_attn<DT, GP, 48, true>), grid, block, smem, s, g, w, scale, q);
    else
        hipLaunchKernelGGL((k_attn<DT, GP, 128, false>), grid, block, smem, s, g, w, scale, q);
    return hipGetLastError();
}

template <int GP>
hipError_t launch_decode_t(const Geom &g, const WsGeom &w, const uint16_t *q, float *out, float scale,
                           int max_desc_used, int max_windows_used, hipStream_t s, hipEvent_t *ev) {
    const int nwq = g.rotated ? max_windows_used : 1;
    if (ev) hipEventRecord(ev[0], s);
    hipLaunchKernelGGL(k_qrot, dim3(nwq, g.npairs), dim3(256), 0, s, g, w, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // block scoring: stage at most 48 KiB of score records per workgroup
    const int maxrec = max_record_bytes(g);
    int minb = g.def_block;
    for (int i = 0; i < 3; ++i) minb = min(minb, g.block_cand[i]);
    const int seg_bytes = (SEG / minb) * maxrec;
    int spw = min(SCORE_SEGS, max(1, 49152 / seg_bytes));
    spw = min(spw, max(1, g.W / SEG));
    const int stage_bytes = ((spw * seg_bytes) + 31) & ~15;
    const size_t score_smem = 2 * D * GP * 4 + 32 * sizeof(Desc) + 48 * 4 + stage_bytes;
    if (ev) hipEventRecord(ev[1], s);
    if (max_desc_used > 0) {
        if (maxrec <= 2 * 48 + 16)
            hipLaunchKernelGGL((k_score<GP, 48>), dim3(ceil_div(max_desc_used, spw), g.npairs), dim3(256), score_smem, s,
                               g, w, spw, stage_bytes);
        else
            hipLaunchKernelGGL((k_score<GP, 128>), dim3(ceil_div(max_desc_used, spw), g.npairs), dim3(256), score_smem,
                               s, g, w, spw, stage_bytes);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (ev) hipEventRecord(ev[2], s);
    const size_t topk_smem = (size_t)min(w.max_blocks, TOPK_LDS_KEYS) * 4;
    hipLaunchKernelGGL(k_topk, dim3(g.npairs), dim3(1024), topk_smem, s, g, w);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev) hipEventRecord(ev[3], s);
    e = g.dtype ? launch_attn<1, GP>(g, w, q, scale, s) : launch_attn<0, GP>(g, w, q, scale, s);
    if (e != hipSuccess) return e;
    if (ev) hipEventRecord(ev[4], s);
    const size_t red_smem = (size_t)min(w.max_splits, REDUCE_MAX_SPLITS) * (2 * GP + 1) * 4;
    hipLaunchKernelGGL(k_reduce<GP>, dim3(g.npairs), dim3(256), red_smem, s, g, w, out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev) hipEventRecord(ev[5], s);
    return hipSuccess;
}

}  // namespace

hipError_t launch_decode(const Geom &g, const WsGeom &w, const uint16_t *q, float *out, float scale,
                         int max_desc_used, int max_windows_used, hipStream_t s, hipEvent_t *ev) {
    if (g.GP == 4) return launch_decode_t<4>(g, w, q, out, scale, max_desc_used, max_windows_used, s, ev);
    return launch_decode_t<8>(g, w, q, out, scale, max_desc_used, max_windows_used, s, ev);
}

}  // namespace mosaic
