// decode.hip -- gfx950 kernels of MosaicKV's decode step (PackedAttention,
// Sec. 5.3; stage-2 dynamic sequence compression, Sec. 4.2).
//
//   qrot   : q . R_k^T once per (pair, window): the rotation is merged into
//            the single query vector instead of un-rotating the cache.
//   score  : every block key of a pair streamed once; lane per block key, a
//            packed vector product walking the bitmap's set bits in
//            ascending order, fp32 fused chain, max over the GQA group.
//   topk   : exact radix select of the k-th largest score key (8-bit
//            digits, LDS histograms), then an ordered compaction that breaks
//            ties by the lowest block index.
//   attn   : split-K over the selected list (64 blocks per workgroup, one
//            rotation window per split): lane per token for q . k on the
//            packed key, online softmax in fp32, lane per channel pair for
//            P . V on the packed value; the update buffer is one more split.
//   reduce : log-sum-exp merge of the splits per window, back-rotation of
//            each window's accumulator by R_v, merge of windows and buffer.
#include "mosaic_internal.h"

namespace mosaic {

namespace {

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
__global__ void __launch_bounds__(128) k_qrot(Geom g, WsGeom ws, const uint16_t *q) {
    __shared__ float qs[8][D];
    const int w = blockIdx.x, p = blockIdx.y, j = threadIdx.x;
    const int G = g.G;
    for (int i = threadIdx.x; i < G * D; i += 128) qs[i / D][i % D] = h2f(q[((uint64_t)p * G) * D + i], g.dtype);
    __syncthreads();
    float acc[8];
#pragma unroll
    for (int h = 0; h < 8; ++h) acc[h] = 0.0f;
    if (g.rotated) {
        const float *rt = g.rot_of(p, w);          // R_k^T: rt[c*D + j] = R_k[j][c]
        for (int c = 0; c < D; ++c) {
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
template <int GP>
__global__ void __launch_bounds__(256) k_score(Geom g, WsGeom ws, int spw, int stage_bytes) {
    extern __shared__ __align__(16) uint8_t smem[];
    float *qs = (float *)smem;                                   // [2][D][GP]
    Desc *ds = (Desc *)(smem + 2 * D * GP * 4);                   // [spw]
    int *bpre = (int *)(ds + 32);                                 // [spw + 1]
    uint32_t *arena = (uint32_t *)(bpre + 34);                    // staged score records

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
    const int nwords = (int)((hi - lo) >> 2);
    const uint32_t *src = (const uint32_t *)(g.sc_of(p) + lo);
    for (int i = tid; i < nwords; i += 256) arena[i] = src[i];
    __syncthreads();
    const int nblk = bpre[ns];
    float *out = ws.score + (uint64_t)p * (ws.score_stride / 4);
    for (int b = tid; b < nblk; b += 256) {
        int i = 0;
        while (i + 1 < ns && bpre[i + 1] <= b) ++i;
        const Desc d = ds[i];
        const int j = b - bpre[i];
        const int rec = vec_bytes(d.r, d.log2g);
        const uint32_t off = d.sc_off - lo + (uint32_t)j * rec;
        const uint32_t *bm = arena + (off >> 2);
        const uint16_t *vals = (const uint16_t *)(arena) + ((off + (16 >> d.log2g)) >> 1);
        const int w = ((s0 + i) * SEG) / g.W;
        const float *q = qs + ((g.rotated && w != w0) ? D * GP : 0);
        float acc[GP];
        packed_dot<GP>(bm, vals, d.log2g, g.dtype, q, acc);
        float best = acc[0];
#pragma unroll
        for (int h = 1; h < GP; ++h)
            if (h < g.G) best = fmaxf(best, acc[h]);
        if (__float_as_uint(best) == 0x80000000u) best = 0.0f;
        out[d.first_block + j] = best;
    }
}

// ------------------------------------------------------------------ topk
__device__ uint32_t block_excl_scan_1024(uint32_t v, uint32_t *s) {
    const int tid = threadIdx.x;
    s[tid] = v;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        uint32_t a = (tid >= off) ? s[tid - off] : 0u;
        __syncthreads();
        s[tid] += a;
        __syncthreads();
    }
    uint32_t r = s[tid] - v;
    __syncthreads();
    return r;
}

__global__ void __launch_bounds__(1024) k_topk(Geom g, WsGeom ws) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t scan[1024];
    __shared__ uint32_t s_prefix, s_rem;
    const int p = blockIdx.x, tid = threadIdx.x;
    const PairMeta meta = *g.meta_of(p);
    const int nb = pair_nblocks(g, p, meta);
    int nf, prov, nbuf;
    const int ndesc = pair_ndesc(meta, nf, prov, nbuf);
    int k = 0;
    if (nb > 0) {
        long long kk = ((long long)nb * g.sel_num + g.sel_den - 1) / g.sel_den;
        k = (int)(kk < 1 ? 1 : (kk > nb ? nb : kk));
    }
    const float *sc = ws.score + (uint64_t)p * (ws.score_stride / 4);
    int32_t *sel = ws.sel + (uint64_t)p * (ws.sel_stride / 4);
    int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    if (tid == 0) { s_prefix = 0; s_rem = (uint32_t)k; }
    __syncthreads();
    uint32_t mask = 0;
    for (int pass = 0; pass < 4 && k > 0; ++pass) {
        const int shift = 24 - 8 * pass;
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        const uint32_t prefix = s_prefix;
        for (int i = tid; i < nb; i += 1024) {
            const uint32_t key = score_key(sc[i]);
            if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (tid == 0) {
            uint32_t cum = 0, rem = s_rem;
            for (int dgt = 255; dgt >= 0; --dgt) {
                if (cum + hist[dgt] >= rem) { s_prefix = prefix | ((uint32_t)dgt << shift); s_rem = rem - cum; break; }
                cum += hist[dgt];
            }
        }
        mask |= 255u << shift;
        __syncthreads();
    }
    const uint32_t T = s_prefix, take_eq_total = s_rem;
    // ordered compaction: all keys > T, and the first take_eq_total keys == T
    const int chunk = (nb + 1023) / 1024;
    const int i0 = min(nb, tid * chunk), i1 = min(nb, i0 + chunk);
    uint32_t gt = 0, eq = 0;
    if (k > 0)
        for (int i = i0; i < i1; ++i) {
            const uint32_t key = score_key(sc[i]);
            gt += key > T; eq += key == T;
        }
    const uint32_t eq_before = block_excl_scan_1024(eq, scan);
    uint32_t take = 0;
    if (take_eq_total > eq_before) take = min(eq, take_eq_total - eq_before);
    const uint32_t pos0 = block_excl_scan_1024(gt + take, scan);
    if (k > 0) {
        uint32_t pos = pos0, seen = 0;
        for (int i = i0; i < i1; ++i) {
            const uint32_t key = score_key(sc[i]);
            if (key > T) sel[pos++] = i;
            else if (key == T && seen < take) { sel[pos++] = i; ++seen; }
        }
    }
    __syncthreads();
    // first selected entry of every rotation window
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
struct BlkInfo { uint32_t off; int r, log2g, log2b; };

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

// value of channel c of a packed vector (0 if dropped)
__device__ __forceinline__ float packed_channel(const uint32_t *bm, const uint16_t *vals, int c, int log2g, int dtype) {
    const int gi = c >> log2g, wi = gi >> 5, bit = gi & 31;
    const uint32_t word = bm[wi];
    if (!((word >> bit) & 1u)) return 0.0f;
    int cnt = 0;
    for (int x = 0; x < wi; ++x) cnt += __popc(bm[x]);
    cnt += __popc(word & ((1u << bit) - 1u));
    return h2f(vals[(cnt << log2g) + (c & ((1 << log2g) - 1))], dtype);
}

template <int GP>
__global__ void __launch_bounds__(256) k_attn(Geom g, WsGeom ws, float scale, const uint16_t *qraw, int slot_dw) {
    extern __shared__ __align__(16) uint8_t smem[];
    float *qs = (float *)smem;                                     // [D][GP]
    BlkInfo *blk = (BlkInfo *)(qs + D * GP);                       // [SPLIT_BLOCKS]
    int *tstart = (int *)(blk + SPLIT_BLOCKS);                     // [SPLIT_BLOCKS + 1]
    float *ps = (float *)(tstart + SPLIT_BLOCKS + 2);              // [4][64][GP]
    float *mrg = ps + 4 * 64 * GP;                                 // [4][GP][D + 2]
    int *tl2g = (int *)(mrg + 4 * GP * (D + 2));                   // [256] log2 g of each lane's token
    uint32_t *slots = (uint32_t *)(tl2g + 256);                    // [256][slot_dw]

    const int p = blockIdx.y, s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const PairMeta meta = *g.meta_of(p);
    int nf, prov, nbuf;
    const int ndesc = pair_ndesc(meta, nf, prov, nbuf);
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
    float m_run[GP], l_run[GP], acc[GP][2];
#pragma unroll
    for (int h = 0; h < GP; ++h) { m_run[h] = -INFINITY; l_run[h] = 0.0f; acc[h][0] = acc[h][1] = 0.0f; }

    if (is_buf) {
        // update-buffer tokens: dense, unrotated (Sec. 5.3)
        for (int i = tid; i < D * GP; i += 256) {
            const int c = i / GP, h = i % GP;
            qs[i] = (h < G) ? h2f(qraw[((uint64_t)p * G + h) * D + c], g.dtype) : 0.0f;
        }
        __syncthreads();
        const uint16_t *bk = g.buf_of(p), *bv = bk + UBUF * D;
        if (wave == 0) {
            float z[GP];
#pragma unroll
            for (int h = 0; h < GP; ++h) z[h] = 0.0f;
            const bool valid = lane < nbuf;
            if (valid)
                for (int c = 0; c < D; ++c) {
                    const float kv = h2f(bk[lane * D + c], g.dtype);
#pragma unroll
                    for (int h = 0; h < GP; ++h) z[h] = fmaf(qs[c * GP + h], kv, z[h]);
                }
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                const float zz = valid ? z[h] * scale : -INFINITY;
                const float m = wave_max(zz);
                const float pv = valid ? __expf(zz - m) : 0.0f;
                m_run[h] = m;
                l_run[h] = wave_sum(pv);
                ps[lane * GP + h] = pv;
            }
        }
        __syncthreads();
        if (wave == 0) {
            for (int t = 0; t < nbuf; ++t) {
                const float vlo = h2f(bv[t * D + lane], g.dtype), vhi = h2f(bv[t * D + lane + 64], g.dtype);
#pragma unroll
                for (int h = 0; h < GP; ++h) {
                    const float pv = ps[t * GP + h];
                    acc[h][0] = fmaf(pv, vlo, acc[h][0]);
                    acc[h][1] = fmaf(pv, vhi, acc[h][1]);
                }
            }
        }
    } else {
        const int nbk = e1 - e0;
        if (tid < nbk) {
            const int b = sel[e0 + tid];
            const Desc *gd = g.desc_of(p);
            int lo = 0, hi = ndesc - 1;                 // last descriptor with first_block <= b
            while (lo < hi) { const int mid = (lo + hi + 1) >> 1; if ((int)gd[mid].first_block <= b) lo = mid; else hi = mid - 1; }
            const Desc d = gd[lo];
            const int j = b - (int)d.first_block;
            const int rec = vec_bytes(d.r, d.log2g);
            BlkInfo bi;
            bi.off = d.tok_off + (uint32_t)(j << d.log2b) * (uint32_t)(2 * rec);
            bi.r = d.r; bi.log2g = d.log2g; bi.log2b = d.log2b;
            blk[tid] = bi;
        }
        const int qw = g.rotated ? w : 0;
        const float *src = ws.qrot + (uint64_t)p * (ws.qrot_stride / 4) + (uint64_t)qw * D * GP;
        for (int i = tid; i < D * GP; i += 256) qs[i] = src[i];
        __syncthreads();
        if (tid == 0) {
            int a = 0;
            for (int i = 0; i < nbk; ++i) { tstart[i] = a; a += 1 << blk[i].log2b; }
            tstart[nbk] = a;
        }
        __syncthreads();
        const int T = tstart[nbk];
        const uint8_t *tok = g.tok_of(p);
        uint32_t *myslot = slots + (uint64_t)tid * slot_dw;
        const int nchunks = (T + 63) / 64;
        for (int ch = 0; ch < (nchunks + 3) / 4; ++ch) {     // uniform trip count across waves
            const int c64 = ch * 4 + wave;
            const int tau = c64 * 64 + lane;
            const bool valid = tau < T;
            int i = 0, j = 0;
            BlkInfo bi = blk[0];
            if (valid) {
                while (i + 1 < nbk && tstart[i + 1] <= tau) ++i;
                j = tau - tstart[i];
                bi = blk[i];
            }
            const int bmb = 16 >> bi.log2g, vb = 2 * bi.r, B = 1 << bi.log2b;
            // K record of this token into the lane's slot
            if (valid) {
                const uint32_t *kb = (const uint32_t *)(tok + bi.off + j * bmb);
                const uint32_t *kv = (const uint32_t *)(tok + bi.off + B * bmb + j * vb);
                for (int x = 0; x < (bmb >> 2); ++x) myslot[x] = kb[x];
                for (int x = 0; x < (vb >> 2); ++x) myslot[(bmb >> 2) + x] = kv[x];
            }
            float z[GP];
#pragma unroll
            for (int h = 0; h < GP; ++h) z[h] = 0.0f;
            if (valid) packed_dot<GP>(myslot, (const uint16_t *)(myslot + (bmb >> 2)), bi.log2g, g.dtype, qs, z);
            tl2g[wave * 64 + lane] = bi.log2g;
            // V record into the slot (the K record is no longer needed)
            if (valid) {
                const uint32_t *vbm = (const uint32_t *)(tok + bi.off + B * (bmb + vb) + j * bmb);
                const uint32_t *vv = (const uint32_t *)(tok + bi.off + B * (2 * bmb + vb) + j * vb);
                for (int x = 0; x < (bmb >> 2); ++x) myslot[x] = vbm[x];
                for (int x = 0; x < (vb >> 2); ++x) myslot[(bmb >> 2) + x] = vv[x];
            }
            const bool any = c64 * 64 < T;
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                const float zz = valid ? z[h] * scale : -INFINITY;
                const float mw = wave_max(zz);
                const float mn = fmaxf(m_run[h], mw);
                const float alpha = (m_run[h] == -INFINITY) ? 0.0f : __expf(m_run[h] - mn);
                const float pv = valid ? __expf(zz - mn) : 0.0f;
                if (any) {
                    l_run[h] = l_run[h] * alpha + wave_sum(pv);
                    acc[h][0] *= alpha; acc[h][1] *= alpha;
                    m_run[h] = mn;
                }
                ps[(wave * 64 + lane) * GP + h] = pv;
            }
            __syncthreads();
            const int tmax = any ? min(64, T - c64 * 64) : 0;
            for (int t = 0; t < tmax; ++t) {
                const uint32_t *sl = slots + (uint64_t)(wave * 64 + t) * slot_dw;
                const int l2g = tl2g[wave * 64 + t];
                const int bw = (16 >> l2g) >> 2;
                const float vlo = packed_channel(sl, (const uint16_t *)(sl + bw), lane, l2g, g.dtype);
                const float vhi = packed_channel(sl, (const uint16_t *)(sl + bw), lane + 64, l2g, g.dtype);
#pragma unroll
                for (int h = 0; h < GP; ++h) {
                    const float pv = ps[(wave * 64 + t) * GP + h];
                    acc[h][0] = fmaf(pv, vlo, acc[h][0]);
                    acc[h][1] = fmaf(pv, vhi, acc[h][1]);
                }
            }
            __syncthreads();
        }
    }
    // merge the waves' (m, l, acc) and write the split's partial
#pragma unroll
    for (int h = 0; h < GP; ++h) {
        float *mw = mrg + (wave * GP + h) * (D + 2);
        if (lane == 0) { mw[0] = m_run[h]; mw[1] = l_run[h]; }
        mw[2 + lane] = acc[h][0];
        mw[2 + lane + 64] = acc[h][1];
    }
    __syncthreads();
    const int nwv = is_buf ? 1 : 4;
    for (int i = tid; i < GP * D; i += 256) {
        const int h = i / D, c = i % D;
        float M = -INFINITY;
        for (int x = 0; x < nwv; ++x) M = fmaxf(M, mrg[(x * GP + h) * (D + 2)]);
        float A = 0.0f, Lsum = 0.0f;
        for (int x = 0; x < nwv; ++x) {
            const float *mw = mrg + (x * GP + h) * (D + 2);
            const float f = (mw[0] == -INFINITY) ? 0.0f : __expf(mw[0] - M);
            A += mw[2 + c] * f;
            Lsum += mw[1] * f;
        }
        part[2 * GP + h * D + c] = A;
        if (c == 0) { part[h] = M; part[GP + h] = Lsum; }
    }
    if (tid == 0) tag[s] = is_buf ? -1 : w;
}

// ------------------------------------------------------------------ reduce
template <int GP>
__global__ void __launch_bounds__(128) k_reduce(Geom g, WsGeom ws, float *out) {
    __shared__ float A[GP][D];
    __shared__ float Ms[GP], Ls[GP];
    const int p = blockIdx.x, j = threadIdx.x, G = g.G;
    const PairMeta meta = *g.meta_of(p);
    float *o = out + (uint64_t)p * G * D;
    const int32_t *tag = ws.tag + (uint64_t)p * (ws.tag_stride / 4);
    const float *part = ws.part + (uint64_t)p * (ws.part_stride / 4);
    const int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    int nf, prov, nbuf;
    pair_ndesc(meta, nf, prov, nbuf);
    int w_, e0_, e1_, total;
    split_of(wsel, g.nw, 0, w_, e0_, e1_, total);
    const int nsplit = total + (nbuf > 0 ? 1 : 0);
    float Mg[GP], Lg[GP], Og[GP];
#pragma unroll
    for (int h = 0; h < GP; ++h) { Mg[h] = -INFINITY; Lg[h] = 0.0f; Og[h] = 0.0f; }
    for (int w = -1; w < g.nw; ++w) {             // -1 = update buffer
        float M[GP], Lw[GP], Aw[GP];
        bool any = false;
#pragma unroll
        for (int h = 0; h < GP; ++h) { M[h] = -INFINITY; Lw[h] = 0.0f; Aw[h] = 0.0f; }
        for (int s = 0; s < nsplit; ++s) {
            if (tag[s] != w) continue;
            any = true;
            const float *ps = part + (uint64_t)s * GP * (D + 2);
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                const float m = ps[h];
                if (m == -INFINITY) continue;
                const float mn = fmaxf(M[h], m);
                const float a = (M[h] == -INFINITY) ? 0.0f : __expf(M[h] - mn), b = __expf(m - mn);
                Aw[h] = Aw[h] * a + ps[2 * GP + h * D + j] * b;
                Lw[h] = Lw[h] * a + ps[GP + h] * b;
                M[h] = mn;
            }
        }
        if (!any) continue;
        float Ow[GP];
        if (w >= 0 && g.rotated) {
            __syncthreads();
#pragma unroll
            for (int h = 0; h < GP; ++h) A[h][j] = Aw[h];
            __syncthreads();
            const float *Rv = g.rot_of(p, w) + 2 * D * D;   // R_v[c][j]: x = y . R
#pragma unroll
            for (int h = 0; h < GP; ++h) Ow[h] = 0.0f;
            for (int c = 0; c < D; ++c) {
                const float r = Rv[c * D + j];
#pragma unroll
                for (int h = 0; h < GP; ++h) Ow[h] = fmaf(A[h][c], r, Ow[h]);
            }
        } else {
#pragma unroll
            for (int h = 0; h < GP; ++h) Ow[h] = Aw[h];
        }
#pragma unroll
        for (int h = 0; h < GP; ++h) {
            if (M[h] == -INFINITY) continue;
            const float mn = fmaxf(Mg[h], M[h]);
            const float a = (Mg[h] == -INFINITY) ? 0.0f : __expf(Mg[h] - mn), b = __expf(M[h] - mn);
            Og[h] = Og[h] * a + Ow[h] * b;
            Lg[h] = Lg[h] * a + Lw[h] * b;
            Mg[h] = mn;
        }
    }
#pragma unroll
    for (int h = 0; h < GP; ++h)
        if (h < G) o[h * D + j] = (Lg[h] > 0.0f) ? Og[h] / Lg[h] : 0.0f;
    (void)Ms; (void)Ls;
}

template <int GP>
hipError_t launch_decode_t(const Geom &g, const WsGeom &w, const uint16_t *q, float *out, float scale,
                           int max_desc_used, int max_windows_used, hipStream_t s, hipEvent_t *ev) {
    const int nwq = g.rotated ? max_windows_used : 1;
    if (ev) hipEventRecord(ev[0], s);
    hipLaunchKernelGGL(k_qrot, dim3(nwq, g.npairs), dim3(128), 0, s, g, w, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // block scoring: stage at most 48 KiB of score records per workgroup
    int maxrec = 0, minb = 16;
    for (int i = 0; i < 3; ++i) for (int k = 0; k < 3; ++k) {
        const int l2 = 31 - __builtin_clz(g.group_cand[k]);
        maxrec = max(maxrec, 2 * g.keep_cand[i] + (16 >> l2));
    }
    maxrec = max(maxrec, 2 * g.def_keep + (16 >> (31 - __builtin_clz(g.def_group))));
    for (int i = 0; i < 3; ++i) minb = min(minb, g.block_cand[i]);
    minb = min(minb, g.def_block);
    const int seg_bytes = (SEG / minb) * maxrec;
    int spw = min(SCORE_SEGS, max(1, 49152 / seg_bytes));
    spw = min(spw, max(1, g.W / SEG));
    const int stage_bytes = spw * seg_bytes + 16;
    const size_t score_smem = 2 * D * GP * 4 + 32 * sizeof(Desc) + 34 * 4 + stage_bytes;
    if (ev) hipEventRecord(ev[1], s);
    if (max_desc_used > 0) {
        hipLaunchKernelGGL(k_score<GP>, dim3(ceil_div(max_desc_used, spw), g.npairs), dim3(256), score_smem, s, g, w,
                           spw, stage_bytes);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (ev) hipEventRecord(ev[2], s);
    hipLaunchKernelGGL(k_topk, dim3(g.npairs), dim3(1024), 0, s, g, w);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int slot_dw = (maxrec + 3) / 4;
    if ((slot_dw & 1) == 0) slot_dw += 1;
    const size_t attn_smem = D * GP * 4 + SPLIT_BLOCKS * sizeof(BlkInfo) + (SPLIT_BLOCKS + 2) * 4 +
                             4 * 64 * GP * 4 + 4 * GP * (D + 2) * 4 + 256 * 4 + (size_t)256 * slot_dw * 4;
    if (ev) hipEventRecord(ev[3], s);
    hipLaunchKernelGGL(k_attn<GP>, dim3(w.max_splits, g.npairs), dim3(256), attn_smem, s, g, w, scale, q, slot_dw);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev) hipEventRecord(ev[4], s);
    hipLaunchKernelGGL(k_reduce<GP>, dim3(g.npairs), dim3(128), 0, s, g, w, out);
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
