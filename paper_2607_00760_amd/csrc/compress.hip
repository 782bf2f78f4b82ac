// compress.hip -- gfx950 kernels of the MosaicKV compression pass.
//
//   Stage-1 per-vector channel compression (Sec. 4.2), the packed KV format
//   with variable-granularity bitmaps (Sec. 5.1), compressed KV encoding with
//   mean block keys (Sec. 5.2), per-segment strategy selection (Sec. 4.3,
//   Sec. 5.5), the update buffer (Sec. 5.3) and heterogeneous double
//   compression buffering (Sec. 5.4).
//
// Work decomposition: the prefill runs one 256-thread workgroup per 64-token
// segment, wave w owning tokens [16w, 16w+16); the append path's flush and
// finalize run 16-token workgroups of 8 waves x 2 tokens.  Lane l owns
// channels l and l+64, so a vector's 128 channels live in one wave and
// channel trees, ranks, bitmaps and slot numbers are wave-local (butterflies,
// ballots, mbcnt).  The rotation is an fp32 fused-multiply-add chain over
// ascending input channels per output channel (rows of R^T read from the
// arena, x broadcast from LDS), so every rotated value, kept index and packed
// byte is reproducible bit for bit.
#include "mosaic_internal.h"

namespace mosaic {

namespace {

constexpr int NCAND = 9;

// shared memory of a workgroup of NWV waves: 4 waves x 16 tokens for the
// prefill and the reorder's counting (throughput), 8 waves x 2 tokens for the
// flush and finalize of the append path (latency: short serial work per wave,
// several waves per SIMD to hide it)
template <int NWV>
struct SegSmem {
    float x[SEG * D];              // the segment's input tokens, fp32; then the rotated keys
    float tot[2][SEG];             // per-token energy (K, V)
    float drop[2][NCAND][SEG];     // per-token dropped energy per (r, g) candidate
    float bvar[3][SEG];            // per-token deviation from its block mean, per B candidate
    uint64_t keys[NWV][D];         // per-wave group keys of the vector being ranked
    int strat[4];                  // chosen r, log2 g, log2 B
};

__device__ __forceinline__ int ilog2i(int v) { return 31 - __clz(v); }

// Stage the tokens, then y[i][0..1] = rotated channels (l, l+64) of token
// 16w+i.  y = x . R^T as fp32 fmaf chains over ascending c; the rows of R^T
// (rt_g[c*D + j] = R[j][c]) are read from the arena (cached: a window's R is
// shared by all of its segments), the next four rows while the current four
// are applied, so the workgroup keeps no copy of R in LDS.
template <int TPW, int NWV>
__device__ __forceinline__ void rotate_tile(const uint16_t *src, int ntok, const float *rt_g, int dtype,
                            SegSmem<NWV> &sm, float (&y)[TPW][2]) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int i = tid; i < NWV * TPW * D; i += 64 * NWV) {
        int t = i / D;
        sm.x[i] = (t < ntok) ? h2f(src[i], dtype) : 0.0f;
    }
    __syncthreads();
    const int t0 = wave * TPW;
    if (!rt_g) {
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            y[i][0] = sm.x[(t0 + i) * D + lane];
            y[i][1] = sm.x[(t0 + i) * D + lane + 64];
        }
    } else {
#pragma unroll
        for (int i = 0; i < TPW; ++i) { y[i][0] = 0.0f; y[i][1] = 0.0f; }
        const float *r0 = rt_g + lane, *r1 = rt_g + lane + 64;
        float rl[4], rh[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) { rl[k] = r0[k * D]; rh[k] = r1[k * D]; }
        for (int c = 0; c < D; c += 4) {
            const int cn = (c + 4 < D) ? c + 4 : c;          // the last block reloads itself
            float nl[4], nh[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) { nl[k] = r0[(cn + k) * D]; nh[k] = r1[(cn + k) * D]; }
#pragma unroll
            for (int i = 0; i < TPW; ++i) {
                float4 xv = *(const float4 *)&sm.x[(t0 + i) * D + c];
                float xs[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    y[i][0] = fmaf(xs[k], rl[k], y[i][0]);
                    y[i][1] = fmaf(xs[k], rh[k], y[i][1]);
                }
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) { rl[k] = nl[k]; rh[k] = nh[k]; }
        }
    }
    __syncthreads();
}

// Group scores (L1 of magnitudes, pairwise) and exact ranks by
// (score desc, group index asc) of the groups holding channels lane, lane+64.
// Groups at or past ngt (truncated channels, Sec. 5.2) take key 0, below
// every represented group, so they never rank among the kept ones.
__device__ __forceinline__ void group_ranks(float ylo, float yhi, int log2g, int ngt, uint64_t *keys,
                                            int &rank_lo, int &rank_hi) {
    const int lane = threadIdx.x & 63;
    float slo = fabsf(ylo), shi = fabsf(yhi);
    // group sums of adjacent lanes (lane ^ 1, then lane ^ 2: quad permutes)
    if (log2g >= 1) { slo = slo + dpp_read<0xb1, 0xf>(slo); shi = shi + dpp_read<0xb1, 0xf>(shi); }
    if (log2g >= 2) { slo = slo + dpp_read<0x4e, 0xf>(slo); shi = shi + dpp_read<0x4e, 0xf>(shi); }
    const int ng = D >> log2g;
    const int glo = lane >> log2g, ghi = (64 >> log2g) + (lane >> log2g);
    const uint64_t klo = glo < ngt ? ((uint64_t)__float_as_uint(slo) << 8) | (uint64_t)(255 - glo) : 0ull;
    const uint64_t khi = ghi < ngt ? ((uint64_t)__float_as_uint(shi) << 8) | (uint64_t)(255 - ghi) : 0ull;
    // keys is this wave's own array and a wave's LDS operations complete in
    // order, so keeping the compiler from moving memory operations across
    // these points is all the ordering the exchange needs (no barrier)
    if ((lane & ((1 << log2g) - 1)) == 0) { keys[glo] = klo; keys[ghi] = khi; }
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
    int rl = 0, rh = 0;
#pragma unroll 8
    for (int j = 0; j < ng; j += 2) {                      // ng is a multiple of 16: reads issued 8 at a time
        uint64_t k0 = keys[j], k1 = keys[j + 1];
        rl += (k0 > klo) + (k1 > klo);
        rh += (k0 > khi) + (k1 > khi);
    }
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
    rank_lo = rl; rank_hi = rh;
}

// fp32 mean of the B rotated keys of the block starting at token b0, read
// from the staged keys ys (ascending adds, then times 1 / B)
template <int B>
__device__ __forceinline__ void block_mean_lds(const float *ys, int b0, float &mlo, float &mhi) {
    const int lane = threadIdx.x & 63;
    mlo = ys[b0 * D + lane]; mhi = ys[b0 * D + lane + 64];
#pragma unroll
    for (int t = 1; t < B; ++t) { mlo = mlo + ys[(b0 + t) * D + lane]; mhi = mhi + ys[(b0 + t) * D + lane + 64]; }
    mlo = mlo * (1.0f / (float)B); mhi = mhi * (1.0f / (float)B);
}

// Per-token statistics of one wave's TPW tokens: energy, dropped energy of
// every (r, g) candidate; for K also the block deviation per B candidate
// (blocks longer than a wave's run take their mean from the staged keys ys).
template <int B, int TPW>
__device__ __forceinline__ void block_dev(const float (&y)[TPW][2], float *out_tok, int t0, int valid_ntok,
                                          const float *ys) {
    const int lane = threadIdx.x & 63;
    if constexpr (B > TPW) {
        float mlo, mhi;
        block_mean_lds<B>(ys, t0 / B * B, mlo, mhi);
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            float dl = y[t][0] - mlo, dh = y[t][1] - mhi;
            float v = tree128(dl * dl, dh * dh);
            if (lane == 0 && t0 + t < valid_ntok) out_tok[t0 + t] = v;
        }
        return;
    }
#pragma unroll
    for (int b0 = 0; b0 < TPW; b0 += B) {
        float mlo = y[b0][0], mhi = y[b0][1];
#pragma unroll
        for (int t = 1; t < B; ++t) { mlo = mlo + y[b0 + t][0]; mhi = mhi + y[b0 + t][1]; }
        mlo = mlo * (1.0f / (float)B); mhi = mhi * (1.0f / (float)B);
#pragma unroll
        for (int t = 0; t < B; ++t) {
            float dl = y[b0 + t][0] - mlo, dh = y[b0 + t][1] - mhi;
            float v = tree128(dl * dl, dh * dh);
            if (lane == 0 && t0 + b0 + t < valid_ntok) out_tok[t0 + b0 + t] = v;
        }
    }
}

template <int TPW, int NWV>
__device__ __forceinline__ void token_stats(const Geom &g, const float (&y)[TPW][2], int which, SegSmem<NWV> &sm, int ntok) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, t0 = wave * TPW;
    uint64_t *keys = sm.keys[wave];
    for (int i = 0; i < TPW; ++i) {
        float ylo = 0.0f, yhi = 0.0f;          // static select (no dynamic register indexing)
#pragma unroll
        for (int x = 0; x < TPW; ++x)
            if (x == i) { ylo = y[x][0]; yhi = y[x][1]; }
        const float elo = ylo * ylo, ehi = yhi * yhi;
        const float tot = tree128(elo, ehi);
        if (lane == 0) sm.tot[which][t0 + i] = tot;
        for (int gi = 0; gi < 3; ++gi) {
            const int log2g = ilog2i(g.group_cand[gi]);
            int rlo, rhi;
            group_ranks(ylo, yhi, log2g, g.trunc >> log2g, keys, rlo, rhi);
            for (int ri = 0; ri < 3; ++ri) {
                const int n = g.keep_cand[ri] >> log2g;
                float d = tree128(rlo < n ? 0.0f : elo, rhi < n ? 0.0f : ehi);
                if (lane == 0) sm.drop[which][ri * 3 + gi][t0 + i] = d;
            }
        }
    }
}

template <int TPW, int NWV>
__device__ __forceinline__ void block_stats(const Geom &g, const float (&y)[TPW][2], SegSmem<NWV> &sm, int ntok) {
    const int t0 = (threadIdx.x >> 6) * TPW;
    for (int bi = 0; bi < 3; ++bi) {
        switch (g.block_cand[bi]) {
            case 4: block_dev<4, TPW>(y, sm.bvar[bi], t0, ntok, sm.x); break;
            case 8: block_dev<8, TPW>(y, sm.bvar[bi], t0, ntok, sm.x); break;
            default: block_dev<16, TPW>(y, sm.bvar[bi], t0, ntok, sm.x); break;
        }
    }
}

// tree over the 64 per-token values (wave 0; adjacent pairwise tree)
__device__ __forceinline__ float tree64_lds(const float *v) { return tree64(v[threadIdx.x & 63]); }

// Strategy choice (Sec. 5.5): first (r, g) in candidate order whose dropped
// energy is below tau_ch * energy for K and for V; first B whose block
// deviation is below tau_blk * K energy; fallbacks are the last candidates.
template <int NWV>
__device__ __forceinline__ void choose_strategy(const Geom &g, SegSmem<NWV> &sm) {
    if (threadIdx.x < 64) {
        const float TK = tree64_lds(sm.tot[0]), TV = tree64_lds(sm.tot[1]);
        int chosen = NCAND - 1;
        for (int ci = 0; ci < NCAND; ++ci) {
            const float DK = tree64_lds(sm.drop[0][ci]), DV = tree64_lds(sm.drop[1][ci]);
            const float lk = g.tau_ch * TK, lv = g.tau_ch * TV;
            if (DK < lk && DV < lv) { chosen = ci; break; }
        }
        int bsel = g.block_cand[2];
        for (int bi = 0; bi < 3; ++bi) {
            const float VB = tree64_lds(sm.bvar[bi]);
            const float lim = g.tau_blk * TK;
            if (VB < lim) { bsel = g.block_cand[bi]; break; }
        }
        if (threadIdx.x == 0) {
            sm.strat[0] = g.keep_cand[chosen / 3];
            sm.strat[1] = ilog2i(g.group_cand[chosen % 3]);
            sm.strat[2] = ilog2i(bsel);
        }
    }
    __syncthreads();
}

// Pack one vector held as (lane: channel lane, lane+64): bitmap + values,
// the values as E4M3 codes (one byte each) when e4m3 is set, else 16-bit.
__device__ __forceinline__ void pack_vector(float ylo, float yhi, int r, int log2g, int T, int dtype, bool e4m3,
                                            uint64_t *keys, uint8_t *bm_out, uint8_t *val_out, bool active) {
    const int lane = threadIdx.x & 63;
    int rlo, rhi;
    group_ranks(ylo, yhi, log2g, T >> log2g, keys, rlo, rhi);
    const int n = r >> log2g;
    const bool klo = rlo < n, khi = rhi < n;
    const uint64_t mlo = __ballot(klo), mhi = __ballot(khi);
    // group flags in bitmap order: group i's first channel is src = i * g of
    // its half, whose kept flag is bit src of that half's ballot
    const int gph = 64 >> log2g;                 // groups per half
    const int src = (lane % gph) << log2g;
    const bool flag = (lane < 2 * gph) && ((((lane / gph) ? mhi : mlo) >> src) & 1ull);
    const uint64_t bm = __ballot(flag);
    if (!active) return;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    // with truncated bitmaps of 3 or 6 bytes a block-key record can start at
    // an odd byte: its 16-bit values are then stored a byte at a time
    auto put16 = [&](int slot, uint16_t h) {
        if (T < D) { val_out[2 * slot] = (uint8_t)h; val_out[2 * slot + 1] = (uint8_t)(h >> 8); }
        else *(uint16_t *)(val_out + 2 * slot) = h;
    };
    if (klo) {
        int slot = __popcll(mlo & below);
        if (e4m3) val_out[slot] = (uint8_t)f2e4m3(ylo);
        else put16(slot, f2h(ylo, dtype));
    }
    if (khi) {
        int slot = __popcll(mlo) + __popcll(mhi & below);
        if (e4m3) val_out[slot] = (uint8_t)f2e4m3(yhi);
        else put16(slot, f2h(yhi, dtype));
    }
    if (T < D) {
        // a truncated bitmap (exactly T / g bits, whole bytes): lane i stores byte i
        const uint64_t lo64 = log2g == 0 ? mlo : bm, hi64 = log2g == 0 ? mhi : 0ull;
        const int nbytes = bm_bytes(log2g, T);
        if (lane < nbytes) bm_out[lane] = (uint8_t)((lane < 8 ? lo64 >> (8 * lane) : hi64 >> (8 * (lane - 8))) & 0xffu);
    } else if (lane == 0) {
        uint32_t *w = (uint32_t *)bm_out;
        if (log2g == 0) {
            w[0] = (uint32_t)mlo; w[1] = (uint32_t)(mlo >> 32); w[2] = (uint32_t)mhi; w[3] = (uint32_t)(mhi >> 32);
        } else if (log2g == 1) {
            w[0] = (uint32_t)bm; w[1] = (uint32_t)(bm >> 32);
        } else {
            w[0] = (uint32_t)bm;
        }
    }
}

// Encode the workgroup's tokens (K in yk, V in yv) into the token arena at
// tok and the block keys into the score arena at sc (Sec. 5.2).  Token
// values are E4M3 codes when fp8 is set; block keys keep 16-bit values.  A
// block longer than a wave's run gets its key from the wave holding its first
// token, which reads the block's keys from the staged ys.  The workgroup holds
// tokens tb.. of the ntok being encoded (tb a multiple of every block size).
template <int B, int TPW>
__device__ __forceinline__ void pack_segment_B(const float (&yk)[TPW][2], const float (&yv)[TPW][2], int r, int log2g, int T,
                               int dtype, bool fp8, uint8_t *tok, uint8_t *sc, int ntok, uint64_t *keys,
                               const float *ys, int tb) {
    const int wave = threadIdx.x >> 6, t0 = wave * TPW;
    tok += (uint64_t)(tb / B) * B * 2 * (bm_bytes(log2g, T) + (fp8 ? r : 2 * r));
    sc += (uint64_t)(tb / B) * vec_bytes(r, log2g, T);
    ntok -= tb;
    const int bmb = bm_bytes(log2g, T), vb = fp8 ? r : 2 * r, rec = bmb + vb, srec = vec_bytes(r, log2g, T);
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int t = t0 + i, bi = t / B, j = t % B;
        const bool act = t < ntok;
        uint8_t *blk = tok + (uint64_t)bi * B * 2 * rec;
        pack_vector(yk[i][0], yk[i][1], r, log2g, T, dtype, fp8, keys, blk + j * bmb, blk + B * bmb + j * vb, act);
        pack_vector(yv[i][0], yv[i][1], r, log2g, T, dtype, fp8, keys, blk + B * (bmb + vb) + j * bmb,
                    blk + B * (2 * bmb + vb) + j * vb, act);
    }
    if constexpr (B > TPW) {
        if (t0 % B == 0) {                       // wave-uniform
            float mlo, mhi;
            block_mean_lds<B>(ys, t0, mlo, mhi);
            uint8_t *rp = sc + (uint64_t)(t0 / B) * srec;
            pack_vector(mlo, mhi, r, log2g, T, dtype, false, keys, rp, rp + bmb, t0 < ntok);
        }
        return;
    }
#pragma unroll
    for (int b0 = 0; b0 < TPW; b0 += B) {
        float mlo = yk[b0][0], mhi = yk[b0][1];
#pragma unroll
        for (int t = 1; t < B; ++t) { mlo = mlo + yk[b0 + t][0]; mhi = mhi + yk[b0 + t][1]; }
        mlo = mlo * (1.0f / (float)B); mhi = mhi * (1.0f / (float)B);
        const int bi = (t0 + b0) / B;
        uint8_t *rp = sc + (uint64_t)bi * srec;
        pack_vector(mlo, mhi, r, log2g, T, dtype, false, keys, rp, rp + bmb, t0 + b0 < ntok);
    }
}

template <int TPW>
__device__ __forceinline__ void pack_segment(const float (&yk)[TPW][2], const float (&yv)[TPW][2], int r, int log2g, int log2b,
                             int T, int dtype, bool fp8, uint8_t *tok, uint8_t *sc, int ntok, uint64_t *keys,
                             const float *ys, int tb) {
    switch (log2b) {
        case 2: pack_segment_B<4, TPW>(yk, yv, r, log2g, T, dtype, fp8, tok, sc, ntok, keys, ys, tb); break;
        case 3: pack_segment_B<8, TPW>(yk, yv, r, log2g, T, dtype, fp8, tok, sc, ntok, keys, ys, tb); break;
        default: pack_segment_B<16, TPW>(yk, yv, r, log2g, T, dtype, fp8, tok, sc, ntok, keys, ys, tb); break;
    }
}

// the rotated keys of the wave's tokens into sm.x (after both rotations, when
// the input tokens are no longer needed), for blocks spanning several waves
template <int TPW, int NWV>
__device__ __forceinline__ void stage_keys(const float (&yk)[TPW][2], SegSmem<NWV> &sm) {
    const int lane = threadIdx.x & 63, t0 = (threadIdx.x >> 6) * TPW;
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        sm.x[(t0 + i) * D + lane] = yk[i][0];
        sm.x[(t0 + i) * D + lane + 64] = yk[i][1];
    }
    __syncthreads();
}

// ------------------------------------------------------------------ kernels

// R^T of K and V and R of V of one rotation into a window slot
__device__ __forceinline__ void put_rot(float *dst, const float *Rk, const float *Rv) {
    for (int i = threadIdx.x; i < D * D; i += blockDim.x) {
        const int j = i / D, c = i % D;        // source R[j][c]
        dst[c * D + j] = Rk[i];
        dst[D * D + c * D + j] = Rv[i];
        dst[2 * D * D + i] = Rv[i];
    }
}

// every window slot of every pair, from the caller's nw_src windows per pair
// (slots past them take the last one: windows that close later get their own)
__global__ void k_copy_rot(Geom g, const float *rk, const float *rv, int nw_src) {
    const int p = blockIdx.y, w = blockIdx.x, ws = min(w, nw_src - 1);
    put_rot(g.rot_of(p, w), rk + ((uint64_t)p * nw_src + ws) * D * D, rv + ((uint64_t)p * nw_src + ws) * D * D);
}

__global__ void k_set_meta(Geom g, const int32_t *ctx) {
    const int p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= g.npairs) return;
    PairMeta *m = g.meta_of(p);
    m->L = ctx[p / g.hkv];
    m->nblk_final = 0; m->tok_tail = 0; m->sc_tail = 0;
    m->nwin = 1; m->wloss = 0.0f; m->pend = -1;
    if (g.dyn) {
        // input tokens sit in fixed windows of W tokens (Sec. 4.3); the window
        // holding the first token after the full segments stays open
        const int spw = g.W / SEG, nwin = min((m->L / SEG) / spw + 1, g.nw);
        int32_t *wt = g.wtab_of(p);
        for (int w = 0; w < nwin; ++w) wt[w] = w * spw;
        m->nwin = nwin;
    }
}

// mode 0: choose the segment's strategy; mode 1: pack it at its descriptor's
// offsets (both rotate the tokens); mode 2: both from one rotation, packing
// into the segment's worst-case slot of the workspace (slot_tok + slot_sc
// bytes per (pair, segment)), from where k_compact moves the records to their
// offsets once the offsets are known.  With close set (modes 0 and 1), the
// segments are those of each pair's window awaiting its rotation, and the
// input holds that window's tokens from its first one.
// (one instantiation per mode, so that each gets its own register budget:
// three waves per SIMD)
template <int MODE>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
k_prefill(Geom g, const uint16_t *k, const uint16_t *v, int64_t seq_stride, uint8_t *ws, uint32_t slot_tok,
          uint32_t slot_sc, int close) {
    constexpr int TPW = 16, NWV = 4;
    __shared__ SegSmem<NWV> sm;
    const int p = blockIdx.y;
    const PairMeta *meta = g.meta_of(p);
    int seg = blockIdx.x, win;
    if (close) {
        const int pw = meta->pend;
        if (pw < 0) return;
        const int32_t *wt = g.wtab_of(p);
        seg += wt[pw];
        if (seg >= wt[pw + 1]) return;
        win = pw;
    } else {
        if (seg >= meta->L / SEG) return;
        win = (seg * SEG) / g.W;
    }
    const uint64_t base = ((uint64_t)p * seq_stride + (uint64_t)blockIdx.x * SEG) * D;
    Desc *desc = g.desc_of(p) + seg;
    const float *rot = g.rotated ? g.rot_of(p, win) : nullptr;
    float yk[TPW][2], yv[TPW][2];
    rotate_tile(k + base, SEG, rot, g.dtype, sm, yk);
    rotate_tile(v + base, SEG, rot ? rot + D * D : nullptr, g.dtype, sm, yv);
    const int wave = threadIdx.x >> 6;
    if constexpr (MODE == 2) {
        if (g.force) {
            if (threadIdx.x == 0) { sm.strat[0] = g.def_keep; sm.strat[1] = ilog2i(g.def_group); sm.strat[2] = ilog2i(g.def_block); }
        } else {
            token_stats(g, yk, 0, sm, SEG);
            token_stats(g, yv, 1, sm, SEG);
            block_stats(g, yk, sm, SEG);
            __syncthreads();
            choose_strategy(g, sm);
        }
        __syncthreads();
        const int r = sm.strat[0], l2g = sm.strat[1], l2b = sm.strat[2];
        if (threadIdx.x == 0) {
            desc->r = (uint8_t)r; desc->log2g = (uint8_t)l2g; desc->log2b = (uint8_t)l2b; desc->flags = 0;
        }
        uint8_t *slot = ws + ((uint64_t)p * g.max_desc + seg) * ((uint64_t)slot_tok + slot_sc);
        pack_segment(yk, yv, r, l2g, l2b, g.trunc, g.dtype, g.fp8 != 0, slot, slot + slot_tok, SEG, sm.keys[wave], sm.x, 0);
        return;
    }
    if constexpr (MODE == 0) {
        if (g.force) {
            if (threadIdx.x == 0) {
                desc->r = (uint8_t)g.def_keep; desc->log2g = (uint8_t)ilog2i(g.def_group);
                desc->log2b = (uint8_t)ilog2i(g.def_block); desc->flags = 0;
            }
            return;
        }
        token_stats(g, yk, 0, sm, SEG);
        token_stats(g, yv, 1, sm, SEG);
        block_stats(g, yk, sm, SEG);
        __syncthreads();
        choose_strategy(g, sm);
        if (threadIdx.x == 0) {
            desc->r = (uint8_t)sm.strat[0]; desc->log2g = (uint8_t)sm.strat[1];
            desc->log2b = (uint8_t)sm.strat[2]; desc->flags = 0;
        }
    } else {
        const Desc d = *desc;
        pack_segment(yk, yv, d.r, d.log2g, d.log2b, g.trunc, g.dtype, g.fp8 != 0, g.tok_of(p) + d.tok_off, g.sc_of(p) + d.sc_off,
                     SEG, sm.keys[wave], sm.x, 0);
    }
}

// The records of the single-pass compression from the segments' workspace
// slots to their offsets (dword copies: every record run is a multiple of 4
// bytes at a 4-byte aligned offset).
__global__ void __launch_bounds__(256) k_compact(Geom g, const uint8_t *ws, uint32_t slot_tok, uint32_t slot_sc) {
    const int p = blockIdx.y, seg = blockIdx.x;
    const PairMeta *meta = g.meta_of(p);
    if (seg >= meta->L / SEG) return;
    const Desc d = g.desc_of(p)[seg];
    const uint32_t tb = SEG * 2 * (uint32_t)tok_vec_bytes(d.r, d.log2g, g.trunc, g.fp8);
    const uint32_t sb = (uint32_t)(SEG >> d.log2b) * (uint32_t)vec_bytes(d.r, d.log2g, g.trunc);
    const uint8_t *slot = ws + ((uint64_t)p * g.max_desc + seg) * ((uint64_t)slot_tok + slot_sc);
    const uint32_t *st = (const uint32_t *)slot, *ss = (const uint32_t *)(slot + slot_tok);
    uint32_t *dt = (uint32_t *)(g.tok_of(p) + d.tok_off), *ds = (uint32_t *)(g.sc_of(p) + d.sc_off);
    for (uint32_t i = threadIdx.x; i < tb / 4; i += 256) dt[i] = st[i];
    for (uint32_t i = threadIdx.x; i < sb / 4; i += 256) ds[i] = ss[i];
}

// Exclusive scan of segment sizes per pair -> descriptor offsets and tails.
// With close set, the segments of the window awaiting its rotation, from the
// offsets its first segment already has (every earlier segment is kept).
__global__ void __launch_bounds__(256) k_scan(Geom g, int close) {
    __shared__ uint32_t s_tok[256], s_sc[256], s_blk[256];
    __shared__ uint32_t carry[3];
    const int p = blockIdx.x, tid = threadIdx.x;
    PairMeta *meta = g.meta_of(p);
    int s_first = 0, nfull = meta->L / SEG;
    if (close) {
        const int pw = meta->pend;
        if (pw < 0) return;
        s_first = g.wtab_of(p)[pw];
        nfull = g.wtab_of(p)[pw + 1];
    }
    Desc *desc = g.desc_of(p);
    if (tid == 0) {
        if (close) { carry[0] = desc[s_first].tok_off; carry[1] = desc[s_first].sc_off; carry[2] = desc[s_first].first_block; }
        else { carry[0] = carry[1] = carry[2] = 0; }
    }
    __syncthreads();
    for (int base = s_first; base < nfull; base += 256) {
        const int s = base + tid;
        uint32_t tb = 0, sb = 0, nb = 0;
        if (s < nfull) {
            const Desc d = desc[s];
            tb = SEG * 2 * (uint32_t)tok_vec_bytes(d.r, d.log2g, g.trunc, g.fp8);
            nb = SEG >> d.log2b; sb = nb * (uint32_t)vec_bytes(d.r, d.log2g, g.trunc);
        }
        s_tok[tid] = tb; s_sc[tid] = sb; s_blk[tid] = nb;
        __syncthreads();
        for (int off = 1; off < 256; off <<= 1) {      // inclusive Hillis-Steele (integers: exact)
            uint32_t a = 0, b = 0, c = 0;
            if (tid >= off) { a = s_tok[tid - off]; b = s_sc[tid - off]; c = s_blk[tid - off]; }
            __syncthreads();
            s_tok[tid] += a; s_sc[tid] += b; s_blk[tid] += c;
            __syncthreads();
        }
        if (s < nfull) {
            desc[s].tok_off = carry[0] + s_tok[tid] - tb;
            desc[s].sc_off = carry[1] + s_sc[tid] - sb;
            desc[s].first_block = carry[2] + s_blk[tid] - nb;
        }
        __syncthreads();
        if (tid == 255) { carry[0] += s_tok[255]; carry[1] += s_sc[255]; carry[2] += s_blk[255]; }
        __syncthreads();
    }
    if (tid == 0) { meta->tok_tail = carry[0]; meta->sc_tail = carry[1]; meta->nblk_final = (int32_t)carry[2]; }
}

// Remainder tokens of a prefill (L mod S) into the staging area and the
// update buffer, as if appended one by one.
__global__ void k_stage_tail(Geom g, const uint16_t *k, const uint16_t *v, int64_t seq_stride) {
    const int p = blockIdx.x;
    const int L = g.meta_of(p)->L, nf = L / SEG, m = L % SEG;
    const int prov = m >= UBUF;
    uint16_t *stg = g.stg_of(p), *buf = g.buf_of(p);
    const uint64_t base = ((uint64_t)p * seq_stride + (uint64_t)nf * SEG) * D;
    for (int i = threadIdx.x; i < m * D; i += blockDim.x) {
        stg[i] = k[base + i];
        stg[SEG * D + i] = v[base + i];
        const int t = i / D;
        if (t >= UBUF * prov) {
            buf[i - UBUF * prov * D] = k[base + i];
            buf[UBUF * D + i - UBUF * prov * D] = v[base + i];
        }
    }
}

__global__ void k_append(Geom g, const uint16_t *kn, const uint16_t *vn) {
    const int p = blockIdx.x;
    PairMeta *meta = g.meta_of(p);
    const int L = meta->L, m = L % SEG;
    const int nb = m - (m >= UBUF ? UBUF : 0);
    uint16_t *stg = g.stg_of(p), *buf = g.buf_of(p);
    for (int i = threadIdx.x; i < D; i += blockDim.x) {
        const uint16_t a = kn[(uint64_t)p * D + i], b = vn[(uint64_t)p * D + i];
        stg[m * D + i] = a; stg[SEG * D + m * D + i] = b;
        buf[nb * D + i] = a; buf[UBUF * D + nb * D + i] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) meta->L = L + 1;
}

// Provisional flush (U tokens, previous strategy) and finalize (S tokens, own
// strategy, recompressed in place) of a pair's trailing segment.  Both are
// latency-bound (a few dozen pairs at a time), so a pair's work is spread over
// workgroups of 8 waves x 2 tokens (blockIdx.y: tokens 16 y .. 16 y + 15): two
// for the flush, four for each of the finalize's two kernels.  The finalize's
// strategy needs every token's statistics, so its first kernel writes them to
// the pair's update buffer, which is empty when a segment completes (every
// buffered token belongs to it) and is next written by the following append.
constexpr int MT_TPW = 2, MT_NWV = 8, MT_TOK = MT_TPW * MT_NWV, MT_THREADS = 64 * MT_NWV;
// per-token statistics: tot K/V, drop K/V x 9, bvar x 3, and (dynamic
// windows) the dropped energy of K/V under the provisional strategy
constexpr int FST_PROV = 2 + 2 * NCAND + 3;
constexpr int FST_N = FST_PROV + 2;
static_assert(FST_N * SEG * 4 + 16 <= 2 * UBUF * D * 2, "finalize statistics and offsets fit the update buffer");

// dropped energy of each of the wave's tokens under (r, 2^log2g), from lane 0
// into out[t] (t = token within the workgroup's run)
template <int TPW, int NWV>
__device__ __forceinline__ void prov_drop(const Geom &g, const float (&y)[TPW][2], int r, int log2g,
                                          SegSmem<NWV> &sm, float *out) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, t0 = wave * TPW;
    const int n = r >> log2g;
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        int rlo, rhi;
        group_ranks(y[i][0], y[i][1], log2g, g.trunc >> log2g, sm.keys[wave], rlo, rhi);
        const float d = tree128(rlo < n ? 0.0f : y[i][0] * y[i][0], rhi < n ? 0.0f : y[i][1] * y[i][1]);
        if (lane == 0) out[t0 + i] = d;
    }
}

__device__ __forceinline__ bool maint_due(const Geom &g, int mode, int L, bool fin) {
    const int m = L % SEG;
    if (mode == MAINT_APPEND) {
        if (L <= 0 || (L % UBUF) != 0) return false;
        return fin ? m == 0 : m != 0;
    }
    return !fin && m >= UBUF;
}

// rotate this workgroup's tokens of the trailing segment (K into yk, V into
// yv) and stage the rotated keys for blocks spanning several waves
__device__ __forceinline__ void maint_rotate(const Geom &g, int p, int seg, int tb, int ntok, SegSmem<MT_NWV> &sm,
                                             float (&yk)[MT_TPW][2], float (&yv)[MT_TPW][2]) {
    // the trailing segment belongs to the open window
    const int win = g.dyn ? g.meta_of(p)->nwin - 1 : (seg * SEG) / g.W;
    const float *rot = g.rotated ? g.rot_of(p, win) : nullptr;
    const uint16_t *stg = g.stg_of(p) + (uint64_t)tb * D;
    rotate_tile(stg, ntok - tb, rot, g.dtype, sm, yk);
    rotate_tile(stg + SEG * D, ntok - tb, rot ? rot + D * D : nullptr, g.dtype, sm, yv);
    stage_keys(yk, sm);
}

__device__ __forceinline__ void maint_pack(const Geom &g, int p, int seg, int tb, int ntok, bool fin, int r, int log2g,
                                           int log2b, uint32_t tok_off, uint32_t sc_off, int nblk0,
                                           SegSmem<MT_NWV> &sm, const float (&yk)[MT_TPW][2],
                                           const float (&yv)[MT_TPW][2]) {
    const int wave = threadIdx.x >> 6;
    pack_segment(yk, yv, r, log2g, log2b, g.trunc, g.dtype, g.fp8 != 0, g.tok_of(p) + tok_off, g.sc_of(p) + sc_off, ntok,
                 sm.keys[wave], sm.x, tb);
    if (threadIdx.x == 0 && blockIdx.y == 0) {
        Desc d;
        d.tok_off = tok_off; d.sc_off = sc_off; d.first_block = (uint32_t)nblk0;
        d.r = (uint8_t)r; d.log2g = (uint8_t)log2g; d.log2b = (uint8_t)log2b; d.flags = fin ? 0 : 1;
        g.desc_of(p)[seg] = d;
        if (fin) {
            PairMeta *meta = g.meta_of(p);
            meta->tok_tail = tok_off + SEG * 2 * (uint32_t)tok_vec_bytes(r, log2g, g.trunc, g.fp8);
            meta->sc_tail = sc_off + (SEG >> log2b) * (uint32_t)vec_bytes(r, log2g, g.trunc);
            meta->nblk_final = nblk0 + (SEG >> log2b);
        }
    }
}

__global__ void __launch_bounds__(MT_THREADS) k_flush(Geom g, int mode) {
    __shared__ SegSmem<MT_NWV> sm;
    const int p = blockIdx.x;
    const PairMeta *meta = g.meta_of(p);
    const int L = meta->L;
    if (!maint_due(g, mode, L, false)) return;
    const int seg = L / SEG, tb = (int)blockIdx.y * MT_TOK;
    float yk[MT_TPW][2], yv[MT_TPW][2];
    maint_rotate(g, p, seg, tb, UBUF, sm, yk, yv);
    int r, log2g, log2b;
    if (seg > 0) {
        const Desc pd = g.desc_of(p)[seg - 1];
        r = pd.r; log2g = pd.log2g; log2b = pd.log2b;
    } else {
        r = g.def_keep; log2g = ilog2i(g.def_group); log2b = ilog2i(g.def_block);
    }
    // a flush leaves the tails alone: every workgroup reads the same offsets
    maint_pack(g, p, seg, tb, UBUF, false, r, log2g, log2b, meta->tok_tail, meta->sc_tail, meta->nblk_final, sm, yk, yv);
}

// finalize, first kernel: statistics of this workgroup's 16 tokens into the
// scratch st[FST_N][SEG] (fp32) and, from workgroup 0, the segment's starting
// offsets after it (the second kernel changes the tails)
__global__ void __launch_bounds__(MT_THREADS) k_fin_stats(Geom g) {
    __shared__ SegSmem<MT_NWV> sm;
    const int p = blockIdx.x;
    const PairMeta *meta = g.meta_of(p);
    const int L = meta->L;
    if (!maint_due(g, MAINT_APPEND, L, true)) return;
    const int seg = L / SEG - 1, tb = (int)blockIdx.y * MT_TOK;
    float *st = (float *)g.buf_of(p);
    if (blockIdx.y == 0 && threadIdx.x == 0) {
        uint32_t *off = (uint32_t *)(st + FST_N * SEG);
        off[0] = meta->tok_tail; off[1] = meta->sc_tail; off[2] = (uint32_t)meta->nblk_final;
    }
    if (g.force && !g.dyn) return;
    float yk[MT_TPW][2], yv[MT_TPW][2];
    maint_rotate(g, p, seg, tb, SEG, sm, yk, yv);
    token_stats(g, yk, 0, sm, MT_TOK);
    token_stats(g, yv, 1, sm, MT_TOK);
    block_stats(g, yk, sm, MT_TOK);
    if (g.dyn) {
        // the segment's loss under the provisional strategy (the previous
        // finalized segment's (r, g), else the default): dropped energy per token
        int r = g.def_keep, log2g = ilog2i(g.def_group);
        if (seg > 0) { const Desc pd = g.desc_of(p)[seg - 1]; r = pd.r; log2g = pd.log2g; }
        prov_drop(g, yk, r, log2g, sm, st + FST_PROV * SEG + tb);
        prov_drop(g, yv, r, log2g, sm, st + (FST_PROV + 1) * SEG + tb);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < FST_PROV * MT_TOK; i += MT_THREADS) {
        const int k = i / MT_TOK, t = i % MT_TOK;
        const float v = k < 2 ? sm.tot[k][t] : (k < 2 + 2 * NCAND ? sm.drop[(k - 2) / NCAND][(k - 2) % NCAND][t]
                                                                  : sm.bvar[k - 2 - 2 * NCAND][t]);
        st[k * SEG + tb + t] = v;
    }
}

// finalize, second kernel: every workgroup takes the same strategy from the
// 64 tokens' statistics, then packs its 16 tokens
__global__ void __launch_bounds__(MT_THREADS) k_fin_pack(Geom g) {
    __shared__ SegSmem<MT_NWV> sm;
    const int p = blockIdx.x;
    const int L = g.meta_of(p)->L;
    if (!maint_due(g, MAINT_APPEND, L, true)) return;
    const int seg = L / SEG - 1, tb = (int)blockIdx.y * MT_TOK;
    const float *st = (const float *)g.buf_of(p);
    const uint32_t *off = (const uint32_t *)(st + FST_N * SEG);
    float yk[MT_TPW][2], yv[MT_TPW][2];
    maint_rotate(g, p, seg, tb, SEG, sm, yk, yv);
    int r, log2g, log2b;
    if (g.force) {
        r = g.def_keep; log2g = ilog2i(g.def_group); log2b = ilog2i(g.def_block);
    } else {
        for (int i = threadIdx.x; i < FST_PROV * SEG; i += MT_THREADS) {
            const int k = i / SEG, t = i % SEG;
            const float v = st[i];
            if (k < 2) sm.tot[k][t] = v;
            else if (k < 2 + 2 * NCAND) sm.drop[(k - 2) / NCAND][(k - 2) % NCAND][t] = v;
            else sm.bvar[k - 2 - 2 * NCAND][t] = v;
        }
        __syncthreads();
        choose_strategy(g, sm);
        r = sm.strat[0]; log2g = sm.strat[1]; log2b = sm.strat[2];
    }
    maint_pack(g, p, seg, tb, SEG, true, r, log2g, log2b, off[0], off[1], (int)off[2], sm, yk, yv);
}

// Windows closed by their loss (Sec. 4.3 dynamic compression strategy,
// Sec. 5.5 incremental strategy generation): after a finalize, a wave per
// pair adds the segment's loss under the provisional strategy -- the larger of
// K's and V's relative dropped energy, segment sums as 64-token pairwise trees
// -- to its window's sum, and closes the window after this segment when it
// holds W tokens, or when the sum exceeds tau_win and it holds min_win
// tokens.  The closed window awaits its own rotation (pend); the next segment
// opens a window.  Runs after k_fin_pack, which no longer reads the window.
__global__ void __launch_bounds__(256) k_win_update(Geom g) {
    const int p = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (p >= g.npairs) return;
    PairMeta *meta = g.meta_of(p);
    const int L = meta->L;
    if (!maint_due(g, MAINT_APPEND, L, true)) return;
    const float *st = (const float *)g.buf_of(p);
    const float TK = tree64(st[lane]), TV = tree64(st[SEG + lane]);
    const float DK = tree64(st[FST_PROV * SEG + lane]), DV = tree64(st[(FST_PROV + 1) * SEG + lane]);
    if (lane != 0) return;
    const float lk = TK > 0.0f ? DK / TK : 0.0f, lv = TV > 0.0f ? DV / TV : 0.0f;
    const float loss = lk > lv ? lk : lv;
    const int seg = L / SEG - 1, nwin = meta->nwin;
    int32_t *wt = g.wtab_of(p);
    const int ntok = (seg + 1 - wt[nwin - 1]) * SEG;
    const float acc = meta->wloss + loss;
    const bool close = ntok >= g.W || (acc > g.tau_win && ntok >= g.min_win);
    if (close && nwin < g.nw) {
        wt[nwin] = seg + 1;
        meta->nwin = nwin + 1;
        meta->pend = nwin - 1;
        meta->wloss = 0.0f;
    } else {
        meta->wloss = acc;
    }
}

// Incremental covariance of the open window (Sec. 5.5: updated with each new
// token's outer product; here segment by segment): grid (pairs, K / V, 8
// blocks of 16 rows), 256 threads, thread t owning entries (16 b + t / 16,
// 8 (t % 16) .. + 7).  Per segment, each entry is the fp64 sum over the 64
// tokens in order of x[i] x[j] (products exact), added to the window's running
// entry (replacing it at the window's first segment).  from_input = 0: the
// segment an append just finalized (tokens in the staging area), for pairs
// whose finalize ran; 1: after a prefill, the open window's full segments,
// from the input x (pair p's token s at (p seq_stride + s) D).
__global__ void __launch_bounds__(256) k_cov_seg(Geom g, const uint16_t *kin, const uint16_t *vin, int64_t seq_stride,
                                                 int from_input) {
    __shared__ float xs[SEG][D];
    const int p = blockIdx.x, which = blockIdx.y, tid = threadIdx.x;
    const PairMeta *meta = g.meta_of(p);
    const int L = meta->L, w = meta->nwin - 1;
    const int32_t *wt = g.wtab_of(p);
    int s0, s1;
    if (from_input) {
        s0 = wt[w]; s1 = L / SEG;
    } else {
        if (!maint_due(g, MAINT_APPEND, L, true)) return;
        s0 = L / SEG - 1; s1 = s0 + 1;
    }
    const int i = blockIdx.z * 16 + tid / 16, j0 = (tid % 16) * 8;
    double *C = g.cov_of(p, w, which) + (uint64_t)i * D + j0;
    for (int s = s0; s < s1; ++s) {
        const uint16_t *src = from_input ? (which ? vin : kin) + ((uint64_t)p * seq_stride + (uint64_t)s * SEG) * D
                                         : g.stg_of(p) + (uint64_t)which * SEG * D;
        __syncthreads();
        for (int e = tid; e < SEG * D; e += 256) xs[e / D][e % D] = h2f(src[e], g.dtype);
        __syncthreads();
        double acc[8];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) acc[jj] = 0.0;
        for (int t = 0; t < SEG; ++t) {
            const double xi = (double)xs[t][i];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) acc[jj] = acc[jj] + xi * (double)xs[t][j0 + jj];
        }
        const bool first = s == wt[w];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) C[jj] = (first ? 0.0 : C[jj]) + acc[jj];
    }
}

// The new rotation of each pair's closed window into its slot and the next
// one (the provisional rotation of the window the close opened).
__global__ void k_close_rot(Geom g, const float *rk, const float *rv) {
    const int p = blockIdx.y, pw = g.meta_of(p)->pend;
    if (pw < 0) return;
    const int w = pw + (int)blockIdx.x;
    if (w >= g.nw) return;
    put_rot(g.rot_of(p, w), rk + (uint64_t)p * D * D, rv + (uint64_t)p * D * D);
}

__global__ void k_close_done(Geom g) {
    const int p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p < g.npairs) g.meta_of(p)->pend = -1;
}

// ------------------------------------------------------------------ channel reorder
// Selection-pattern reorder of the rotation rows (Sec. 5.5 asks for channels
// selected alike to become neighbours).  Per window, K and V apart: each
// token selects its default_keep largest magnitudes (the compressor's
// rotation and ranks); C[i][j] counts the tokens selecting channels i and j;
// the rows are then placed in groups of four, each started by the most
// selected channel left and filled by the channels selected most often
// together with the group so far.
constexpr int SEL_SLICE = 4096;    // tokens per masking workgroup
constexpr int CS_CHUNK = 512;      // token masks staged per round of the counting

// R^T of every window of every pair, K and V (matrix (2 pair + which) nw + w),
// for the compressor's rotation loop
__global__ void k_sel_transpose(const float *rk, const float *rv, int npairs, int nw, float *rt) {
    const int m = blockIdx.x, pw = m >> 1, which = m & 1;      // m = 2 pair + which
    const int w = blockIdx.y;
    const float *R = (which ? rv : rk) + ((uint64_t)pw * nw + w) * D * D;
    float *dst = rt + ((uint64_t)m * nw + w) * D * D;
    for (int i = threadIdx.x; i < D * D; i += blockDim.x) {
        const int j = i / D, c = i % D;
        dst[c * D + j] = R[i];
    }
}

// grid (slices, windows, 2 pairs): every token of the slice rotated with the
// window's R (the compressor's chain) and ranked; its selected channels (the
// r largest magnitudes, lower channel first on ties) as a 128-bit mask at
// masks[(m nw + w) wtok + token in window]
__global__ void __launch_bounds__(256) k_sel_mask(const uint16_t *k, const uint16_t *v, int64_t seq_stride, int hkv,
                                                  int dtype, const int32_t *ctx, int W, int nw, int r,
                                                  const float *rt, uint4 *masks, int wtok) {
    constexpr int TPW = 16, NWV = 4;
    __shared__ SegSmem<NWV> sm;
    const int sl = blockIdx.x, w = blockIdx.y, m = blockIdx.z, pair = m >> 1, which = m & 1;
    const int L = ctx[pair / hkv];
    const int64_t a = (int64_t)w * W + (int64_t)sl * SEL_SLICE;
    const int64_t e = min(min((int64_t)(w + 1) * W, (int64_t)L), a + SEL_SLICE);
    if (a >= e) return;
    const uint16_t *src = (which ? v : k) + ((uint64_t)pair * seq_stride + (uint64_t)a) * D;
    const float *rtw = rt + ((uint64_t)m * nw + w) * D * D;
    uint4 *dst = masks + ((uint64_t)m * nw + w) * (uint64_t)wtok + (uint64_t)sl * SEL_SLICE;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int64_t t0 = 0; t0 < e - a; t0 += SEG) {
        const int ntok = (int)min((int64_t)SEG, e - a - t0);
        float y[TPW][2];
        rotate_tile(src + (uint64_t)t0 * D, ntok, rtw, dtype, sm, y);
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            if (wave * TPW + i < ntok) {                     // wave-uniform
                int rlo, rhi;
                group_ranks(y[i][0], y[i][1], 0, D, sm.keys[wave], rlo, rhi);
                const uint64_t mlo = __ballot(rlo < r), mhi = __ballot(rhi < r);
                if (lane == 0)
                    dst[t0 + wave * TPW + i] = make_uint4((uint32_t)mlo, (uint32_t)(mlo >> 32), (uint32_t)mhi,
                                                          (uint32_t)(mhi >> 32));
            }
        }
    }
}

// grid (2 pairs x windows, 8 blocks of 16 rows), 256 threads: co-selection
// counts of one window's tokens, thread t owning C[16 b + t / 16][8 (t % 16)
// .. + 7]; the masks are staged in LDS 512 tokens at a time.  Integer counts:
// exact in any order.  A window without tokens gets zeros.
__global__ void __launch_bounds__(256) k_cosel(const uint4 *masks, int hkv, const int32_t *ctx, int W, int nw,
                                               int wtok, uint32_t *cos) {
    __shared__ uint32_t ms[CS_CHUNK][4];
    const int mw = blockIdx.x, m = mw / nw, w = mw % nw, tid = threadIdx.x;
    const int L = ctx[(m >> 1) / hkv];
    const int ntok = (int)max((int64_t)0, min((int64_t)W, (int64_t)L - (int64_t)w * W));
    const int i = blockIdx.y * 16 + tid / 16, j0 = (tid % 16) * 8;
    const int wi = i >> 5, si = i & 31, wj = j0 >> 5, sj = j0 & 31;
    const uint4 *src = masks + (uint64_t)mw * (uint64_t)wtok;
    uint32_t cnt[8];
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) cnt[jj] = 0u;
    for (int t0 = 0; t0 < ntok; t0 += CS_CHUNK) {
        const int n = min(CS_CHUNK, ntok - t0);
        __syncthreads();
        for (int e = tid; e < n; e += 256) {
            const uint4 x = src[t0 + e];
            ms[e][0] = x.x; ms[e][1] = x.y; ms[e][2] = x.z; ms[e][3] = x.w;
        }
        __syncthreads();
        for (int t = 0; t < n; ++t) {
            const uint32_t sel = ((ms[t][wi] >> si) & 1u) ? (ms[t][wj] >> sj) : 0u;
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) cnt[jj] += (sel >> jj) & 1u;
        }
    }
    uint32_t *dst = cos + ((uint64_t)mw * D + i) * D + j0;
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) dst[jj] = cnt[jj];
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t y = __shfl_xor(x, o);
        x = x > y ? x : y;
    }
    return x;
}

// grid (windows, 2 pairs), 1024 threads: the new row order from the window's
// co-selection counts, then the rows of R moved in place; a window without
// tokens takes the order of the last window with tokens, and a pair with no
// tokens keeps R.  Each of the 128 placements takes the unplaced channel of
// the largest key (summed co-selection with the group so far, own count,
// lower channel): threads 0..127 hold one candidate each and two waves'
// maxima meet in LDS.
__global__ void __launch_bounds__(1024) k_sel_permute(float *rk, float *rv, int hkv, const int32_t *ctx, int W, int nw,
                                                      const uint32_t *cos) {
    __shared__ uint32_t Cs[D * D];
    __shared__ uint64_t best[2];
    __shared__ int pos[D];
    const int w = blockIdx.x, m = blockIdx.y, pair = m >> 1, which = m & 1, tid = threadIdx.x;
    const int L = ctx[pair / hkv];
    const int nwt = min(nw, (L + W - 1) / W);                 // windows with tokens
    if (nwt == 0) return;
    const int ws = min(w, nwt - 1);
    const uint32_t *cw = cos + ((uint64_t)m * nw + ws) * D * D;
    for (int e = tid; e < D * D; e += 1024) Cs[e] = cw[e];
    __syncthreads();
    const bool cand = tid < D;
    const uint32_t nj = cand ? Cs[tid * D + tid] : 0u;
    uint32_t gsum = 0u;
    bool placed = false;
    for (int k = 0; k < D; ++k) {
        if ((k & 3) == 0) gsum = 0u;                           // a new group of four
        uint64_t key = (cand && !placed) ? (((uint64_t)gsum << 32) | ((uint64_t)nj << 8) | (uint64_t)(D - tid)) : 0ull;
        key = wave_max_u64(key);
        if (tid < D && (tid & 63) == 0) best[tid >> 6] = key;
        __syncthreads();
        const uint64_t b = best[0] > best[1] ? best[0] : best[1];
        const int pick = D - (int)(b & 0xffu);
        if (cand) {
            if (tid == pick) { placed = true; pos[tid] = k; }
            gsum += Cs[pick * D + tid];
        }
        __syncthreads();
    }
    float *R = (which ? rv : rk) + ((uint64_t)pair * nw + w) * D * D;
    const int row = tid >> 3, part = (tid & 7) * 16;        // 128 rows x 8 parts of 16 values
    float4 t[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = *(const float4 *)(R + row * D + part + 4 * i);
    __syncthreads();                                         // every row read before any is written
#pragma unroll
    for (int i = 0; i < 4; ++i) *(float4 *)(R + pos[row] * D + part + 4 * i) = t[i];
}

}  // namespace

// the context lengths of a compress call, from the caller's host array into the arena
hipError_t launch_ctx_copy(int32_t *dst_dev, const int32_t *src_host, int n, hipStream_t s) {
    return hipMemcpyAsync(dst_dev, src_host, sizeof(int32_t) * (size_t)n, hipMemcpyHostToDevice, s);
}

hipError_t launch_pairs_copy(uint64_t *dst_dev, const uint64_t *src_host, int npairs, hipStream_t s) {
    return hipMemcpyAsync(dst_dev, src_host, sizeof(uint64_t) * 4 * (size_t)npairs, hipMemcpyHostToDevice, s);
}

hipError_t launch_copy_rot(const Geom &g, const float *rk, const float *rv, int nw_src, hipStream_t s) {
    hipLaunchKernelGGL(k_copy_rot, dim3(g.nw, g.npairs), dim3(256), 0, s, g, rk, rv, nw_src);
    return hipGetLastError();
}

hipError_t launch_close(const Geom &g, const float *rk, const float *rv, const uint16_t *k, const uint16_t *v,
                        int64_t seq_stride, int max_segs, hipStream_t s) {
    hipLaunchKernelGGL(k_close_rot, dim3(2, g.npairs), dim3(256), 0, s, g, rk, rv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 grid(max_segs, g.npairs);
    if (max_segs > 0) {
        hipLaunchKernelGGL(k_prefill<0>, grid, dim3(256), 0, s, g, k, v, seq_stride, (uint8_t *)nullptr, 0u, 0u, 1);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(k_scan, dim3(g.npairs), dim3(256), 0, s, g, 1);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(k_prefill<1>, grid, dim3(256), 0, s, g, k, v, seq_stride, (uint8_t *)nullptr, 0u, 0u, 1);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_close_done, dim3(ceil_div(g.npairs, 256)), dim3(256), 0, s, g);
    return hipGetLastError();
}

hipError_t launch_set_meta(const Geom &g, const int32_t *ctx_dev, hipStream_t s) {
    hipLaunchKernelGGL(k_set_meta, dim3(ceil_div(g.npairs, 256)), dim3(256), 0, s, g, ctx_dev);
    return hipGetLastError();
}

hipError_t launch_compress(const Geom &g, const uint16_t *k, const uint16_t *v, int64_t seq_stride,
                           const int32_t *ctx_dev, int max_full_segs, int any_tail, uint8_t *ws, uint32_t slot_tok,
                           uint32_t slot_sc, hipStream_t s) {
    hipError_t e = launch_set_meta(g, ctx_dev, s);
    if (e != hipSuccess) return e;
    if (g.dyn) {
        hipLaunchKernelGGL(k_cov_seg, dim3(g.npairs, 2, D / 16), dim3(256), 0, s, g, k, v, seq_stride, 1);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const dim3 grid(max_full_segs, g.npairs);
    if (max_full_segs > 0) {
        if (ws) hipLaunchKernelGGL(k_prefill<2>, grid, dim3(256), 0, s, g, k, v, seq_stride, ws, slot_tok, slot_sc, 0);
        else hipLaunchKernelGGL(k_prefill<0>, grid, dim3(256), 0, s, g, k, v, seq_stride, ws, slot_tok, slot_sc, 0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_scan, dim3(g.npairs), dim3(256), 0, s, g, 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (max_full_segs > 0) {
        if (ws) hipLaunchKernelGGL(k_compact, grid, dim3(256), 0, s, g, (const uint8_t *)ws, slot_tok, slot_sc);
        else hipLaunchKernelGGL(k_prefill<1>, grid, dim3(256), 0, s, g, k, v, seq_stride, ws, slot_tok, slot_sc, 0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (any_tail) {
        hipLaunchKernelGGL(k_stage_tail, dim3(g.npairs), dim3(256), 0, s, g, k, v, seq_stride);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = launch_maintain(g, MAINT_AFTER_PREFILL, MAINT_FLUSH, s)) != hipSuccess) return e;
    }
    return hipSuccess;
}

// reorder workspace: context lengths, then per matrix (2 pairs x windows) the
// token masks (wtok per window), the co-selection counts and R^T
size_t reorder_ws_bytes(int num_seqs, int hkv, int nw, int wtok) {
    const size_t mats = (size_t)num_seqs * hkv * 2 * nw;
    return ((size_t)num_seqs * sizeof(int32_t) + 255) / 256 * 256 + (mats * wtok * 16 + 255) / 256 * 256 +
           mats * D * D * sizeof(uint32_t) + mats * D * D * sizeof(float);
}

hipError_t launch_reorder(const uint16_t *k, const uint16_t *v, int64_t seq_stride, int num_seqs, int hkv, int dtype,
                          const int32_t *ctx_dev, int W, int nw, int wtok, int r, float *rot_k, float *rot_v,
                          uint8_t *ws, hipStream_t s) {
    const int npairs = num_seqs * hkv, m = npairs * 2;
    uint4 *masks = (uint4 *)(ws + ((size_t)num_seqs * sizeof(int32_t) + 255) / 256 * 256);
    uint32_t *cos = (uint32_t *)((uint8_t *)masks + ((size_t)m * nw * wtok * 16 + 255) / 256 * 256);
    float *rt = (float *)((uint8_t *)cos + (size_t)m * nw * D * D * sizeof(uint32_t));
    hipLaunchKernelGGL(k_sel_transpose, dim3(m, nw), dim3(256), 0, s, rot_k, rot_v, npairs, nw, rt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_sel_mask, dim3(ceil_div(W < wtok ? W : wtok, SEL_SLICE), nw, m), dim3(256), 0, s, k, v,
                       seq_stride, hkv, dtype, ctx_dev, W, nw, r, rt, masks, wtok);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_cosel, dim3(m * nw, D / 16), dim3(256), 0, s, masks, hkv, ctx_dev, W, nw, wtok, cos);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_sel_permute, dim3(nw, m), dim3(1024), 0, s, rot_k, rot_v, hkv, ctx_dev, W, nw, cos);
    return hipGetLastError();
}

hipError_t launch_append(const Geom &g, const uint16_t *k, const uint16_t *v, hipStream_t s) {
    hipLaunchKernelGGL(k_append, dim3(g.npairs), dim3(128), 0, s, g, k, v);
    return hipGetLastError();
}

hipError_t launch_maintain(const Geom &g, int mode, int what, hipStream_t s) {
    hipError_t e;
    if (what & MAINT_FLUSH) {
        hipLaunchKernelGGL(k_flush, dim3(g.npairs, UBUF / MT_TOK), dim3(MT_THREADS), 0, s, g, mode);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if ((what & MAINT_FINALIZE) && mode == MAINT_APPEND) {
        hipLaunchKernelGGL(k_fin_stats, dim3(g.npairs, SEG / MT_TOK), dim3(MT_THREADS), 0, s, g);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(k_fin_pack, dim3(g.npairs, SEG / MT_TOK), dim3(MT_THREADS), 0, s, g);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (g.dyn) {
            hipLaunchKernelGGL(k_cov_seg, dim3(g.npairs, 2, D / 16), dim3(256), 0, s, g, (const uint16_t *)nullptr,
                               (const uint16_t *)nullptr, (int64_t)0, 0);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            hipLaunchKernelGGL(k_win_update, dim3(ceil_div(g.npairs, 4)), dim3(256), 0, s, g);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

}  // namespace mosaic
