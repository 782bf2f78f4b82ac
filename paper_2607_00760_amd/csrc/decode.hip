// decode.hip -- gfx950 kernels of MosaicKV's decode step (PackedAttention,
// Sec. 5.3; stage-2 dynamic sequence compression, Sec. 4.2).
//
//   qrot   : q . R_k^T once per (pair, window) -- the rotation is merged into
//            the single query vector instead of un-rotating the cache.  Each
//            workgroup produces 16 output channels from an LDS slice of R_k^T;
//            every output is one fp32 fused chain over the input channels.
//   score  : lane per block key.  The packed record (bitmap + values) is read
//            straight into registers; a fixed, unrolled slot sequence walks
//            the bitmap's set bits in ascending order (v_ffbl on the current
//            word), fp32 fused chain over the kept channels, max over the GQA
//            group.  These scores decide the selection, so their arithmetic
//            order is fixed.
//   topk   : exact selection of the k-th largest score key: passes over the
//            range [min, max] of the keys still in play, 2048 bins each, so
//            the bins follow the keys that are present (at most three passes
//            reach a single key), then an ordered compaction that breaks ties
//            by the lowest block index.  Up to 32768 blocks per pair the keys
//            stay in registers (16 or 32 per thread, one workgroup per pair);
//            scans and reductions use lane shifts inside the wave.  Longer
//            pairs are spread over workgroups of 4096 blocks, one kernel per
//            phase.
//   attn   : split-K over the selected list (up to 128 blocks of one rotation
//            window per split).  The split's blocks are ordered by size, so a
//            64-token chunk never cuts a block and a token finds its block by
//            a closed form.  Lane per token: the packed K record is expanded
//            from registers into an LDS tile with the same bitmap walk,
//            logits K . q^T on the matrix cores (16x16x32, q split into two
//            16-bit halves), online softmax in fp32 on the accumulator layout,
//            then V expanded the same way and P . V on the matrix cores.  The
//            matrix-core operand reads zero what they read, so the tile is
//            zero again for the next expansion without a clearing pass.  The
//            next chunk's records are loaded while the current one is
//            processed.  The update buffer is one more split (dense, unrotated).
//            Each window split rotates its accumulator back by R_v before
//            writing it (the rotation stays merged into one vector per split).
//   combine: log-sum-exp merge of every split of a pair into the output.
#include "mosaic_internal.h"

namespace mosaic {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 halfx8;
typedef __attribute__((ext_vector_type(4))) float floatx4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

template <int DT> struct Mma;
template <> struct Mma<1> {
    using v8 = bf16x8;
    using el = __bf16;
    static __device__ __forceinline__ floatx4 run(v8 a, v8 b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mma<0> {
    using v8 = halfx8;
    using el = _Float16;
    static __device__ __forceinline__ floatx4 run(v8 a, v8 b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};

template <int DT> __device__ __forceinline__ float h2f_t(uint32_t h16) {
    if (DT) return __uint_as_float(h16 << 16);
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h16);
}

__device__ __forceinline__ void wave_sync() { __builtin_amdgcn_wave_barrier(); }

// LDS byte addresses as plain integers (so that address arithmetic folds into
// single mad/shift-add instructions) and accesses through them
typedef __attribute__((address_space(3))) uint8_t lds_u8;
__device__ __forceinline__ uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)(const lds_u8 *)p; }
template <typename T> __device__ __forceinline__ T lds_ld(uint32_t a) {
    return *(const __attribute__((address_space(3))) T *)(uintptr_t)a;
}
template <typename T> __device__ __forceinline__ void lds_st(uint32_t a, T v) {
    *(__attribute__((address_space(3))) T *)(uintptr_t)a = v;
}
// keep the compiler from moving memory operations across this point
__device__ __forceinline__ void mem_fence_compiler() { asm volatile("" ::: "memory"); }

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

// ------------------------------------------------------------------ qrot
// grid (windows * 2, pairs), 256 threads: a workgroup produces 64 output
// channels j0..j0+63 of every query head of one (pair, window).  It stages the
// matching 256-byte half of every row of R_k^T (32 KB, each 128-byte line read
// by one workgroup only) and the pair's queries in LDS; thread (j, h) then runs
// the fp32 fused chain over the input channels c for head h (and h + 4).
constexpr int QROT_COLS = 64;

__global__ void __launch_bounds__(256) k_qrot(Geom g, WsGeom ws, const uint16_t *q) {
    __shared__ __align__(16) float rt[D][QROT_COLS];      // R_k^T[c][j0 + jj] = R_k[j0 + jj][c]
    __shared__ float qs[8][D];
    constexpr int NCG = D / QROT_COLS;
    const int w = blockIdx.x / NCG, j0 = (blockIdx.x % NCG) * QROT_COLS;
    const int p = blockIdx.y, tid = threadIdx.x, G = g.G;
    if (ws.tkx && blockIdx.x == 0) {        // the multi-workgroup top-k's histograms of this call
        uint32_t *h = ws.tkx + (uint64_t)p * (ws.tkx_stride / 4);
        for (int i = tid; i < 3 * 2048; i += 256) h[i] = 0u;
    }
    if (g.rotated) {
        const float *src = g.rot_of(p, w);
        constexpr int PER = D * QROT_COLS / 4 / 256;       // 16-byte pieces per thread
        uint4 t[PER];
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int idx = tid + 256 * k, c = idx / (QROT_COLS / 4), part = idx % (QROT_COLS / 4);
            t[k] = *(const uint4 *)(src + c * D + j0 + 4 * part);
        }
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int idx = tid + 256 * k, c = idx / (QROT_COLS / 4), part = idx % (QROT_COLS / 4);
            *(uint4 *)&rt[c][4 * part] = t[k];
        }
    }
    for (int i = tid; i < G * D; i += 256) qs[i / D][i % D] = h2f(q[(uint64_t)p * G * D + i], g.dtype);
    __syncthreads();
    const int jj = tid & (QROT_COLS - 1), h0 = tid / QROT_COLS;   // heads h0 and h0 + 4
    float a0 = 0.0f, a1 = 0.0f;
    if (g.rotated) {
        if (h0 + 4 < G) {
#pragma unroll 8
            for (int c = 0; c < D; ++c) {
                const float r = rt[c][jj];
                a0 = fmaf(qs[h0][c], r, a0);
                a1 = fmaf(qs[h0 + 4][c], r, a1);
            }
        } else if (h0 < G) {
#pragma unroll 8
            for (int c = 0; c < D; ++c) a0 = fmaf(qs[h0][c], rt[c][jj], a0);
        }
    } else {
        a0 = (h0 < G) ? qs[h0][j0 + jj] : 0.0f;
        a1 = (h0 + 4 < G) ? qs[h0 + 4][j0 + jj] : 0.0f;
    }
    float *dst = ws.qrot + (uint64_t)p * (ws.qrot_stride / 4) + ((uint64_t)w * D + j0 + jj) * g.GP;
    if (h0 < g.GP) dst[h0] = (h0 < G) ? a0 : 0.0f;
    if (h0 + 4 < g.GP) dst[h0 + 4] = (h0 + 4 < G) ? a1 : 0.0f;
}

// ------------------------------------------------------------------ bitmap walk
// A packed vector keeps r values in ascending channel order; its bitmap marks
// the kept groups of 1 << log2g channels.  The walk visits the set bits in
// ascending order, one per step, so that a fixed, unrolled slot sequence can
// take the values from registers.  The position is v_ffbl of the current
// bitmap word; the words are walked in order, with empty words in the middle
// squeezed out first so that a step moves on by at most one word.  Each word
// carries the caller's address of its first group.
struct Walk {
    uint32_t cur, n1, n2, n3;
    uint32_t a, a1, a2, a3;
    __device__ __forceinline__ uint32_t pos() const { return (uint32_t)__builtin_ctz(cur); }
    template <int NWD>
    __device__ __forceinline__ void step() {
        cur &= cur - 1u;
        if (NWD > 1) {
            const bool z = cur == 0u;
            cur = z ? n1 : cur;
            a = z ? a1 : a;
            if (NWD > 2) {
                n1 = z ? n2 : n1; a1 = z ? a2 : a1;
                n2 = z ? n3 : n2; a2 = z ? a3 : a2;
            }
        }
    }
};

__device__ __forceinline__ void cswap_empty(uint32_t &wa, uint32_t &aa, uint32_t &wb, uint32_t &ab) {
    const bool z = wa == 0u;
    wa = z ? wb : wa;
    aa = z ? ab : aa;
    wb = z ? 0u : wb;
}

template <int NWD>
__device__ __forceinline__ Walk make_walk(const uint32_t (&bw)[4], uint32_t a0, uint32_t astep) {
    uint32_t w[4], a[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) { w[k] = k < NWD ? bw[k] : 0u; a[k] = a0 + (uint32_t)k * astep; }
    if (NWD == 2) {
        const bool hole = w[0] == 0u && w[1] != 0u;
        if (__ballot(hole)) cswap_empty(w[0], a[0], w[1], a[1]);
    } else if (NWD == 4) {
        const bool hole = (w[0] == 0u && (w[1] | w[2] | w[3]) != 0u) || (w[1] == 0u && (w[2] | w[3]) != 0u) ||
                          (w[2] == 0u && w[3] != 0u);
        if (__ballot(hole)) {                      // stable: non-empty words to the front
#pragma unroll
            for (int round = 0; round < 2; ++round) {
                cswap_empty(w[0], a[0], w[1], a[1]);
                cswap_empty(w[2], a[2], w[3], a[3]);
                cswap_empty(w[1], a[1], w[2], a[2]);
            }
        }
    }
    Walk wk;
    wk.cur = w[0]; wk.n1 = w[1]; wk.n2 = w[2]; wk.n3 = w[3];
    wk.a = a[0]; wk.a1 = a[1]; wk.a2 = a[2]; wk.a3 = a[3];
    return wk;
}

// A truncated bitmap (Sec. 5.2: only the first T channels are represented)
// has T / g bits; the whole 16-byte bitmap loads read the values after it
// as well, so the words are cut to the first nbits bits before a walk.
__device__ __forceinline__ void mask_words(uint32_t (&bw)[4], int nbits) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int lo = 32 * k;
        bw[k] = nbits >= lo + 32 ? bw[k] : (nbits <= lo ? 0u : bw[k] & ((1u << (nbits - lo)) - 1u));
    }
}

// element s (static) of packed 16-bit values held two per dword
template <int N>
__device__ __forceinline__ uint32_t half_at(const uint32_t (&v)[N], int s) {
    return (s & 1) ? (v[s >> 1] >> 16) : (v[s >> 1] & 0xffffu);
}

// 16 bytes at a 4-byte aligned address: every record is 4-byte aligned, and
// the target runs vector memory loads in unaligned mode, so one dwordx4 load
// serves any record (the compiler merges plain dword runs the same way)
typedef uint32_t u32x4a4 __attribute__((ext_vector_type(4), aligned(4)));

// N dwords starting at any byte p: the N + 1 aligned dwords that cover them,
// joined pairwise by byte shifts (v_alignbyte).  Truncated bitmaps of 3 or 6
// bytes put token bitmaps and block-key records at any byte; the one dword
// read past the end stays inside the arena's slack.
template <int N>
__device__ __forceinline__ void load_dwords_any(const uint8_t *p, uint32_t (&out)[N]) {
    const uintptr_t a = (uintptr_t)p;
    const uint32_t *b = (const uint32_t *)(a & ~(uintptr_t)3);
    const uint32_t sh = (uint32_t)(a & 3u);
    uint32_t w[N + 1];
#pragma unroll
    for (int k = 0; k <= N; ++k) w[k] = b[k];
#pragma unroll
    for (int k = 0; k < N; ++k) out[k] = __builtin_amdgcn_alignbyte(w[k + 1], w[k], sh);
}

// A packed vector (bitmap words + values) held in registers.
template <int RMAX>
struct PVec {
    uint32_t bw[4];
    uint32_t v[RMAX / 2];
};

// A token record with one-byte E4M3 values, as loaded (four codes per word,
// slot order from the low byte); widened to the dtype just before its walk,
// so that the loads of a prefetch are not waited on where they are issued.
template <int RMAX>
struct PVec8 {
    uint32_t bw[4];
    uint32_t v[RMAX / 4];
};

// codes 2 HI and 2 HI + 1 of w -> the two 16-bit values of the dtype (exact:
// every E4M3 value is a bf16 and an fp16 value), the first in the low half
template <int DT, bool HI>
__device__ __forceinline__ uint32_t e4m3x2(uint32_t w) {
    if constexpr (DT) return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
    else return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, HI));
}

// the first NW words of codes (4 NW values) widened into a 16-bit vector
template <int DT, int RMAX, int NW>
__device__ __forceinline__ void widen(const PVec8<RMAX> &c, PVec<RMAX> &x) {
    static_assert(NW <= RMAX / 4, "code words");
#pragma unroll
    for (int k = 0; k < 4; ++k) x.bw[k] = c.bw[k];
#pragma unroll
    for (int k = 0; k < NW; ++k) {
        x.v[2 * k] = e4m3x2<DT, false>(c.v[k]);
        x.v[2 * k + 1] = e4m3x2<DT, true>(c.v[k]);
    }
}

// bm and val point at the vector's bitmap and values; rmax is the largest r
// in the wave (uniform) and a16 (uniform) says both pointers are 16-byte
// aligned (A16: always so).  The loads take a fixed 16-byte bitmap and rmax
// values: what lies past a vector's own bitmap or values is read (inside the
// arena's slack) and never used.  Value slots at or past rmax keep what they
// held: a walk reads only its first r slots, and leaving them unwritten keeps
// the registers of earlier, still outstanding loads free of write-after-write
// waits.
//
// A16: 1 = the pointers are known 16-byte aligned, 0 = dword loads, -1 = chosen
// by a16 at run time.  ZF zero-fills the slots past rmax.  Without it every
// slot is loaded, those past rmax from the start of the values again (lines
// the wave reads anyway): straight-line loads with no branch, so that a
// prefetch into loop-carried registers leaves no join whose bookkeeping would
// make the wave wait on loads that are still in flight.
//
// RL > 0: exactly the first RL 16-byte granules of values and a 16-byte
// bitmap, with no condition (the caller knows r <= 8 RL for every lane of the
// wave), at any 4-byte aligned record.
template <int RMAX, int A16, bool ZF, int RL = 0>
__device__ __forceinline__ void load_pvec(PVec<RMAX> &x, const uint8_t *bm, const uint8_t *val, int rmax, bool a16) {
    static_assert(RL == 0 || (A16 == 1 && RL <= RMAX / 8), "fixed granule count");
    if (RL > 0) {
        const u32x4a4 b = *(const u32x4a4 *)bm;
        x.bw[0] = b.x; x.bw[1] = b.y; x.bw[2] = b.z; x.bw[3] = b.w;
        const u32x4a4 *v4 = (const u32x4a4 *)val;
#pragma unroll
        for (int k = 0; k < RL; ++k) {
            const u32x4a4 t = v4[k];
            x.v[4 * k] = t.x; x.v[4 * k + 1] = t.y; x.v[4 * k + 2] = t.z; x.v[4 * k + 3] = t.w;
        }
    } else if (A16 == 1 || (A16 == -1 && a16)) {
        const uint4 b = *(const uint4 *)bm;
        x.bw[0] = b.x; x.bw[1] = b.y; x.bw[2] = b.z; x.bw[3] = b.w;
        const uint4 *v4 = (const uint4 *)val;
#pragma unroll
        for (int k = 0; k < RMAX / 8; ++k) {
            uint4 t;
            if (ZF) {
                t = make_uint4(0u, 0u, 0u, 0u);
                if (8 * k < rmax) t = v4[k];
            } else {
                t = v4[(8 * k < rmax) ? k : 0];
            }
            x.v[4 * k] = t.x; x.v[4 * k + 1] = t.y; x.v[4 * k + 2] = t.z; x.v[4 * k + 3] = t.w;
        }
    } else {
        // dword loads at any byte: the bitmap, then the values below rmax
        // (those past it from the start of the values again, or zero with ZF)
        load_dwords_any<4>(bm, x.bw);
        const uintptr_t va = (uintptr_t)val;
        const uint32_t *v = (const uint32_t *)(va & ~(uintptr_t)3);
        const uint32_t sh = (uint32_t)(va & 3u);
        uint32_t u[RMAX / 2 + 1];
#pragma unroll
        for (int k = 0; k <= RMAX / 2; ++k) u[k] = v[(2 * k < rmax + 2) ? k : 0];
#pragma unroll
        for (int k = 0; k < RMAX / 2; ++k) {
            const uint32_t t = __builtin_amdgcn_alignbyte(u[k + 1], u[k], sh);
            x.v[k] = (ZF && 2 * k >= rmax) ? 0u : t;
        }
    }
}

// maximum over the wave of 0 <= v < 256 (every lane active): eight ballots,
// no cross-lane data movement
__device__ __forceinline__ int wave_max_i(int v) {
    int m = 0;
#pragma unroll
    for (int b = 7; b >= 0; --b) {
        const int c = m | (1 << b);
        if (__ballot(v >= c)) m = c;
    }
    return m;
}

template <int V> struct IntC { static constexpr int value = V; };

// ------------------------------------------------------------------ score
// One walk: acc[h] += q[c][h] * value over the kept channels c, ascending.
// qs + qoff is the [D][GP] fp32 query of the vector's window.  RV is the
// number of kept values when it is a compile-time constant, else 0 and r
// (wave-uniform over the calling lanes) gives it.  The LDS reads of q run SA
// steps ahead of their products (the positions do not depend on q), so a
// step does not wait for its own read.
template <int DT, int GP, int RMAX, int L2G, int RV>
__device__ __forceinline__ void score_walk(const PVec<RMAX> &x, int r, uint32_t qaddr, float (&acc)[GP]) {
    constexpr int GS = 1 << L2G, NWD = 4 >> L2G;
    constexpr uint32_t QB = GP * 4;                           // bytes of q per channel
    constexpr int NS = (RV ? RV : RMAX) / GS;                 // most steps
    constexpr int SA = GS == 1 ? 2 : 0;                       // reads in flight ahead of use
    constexpr int NQ = GS * (GP / 4);                         // 16-byte reads per step
    Walk wk = make_walk<NWD>(x.bw, qaddr, 32u * GS * QB);      // LDS address of group 0 of word k
    const int n = RV ? RV : r;
    floatx4 ring[SA + 1][NQ];
    auto issue = [&](int j) {                                 // j static in the unrolled code
        const uint32_t qc = wk.a + wk.pos() * (GS * QB);
#pragma unroll
        for (int e = 0; e < GS; ++e)
#pragma unroll
            for (int h4 = 0; h4 < GP; h4 += 4)
                ring[j % (SA + 1)][e * (GP / 4) + h4 / 4] = lds_ld<floatx4>(qc + e * QB + h4 * 4);
        wk.template step<NWD>();
    };
#pragma unroll
    for (int j = 0; j < SA; ++j)
        if (j < NS && (RV || j * GS < n)) issue(j);
#pragma unroll
    for (int k = 0; k < NS; ++k) {
        if (RV || k * GS < n) {                               // wave-uniform
            if (k + SA < NS && (RV || (k + SA) * GS < n)) issue(k + SA);
#pragma unroll
            for (int e = 0; e < GS; ++e) {
                const float xv = h2f_t<DT>(half_at(x.v, k * GS + e));
#pragma unroll
                for (int h4 = 0; h4 < GP; h4 += 4) {
                    const floatx4 q4 = ring[k % (SA + 1)][e * (GP / 4) + h4 / 4];
                    acc[h4] = fmaf(q4[0], xv, acc[h4]);
                    acc[h4 + 1] = fmaf(q4[1], xv, acc[h4 + 1]);
                    acc[h4 + 2] = fmaf(q4[2], xv, acc[h4 + 2]);
                    acc[h4 + 3] = fmaf(q4[3], xv, acc[h4 + 3]);
                }
            }
            if ((k & 3) == 3) __builtin_amdgcn_sched_barrier(0);   // bound the look-ahead
        }
    }
}

// FR: every kept count is 16, 32 or 48 (checked on the host), each with its
// own fully unrolled walk; otherwise one walk with a runtime trip count.  The
// two kinds live in different kernels so that the compiler cannot fold the
// fixed walks into the general one.
template <int DT, int GP, int RMAX, int L2G, bool FR>
__device__ __forceinline__ void score_r(const PVec<RMAX> &x, int r, uint32_t qaddr, float (&acc)[GP]) {
    if (FR) {
        if (r == 32) score_walk<DT, GP, RMAX, L2G, 32>(x, r, qaddr, acc);
        else if (r == 16) score_walk<DT, GP, RMAX, L2G, 16>(x, r, qaddr, acc);
        else score_walk<DT, GP, RMAX, L2G, (RMAX >= 48 ? 48 : 16)>(x, r, qaddr, acc);
    } else {
        score_walk<DT, GP, RMAX, L2G, 0>(x, r, qaddr, acc);
    }
}

// One pass per distinct (r, log2g) among the active lanes, so that every walk
// runs with a wave-uniform trip count and no per-step predicate.
template <int DT, int GP, int RMAX, bool FR>
__device__ __forceinline__ void score_any(const PVec<RMAX> &x, int r, int l2g, uint32_t qaddr, float (&acc)[GP]) {
    const int key = (r << 2) | l2g;
    uint64_t todo = __ballot(1);
    while (todo) {
        const int kv = __builtin_amdgcn_readlane(key, (int)__builtin_ctzll(todo));
        const bool mine = key == kv;
        todo &= ~__ballot(mine);
        if (mine) {
            const int rv = kv >> 2;
            if ((kv & 3) == 0) score_r<DT, GP, RMAX, 0, FR>(x, rv, qaddr, acc);
            else if ((kv & 3) == 1) score_r<DT, GP, RMAX, 1, FR>(x, rv, qaddr, acc);
            else score_r<DT, GP, RMAX, 2, FR>(x, rv, qaddr, acc);
        }
    }
}

// grid (ceil(max segments / spw), pairs): a workgroup scores the block keys of
// spw <= SCORE_SEGS consecutive segments, one lane per block key; spw is at
// most the segments of every window but a pair's last (W, or the least a
// window closed by its loss holds), so a workgroup sees at most two windows.
template <int DT, int GP, int RMAX, bool FR>
__global__ void __launch_bounds__(256) k_score(Geom g, WsGeom ws, int spw) {
    __shared__ __align__(16) float qs[2][D * GP];
    __shared__ Desc ds[SCORE_SEGS];
    __shared__ uint8_t b2s[SCORE_SEGS * 16];                 // block (relative) -> segment (relative)
    __shared__ int s_nblk;

    const int p = blockIdx.y, tid = threadIdx.x;
    const PairMeta meta = *g.meta_of(p);
    int nf, prov, nbuf;
    const int ndesc = pair_ndesc(meta, nf, prov, nbuf);
    const int s0 = blockIdx.x * spw;
    if (s0 >= ndesc) return;
    const int ns = min(spw, ndesc - s0);
    const Desc *gd = g.desc_of(p);
    const uint32_t fb0 = gd[s0].first_block;
    bool plain = true;                      // one channel per group, r a multiple of 8 up to 32, aligned records
    bool dense = true;                      // every channel kept (r = D), aligned records
    if (tid < ns) {
        const Desc d = gd[s0 + tid];
        ds[tid] = d;
        const int nb = ((d.flags & 1) ? UBUF : SEG) >> d.log2b;
        const int o = (int)(d.first_block - fb0);
        for (int j = 0; j < nb; ++j) b2s[o + j] = (uint8_t)tid;
        if (tid == ns - 1) s_nblk = o + nb;
        plain = d.log2g == 0 && d.r <= 32 && (d.sc_off & 3u) == 0;
        dense = d.log2g == 0 && d.r == D && (d.sc_off & 15u) == 0;
    }
    // the window of the first segment and the first segment of the next one
    const int w0 = g.rotated ? win_of_seg(g, p, s0) : 0;
    const int nxt = g.rotated ? win_first_seg(g, p, w0 + 1) : 0x7fffffff;
    const int w1 = (s0 + ns - 1 >= nxt) ? w0 + 1 : w0;
    {
        const float4 *src = (const float4 *)(ws.qrot + (uint64_t)p * (ws.qrot_stride / 4));
        float4 *d0 = (float4 *)qs[0], *d1 = (float4 *)qs[1];
        for (int i = tid; i < D * GP / 4; i += 256) {
            const float4 x0 = src[(uint64_t)w0 * D * GP / 4 + i], x1 = src[(uint64_t)w1 * D * GP / 4 + i];
            d0[i] = x0;
            d1[i] = x1;
        }
    }
    plain = __syncthreads_and(plain);
    if (RMAX >= D) dense = __syncthreads_and(dense);
    const int nblk = s_nblk;
    float *out = ws.score + (uint64_t)p * (ws.score_stride / 4);
    uint2 *binfo = ws.binfo + (uint64_t)p * (ws.binfo_stride / 8);
    uint8_t *bsize = ws.bsize + (uint64_t)p * ws.bsize_stride;
    // a block's token-record offset and strategy (what the selection hands to the attention)
    auto info_of = [&](const Desc &d, int j) {
        return blk_info(d.tok_off + (uint32_t)(j << d.log2b) * (uint32_t)(2 * tok_vec_bytes(d.r, d.log2g, g.trunc, g.fp8)),
                        d.r, d.log2g, d.log2b);
    };
    const uint8_t *sc = g.sc_of(p);
    if constexpr (RMAX >= D) {
        if (dense) {
            // every channel kept: the values are the dense key in channel
            // order; the same ascending fp32 chain reads q row by row (one
            // address for the whole wave)
            for (int b0 = 0; b0 < nblk; b0 += 256) {
                const int b = b0 + tid;
                const bool valid = b < nblk;
                const int i = valid ? b2s[b] : 0;
                const Desc d = ds[i];
                const int j = b - (int)(d.first_block - fb0);
                const uint8_t *rec = valid ? sc + d.sc_off + (uint32_t)j * (uint32_t)vec_bytes(D, 0, g.trunc) : sc;
                const uint4 *v4 = (const uint4 *)(rec + 16);
                uint4 t[D / 8];
#pragma unroll
                for (int k = 0; k < D / 8; ++k) t[k] = v4[k];
                const uint32_t qa = lds_addr(qs) + ((s0 + i >= nxt) ? D * GP * 4 : 0);
                float acc[GP];
#pragma unroll
                for (int h = 0; h < GP; ++h) acc[h] = 0.0f;
#pragma unroll
                for (int k = 0; k < D / 8; ++k) {
                    const uint32_t w4[4] = {t[k].x, t[k].y, t[k].z, t[k].w};
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float xv = h2f_t<DT>((e & 1) ? (w4[e >> 1] >> 16) : (w4[e >> 1] & 0xffffu));
#pragma unroll
                        for (int h4 = 0; h4 < GP; h4 += 4) {
                            const floatx4 q4v = lds_ld<floatx4>(qa + (uint32_t)(((8 * k + e) * GP + h4) * 4));
                            acc[h4] = fmaf(q4v[0], xv, acc[h4]);
                            acc[h4 + 1] = fmaf(q4v[1], xv, acc[h4 + 1]);
                            acc[h4 + 2] = fmaf(q4v[2], xv, acc[h4 + 2]);
                            acc[h4 + 3] = fmaf(q4v[3], xv, acc[h4 + 3]);
                        }
                    }
                }
                float best = acc[0];
#pragma unroll
                for (int h = 1; h < GP; ++h)
                    if (h < g.G) best = fmaxf(best, acc[h]);
                if (__float_as_uint(best) == 0x80000000u) best = 0.0f;
                if (valid) {
                    out[d.first_block + j] = best;
                    binfo[d.first_block + j] = info_of(d, j);
            bsize[d.first_block + j] = d.log2b;
                    bsize[d.first_block + j] = d.log2b;
                }
            }
            return;
        }
    }
    if (plain) {
        // one channel per group and at most 32 values: a 16-byte bitmap and
        // four fixed 16-byte value loads at any 4-byte aligned record, and the
        // next key's record is loaded while the current one is scored (one
        // load form, so no join waits on it)
        auto where = [&](int b, int &i, int &j, int &r) {
            const bool valid = b < nblk;
            i = valid ? b2s[b] : 0;
            const Desc d = ds[i];
            j = b - (int)(d.first_block - fb0);
            r = valid ? d.r : 0;
            return valid ? sc + d.sc_off + (uint32_t)j * (uint32_t)vec_bytes(d.r, 0, g.trunc) : sc;
        };
        const int bmb = bm_bytes(0, g.trunc);
        int i, j, r;
        const uint8_t *rec = where(tid, i, j, r);
        PVec<RMAX> x;
        load_pvec<RMAX, 1, false, 4>(x, rec, rec + bmb, 32, true);
        for (int b0 = 0; b0 < nblk; b0 += 256) {
            int in, jn, rn;
            const uint8_t *recn = where(b0 + 256 + tid, in, jn, rn);
            PVec<RMAX> xn;
            __builtin_amdgcn_sched_barrier(0);
            load_pvec<RMAX, 1, false, 4>(xn, recn, recn + bmb, 32, true);
            __builtin_amdgcn_sched_barrier(0);
            if (g.trunc < D) mask_words(x.bw, g.trunc);       // a truncated bitmap's bytes past T bits are values
            const uint32_t qoff = (s0 + i >= nxt) ? D * GP * 4 : 0;
            float acc[GP];
#pragma unroll
            for (int h = 0; h < GP; ++h) acc[h] = 0.0f;
            score_any<DT, GP, RMAX, FR>(x, r, 0, lds_addr(qs) + qoff, acc);
            float best = acc[0];
#pragma unroll
            for (int h = 1; h < GP; ++h)
                if (h < g.G) best = fmaxf(best, acc[h]);
            if (__float_as_uint(best) == 0x80000000u) best = 0.0f;
            if (b0 + tid < nblk) {
                const uint32_t fb = ds[i].first_block;
                out[fb + j] = best;
                binfo[fb + j] = info_of(ds[i], j);
                bsize[fb + j] = ds[i].log2b;
            }
            x = xn; i = in; j = jn; r = rn;
        }
        return;
    }
    for (int b0 = 0; b0 < nblk; b0 += 256) {
        const int b = b0 + tid;
        const bool valid = b < nblk;
        const int i = valid ? b2s[b] : 0;
        const Desc d = ds[i];
        const int j = b - (int)(d.first_block - fb0);
        const int r = valid ? d.r : 0, l2g = d.log2g;
        const uint8_t *rec = valid ? sc + d.sc_off + (uint32_t)j * (uint32_t)vec_bytes(r, l2g, g.trunc) : sc;
        const uint32_t qoff = (s0 + i >= nxt) ? D * GP * 4 : 0;
        const bool a16 = __all(!valid || (l2g == 0 && ((uintptr_t)rec & 15u) == 0 && g.trunc == D));
        PVec<RMAX> x;
        load_pvec<RMAX, -1, true>(x, rec, rec + bm_bytes(l2g, g.trunc), wave_max_i(r), a16);
        if (g.trunc < D) mask_words(x.bw, g.trunc >> l2g);
        float acc[GP];
#pragma unroll
        for (int h = 0; h < GP; ++h) acc[h] = 0.0f;
        score_any<DT, GP, RMAX, FR>(x, r, l2g, lds_addr(qs) + qoff, acc);
        float best = acc[0];
#pragma unroll
        for (int h = 1; h < GP; ++h)
            if (h < g.G) best = fmaxf(best, acc[h]);
        if (__float_as_uint(best) == 0x80000000u) best = 0.0f;
        if (valid) {
            out[d.first_block + j] = best;
            binfo[d.first_block + j] = info_of(d, j);
            bsize[d.first_block + j] = d.log2b;
        }
    }
}

// ------------------------------------------------------------------ topk
constexpr int TOPK_BINS = 2048;
constexpr int TOPK_KPT_MAX = 32;                           // keys per thread held in registers, at most

// wave-level inclusive scans on the data-parallel-primitive lane shifts (no
// LDS round trips): shifts by 1, 2, 4, 8 inside each 16-lane row, then the
// row broadcasts of lanes 15 and 31
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_u(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xf, false);
}
// x combined with its value in lane ^ 16 or lane ^ 32, on the cross-row
// swap instructions (no LDS round trip): the swap leaves each lane holding
// its own value and its partner's
template <int X>
__device__ __forceinline__ void xor_pair(float x, float &a, float &b) {
    static_assert(X == 16 || X == 32, "row pairs or wave halves");
    const uint32_t u = __float_as_uint(x);
    if (X == 16) { const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false); a = __uint_as_float(r[0]); b = __uint_as_float(r[1]); }
    else { const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false); a = __uint_as_float(r[0]); b = __uint_as_float(r[1]); }
}
template <int X> __device__ __forceinline__ float xor_max(float x) { float a, b; xor_pair<X>(x, a, b); return fmaxf(a, b); }
template <int X> __device__ __forceinline__ float xor_sum(float x) { float a, b; xor_pair<X>(x, a, b); return a + b; }

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ uint32_t wave_scan_add(uint32_t x) {
    x += dpp_u<0x111, 0xf>(x);
    x += dpp_u<0x112, 0xf>(x);
    x += dpp_u<0x114, 0xf>(x);
    x += dpp_u<0x118, 0xf>(x);
    x += dpp_u<0x142, 0xa>(x);
    x += dpp_u<0x143, 0xc>(x);
    return x;
}
// maximum over the wave (every lane active); lanes that read out of range get 0
__device__ __forceinline__ uint32_t wave_max_u(uint32_t x) {
    x = max(x, dpp_u<0x111, 0xf>(x));
    x = max(x, dpp_u<0x112, 0xf>(x));
    x = max(x, dpp_u<0x114, 0xf>(x));
    x = max(x, dpp_u<0x118, 0xf>(x));
    x = max(x, dpp_u<0x142, 0xa>(x));
    x = max(x, dpp_u<0x143, 0xc>(x));
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// sum of s[0 .. n) for n <= 64 (wave-uniform): one read per lane, then the
// lane shifts and the last lane's total (no chain of dependent LDS reads)
__device__ __forceinline__ uint32_t sum_below(const uint32_t *s, int n) {
    const int lane = threadIdx.x & 63;
    const uint32_t x = lane < n ? s[lane] : 0u;
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_scan_add(x), 63);
}

// exclusive prefix sums over the 1024 threads of the block of N values per
// thread, and their block totals; s: 16 N words of LDS
template <int N>
__device__ __forceinline__ void block_excl_scan_1024(uint32_t (&v)[N], uint32_t (&tot)[N], uint32_t *s) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    uint32_t x[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        x[i] = wave_scan_add(v[i]);
        if (lane == 63) s[16 * i + wv] = x[i];
    }
    lds_barrier();
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const uint32_t y = wave_scan_add(lane < 16 ? s[16 * i + lane] : 0u);   // inclusive over the waves
        const uint32_t base = wv ? (uint32_t)__builtin_amdgcn_readlane((int)y, wv - 1) : 0u;
        tot[i] = (uint32_t)__builtin_amdgcn_readlane((int)y, 15);
        v[i] = base + x[i] - v[i];
    }
    lds_barrier();
}

// block-wide minimum of lo and maximum of hi (1024 threads); s: 32 words
__device__ __forceinline__ void block_minmax_1024(uint32_t &lo, uint32_t &hi, uint32_t *s) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const uint32_t l = ~wave_max_u(~lo), h = wave_max_u(hi);
    if (lane == 0) { s[wv] = l; s[16 + wv] = h; }
    lds_barrier();
    lo = s[0]; hi = s[16];
    for (int i = 1; i < 16; ++i) { lo = min(lo, s[i]); hi = max(hi, s[16 + i]); }
    lds_barrier();
}

// The bin holding the rem-th token from the top of a filled histogram hc
// (2048 bins of width 2^sh over [base, base + span]); zeroes hn for the next
// pass, narrows base / span to that bin and rem to the tokens still needed
// inside it.  True when the bins were single keys (the threshold is base).
__device__ __forceinline__ bool radix_pick(const uint32_t *hc, uint32_t *hn, uint32_t *sbuf, int sh, uint32_t &base,
                                           uint32_t &span, uint32_t &rem) {
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    // bins from the top: thread t owns bins 2047 - 2t and 2046 - 2t
    const uint32_t h0 = hc[TOPK_BINS - 1 - 2 * tid], h1 = hc[TOPK_BINS - 2 - 2 * tid];
    hn[2 * tid] = 0;
    hn[2 * tid + 1] = 0;
    const uint32_t x = wave_scan_add(h0 + h1);
    if (lane == 63) sbuf[wv] = x;
    lds_barrier();
    uint32_t above = x - (h0 + h1);
    above += sum_below(sbuf, wv);
    if (above < rem && above + h0 + h1 >= rem) {
        if (above + h0 >= rem) { sbuf[32] = TOPK_BINS - 1 - 2 * tid; sbuf[33] = rem - above; }
        else { sbuf[32] = TOPK_BINS - 2 - 2 * tid; sbuf[33] = rem - above - h0; }
    }
    lds_barrier();
    const uint32_t b = sbuf[32];
    rem = sbuf[33];
    base += b << sh;
    const uint32_t width = sh ? ((1u << sh) - 1u) : 0u;
    span = min(span - (b << sh), width);
    return sh == 0;
}

// Token-budget selection (Sec. 4.2 stage 2; Sec. 6.1 selects 10 % of tokens):
// blocks are taken in (score desc, block index asc) order while the tokens
// already taken are fewer than the budget.  The last block taken has the
// threshold key T: a radix selection over the range of the keys finds it,
// each pass histogramming the candidates' TOKENS (block sizes) into 2048 bins
// of width 2^s over the keys still in play, so at most three passes narrow
// the range to T.  Every block above T is taken; the blocks equal to T are
// taken in block order while the tokens taken among them are fewer than what
// the budget still needs (one scan of their tokens).  The selected list is
// written in ascending block order (one scan of the taken counts) together
// with each entry's record info, and the list position where each rotation
// window starts.
constexpr int TOPK_MAXW = MAX_WINDOWS;                     // rotation windows tracked in LDS

// first block of each of the first nwl rotation windows (windows past the
// last segment start at nb)
__device__ __forceinline__ void window_firsts(const Geom &g, int p, int nb, int ndesc, int nwl, int *fbw) {
    const Desc *gd = g.desc_of(p);
    for (int w = threadIdx.x; w < nwl; w += 1024) {
        const int s0 = win_first_seg(g, p, w);
        fbw[w] = (s0 < ndesc) ? (int)gd[s0].first_block : nb;
    }
}

// k and the block count after the window starts
__device__ __forceinline__ void window_tail(const Geom &g, int nb, int k, int32_t *wsel) {
    if (threadIdx.x == 0) { wsel[g.nw] = k; wsel[g.nw + 1] = nb; }
}

// Up to 1024 KPT keys (KPT = 16 or 32): thread t owns the blocks [KPT t,
// KPT t + KPT); their keys and sizes stay in registers and the taken ones are
// a KPT-bit mask.
template <int KPT>
__device__ __forceinline__ void topk_reg(const Geom &g, const WsGeom &ws, int p, int nb, int ndesc, int budget,
                                         uint32_t *hist, uint32_t *sbuf, int *fbw) {
    const int tid = threadIdx.x;
    const float *sc = ws.score + (uint64_t)p * (ws.score_stride / 4);
    const uint2 *bi = ws.binfo + (uint64_t)p * (ws.binfo_stride / 8);
    int32_t *sel = ws.sel + (uint64_t)p * (ws.sel_stride / 4);
    int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    uint2 *sinfo = ws.selinfo + (uint64_t)p * (ws.selinfo_stride / 8);
    const int i0 = min(nb, tid * KPT), i1 = min(nb, i0 + KPT), n_own = i1 - i0;
    const int nwl = min(g.nw, TOPK_MAXW);
    window_firsts(g, p, nb, ndesc, nwl, fbw);              // published by the first barrier
    const uint8_t *bz = ws.bsize + (uint64_t)p * ws.bsize_stride;
    uint32_t kr[KPT];
    uint32_t zr[KPT / 4];                             // log2 block sizes, four per word
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    {
        const float4 *s4 = (const float4 *)(sc + i0);
#pragma unroll
        for (int h = 0; h < KPT / 16; ++h) {
            const uint4 z4 = 16 * h < n_own ? *(const uint4 *)(bz + i0 + 16 * h) : make_uint4(0u, 0u, 0u, 0u);
            zr[4 * h] = z4.x; zr[4 * h + 1] = z4.y; zr[4 * h + 2] = z4.z; zr[4 * h + 3] = z4.w;
        }
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q) {
            float4 f = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (4 * q < n_own) f = s4[q];
            kr[4 * q] = score_key(f.x); kr[4 * q + 1] = score_key(f.y);
            kr[4 * q + 2] = score_key(f.z); kr[4 * q + 3] = score_key(f.w);
        }
#pragma unroll
        for (int j = 0; j < KPT; ++j)
            if (j < n_own) { kmin = min(kmin, kr[j]); kmax = max(kmax, kr[j]); }
    }
    // tokens of owned block j: 2^(log2 size)
    auto tok_reg = [&](int j) -> uint32_t { return 1u << ((zr[j >> 2] >> (8 * (j & 3))) & 7u); };
    // two histograms in turn: a pass zeroes the next one while it reads its own
    for (int i = tid; i < TOPK_BINS; i += 1024) hist[i] = 0;
    block_minmax_1024(kmin, kmax, sbuf);                          // (its barriers publish the zeros and fbw)
    uint32_t base = kmin, span = kmax - kmin;                     // candidates: [base, base + span]
    uint32_t rem = (uint32_t)budget;                               // tokens still to take
    for (int pass = 0; budget > 0; ++pass) {
        uint32_t *hc = hist + (pass & 1) * TOPK_BINS, *hn = hist + ((pass + 1) & 1) * TOPK_BINS;
        const int bits = 32 - (span ? __builtin_clz(span) : 32);
        const int sh = bits > 11 ? bits - 11 : 0;                 // (span >> sh) < 2048
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const uint32_t d = kr[j] - base;
            if (j < n_own && kr[j] >= base && d <= span) atomicAdd(&hc[d >> sh], tok_reg(j));
        }
        lds_barrier();
        if (radix_pick(hc, hn, sbuf, sh, base, span, rem)) break;
    }
    // T = base; need = tokens the budget still needs among the blocks equal to T
    const uint32_t T = base, need = rem;
    uint32_t v[1] = {0u}, tot[1];
    if (budget > 0) {                                      // this thread's tokens equal to T
#pragma unroll
        for (int j = 0; j < KPT; ++j) v[0] += (j < n_own && kr[j] == T) ? tok_reg(j) : 0u;
    }
    block_excl_scan_1024<1>(v, tot, sbuf);                 // -> equal tokens before this thread
    // taken blocks: above T, or equal to T while the equal tokens before are below need
    uint32_t tmask = 0;
    if (budget > 0) {
        uint32_t acc = v[0];
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const bool eq = j < n_own && kr[j] == T;
            const bool t = j < n_own && (kr[j] > T || (eq && acc < need));
            acc += eq ? tok_reg(j) : 0u;
            tmask |= t ? (1u << j) : 0u;
        }
    }
    v[0] = (uint32_t)__popc(tmask);
    block_excl_scan_1024<1>(v, tot, sbuf);                 // -> list position of this thread's first
    const uint32_t pos0 = v[0];
    const int k = budget > 0 ? (int)tot[0] : 0;            // blocks selected
    // the record info of the taken blocks only: all loads issued, then the stores
    uint2 br[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) br[j] = ((tmask >> j) & 1u) ? bi[i0 + j] : make_uint2(0u, 0u);
    uint32_t pos = pos0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        if ((tmask >> j) & 1u) { sel[pos] = i0 + j; sinfo[pos] = br[j]; }
        pos += (tmask >> j) & 1u;
    }
    // window starts: the position of the first block at or after each
    // start, from the owning thread's first position and taken mask
    uint32_t *tpos = hist, *tmk = hist + 1024;              // (the histograms are no longer needed)
    tpos[tid] = pos0;
    tmk[tid] = tmask;
    lds_barrier();
    for (int w = tid; w < nwl; w += 1024) {
        const int f = fbw[w];
        if (f >= nb) { wsel[w] = k; continue; }
        const int t = f / KPT, off = f % KPT;
        wsel[w] = (int)(tpos[t] + (uint32_t)__popc(tmk[t] & ((1u << off) - 1u)));
    }
    window_tail(g, nb, k, wsel);
}

// four consecutive keys and their log2 block sizes from index i (a multiple
// of 4 below nb; the lanes past nb read the rest of the arrays' slack)
struct Key4 {
    uint32_t k[4];
    uint32_t z;                                             // four log2 sizes, one per byte
    __device__ __forceinline__ uint32_t tok(int e) const { return 1u << ((z >> (8 * e)) & 7u); }
};
__device__ __forceinline__ Key4 load_key4(const float *sc, const uint8_t *bz, int i) {
    const float4 f = *(const float4 *)(sc + i);
    Key4 r;
    r.k[0] = score_key(f.x); r.k[1] = score_key(f.y); r.k[2] = score_key(f.z); r.k[3] = score_key(f.w);
    r.z = *(const uint32_t *)(bz + i);
    return r;
}

// the token budget of pair p: ceil(rho * scoreable tokens), at least one
// token (0 without scoreable blocks)
__device__ __forceinline__ int pair_budget(const Geom &g, int nb, int nf, int prov) {
    const int ntok = nf * SEG + prov * UBUF;
    if (nb <= 0 || ntok <= 0) return 0;
    const long long bb = ((long long)ntok * g.sel_num + g.sel_den - 1) / g.sel_den;
    return (int)(bb < 1 ? 1 : (bb > ntok ? ntok : bb));
}

// one workgroup per pair, for calls whose pairs hold at most 32 K blocks
// (longer ones take the multi-workgroup kernels below): 16 keys per thread
// when the pair's blocks fit, else 32
__global__ void __launch_bounds__(1024) k_topk(Geom g, WsGeom ws) {
    __shared__ uint32_t hist[2 * TOPK_BINS];
    __shared__ uint32_t sbuf[64];
    __shared__ int fbw[TOPK_MAXW];
    const int p = blockIdx.x;
    const PairMeta meta = *g.meta_of(p);
    const int nb = pair_nblocks(g, p, meta);
    int nf, prov, nbuf;
    const int ndesc = pair_ndesc(meta, nf, prov, nbuf);
    const int budget = pair_budget(g, nb, nf, prov);
    if (nb <= 1024 * 16) topk_reg<16>(g, ws, p, nb, ndesc, budget, hist, sbuf, fbw);
    else topk_reg<32>(g, ws, p, min(nb, 1024 * TOPK_KPT_MAX), ndesc, budget, hist, sbuf, fbw);
}

// ------------------------------------------------------------------ top-k over many workgroups
// Calls whose pairs can hold more than 32 K blocks: the same token-budget
// selection, spread over workgroups of TKM_CHUNK consecutive blocks of a pair
// and one kernel per phase, so that a long pair's keys are read by dozens of
// CUs instead of one.  Three radix passes of 11, 11 and 10 bits over the
// key: kernel k first takes the pick of pass k - 1 from the pair's histogram
// of that pass (every workgroup the same, workgroup 0 records the state),
// then adds its chunk's candidates' tokens to the pair's histogram of pass k
// (per-chunk LDS bins, then integer atomics: exact in any order).  After the
// last pick (threshold T, tokens still needed at T) one kernel sums the
// tokens equal to T per chunk, the next counts each chunk's taken blocks
// (blocks above T, and blocks equal to T while the equal tokens before them,
// over the chunks before and the block order inside, are below the need), and
// the last writes the list in block order and the windows' starts.  Chunk
// prefixes are sums over the chunks before (a few dozen).
// Per-pair state (WsGeom::tkx): hist[3][2048] | TkmHdr[4] | eq[nch] | tk[nch];
// the three histograms are zeroed by k_qrot earlier in the same call.
constexpr int TKM_CHUNK = 4096;                            // blocks per workgroup: 1024 threads x 4

struct TkmHdr { uint32_t base, span, rem, done; };          // radix state after each pick

__device__ __forceinline__ uint32_t *tkm_of(const WsGeom &ws, int p) { return ws.tkx + (uint64_t)p * (ws.tkx_stride / 4); }

// this workgroup's view of pair p: blocks, budget, its chunk's keys (four
// consecutive per thread) and the radix state after `npicks` picks
struct TkmCtx {
    int nb, ndesc, budget, i0, n_own;
    Key4 x;
    uint32_t *st;
    __device__ __forceinline__ bool in(int e) const { return e < n_own; }
};

__device__ __forceinline__ bool tkm_setup(const Geom &g, const WsGeom &ws, int p, int c, TkmCtx &t) {
    const PairMeta meta = *g.meta_of(p);
    int nf, prov, nbuf;
    t.ndesc = pair_ndesc(meta, nf, prov, nbuf);
    t.nb = pair_nblocks(g, p, meta);
    t.budget = pair_budget(g, t.nb, nf, prov);
    t.st = tkm_of(ws, p);
    t.i0 = c * TKM_CHUNK + 4 * (int)threadIdx.x;
    t.n_own = max(0, min(4, t.nb - t.i0));
    const float *sc = ws.score + (uint64_t)p * (ws.score_stride / 4);
    const uint8_t *bz = ws.bsize + (uint64_t)p * ws.bsize_stride;
    if (t.n_own > 0) t.x = load_key4(sc, bz, t.i0);
    else { t.x.k[0] = t.x.k[1] = t.x.k[2] = t.x.k[3] = 0u; t.x.z = 0u; }
    return c * TKM_CHUNK < t.nb;                             // the chunk holds blocks of the pair
}

// the state after pick `pass - 1` (pass >= 1) from the state before it and the
// histogram of that pass; the initial state for pass 0.  hl, hd: 2048 words
// of LDS each.
__device__ __forceinline__ TkmHdr tkm_state(const TkmCtx &t, int pass, uint32_t *hl, uint32_t *hd, uint32_t *sbuf) {
    TkmHdr h;
    if (pass == 0) {
        h.base = 0u; h.span = 0xffffffffu; h.rem = (uint32_t)max(t.budget, 0); h.done = t.budget <= 0;
        return h;
    }
    h = ((const TkmHdr *)(t.st + 3 * TOPK_BINS))[pass - 1];
    if (h.done) return h;
    for (int i = threadIdx.x; i < TOPK_BINS; i += 1024) hl[i] = t.st[(pass - 1) * TOPK_BINS + i];
    lds_barrier();
    const int bits = 32 - (h.span ? __builtin_clz(h.span) : 32);
    const int sh = bits > 11 ? bits - 11 : 0;
    h.done = radix_pick(hl, hd, sbuf, sh, h.base, h.span, h.rem) ? 1u : 0u;
    return h;
}

// grid (chunks, pairs): pass 0, 1 or 2 of the radix selection
__global__ void __launch_bounds__(1024) k_tkm_pass(Geom g, WsGeom ws, int pass) {
    __shared__ uint32_t hl[TOPK_BINS], hd[TOPK_BINS], sbuf[64];
    const int p = blockIdx.y, c = blockIdx.x, tid = threadIdx.x;
    TkmCtx t;
    const bool mine = tkm_setup(g, ws, p, c, t);
    if (!mine && c != 0) return;                            // past the pair's blocks (workgroup 0 records the state)
    const TkmHdr h = tkm_state(t, pass, hl, hd, sbuf);
    if (c == 0 && tid == 0) ((TkmHdr *)(t.st + 3 * TOPK_BINS))[pass] = h;
    if (h.done || !mine) return;
    const int bits = 32 - (h.span ? __builtin_clz(h.span) : 32);
    const int sh = bits > 11 ? bits - 11 : 0;
    lds_barrier();                                          // hl (the previous pick's bins) is reused
    for (int i = tid; i < TOPK_BINS; i += 1024) hl[i] = 0u;
    lds_barrier();
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const uint32_t key = t.x.k[e], d = key - h.base;
        if (t.in(e) && key >= h.base && d <= h.span) atomicAdd(&hl[d >> sh], t.x.tok(e));
    }
    lds_barrier();
    uint32_t *hg = t.st + pass * TOPK_BINS;
    for (int i = tid; i < TOPK_BINS; i += 1024)
        if (hl[i]) atomicAdd(&hg[i], hl[i]);
}

// tokens equal to T among the chunk's blocks, in block order: v (this
// thread's four blocks), then the exclusive prefix over the workgroup
__device__ __forceinline__ uint32_t tkm_eq4(const TkmCtx &t, uint32_t T) {
    uint32_t v = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) v += (t.in(e) && t.x.k[e] == T) ? t.x.tok(e) : 0u;
    return v;
}

// grid (chunks, pairs): the last pick (T = base, need = rem), then the tokens
// equal to T per chunk
__global__ void __launch_bounds__(1024) k_tkm_eq(Geom g, WsGeom ws, int nch) {
    __shared__ uint32_t hl[TOPK_BINS], hd[TOPK_BINS], sbuf[64];
    const int p = blockIdx.y, c = blockIdx.x, tid = threadIdx.x;
    TkmCtx t;
    const bool mine = tkm_setup(g, ws, p, c, t);
    if (!mine && c != 0) return;
    const TkmHdr h = tkm_state(t, 3, hl, hd, sbuf);
    if (c == 0 && tid == 0) ((TkmHdr *)(t.st + 3 * TOPK_BINS))[3] = h;
    if (!mine) return;
    uint32_t v[1] = {t.budget > 0 ? tkm_eq4(t, h.base) : 0u}, tot[1];
    block_excl_scan_1024<1>(v, tot, sbuf);
    if (tid == 0) t.st[3 * TOPK_BINS + 16 + c] = tot[0];
}

// the taken mask (bit e: block i0 + e) of this thread's blocks
__device__ __forceinline__ uint32_t tkm_taken(const TkmCtx &t, const TkmHdr &h, int c, uint32_t *sbuf) {
    const uint32_t *eq = t.st + 3 * TOPK_BINS + 16;
    uint32_t before = 0u;                                   // equal tokens of the chunks before
    for (int i = 0; i < c; ++i) before += eq[i];
    const uint32_t T = h.base, need = h.rem;
    uint32_t v[1] = {t.budget > 0 ? tkm_eq4(t, T) : 0u}, tot[1];
    block_excl_scan_1024<1>(v, tot, sbuf);
    uint32_t acc = before + v[0], m = 0u;
    if (t.budget > 0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t key = t.x.k[e];
            const bool eqk = t.in(e) && key == T;
            const bool tk = t.in(e) && (key > T || (eqk && acc < need));
            acc += eqk ? t.x.tok(e) : 0u;
            m |= tk ? (1u << e) : 0u;
        }
    }
    return m;
}

// grid (chunks, pairs): each chunk's taken blocks
__global__ void __launch_bounds__(1024) k_tkm_taken(Geom g, WsGeom ws, int nch) {
    __shared__ uint32_t sbuf[64];
    const int p = blockIdx.y, c = blockIdx.x, tid = threadIdx.x;
    TkmCtx t;
    if (!tkm_setup(g, ws, p, c, t)) return;
    const TkmHdr h = ((const TkmHdr *)(t.st + 3 * TOPK_BINS))[3];
    const uint32_t m = tkm_taken(t, h, c, sbuf);
    uint32_t v[1] = {(uint32_t)__popc(m)}, tot[1];
    block_excl_scan_1024<1>(v, tot, sbuf);
    if (tid == 0) t.st[3 * TOPK_BINS + 16 + nch + c] = tot[0];
}

// grid (chunks, pairs): the list entries of each chunk in block order, their
// record info, and the list position where each window starts
__global__ void __launch_bounds__(1024) k_tkm_write(Geom g, WsGeom ws, int nch) {
    __shared__ uint32_t sbuf[64], tpos[1024], tmk[1024];
    __shared__ int fbw[TOPK_MAXW];
    const int p = blockIdx.y, c = blockIdx.x, tid = threadIdx.x;
    TkmCtx t;
    const bool mine = tkm_setup(g, ws, p, c, t);
    // the record info of this thread's four blocks, loaded with the keys
    // (taken or not): it is not waited on until the list is written
    const uint2 *bi = ws.binfo + (uint64_t)p * (ws.binfo_stride / 8);
    uint2 br[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) br[e] = t.in(e) ? bi[t.i0 + e] : make_uint2(0u, 0u);
    const int nvalid = (t.nb + TKM_CHUNK - 1) / TKM_CHUNK;  // chunks holding blocks
    const uint32_t *tk = t.st + 3 * TOPK_BINS + 16 + nch;
    uint32_t before = 0u, k = 0u;
    for (int i = 0; i < nvalid; ++i) { k += tk[i]; before += i < c ? tk[i] : 0u; }
    if (t.budget <= 0) k = 0u;
    int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    const int nwl = min(g.nw, TOPK_MAXW);
    if (c == 0) window_tail(g, t.nb, (int)k, wsel);
    if (!mine && c != 0) return;
    window_firsts(g, p, t.nb, t.ndesc, nwl, fbw);
    const TkmHdr h = ((const TkmHdr *)(t.st + 3 * TOPK_BINS))[3];
    const uint32_t m = mine ? tkm_taken(t, h, c, sbuf) : 0u;
    uint32_t v[1] = {(uint32_t)__popc(m)}, tot[1];
    block_excl_scan_1024<1>(v, tot, sbuf);                  // (its barriers also publish fbw)
    const uint32_t pos0 = before + v[0];
    int32_t *sel = ws.sel + (uint64_t)p * (ws.sel_stride / 4);
    uint2 *sinfo = ws.selinfo + (uint64_t)p * (ws.selinfo_stride / 8);
    uint32_t pos = pos0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if ((m >> e) & 1u) { sel[pos] = t.i0 + e; sinfo[pos] = br[e]; }
        pos += (m >> e) & 1u;
    }
    tpos[tid] = pos0;
    tmk[tid] = m;
    lds_barrier();
    const int lo = c * TKM_CHUNK, hi = min(lo + TKM_CHUNK, t.nb);
    for (int w = tid; w < nwl; w += 1024) {
        const int f = fbw[w];
        if (f >= lo && f < hi) {
            const int o = f - lo, th = o >> 2, e0 = o & 3;
            wsel[w] = (int)(tpos[th] + (uint32_t)__popc(tmk[th] & ((1u << e0) - 1u)));
        } else if (c == 0 && (f >= t.nb || t.budget <= 0)) {
            wsel[w] = (int)k;
        }
    }
}

// ------------------------------------------------------------------ attention
// a selected block in the attention kernel's LDS table: byte offset in the
// pair's token arena, and r << 8 | log2g << 16 | log2b << 20
typedef uint2 BlkInfo;

// Split-K plan of a call.  The selected blocks of all pairs are spread over
// the attention workgroups that the device runs at once (split_slots), so
// that the attention runs as one round of workgroups: bps blocks per split,
// bps = ceil(selected blocks / slots left once every non-empty window and
// every update buffer has its rounding split), within [SPLIT_MIN,
// SPLIT_MAX].  Window w of a pair with n selected entries gets ceil(n / bps)
// splits dealt round-robin, so every split of a window holds the same mix of
// 16-, 8- and 4-token blocks (the list is in block order, where blocks of one
// size cluster); a pair's splits are its windows' in order, then one for its
// update buffer.  Every kernel that numbers splits derives the same plan from
// the top-k's window bounds.  List bounds are clamped to [0, lim] (the list's
// capacity), so that no workspace content can send an index outside it.

// f(n) for the selected entries n of each window of a pair, in window order
// (eight windows' bounds per round trip)
template <typename F>
__device__ __forceinline__ void for_windows(const int32_t *wsel, int nw, int lim, F f) {
    for (int w0 = 0; w0 < nw; w0 += 8) {
        int v[9];
#pragma unroll
        for (int i = 0; i <= 8; ++i) v[i] = wsel[min(w0 + i, nw)];
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (w0 + i < nw) {
                const int a = min(max(v[i], 0), lim), b = min(max(v[i + 1], a), lim);
                f(b - a);
            }
    }
}

// block-wide sum over blockDim.x threads (a multiple of 64); red: 16 words of LDS
__device__ __forceinline__ int block_sum(int v, int *red) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nwv = blockDim.x >> 6;
    const int x = (int)__builtin_amdgcn_readlane((int)wave_scan_add((uint32_t)v), 63);
    if (lane == 0) red[wv] = x;
    __syncthreads();
    int t = 0;
    for (int i = 0; i < nwv; ++i) t += red[i];
    __syncthreads();
    return t;
}

__device__ __forceinline__ bool pair_has_buf(const Geom &g, int p) {
    int nf, prov, nbuf;
    pair_ndesc(*g.meta_of(p), nf, prov, nbuf);
    return nbuf > 0;
}

__device__ __forceinline__ const int32_t *wsel_of(const WsGeom &ws, int p) { return ws.wsel + (uint64_t)p * (ws.wsel_stride / 4); }

// blocks per split of this call (every thread of the block gets it)
__device__ __forceinline__ int split_blocks(const Geom &g, const WsGeom &ws, int *red) {
    int ksum = 0, extra = 0;
    for (int p = threadIdx.x; p < g.npairs; p += blockDim.x) {
        const bool buf = pair_has_buf(g, p);
        for_windows(wsel_of(ws, p), g.nw, ws.max_blocks, [&](int n) { ksum += n; extra += n > 0 ? 1 : 0; });
        extra += buf ? 1 : 0;
    }
    ksum = block_sum(ksum, red);
    extra = block_sum(extra, red);
    const int avail = max(ws.split_slots - extra, max(ws.split_slots / 4, 1));
    return min(max((ksum + avail - 1) / avail, SPLIT_MIN), SPLIT_MAX);
}

// splits of pair p's windows (nbuf > 0 adds the buffer's)
__device__ __forceinline__ int pair_splits(const Geom &g, const WsGeom &ws, int p, int bps) {
    const bool buf = pair_has_buf(g, p);
    int t = 0;
    for_windows(wsel_of(ws, p), g.nw, ws.max_blocks, [&](int n) { t += (n + bps - 1) / bps; });
    return t + (buf ? 1 : 0);
}

// workgroup gidx of the flattened plan -> its pair and the split's index in
// the pair, or p = -1 past the last split; scan: 16 words of LDS
__device__ __forceinline__ void plan_locate(const Geom &g, const WsGeom &ws, int bps, int gidx, int *scan,
                                            int &p_out, int &s_out) {
    __shared__ int loc[2];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, nwv = blockDim.x >> 6;
    if (tid == 0) { loc[0] = -1; loc[1] = 0; }
    int carry = 0;
    for (int p0 = 0; p0 < g.npairs; p0 += blockDim.x) {     // block order: uniform trip count
        const int p = p0 + tid;
        const int n = p < g.npairs ? pair_splits(g, ws, p, bps) : 0;
        const uint32_t x = wave_scan_add((uint32_t)n);
        if (lane == 63) scan[wv] = (int)x;
        __syncthreads();
        int before = carry, tot = 0;
        for (int i = 0; i < nwv; ++i) { before += i < wv ? scan[i] : 0; tot += scan[i]; }
        const int first = before + (int)x - n;                 // this pair's first workgroup
        if (n > 0 && gidx >= first && gidx < first + n) { loc[0] = p; loc[1] = gidx - first; }
        carry += tot;
        __syncthreads();
    }
    p_out = loc[0];
    s_out = loc[1];
}

// split s of pair p: window w and its entries e0, e0 + stride, e0 + 2 stride,
// ... (cnt of them); w = -2 past the windows' splits (total of them)
__device__ __forceinline__ void split_of(const int32_t *wsel, int nw, int s, int lim, int bps, int &w_out, int &e0,
                                         int &stride, int &cnt, int &total) {
    int acc = 0;
    w_out = -2; e0 = 0; stride = 1; cnt = 0;
    for (int w = 0; w < nw; ++w) {
        const int a = min(max(wsel[w], 0), lim), b = min(max(wsel[w + 1], a), lim);
        const int nsp = (b - a + bps - 1) / bps;
        if (w_out == -2 && s < acc + nsp) {
            const int k = s - acc;
            w_out = w;
            e0 = a + k;
            stride = nsp;
            cnt = (b - a - k + nsp - 1) / nsp;
        }
        acc += nsp;
    }
    total = acc;
}

constexpr int CH_TOK = 64;           // tokens per chunk (one wave, lane per token)
constexpr int KT_STRIDE = 136;       // u16 per token row of the K tile (128 + 8 pad)
constexpr int VT_STRIDE = 68;        // u16 per channel row of the V tile (64 + 4 pad)
constexpr int TILE_BYTES = 17408;    // max(64 * 272, 128 * 136)
#ifndef MOSAIC_ATTN_WAVES
#define MOSAIC_ATTN_WAVES 2
#endif
constexpr int ATTN_NWV = MOSAIC_ATTN_WAVES;  // waves per attention workgroup
#ifndef MOSAIC_ATTN_WPE
#define MOSAIC_ATTN_WPE 2
#endif
#define ATTN_WPE MOSAIC_ATTN_WPE             // waves per SIMD the attention's registers allow
// block table [SPLIT_MAX] + per-wave class counts (16-byte multiple)
constexpr int ATTN_HDR_BYTES = (8 * SPLIT_MAX + ATTN_NWV * 4 * 4 + 15) / 16 * 16;
static_assert(SPLIT_MAX <= 64 * ATTN_NWV, "one setup thread per block of a split");

// x = hi + lo with hi, lo in the MFMA's 16-bit type (round to nearest even);
// hi + lo carries x to ~16 (bf16) or ~22 (fp16) significant bits
template <int DT>
__device__ __forceinline__ void split8(const float (&x)[8], typename Mma<DT>::v8 &hi, typename Mma<DT>::v8 &lo) {
    using M8 = typename Mma<DT>::v8;
    using E = typename Mma<DT>::el;
    M8 h, l;
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (E)x[i];
#pragma unroll
    for (int i = 0; i < 8; ++i) l[i] = (E)(x[i] - (float)h[i]);
    hi = h;
    lo = l;
}

// Expand a packed vector into an LDS tile at base + off: COL = false puts
// channel c at + 2c (a token-major row of the K tile), COL = true at
// + c * VT_STRIDE * 2 (a column of the channel-major V tile).  RV as in the
// score walk.
template <int RMAX, int L2G, int RV, bool COL>
__device__ __forceinline__ void scatter_walk(const PVec<RMAX> &x, int r, uint32_t addr) {
    constexpr int GS = 1 << L2G, NWD = 4 >> L2G;
    constexpr uint32_t CB = COL ? VT_STRIDE * 2 : 2;           // bytes per channel
    Walk wk = make_walk<NWD>(x.bw, addr, 32u * GS * CB);
    const int n = RV ? RV : r;
#pragma unroll
    for (int k = 0; k < (RV ? RV : RMAX) / GS; ++k) {
        if (RV || k * GS < n) {                               // wave-uniform
            const uint32_t dst = wk.a + wk.pos() * (GS * CB);
            if (!COL && GS == 1) lds_st<uint16_t>(dst, (uint16_t)half_at(x.v, k));
            else if (!COL && GS == 2) lds_st<uint32_t>(dst, x.v[k]);
            else if (!COL) lds_st<u32x2>(dst, u32x2{x.v[2 * k], x.v[2 * k + 1]});
            else {
#pragma unroll
                for (int e = 0; e < GS; ++e) lds_st<uint16_t>(dst + e * CB, (uint16_t)half_at(x.v, k * GS + e));
            }
            wk.template step<NWD>();
            __builtin_amdgcn_sched_barrier(0);       // keep the steps in order: short live ranges
        }
    }
}

template <int RMAX, int L2G, bool COL, bool FR>
__device__ __forceinline__ void scatter_r(const PVec<RMAX> &x, int r, uint32_t addr) {
    if (FR) {
        if (r == 32) scatter_walk<RMAX, L2G, 32, COL>(x, r, addr);
        else if (r == 16) scatter_walk<RMAX, L2G, 16, COL>(x, r, addr);
        else scatter_walk<RMAX, L2G, (RMAX >= 48 ? 48 : 16), COL>(x, r, addr);
    } else {
        scatter_walk<RMAX, L2G, 0, COL>(x, r, addr);
    }
}

// called by the lanes that hold a token; one pass per distinct (r, log2g)
template <int RMAX, bool COL, bool FR>
__device__ __forceinline__ void scatter_any(const PVec<RMAX> &x, int r, int l2g, uint32_t addr) {
    const int key = (r << 2) | l2g;
    uint64_t todo = __ballot(1);
    while (todo) {
        const int kv = __builtin_amdgcn_readlane(key, (int)__builtin_ctzll(todo));
        const bool mine = key == kv;
        todo &= ~__ballot(mine);
        if (mine) {
            const int rv = kv >> 2;
            if ((kv & 3) == 0) scatter_r<RMAX, 0, COL, FR>(x, rv, addr);
            else if ((kv & 3) == 1) scatter_r<RMAX, 1, COL, FR>(x, rv, addr);
            else scatter_r<RMAX, 2, COL, FR>(x, rv, addr);
        }
    }
}

// where this lane's token of a chunk lives: its block's byte offset in the
// pair's token arena and (token in block, r, log2g, log2b) packed in a word
struct TokLoc {
    uint32_t base, info;
    bool valid;
    __device__ __forceinline__ int j() const { return info & 0xff; }
    __device__ __forceinline__ int r() const { return (info >> 8) & 0xff; }
    __device__ __forceinline__ int l2g() const { return (info >> 16) & 0xf; }
    __device__ __forceinline__ int l2b() const { return info >> 20; }
};

// load the packed K (V when V_ is set) vector of a located token
template <int RMAX, int RL>
__device__ __forceinline__ void load_tok(PVec<RMAX> &x, const uint8_t *tokg, const TokLoc &L, bool V_, int rmax, int T) {
    const int r = L.r(), l2g = L.l2g(), B = 1 << L.l2b(), bmb = bm_bytes(l2g, T), j = L.j();
    const uint32_t half = V_ ? (uint32_t)(B * (bmb + 2 * r)) : 0u;
    const uint8_t *b = tokg + L.base + half;
    load_pvec<RMAX, RL ? 1 : 0, false, RL>(x, b + j * bmb, b + B * bmb + j * 2 * r, rmax, false);
}

// the same for a record with E4M3 values: r bytes of values.  RL > 0: the
// first RL / 2 16-byte granules (8 RL codes, as many values as RL granules
// of 16-bit values), at any 4-byte aligned record; else dword loads of every
// word below rmax, the others from the start of the values again.
template <int RMAX, int RL>
__device__ __forceinline__ void load_tok(PVec8<RMAX> &x, const uint8_t *tokg, const TokLoc &L, bool V_, int rmax, int T) {
    static_assert(RL % 2 == 0 && RL <= RMAX / 8, "whole 16-byte granules of codes");
    const int r = L.r(), l2g = L.l2g(), B = 1 << L.l2b(), bmb = bm_bytes(l2g, T), j = L.j();
    const uint8_t *b = tokg + L.base + (V_ ? (uint32_t)(B * (bmb + r)) : 0u);
    const uint8_t *bm = b + j * bmb, *val = b + B * bmb + j * r;
    if constexpr (RL > 0) {
        const u32x4a4 bb = *(const u32x4a4 *)bm;
        x.bw[0] = bb.x; x.bw[1] = bb.y; x.bw[2] = bb.z; x.bw[3] = bb.w;
        const u32x4a4 *v4 = (const u32x4a4 *)val;
#pragma unroll
        for (int k = 0; k < RL / 2; ++k) {
            const u32x4a4 t = v4[k];
            x.v[4 * k] = t.x; x.v[4 * k + 1] = t.y; x.v[4 * k + 2] = t.z; x.v[4 * k + 3] = t.w;
        }
    } else {
        load_dwords_any<4>(bm, x.bw);                    // a truncated bitmap can sit at any byte
        const uint32_t *v = (const uint32_t *)val;       // token values stay 4-byte aligned
#pragma unroll
        for (int k = 0; k < RMAX / 4; ++k) x.v[k] = v[(4 * k < rmax) ? k : 0];
    }
}

// walk a loaded record into the tile (widening E4M3 codes first)
template <int DT, int RMAX, int RL, bool COL, bool FR>
__device__ __forceinline__ void scatter_rec(const PVec<RMAX> &x, int r, int l2g, uint32_t addr) {
    scatter_any<RMAX, COL, FR>(x, r, l2g, addr);
}
template <int DT, int RMAX, int RL, bool COL, bool FR>
__device__ __forceinline__ void scatter_rec(const PVec8<RMAX> &c, int r, int l2g, uint32_t addr) {
    PVec<RMAX> x;
    widen<DT, RMAX, (RL > 0 ? 2 * RL : RMAX / 4)>(c, x);
    scatter_any<RMAX, COL, FR>(x, r, l2g, addr);
}

// A vector that keeps every channel (r = D, one channel per group): its
// values are the dense row in channel order, so no walk is needed.  K goes to
// the token-major row at addr with 16-byte stores, V to the channel-major
// column at addr with one 16-bit store per channel (the wave's lanes write
// consecutive columns of one row per store).  vals is 16-byte aligned.
template <bool COL>
__device__ __forceinline__ void dense_put(const uint8_t *vals, uint32_t addr) {
    const uint4 *v4 = (const uint4 *)vals;
    uint4 t[D / 8];
#pragma unroll
    for (int k = 0; k < D / 8; ++k) t[k] = v4[k];
#pragma unroll
    for (int k = 0; k < D / 8; ++k) {
        if (!COL) {
            lds_st<u32x4>(addr + (uint32_t)(16 * k), u32x4{t[k].x, t[k].y, t[k].z, t[k].w});
        } else {
            const uint32_t w[4] = {t[k].x, t[k].y, t[k].z, t[k].w};
#pragma unroll
            for (int h = 0; h < 8; ++h)
                lds_st<uint16_t>(addr + (uint32_t)((8 * k + h) * VT_STRIDE * 2),
                                 (uint16_t)((h & 1) ? (w[h >> 1] >> 16) : w[h >> 1]));
        }
    }
}

template <int DT, int GP, int RMAX, bool FR, bool F8>
__global__ void __launch_bounds__(64 * ATTN_NWV) __attribute__((amdgpu_waves_per_eu(ATTN_WPE)))
k_attn(Geom g, WsGeom ws, float scale, const uint16_t *qraw) {
    using M8 = typename Mma<DT>::v8;
    constexpr int NWV = ATTN_NWV;
    extern __shared__ __align__(16) uint8_t smem[];
    BlkInfo *blk = (BlkInfo *)smem;                         // [SPLIT_MAX], ordered 16, 8, 4
    int *wcnt = (int *)(smem + 8 * SPLIT_MAX);              // [NWV][4] blocks per size class
    uint8_t *wbase = smem + ATTN_HDR_BYTES;                 // [NWV] tiles
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, q4 = lane >> 4;
    uint8_t *tile = wbase + wave * TILE_BYTES;

    // the call's plan: workgroup b takes the b-th split of the flattened list
    // (pairs in order, each pair's splits in order); the grid covers every plan
    const int bps = split_blocks(g, ws, wcnt);
    if (blockIdx.x == 0 && tid == 0) ws.wsel[g.nw + 2] = bps;    // for the combine (pair 0's list header)
    int p, s;
    plan_locate(g, ws, bps, blockIdx.x, wcnt, p, s);
    if (p < 0 || s >= ws.max_splits) return;

    const PairMeta meta = *g.meta_of(p);
    int nf, prov, nbuf;
    pair_ndesc(meta, nf, prov, nbuf);
    const int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    int w, e0, estride, nbk, total;
    split_of(wsel, g.nw, s, ws.max_blocks, bps, w, e0, estride, nbk, total);
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

    // ---- split setup: one thread per selected block; blocks ordered by size
    // (16, then 8, then 4; ascending index inside a size), so every block
    // starts at a multiple of its size and none straddles a 64-token chunk
    bool all16;                                     // every record of the split 4-byte aligned (granule loads)
    bool dense = false;                             // every block keeps all D channels (RMAX = D kernels)
    int rsplit;                                     // largest kept count in the split
    {
        const bool on = tid < nbk;
        uint32_t goff = 0; int r = 0, l2g = 0, l2b = 2;
        if (on) {                                   // the entry's record offset and strategy (top-k wrote them)
            const uint2 si = ws.selinfo[(uint64_t)p * (ws.selinfo_stride / 8) + e0 + tid * estride];
            r = (int)((si.y >> 8) & 0xffu); l2g = (int)((si.y >> 16) & 3u); l2b = (int)min(max((si.y >> 20) & 7u, 2u), 4u);
            goff = min(si.x, (uint32_t)g.tok_size(p));     // keeps every read inside the arena
        }
        const int cls = on ? 4 - l2b : 3;
        const uint64_t m0 = __ballot(cls == 0), m1 = __ballot(cls == 1), m2 = __ballot(cls == 2);
        if (lane == 0) {
            wcnt[wave * 4 + 0] = __popcll(m0);
            wcnt[wave * 4 + 1] = __popcll(m1);
            wcnt[wave * 4 + 2] = __popcll(m2);
        }
        const int rw = wave_max_i(on ? r : 0);
        if (lane == 0) wcnt[wave * 4 + 3] = rw;
        // granule loads take a fixed 16-byte bitmap and whole 16-byte runs of
        // values at any 4-byte aligned record (what lies past a record is read
        // inside the arena's slack and never used; a walk reads D / g bits)
        all16 = __syncthreads_and(!on || ((goff & 3u) == 0 && (bm_bytes(l2g, g.trunc) & 3) == 0));
        if (RMAX >= D && !F8) dense = __syncthreads_and(!on || (l2g == 0 && r == D && (goff & 15u) == 0));
        if (on) {
            const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
            int c16 = 0, c8 = 0, before = 0;
#pragma unroll
            for (int x = 0; x < NWV; ++x) {
                c16 += wcnt[x * 4];
                c8 += wcnt[x * 4 + 1];
                before += x < wave ? wcnt[x * 4 + cls] : 0;
            }
            const int base = cls == 0 ? 0 : (cls == 1 ? c16 : c16 + c8);
            const uint64_t mc = cls == 0 ? m0 : (cls == 1 ? m1 : m2);
            const int pos = base + before + __popcll(mc & below);
            blk[pos] = make_uint2(goff, ((uint32_t)r << 8) | ((uint32_t)l2g << 16) | ((uint32_t)l2b << 20));
        }
    }
    // q operand: B[k = channel][n] of the logits K . q^T.  Column n < GP holds
    // the 16-bit high part of head n's query, column GP + n its residual, so
    // one product gives both halves of every head's logit (added across the
    // lanes afterwards): the matrix-core columns past the group are not idle.
    static_assert(2 * GP <= 16, "high and low query parts share the 16 columns");
    M8 qhl[4];
    {
        const int qw = g.rotated ? w : 0;
        const float *src = ws.qrot + (uint64_t)p * (ws.qrot_stride / 4) + (uint64_t)qw * D * GP;
        const int hq = l16 < GP ? l16 : l16 - GP;           // head of this column
        const bool live = l16 < 2 * GP && hq < G;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            float xs[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = ks * 32 + q4 * 8 + i;
                xs[i] = live ? src[c * GP + hq] : 0.0f;
            }
            M8 hi, lo;
            split8<DT>(xs, hi, lo);
            qhl[ks] = (l16 < GP) ? hi : lo;
        }
    }
    __syncthreads();
    // uniform counts (scalar registers)
    int n16 = 0, n8 = 0, n4 = 0;
    rsplit = 0;
#pragma unroll
    for (int x = 0; x < NWV; ++x) {
        n16 += wcnt[x * 4]; n8 += wcnt[x * 4 + 1]; n4 += wcnt[x * 4 + 2]; rsplit = max(rsplit, wcnt[x * 4 + 3]);
    }
    n16 = __builtin_amdgcn_readfirstlane(n16);
    n8 = __builtin_amdgcn_readfirstlane(n8);
    n4 = __builtin_amdgcn_readfirstlane(n4);
    rsplit = __builtin_amdgcn_readfirstlane(rsplit);
    const int T16 = 16 * n16, T8 = T16 + 8 * n8, T = T8 + 4 * n4;
    const int nch = (T + CH_TOK - 1) / CH_TOK;
    const uint8_t *tokg = g.tok_of(p);

    // token t of the split's ordered run -> its packed records
    auto locate = [&](int c) {
        TokLoc L;
        const int t = c * CH_TOK + lane;
        L.valid = c < nch && t < T;
        int bi, j;
        if (t < T16) { bi = t >> 4; j = t & 15; }
        else if (t < T8) { bi = n16 + ((t - T16) >> 3); j = (t - T16) & 7; }
        else { bi = n16 + n8 + ((t - T8) >> 2); j = (t - T8) & 3; }
        if (!L.valid) { bi = 0; j = 0; }
        const BlkInfo b = blk[bi];
        L.base = b.x;
        L.info = (uint32_t)j | (L.valid ? b.y : (b.y & ~0xff00u));
        return L;
    };

    float m_run = -INFINITY, l_run = 0.0f;                  // head l16
    floatx4 acc_o[8];                                       // [channel tile][head 4*q4 + r]
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) acc_o[ct] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    // the chunk loop, compiled for aligned records (a fixed number RL of 16-byte
    // value loads per vector: 4 when no kept count of the split exceeds 32) and
    // for any records (dword loads): one straight-line load form per copy keeps
    // the prefetched registers free of copies at joins, which would wait on them
    auto chunks = [&](auto rlc) {
        constexpr int RL = decltype(rlc)::value;            // < 0: dense blocks, no walk, no prefetch
        int c = wave;
        TokLoc cur = locate(c);
        using PV = std::conditional_t<F8, PVec8<RMAX>, PVec<RMAX>>;
        PV kx, vx;
        if constexpr (RL >= 0) {
            const int rm = wave_max_i(cur.r());
            __builtin_amdgcn_sched_barrier(0);
            load_tok<RMAX, RL>(kx, tokg, cur, false, rm, g.trunc);
            __builtin_amdgcn_sched_barrier(0);          // K's loads before V's, as in the loop
            load_tok<RMAX, RL>(vx, tokg, cur, true, rm, g.trunc);
            __builtin_amdgcn_sched_barrier(0);
        }
        // the tile starts zero; every MFMA operand read below zeroes what it
        // read, and the reads cover every position a scatter can write, so
        // each scatter finds the tile zero again (dense blocks overwrite the
        // rows and columns of their tokens instead; a last chunk's unused rows
        // hold finite values of earlier tokens, whose weights are zero)
        {
            uint4 *t4 = (uint4 *)tile;
            const uint4 zz = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int k = 0; k < TILE_BYTES / 16 / 64; ++k) t4[lane + k * 64] = zz;
        }
        wave_sync();
        for (; c < nch; c += NWV) {
            const int ntok = min(CH_TOK, T - c * CH_TOK);
            const TokLoc nxt = locate(c + NWV);
            const int rmn = RL >= 0 ? wave_max_i(nxt.r()) : 0;
            // ---- K: expand packed keys (token-major rows), logits on MFMA
            if constexpr (RL < 0) {
                if (cur.valid)
                    dense_put<false>(tokg + cur.base + (16 << cur.l2b()) + cur.j() * 2 * D,
                                     lds_addr(tile) + lane * (KT_STRIDE * 2));
            } else if (cur.valid) {
                if (g.trunc < D) mask_words(kx.bw, g.trunc >> cur.l2g());
                scatter_rec<DT, RMAX, RL, false, FR>(kx, cur.r(), cur.l2g(), lds_addr(tile) + lane * (KT_STRIDE * 2));
            }
            wave_sync();
            mem_fence_compiler();
            if constexpr (RL >= 0) load_tok<RMAX, RL>(kx, tokg, nxt, false, rmn, g.trunc);
            float z[4][4];
            {
                // four independent accumulators (token groups n), so no
                // product waits on the one before it
                const uint32_t tb = lds_addr(tile);
                floatx4 a4[4];
#pragma unroll
                for (int n = 0; n < 4; ++n) a4[n] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    M8 a[4];
#pragma unroll
                    for (int n = 0; n < 4; ++n) {
                        const uint32_t ad = tb + (uint32_t)(((n * 16 + l16) * KT_STRIDE + ks * 32 + q4 * 8) * 2);
                        a[n] = __builtin_bit_cast(M8, lds_ld<u32x4>(ad));
                        if (RL >= 0) lds_st<u32x4>(ad, u32x4{0u, 0u, 0u, 0u});
                    }
#pragma unroll
                    for (int n = 0; n < 4; ++n) a4[n] = Mma<DT>::run(a[n], qhl[ks], a4[n]);
                }
                // head l16 < GP: high-part logit + residual logit of column l16 + GP
#pragma unroll
                for (int n = 0; n < 4; ++n)
#pragma unroll
                    for (int r = 0; r < 4; ++r) z[n][r] = (a4[n][r] + dpp_f<0x100 + GP>(a4[n][r])) * scale;
            }
            if (ntok < CH_TOK) {                                  // the split's last chunk
#pragma unroll
                for (int n = 0; n < 4; ++n)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (n * 16 + q4 * 4 + r >= ntok) z[n][r] = -INFINITY;
            }
            // ---- online softmax for head l16 (tokens across r, n and the lane quarters)
            float cm = -INFINITY;
#pragma unroll
            for (int n = 0; n < 4; ++n)
#pragma unroll
                for (int r = 0; r < 4; ++r) cm = fmaxf(cm, z[n][r]);
            cm = xor_max<16>(cm);
            cm = xor_max<32>(cm);
            // every chunk holds a valid token, so mn is finite: exp(-inf - mn) = 0
            // covers the masked tokens and the first chunk's alpha
            const float mn = fmaxf(m_run, cm);
            const float alpha = __expf(m_run - mn);
            float ls = 0.0f;
#pragma unroll
            for (int n = 0; n < 4; ++n)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    z[n][r] = __expf(z[n][r] - mn);
                    ls += z[n][r];
                }
            ls = xor_sum<16>(ls);
            ls = xor_sum<32>(ls);
            l_run = l_run * alpha + ls;
            m_run = mn;
            // ---- V: expand packed values (channel-major rows)
            wave_sync();
            if constexpr (RL < 0) {
                if (cur.valid) {
                    const int B = 1 << cur.l2b();
                    dense_put<true>(tokg + cur.base + B * (16 + 2 * D) + 16 * B + cur.j() * 2 * D, lds_addr(tile) + lane * 2);
                }
            } else if (cur.valid) {
                if (g.trunc < D) mask_words(vx.bw, g.trunc >> cur.l2g());
                scatter_rec<DT, RMAX, RL, true, FR>(vx, cur.r(), cur.l2g(), lds_addr(tile) + lane * 2);
            }
            wave_sync();
            mem_fence_compiler();
            if constexpr (RL >= 0) load_tok<RMAX, RL>(vx, tokg, nxt, true, rmn, g.trunc);
            // ---- P . V on MFMA: A = P[head l16][tokens], B = V[tokens][channel tile]
            if (!__all(alpha == 1.0f)) {                      // some head's running max moved
                float ar[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {                  // alpha of head (q4 * 4 + r) % GP
                    const float a0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), r));
                    if (GP == 4) {
                        ar[r] = a0;
                    } else {
                        const float a1 =
                            __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), 4 + r));
                        ar[r] = (q4 & 1) ? a1 : a0;
                    }
                }
#pragma unroll
                for (int ct = 0; ct < 8; ++ct)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc_o[ct][r] *= ar[r];
            }
            const uint32_t tb = lds_addr(tile);
#pragma unroll
            for (int kv = 0; kv < 2; ++kv) {
                float xs[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) xs[i] = z[2 * kv + (i >> 2)][i & 3];
                // A rows n < GP: P's 16-bit high part for head n; rows GP + n:
                // its residual, moved over from lane n (one product for both)
                M8 ah, al;
                split8<DT>(xs, ah, al);
                u32x4 alw = __builtin_bit_cast(u32x4, al), ahw = __builtin_bit_cast(u32x4, ah);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t sh = dpp_u<0x110 + GP, 0xf>(alw[e]);
                    ahw[e] = (l16 < GP) ? ahw[e] : sh;
                }
                const M8 apl = __builtin_bit_cast(M8, ahw);
                M8 bv[8];
#pragma unroll
                for (int ct = 0; ct < 8; ++ct) {
                    const uint32_t ad = tb + (uint32_t)(((ct * 16 + l16) * VT_STRIDE + kv * 32 + q4 * 4) * 2);
                    const u32x2 v0 = lds_ld<u32x2>(ad), v1 = lds_ld<u32x2>(ad + 32);
                    if (RL >= 0) {
                        lds_st<u32x2>(ad, u32x2{0u, 0u});
                        lds_st<u32x2>(ad + 32, u32x2{0u, 0u});
                    }
                    bv[ct] = __builtin_bit_cast(M8, u32x4{v0.x, v0.y, v1.x, v1.y});
                }
#pragma unroll
                for (int ct = 0; ct < 8; ++ct) acc_o[ct] = Mma<DT>::run(apl, bv[ct], acc_o[ct]);
            }
            wave_sync();
            cur = nxt;
        }
    };
    bool done = false;
    if constexpr (RMAX >= D && !F8) {
        if (all16 && dense) { chunks(IntC<-1>{}); done = true; }
    }
    if (!done) {
        if (!all16) chunks(IntC<0>{});
        else if (RMAX > 32 && rsplit <= 32) chunks(IntC<4>{});
        else chunks(IntC<RMAX / 8>{});
    }
    // ---- merge the waves' (m, l, acc) and write the split's partial
    lds_barrier();
    float *mrg = (float *)(wbase + wave * TILE_BYTES);      // [16][D + 2]
    if (q4 == 0) { mrg[l16 * (D + 2)] = m_run; mrg[l16 * (D + 2) + 1] = l_run; }
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
        for (int r = 0; r < 4; ++r) mrg[(q4 * 4 + r) * (D + 2) + 2 + ct * 16 + l16] = acc_o[ct][r];
    lds_barrier();
    // the merged (max, sum, accumulator) of the split, in the window's rotated
    // space (the combine rotates each window's sum back once)
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
            A += (mw[h * (D + 2) + 2 + cc] + mw[(h + GP) * (D + 2) + 2 + cc]) * f;   // high + residual rows
            Ls += mw[h * (D + 2) + 1] * f;
        }
        part[2 * GP + h * D + cc] = A;
        if (cc == 0) { part[h] = Mx; part[GP + h] = Ls; }
    }
    if (tid == 0) tag[s] = w;
}

// ------------------------------------------------------------------ combine
// Two kernels.  k_combine: one workgroup per (pair p, block of 16 output
// columns j0.., window slot w), 256 threads; slot w = windows is the update
// buffer's split.  It merges the window's splits' (max, sum, accumulator) by
// log-sum-exp, rotates the merged accumulator back once with the window's R_v
// for its columns (x_j = sum_c a_c R_v[c][j]: rows j0.. of the stored R_v^T,
// 8 KB; the rotation stays merged into one vector per window, Sec. 5.3) and
// stores the window's (max, sum, columns) per head.  k_merge then merges the
// windows' results of each output by log-sum-exp.  Kernel boundaries make the
// attention's partials and the window results visible.  Blocks are ordered
// so that b % 8, the XCD a block runs on, is p % 8, as in the attention.
constexpr int CMB_THREADS = 256;

template <int GP>
__global__ void __launch_bounds__(CMB_THREADS) k_combine(Geom g, WsGeom ws, float *out) {
    constexpr int PS = GP * (D + 2);
    constexpr int NPART = CMB_THREADS / (GP * CMB_COLS);     // threads per output in the rotation
    constexpr int CPP = D / NPART;                            // channels per thread
    constexpr int NE = GP * D / CMB_THREADS;                  // merged elements per thread
    constexpr int CH = 16;                                    // splits merged per round trip
    static_assert(CMB_COLS * D / 4 == 2 * CMB_THREADS, "two 16-byte pieces of R_v^T rows per thread");
    __shared__ float am[GP][D];                               // merged accumulator of the window
    __shared__ float rv[CMB_COLS][D + 4];                     // R_v[c][j0 + jj] as rows jj
    __shared__ float sm[CH][GP], sl[CH][GP];                  // staged split maxima and sums
    __shared__ float wml[2][GP], wsc[GP];                     // the window's running max, sum, rescale
    const int np8 = (g.npairs + 7) / 8 * 8;
    const int bid = blockIdx.x, p = bid % np8, cc = (bid / np8) % CMB_NCC, w = bid / (np8 * CMB_NCC);
    if (p >= g.npairs) return;
    const int j0 = cc * CMB_COLS, tid = threadIdx.x;
    const int oi = tid / NPART, part_i = tid % NPART;         // output (head, column) and channel part
    const int oh = oi / CMB_COLS, oj = oi % CMB_COLS;
    const PairMeta meta = *g.meta_of(p);
    int nf, prov, nbuf;
    pair_ndesc(meta, nf, prov, nbuf);
    const int32_t *wsel = ws.wsel + (uint64_t)p * (ws.wsel_stride / 4);
    const float *part = ws.part + (uint64_t)p * (ws.part_stride / 4);
    const int lim = ws.max_blocks;
    // this slot's splits: the windows' splits are numbered window by window,
    // then the buffer's (the attention's numbering), s0 = those before it
    int s0 = 0, nsp = 0;
    const int bps = min(max(ws.wsel[g.nw + 2], SPLIT_MIN), SPLIT_MAX);   // the attention's plan
    for (int x = 0; x <= min(w, g.nw - 1); ++x) {
        const int a = min(max(wsel[x], 0), lim), b = min(max(wsel[x + 1], a), lim);
        const int n = (b - a + bps - 1) / bps;
        if (x < w) s0 += n; else nsp = n;
    }
    if (w == g.nw) nsp = nbuf > 0 ? 1 : 0;
    if (s0 + nsp > ws.max_splits) nsp = 0;                    // (cannot happen: the attention had this many)
    const bool rot = w < g.nw && g.rotated && nsp > 0;
    float4 rq0 = make_float4(0.0f, 0.0f, 0.0f, 0.0f), rq1 = rq0;   // R_v[c][j0 .. j0 + 15], loaded now
    if (rot) {
        const float4 *rvt = (const float4 *)(g.rot_of(p, w) + D * D + (uint64_t)j0 * D);
        rq0 = rvt[tid];
        rq1 = rvt[tid + CMB_THREADS];
    }
    float *res = ws.wres + (uint64_t)p * (ws.wres_stride / 4) + ((uint64_t)cc * (g.nw + 1) + w) * (GP * CMB_RES);
    if (nsp > 0) {
        float A[NE];
#pragma unroll
        for (int e = 0; e < NE; ++e) A[e] = 0.0f;
        for (int c0 = 0; c0 < nsp; c0 += CH) {
            const int n = min(CH, nsp - c0);
            // one round trip: this thread's accumulator elements of the n
            // splits, and the splits' maxima and sums into LDS
            float av[CH][NE];
#pragma unroll
            for (int j = 0; j < CH; ++j)
#pragma unroll
                for (int e = 0; e < NE; ++e) {
                    const int i = tid + e * CMB_THREADS;
                    av[j][e] = j < n ? part[(uint64_t)(s0 + c0 + j) * PS + 2 * GP + i] : 0.0f;
                }
            if (tid < n * GP) {
                const float *ps = part + (uint64_t)(s0 + c0 + tid / GP) * PS;
                sm[tid / GP][tid % GP] = ps[tid % GP];
                sl[tid / GP][tid % GP] = ps[GP + tid % GP];
            }
            if (c0 == 0 && tid < GP) { wml[0][tid] = -INFINITY; wml[1][tid] = 0.0f; }
            lds_barrier();
            if (tid < GP) {                                   // new running max, rescale, sum
                const float Mo = wml[0][tid];
                float Mc = Mo;
                for (int j = 0; j < n; ++j) Mc = fmaxf(Mc, sm[j][tid]);
                const float sc = (Mo == -INFINITY || Mc == -INFINITY) ? 0.0f : __expf(Mo - Mc);
                float Ls = wml[1][tid] * sc;
                for (int j = 0; j < n; ++j) Ls += sm[j][tid] == -INFINITY ? 0.0f : sl[j][tid] * __expf(sm[j][tid] - Mc);
                wml[0][tid] = Mc; wml[1][tid] = Ls; wsc[tid] = sc;
            }
            lds_barrier();
#pragma unroll
            for (int e = 0; e < NE; ++e) {
                const int h = (tid + e * CMB_THREADS) / D;
                const float Mc = wml[0][h];
                float a = A[e] * wsc[h];
#pragma unroll
                for (int j = 0; j < CH; ++j)
                    if (j < n && sm[j][h] != -INFINITY) a = fmaf(av[j][e], __expf(sm[j][h] - Mc), a);
                A[e] = a;
            }
            lds_barrier();                                    // sm / sl / wml are rewritten next
        }
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const int i = tid + e * CMB_THREADS;
            am[i / D][i % D] = A[e];
        }
        if (rot) {                                            // (rows of R_v^T: 16 x 32 pieces)
            *(float4 *)&rv[tid / (D / 4)][4 * (tid % (D / 4))] = rq0;
            *(float4 *)&rv[(tid + CMB_THREADS) / (D / 4)][4 * ((tid + CMB_THREADS) % (D / 4))] = rq1;
        }
        lds_barrier();
        float y = 0.0f;
        if (rot) {
#pragma unroll 8
            for (int c = part_i * CPP; c < (part_i + 1) * CPP; ++c) y = fmaf(am[oh][c], rv[oj][c], y);
#pragma unroll
            for (int m = 1; m < NPART; m <<= 1) y += __shfl_xor(y, m, WAVE);
        } else {
            y = am[oh][j0 + oj];
        }
        if (part_i == 0) res[oh * CMB_RES + 2 + oj] = y;
        if (tid < GP) { res[tid * CMB_RES] = wml[0][tid]; res[tid * CMB_RES + 1] = wml[1][tid]; }
    } else if (tid < GP) {                                    // an empty slot
        res[tid * CMB_RES] = -INFINITY;
        res[tid * CMB_RES + 1] = 0.0f;
    }
}

// one thread per output (pair, head, column): the log-sum-exp merge of its
// window slots' results, in slot order; the slots are read eight per round
// trip (a long context has dozens of windows)
template <int GP>
__global__ void __launch_bounds__(256) k_merge(Geom g, WsGeom ws, float *out) {
    constexpr int MU = 8;
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int p = i / (GP * D), h = (i / D) % GP, j = i % D;
    if (p >= g.npairs || h >= g.G) return;
    const int cc = j / CMB_COLS, jj = j % CMB_COLS;
    const float *r = ws.wres + (uint64_t)p * (ws.wres_stride / 4) + (uint64_t)cc * (g.nw + 1) * (GP * CMB_RES)
                     + h * CMB_RES;
    float M = -INFINITY, Lsum = 0.0f, o = 0.0f;
    for (int x0 = 0; x0 <= g.nw; x0 += MU) {
        float wm[MU], wl[MU], y[MU];
#pragma unroll
        for (int u = 0; u < MU; ++u) {
            wm[u] = -INFINITY; wl[u] = 0.0f; y[u] = 0.0f;
            if (x0 + u <= g.nw) {
                const float *rr = r + (uint64_t)(x0 + u) * (GP * CMB_RES);
                wm[u] = rr[0]; wl[u] = rr[1]; y[u] = rr[2 + jj];
            }
        }
#pragma unroll
        for (int u = 0; u < MU; ++u) {
            if (wm[u] == -INFINITY) continue;
            const float mn = fmaxf(M, wm[u]);
            const float a = __expf(M - mn), b = __expf(wm[u] - mn);    // M = -inf: a = 0
            o = o * a + y[u] * b;
            Lsum = Lsum * a + wl[u] * b;
            M = mn;
        }
    }
    out[((uint64_t)p * g.G + h) * D + j] = (Lsum > 0.0f) ? o / Lsum : 0.0f;
}

int max_keep(const Geom &g) {
    int r = g.def_keep;
    for (int i = 0; i < 3; ++i) r = max(r, g.keep_cand[i]);
    return r;
}

// attention workgroups the device holds at once: ATTN_WPE waves per SIMD,
// four SIMDs per compute unit, ATTN_NWV waves per workgroup
int attn_slots() {
    static int cached[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
    const int d = dev & 63;
    if (cached[d] == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
        cached[d] = cus * 4 * ATTN_WPE / ATTN_NWV;
    }
    return cached[d];
}

template <int DT, int GP>
hipError_t launch_decode_dt(const Geom &g, const WsGeom &w_in, const uint16_t *q, float *out, float scale,
                            int max_desc_used, int max_windows_used, hipStream_t s, hipEvent_t *ev) {
    WsGeom w = w_in;
    w.split_slots = attn_slots();
    const int nwq = g.rotated ? max_windows_used : 1;
    const bool small = max_keep(g) <= 48;
    bool fixed = true;                         // every possible kept count in {16, 32, 48}
    for (int i = 0; i < 4; ++i) {
        const int r = i < 3 ? g.keep_cand[i] : g.def_keep;
        fixed = fixed && (r == 16 || r == 32 || r == 48);
    }
    if (ev) hipEventRecord(ev[0], s);
    hipLaunchKernelGGL(k_qrot, dim3(nwq * (D / QROT_COLS), g.npairs), dim3(256), 0, s, g, w, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (ev) hipEventRecord(ev[1], s);
    if (max_desc_used > 0) {
        const int spw = max(1, min(SCORE_SEGS, (g.dyn ? g.min_win : g.W) / SEG));
        const dim3 grid(ceil_div(max_desc_used, spw), g.npairs);
        if (fixed) hipLaunchKernelGGL((k_score<DT, GP, 48, true>), grid, dim3(256), 0, s, g, w, spw);
        else if (small) hipLaunchKernelGGL((k_score<DT, GP, 48, false>), grid, dim3(256), 0, s, g, w, spw);
        else hipLaunchKernelGGL((k_score<DT, GP, 128, false>), grid, dim3(256), 0, s, g, w, spw);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (ev) hipEventRecord(ev[2], s);
    // blocks of a pair at most in this call: its segments times the most
    // blocks a segment can have
    int minb = g.def_block;
    for (int i = 0; i < 3; ++i) minb = min(minb, g.block_cand[i]);
    const long long maxb = (long long)max_desc_used * (SEG / minb);
    if (maxb > 1024 * TOPK_KPT_MAX) {
        if (!w.tkx) return hipErrorInvalidValue;               // the workspace has no multi-workgroup state
        const int nch = ceil_div(w.max_blocks, TKM_CHUNK);
        const dim3 grid(nch, g.npairs);
        for (int pass = 0; pass < 3; ++pass) {
            hipLaunchKernelGGL(k_tkm_pass, grid, dim3(1024), 0, s, g, w, pass);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        hipLaunchKernelGGL(k_tkm_eq, grid, dim3(1024), 0, s, g, w, nch);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(k_tkm_taken, grid, dim3(1024), 0, s, g, w, nch);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(k_tkm_write, grid, dim3(1024), 0, s, g, w, nch);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
        hipLaunchKernelGGL(k_topk, dim3(g.npairs), dim3(1024), 0, s, g, w);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (ev) hipEventRecord(ev[3], s);
    {
        // the plan has at most max(slots, selected blocks / SPLIT_MAX) splits
        // of whole blocks plus one rounding split per window and per buffer,
        // and never more than every pair's whole partial array
        const size_t smem = ATTN_HDR_BYTES + (size_t)ATTN_NWV * TILE_BYTES;
        const long long extra = (long long)g.npairs * (g.nw + 1);
        const long long whole = std::max<long long>(w.split_slots, (long long)g.npairs * ceil_div(w.max_sel, SPLIT_MAX));
        const long long nwg = std::min<long long>(whole + extra, (long long)g.npairs * w.max_splits);
        const dim3 grid((unsigned)nwg), block(64 * ATTN_NWV);
        if (g.fp8) {
            if (fixed) hipLaunchKernelGGL((k_attn<DT, GP, 48, true, true>), grid, block, smem, s, g, w, scale, q);
            else if (small) hipLaunchKernelGGL((k_attn<DT, GP, 48, false, true>), grid, block, smem, s, g, w, scale, q);
            else hipLaunchKernelGGL((k_attn<DT, GP, 128, false, true>), grid, block, smem, s, g, w, scale, q);
        } else {
            if (fixed) hipLaunchKernelGGL((k_attn<DT, GP, 48, true, false>), grid, block, smem, s, g, w, scale, q);
            else if (small) hipLaunchKernelGGL((k_attn<DT, GP, 48, false, false>), grid, block, smem, s, g, w, scale, q);
            else hipLaunchKernelGGL((k_attn<DT, GP, 128, false, false>), grid, block, smem, s, g, w, scale, q);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (ev) hipEventRecord(ev[4], s);
    hipLaunchKernelGGL(k_combine<GP>, dim3((g.npairs + 7) / 8 * 8 * CMB_NCC * (g.nw + 1)), dim3(CMB_THREADS), 0, s,
                       g, w, out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_merge<GP>, dim3(ceil_div(g.npairs * GP * D, 256)), dim3(256), 0, s, g, w, out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev) hipEventRecord(ev[5], s);
    return hipSuccess;
}

}  // namespace

hipError_t launch_decode(const Geom &g, const WsGeom &w, const uint16_t *q, float *out, float scale,
                         int max_desc_used, int max_windows_used, hipStream_t s, hipEvent_t *ev) {
    if (g.dtype) {
        if (g.GP == 4) return launch_decode_dt<1, 4>(g, w, q, out, scale, max_desc_used, max_windows_used, s, ev);
        return launch_decode_dt<1, 8>(g, w, q, out, scale, max_desc_used, max_windows_used, s, ev);
    }
    if (g.GP == 4) return launch_decode_dt<0, 4>(g, w, q, out, scale, max_desc_used, max_windows_used, s, ev);
    return launch_decode_dt<0, 8>(g, w, q, out, scale, max_desc_used, max_windows_used, s, ev);
}

}  // namespace mosaic
