// api.hip -- C ABI of libmosaic (see include/mosaic.h): argument validation,
// host-side bookkeeping of sequence lengths (the paper's CPU-side management
// of Sec. 5.4, reduced to deciding which kernels run), arena and workspace
// layout, and kernel launches.  No C++ exception crosses the ABI.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/mosaic.h"
#include "mosaic_internal.h"

using namespace mosaic;

namespace {

thread_local std::string g_err;

mosaic_status fail(mosaic_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

mosaic_status ok() {
    g_err.clear();
    return MOSAIC_OK;
}

mosaic_status hip_fail(hipError_t e, const char *what) {
    return fail(MOSAIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }
// window rotations: int32 [pairs] flags, then fp32 [pairs][K, V][D][D]
size_t window_rot_ws_bytes(int npairs) { return align256((uint64_t)npairs * 4) + (size_t)npairs * 2 * D * D * 4; }
int ilog2(int v) { int l = 0; while ((1 << l) < v) ++l; return l; }

}  // namespace

struct mosaic_cache {
    mosaic_params P;
    int num_seqs, max_tokens, rotated, npairs, GP, nw, max_desc, max_blocks, max_sel, max_splits;
    int maxrec, minb;
    uint32_t slot_tok, slot_sc;  // single-pass compression: worst-case bytes of a segment's records
    mosaic_layout lay;
    mosaic_ws_layout wsl;
    uint64_t ctx_off;            // device int32 [num_seqs] (inside the arena)
    uint8_t *arena;
    bool compressed;
    bool timing = false, timed_once = false;
    hipEvent_t ev[6] = {};
    std::vector<int32_t> L;      // host mirror of each sequence's length
    // dynamic windows: nw_src = rotations per pair mosaic_compress receives;
    // poll_due = a segment completed since the last poll (a window may have
    // closed); per pair the windows in use, the window awaiting its rotation
    // and that window's token count, as of the last poll
    bool dyn = false, poll_due = false;
    int nw_src = 1;
    std::vector<int32_t> nwin, pend, pend_len;
    // capacities: per sequence; with ragged capacities the desc, score and
    // token regions of a pair are sized for its sequence and located by the
    // pair table [npairs][4] (offsets from each region's start, token bytes)
    std::vector<int32_t> cap;
    bool ragged = false;
    std::vector<uint64_t> pairs;
    Geom geom() const {
        Geom g{};
        g.npairs = npairs; g.hkv = P.num_kv_heads; g.G = P.group_size; g.GP = GP; g.dtype = P.dtype;
        g.W = P.rot_window; g.nw = nw; g.cap = max_tokens; g.max_desc = max_desc; g.rotated = rotated;
        g.meta = arena + lay.meta_off; g.desc = arena + lay.desc_off; g.sc = arena + lay.score_off;
        g.tok = arena + lay.token_off; g.buf = (uint16_t *)(arena + lay.buf_off);
        g.stg = (uint16_t *)(arena + lay.stage_off); g.rot = (float *)(arena + lay.rot_off);
        g.meta_stride = lay.meta_stride; g.desc_stride = lay.desc_stride; g.sc_stride = lay.score_stride;
        g.tok_stride = lay.token_stride; g.buf_stride = lay.buf_stride; g.stg_stride = lay.stage_stride;
        g.rot_stride = lay.rot_stride;
        g.cov = (double *)(arena + lay.cov_off); g.cov_stride = lay.cov_stride;
        g.poff = (const uint64_t *)(arena + lay.pairs_off);
        for (int i = 0; i < 3; ++i) {
            g.keep_cand[i] = P.keep_cand[i]; g.group_cand[i] = P.group_cand[i]; g.block_cand[i] = P.block_cand[i];
        }
        g.def_keep = P.default_keep; g.def_group = P.default_group; g.def_block = P.default_block;
        g.tau_ch = P.tau_channel; g.tau_blk = P.tau_block;
        g.sel_num = P.select_num; g.sel_den = P.select_den; g.force = P.force_default_strategy;
        g.trunc = P.trunc_channels;
        g.fp8 = P.value_fp8;
        g.dyn = dyn ? 1 : 0; g.min_win = P.min_window; g.tau_win = P.tau_window;
        return g;
    }
    WsGeom wsgeom(void *ws) const {
        uint8_t *b = (uint8_t *)ws;
        WsGeom w{};
        w.qrot = (float *)(b + wsl.qrot_off); w.qrot_stride = wsl.qrot_stride;
        w.score = (float *)(b + wsl.score_off); w.score_stride = wsl.score_stride;
        w.sel = (int32_t *)(b + wsl.sel_off); w.sel_stride = wsl.sel_stride;
        w.wsel = (int32_t *)(b + wsl.wsel_off); w.wsel_stride = wsl.wsel_stride;
        w.part = (float *)(b + wsl.part_off); w.part_stride = wsl.part_stride;
        w.tag = (int32_t *)(b + wsl.tag_off); w.tag_stride = wsl.tag_stride;
        w.binfo = (uint2 *)(b + wsl.binfo_off); w.binfo_stride = wsl.binfo_stride;
        w.bsize = b + wsl.bsize_off; w.bsize_stride = wsl.bsize_stride;
        w.selinfo = (uint2 *)(b + wsl.selinfo_off); w.selinfo_stride = wsl.selinfo_stride;
        w.wres = (float *)(b + wsl.wres_off); w.wres_stride = wsl.wres_stride;
        w.tkx = wsl.tkx_stride ? (uint32_t *)(b + wsl.tkx_off) : nullptr; w.tkx_stride = wsl.tkx_stride;
        w.max_blocks = max_blocks; w.max_splits = max_splits; w.max_sel = max_sel;
        return w;
    }
};

// Fixed decode workspace of mosaic_decode_attention_noalloc: one copy per GPU,
// reserved when the library's code object is loaded on that GPU and held
// until the process ends.  Host code uses only the device address that
// hipGetSymbolAddress returns for the current GPU (the array's name is a
// host-side stand-in); nothing in it needs to start at zero, because every
// region of the decode workspace is written before it is read within a call.
static __device__ __align__(256) uint8_t scratch[MOSAIC_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};

// the address of this GPU's scratch array (resolved once per device, with
// that device current)
mosaic_status scratch_of_current_device(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= MAX_DEVICES) return fail(MOSAIC_ERR_UNSUPPORTED, "device %d beyond %d devices", dev, MAX_DEVICES);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "scratch address");
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return MOSAIC_OK;
}
}  // namespace

extern "C" {

void mosaic_params_default(mosaic_params *p) {
    if (!p) return;
    std::memset(p, 0, sizeof(*p));
    p->head_dim = 128; p->num_kv_heads = 8; p->group_size = 4; p->dtype = MOSAIC_FP16;
    p->seg_len = 64; p->rot_window = 65536; p->update_buf = 32;
    p->keep_cand[0] = 16; p->keep_cand[1] = 32; p->keep_cand[2] = 48;
    p->group_cand[0] = 4; p->group_cand[1] = 2; p->group_cand[2] = 1;
    p->block_cand[0] = 16; p->block_cand[1] = 8; p->block_cand[2] = 4;
    p->default_keep = 32; p->default_group = 1; p->default_block = 8;
    p->tau_channel = 0.30f; p->tau_block = 0.90f;
    p->select_num = 1; p->select_den = 10;
    p->force_default_strategy = 0;
    p->trunc_channels = 128;
    p->value_fp8 = 0;
    p->dyn_windows = 0;
    p->tau_window = 8.0f;
    p->min_window = 1024;
}

static mosaic_status check_params(const mosaic_params *p) {
    if (p->head_dim != 128) return fail(MOSAIC_ERR_UNSUPPORTED, "head_dim %d: only 128 is supported", p->head_dim);
    if (p->seg_len != SEG) return fail(MOSAIC_ERR_UNSUPPORTED, "seg_len %d: only 64 is supported", p->seg_len);
    if (p->update_buf != UBUF) return fail(MOSAIC_ERR_UNSUPPORTED, "update_buf %d: only 32 is supported", p->update_buf);
    if (p->num_kv_heads < 1) return fail(MOSAIC_ERR_INVALID, "num_kv_heads %d < 1", p->num_kv_heads);
    if (p->group_size < 1 || p->group_size > 8) return fail(MOSAIC_ERR_INVALID, "group_size %d not in 1..8", p->group_size);
    if (p->dtype != MOSAIC_FP16 && p->dtype != MOSAIC_BF16) return fail(MOSAIC_ERR_INVALID, "dtype %d", p->dtype);
    if (p->rot_window < SEG || p->rot_window % SEG) return fail(MOSAIC_ERR_INVALID, "rot_window %d: multiple of 64 required", p->rot_window);
    auto okg = [](int g) { return g == 1 || g == 2 || g == 4; };
    auto okb = [](int b) { return b == 4 || b == 8 || b == 16; };
    auto okr = [](int r, int g) { return r >= 2 && r <= 128 && r % g == 0 && r % 2 == 0; };
    for (int i = 0; i < 3; ++i) {
        if (!okg(p->group_cand[i])) return fail(MOSAIC_ERR_INVALID, "group_cand[%d] = %d not in {1,2,4}", i, p->group_cand[i]);
        if (!okb(p->block_cand[i])) return fail(MOSAIC_ERR_INVALID, "block_cand[%d] = %d not in {4,8,16}", i, p->block_cand[i]);
    }
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j)
            if (!okr(p->keep_cand[i], p->group_cand[j]))
                return fail(MOSAIC_ERR_INVALID, "keep_cand[%d] = %d: even, 2..128 and a multiple of every group size",
                            i, p->keep_cand[i]);
    if (!okg(p->default_group) || !okb(p->default_block) || !okr(p->default_keep, p->default_group))
        return fail(MOSAIC_ERR_INVALID, "default strategy (%d, %d, %d) invalid", p->default_keep, p->default_group,
                    p->default_block);
    if (std::isnan(p->tau_channel) || std::isnan(p->tau_block) || p->tau_channel < 0 || p->tau_block < 0)
        return fail(MOSAIC_ERR_INVALID, "thresholds must be >= 0");
    if (p->select_num < 1 || p->select_den < 1) return fail(MOSAIC_ERR_INVALID, "select ratio %d/%d", p->select_num, p->select_den);
    const int T = p->trunc_channels;
    if (T < 32 || T > 128 || T % 32) return fail(MOSAIC_ERR_INVALID, "trunc_channels %d: 32, 64, 96 or 128", T);
    for (int i = 0; i < 3; ++i)
        if (p->keep_cand[i] > T) return fail(MOSAIC_ERR_INVALID, "keep_cand[%d] = %d > trunc_channels %d", i, p->keep_cand[i], T);
    if (p->default_keep > T) return fail(MOSAIC_ERR_INVALID, "default_keep %d > trunc_channels %d", p->default_keep, T);
    if (p->value_fp8 != 0 && p->value_fp8 != 1) return fail(MOSAIC_ERR_INVALID, "value_fp8 %d: 0 or 1", p->value_fp8);
    if (p->value_fp8) {                     // one-byte values: records stay 4-byte aligned
        for (int i = 0; i < 3; ++i)
            if (p->keep_cand[i] % 4)
                return fail(MOSAIC_ERR_INVALID, "keep_cand[%d] = %d: a multiple of 4 with value_fp8", i, p->keep_cand[i]);
        if (p->default_keep % 4) return fail(MOSAIC_ERR_INVALID, "default_keep %d: a multiple of 4 with value_fp8", p->default_keep);
    }
    if (p->dyn_windows != 0 && p->dyn_windows != 1) return fail(MOSAIC_ERR_INVALID, "dyn_windows %d: 0 or 1", p->dyn_windows);
    if (p->dyn_windows) {
        if (!std::isfinite(p->tau_window) || p->tau_window < 0)
            return fail(MOSAIC_ERR_INVALID, "tau_window must be finite and >= 0");
        if (p->min_window < SEG || p->min_window % SEG || p->min_window > p->rot_window)
            return fail(MOSAIC_ERR_INVALID, "min_window %d: a multiple of 64 in [64, rot_window]", p->min_window);
    }
    return MOSAIC_OK;
}

static mosaic_status cache_create(const mosaic_params *params, int32_t num_seqs, const int32_t *caps, bool ragged,
                                  int32_t rotated, mosaic_cache **out) {
    mosaic_status st = check_params(params);
    if (st != MOSAIC_OK) return st;
    int max_tokens = 0;
    for (int q = 0; q < num_seqs; ++q) {
        if (caps[q] < 1) return fail(MOSAIC_ERR_INVALID, "max_tokens[%d] = %d < 1", q, caps[q]);
        max_tokens = std::max(max_tokens, caps[q]);
    }
    mosaic_cache *c = new (std::nothrow) mosaic_cache();
    if (!c) return fail(MOSAIC_ERR_INVALID, "out of host memory");
    c->P = *params;
    c->num_seqs = num_seqs; c->max_tokens = max_tokens; c->rotated = rotated ? 1 : 0;
    c->cap.assign(caps, caps + num_seqs);
    c->ragged = ragged;
    c->npairs = num_seqs * params->num_kv_heads;
    c->GP = params->group_size <= 4 ? 4 : 8;
    c->nw = (max_tokens + params->rot_window - 1) / params->rot_window;
    c->nw_src = c->nw;
    c->dyn = params->dyn_windows != 0;
    if (c->dyn) {
        if (!c->rotated) {
            delete c;
            return fail(MOSAIC_ERR_INVALID, "dynamic windows need rotations (rotated = 1)");
        }
        // every closed window holds at least min_window tokens; one is open
        c->nw = std::max(c->nw, max_tokens / params->min_window + 1);
    }
    if (c->nw > MAX_WINDOWS) {
        const int nw = c->nw;
        delete c;
        return fail(MOSAIC_ERR_UNSUPPORTED, "%d rotation windows per sequence (at most %d)", nw, MAX_WINDOWS);
    }
    c->max_desc = max_tokens / SEG + 2;
    int maxrec = 0, maxtok = 0, minb = params->default_block;
    const int eb = params->value_fp8 ? 1 : 2;          // bytes per value of a token record
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j) {
            maxrec = std::max(maxrec, 2 * params->keep_cand[i] + 16 / params->group_cand[j]);
            maxtok = std::max(maxtok, eb * params->keep_cand[i] + 16 / params->group_cand[j]);
        }
    maxrec = std::max(maxrec, 2 * params->default_keep + 16 / params->default_group);
    maxtok = std::max(maxtok, eb * params->default_keep + 16 / params->default_group);
    for (int i = 0; i < 3; ++i) minb = std::min(minb, params->block_cand[i]);
    c->maxrec = maxrec; c->minb = minb;
    c->slot_tok = (uint32_t)(SEG * 2 * maxtok + 15) / 16 * 16;
    c->slot_sc = (uint32_t)((SEG / minb) * maxrec + 15) / 16 * 16;
    // + 256: the decode kernels read whole 16-byte bitmaps and up to 2 * 128 bytes
    // of values past a vector (never used), which must stay inside the arena
    const uint64_t tok_bytes = (uint64_t)c->max_desc * SEG * 2 * maxtok + 256;
    const uint64_t sc_bytes = (uint64_t)c->max_desc * (SEG / minb) * maxrec + 256;
    if (tok_bytes >= (1ull << 32)) {
        delete c;
        return fail(MOSAIC_ERR_CAPACITY, "max_tokens %d: a pair's token arena would exceed 4 GiB", max_tokens);
    }
    c->max_blocks = c->max_desc * (SEG / minb);
    // the selection takes blocks until ceil(rho * scoreable tokens) tokens: at
    // most ceil(budget / smallest block) of them
    const int64_t max_budget = ((int64_t)c->max_desc * SEG * params->select_num + params->select_den - 1) /
                               params->select_den;
    c->max_sel = (int)std::min<int64_t>(c->max_blocks, (max_budget + minb - 1) / minb + 1);
    c->max_splits = (c->max_sel + SPLIT_MIN - 1) / SPLIT_MIN + c->nw + 1;
    // arena layout
    mosaic_layout &l = c->lay;
    std::memset(&l, 0, sizeof(l));
    uint64_t off = 0;
    auto region = [&](uint64_t &o, uint64_t &stride, uint64_t per_pair) {
        stride = align256(per_pair);
        o = off;
        off = align256(off + stride * (uint64_t)c->npairs);
    };
    // meta: the counters, then (dynamic windows) the window table
    region(l.meta_off, l.meta_stride, sizeof(PairMeta) + (c->dyn ? (uint64_t)(c->nw + 1) * 4 : 0));
    c->pairs.assign((size_t)c->npairs * 4, 0);
    if (!ragged) {
        region(l.desc_off, l.desc_stride, (uint64_t)c->max_desc * sizeof(Desc));
        region(l.score_off, l.score_stride, sc_bytes);
        region(l.token_off, l.token_stride, tok_bytes);
        for (int p = 0; p < c->npairs; ++p) {
            c->pairs[4 * p] = p * l.desc_stride; c->pairs[4 * p + 1] = p * l.score_stride;
            c->pairs[4 * p + 2] = p * l.token_stride; c->pairs[4 * p + 3] = l.token_stride;
        }
    } else {
        // each pair's regions sized for its own sequence, pair after pair
        uint64_t *dst_off[3] = {&l.desc_off, &l.score_off, &l.token_off};
        for (int r = 0; r < 3; ++r) {
            *dst_off[r] = off;
            uint64_t o = 0;
            for (int p = 0; p < c->npairs; ++p) {
                const uint64_t nd = (uint64_t)c->cap[p / params->num_kv_heads] / SEG + 2;
                const uint64_t bytes = r == 0 ? nd * sizeof(Desc)
                                     : r == 1 ? nd * (SEG / minb) * maxrec + 256 : nd * SEG * 2 * maxtok + 256;
                c->pairs[4 * p + r] = o;
                if (r == 2) c->pairs[4 * p + 3] = align256(bytes);
                o += align256(bytes);
            }
            off = align256(off + o);
        }
        l.desc_stride = l.score_stride = l.token_stride = 0;
    }
    region(l.buf_off, l.buf_stride, 2ull * UBUF * D * 2);
    region(l.stage_off, l.stage_stride, 2ull * SEG * D * 2);
    region(l.rot_off, l.rot_stride, c->rotated ? (uint64_t)c->nw * 3 * D * D * 4 : 0);
    if (c->dyn) region(l.cov_off, l.cov_stride, 4ull * D * D * 8);
    l.pairs_off = off;
    off = align256(off + (uint64_t)c->npairs * 4 * sizeof(uint64_t));
    c->ctx_off = off;
    off = align256(off + (uint64_t)num_seqs * 4);
    l.total = off;
    l.num_pairs = c->npairs; l.max_desc = c->max_desc; l.num_windows = c->nw;
    // decode workspace layout
    mosaic_ws_layout &w = c->wsl;
    std::memset(&w, 0, sizeof(w));
    off = 0;
    auto wregion = [&](uint64_t &o, uint64_t &stride, uint64_t per_pair) {
        stride = align256(per_pair);
        o = off;
        off = align256(off + stride * (uint64_t)c->npairs);
    };
    wregion(w.qrot_off, w.qrot_stride, (uint64_t)c->nw * D * c->GP * 4);
    wregion(w.score_off, w.score_stride, (uint64_t)c->max_blocks * 4);
    wregion(w.sel_off, w.sel_stride, (uint64_t)c->max_blocks * 4);
    // wsel: window starts in the selected list, k, block count (pair 0: and
    // the call's blocks per split)
    wregion(w.wsel_off, w.wsel_stride, (uint64_t)(c->nw + 3) * 4);
    // part: split partials (max, sum, unrotated accumulator per head)
    wregion(w.part_off, w.part_stride, (uint64_t)c->max_splits * c->GP * (D + 2) * 4);
    wregion(w.tag_off, w.tag_stride, (uint64_t)c->max_splits * 4);
    wregion(w.binfo_off, w.binfo_stride, (uint64_t)c->max_blocks * 8);
    wregion(w.bsize_off, w.bsize_stride, (uint64_t)c->max_blocks);
    wregion(w.selinfo_off, w.selinfo_stride, (uint64_t)c->max_blocks * 8);
    // wres: each window's merged, back-rotated result per column block
    wregion(w.wres_off, w.wres_stride, (uint64_t)CMB_NCC * (c->nw + 1) * c->GP * CMB_RES * 4);
    // pairs of more than 32 K blocks: the multi-workgroup top-k's histograms,
    // radix states and per-chunk counts (chunks of 4096 blocks)
    if (c->max_blocks > 32768) {
        const uint64_t nch = ((uint64_t)c->max_blocks + 4095) / 4096;
        wregion(w.tkx_off, w.tkx_stride, (3ull * 2048 + 16 + 2 * nch) * 4);
    }
    w.total = off + 256;                     // whole 16-byte loads of the last pair's arrays stay inside
    w.max_blocks = c->max_blocks; w.max_splits = c->max_splits; w.gp = c->GP;
    c->arena = nullptr;
    c->compressed = false;
    c->L.assign(num_seqs, 0);
    c->nwin.assign(c->npairs, 1);
    c->pend.assign(c->npairs, -1);
    c->pend_len.assign(c->npairs, 0);
    *out = c;
    return ok();
}

mosaic_status mosaic_cache_create(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                  int32_t rotated, mosaic_cache **out) {
    if (!params || !out) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (num_seqs < 1 || max_tokens < 1) return fail(MOSAIC_ERR_INVALID, "num_seqs %d, max_tokens %d", num_seqs, max_tokens);
    const std::vector<int32_t> caps((size_t)num_seqs, max_tokens);
    return cache_create(params, num_seqs, caps.data(), false, rotated, out);
}

mosaic_status mosaic_cache_create_ragged(const mosaic_params *params, int32_t num_seqs,
                                         const int32_t *max_tokens_host, int32_t rotated, mosaic_cache **out) {
    if (!params || !out || !max_tokens_host) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (num_seqs < 1) return fail(MOSAIC_ERR_INVALID, "num_seqs %d", num_seqs);
    return cache_create(params, num_seqs, max_tokens_host, true, rotated, out);
}

mosaic_status mosaic_cache_pair_regions(const mosaic_cache *c, uint64_t *out_host) {
    if (!c || !out_host) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    std::memcpy(out_host, c->pairs.data(), c->pairs.size() * sizeof(uint64_t));
    return ok();
}

mosaic_status mosaic_cache_arena_bytes(const mosaic_cache *c, size_t *bytes) {
    if (!c || !bytes) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    *bytes = c->lay.total;
    return ok();
}

mosaic_status mosaic_cache_bind(mosaic_cache *c, void *arena, size_t bytes) {
    if (!c || !arena) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if ((uintptr_t)arena % 256) return fail(MOSAIC_ERR_INVALID, "arena not 256-byte aligned");
    if (bytes < c->lay.total) return fail(MOSAIC_ERR_INVALID, "arena %zu bytes < %llu required", bytes,
                                          (unsigned long long)c->lay.total);
    c->arena = (uint8_t *)arena;
    c->compressed = false;
    return ok();
}

mosaic_status mosaic_cache_destroy(mosaic_cache *c) {
    if (c && c->ev[0])
        for (auto &e : c->ev) hipEventDestroy(e);
    delete c;
    return ok();
}

mosaic_status mosaic_cache_layout(const mosaic_cache *c, mosaic_layout *out) {
    if (!c || !out) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    *out = c->lay;
    return ok();
}

mosaic_status mosaic_decode_ws_layout(const mosaic_cache *c, mosaic_ws_layout *out) {
    if (!c || !out) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    *out = c->wsl;
    return ok();
}

mosaic_status mosaic_workspace_bytes(const mosaic_cache *c, int32_t op, size_t *bytes) {
    if (!c || !bytes) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (op == MOSAIC_OP_COMPRESS) *bytes = (size_t)c->npairs * c->max_desc * ((size_t)c->slot_tok + c->slot_sc);
    else if (op == MOSAIC_OP_APPEND) *bytes = 0;
    else if (op == MOSAIC_OP_DECODE) *bytes = c->wsl.total;
    else if (op == MOSAIC_OP_WINDOW_ROTATIONS) *bytes = c->dyn ? window_rot_ws_bytes(c->npairs) : 0;
    else return fail(MOSAIC_ERR_INVALID, "unknown op %d", op);
    return ok();
}

int32_t mosaic_seq_tokens(const mosaic_cache *c, int32_t seq) {
    if (!c || seq < 0 || seq >= c->num_seqs) return -1;
    return c->L[seq];
}

mosaic_status mosaic_compress(mosaic_cache *c, const void *k, const void *v, int64_t seq_stride,
                              const int32_t *ctx_lens_host, const float *rot_k, const float *rot_v, void *ws,
                              size_t ws_bytes, void *stream) {
    if (!c) return fail(MOSAIC_ERR_INVALID, "NULL cache");
    if (!c->arena) return fail(MOSAIC_ERR_STATE, "cache not bound to an arena");
    if (!k || !v || !ctx_lens_host) return fail(MOSAIC_ERR_INVALID, "NULL k, v or ctx_lens_host");
    if (((uintptr_t)k | (uintptr_t)v) % 16) return fail(MOSAIC_ERR_INVALID, "k/v must be 16-byte aligned");
    if (c->rotated && (!rot_k || !rot_v)) return fail(MOSAIC_ERR_INVALID, "cache is rotated: rot_k and rot_v required");
    if (!c->rotated && (rot_k || rot_v)) return fail(MOSAIC_ERR_INVALID, "cache created without rotation");
    if (c->rotated && (((uintptr_t)rot_k | (uintptr_t)rot_v) % 16)) return fail(MOSAIC_ERR_INVALID, "rot must be 16-byte aligned");
    int maxL = 0, any_tail = 0;
    for (int s = 0; s < c->num_seqs; ++s) {
        const int L = ctx_lens_host[s];
        if (L < 0) return fail(MOSAIC_ERR_INVALID, "ctx_lens[%d] = %d < 0", s, L);
        if (L > c->cap[s]) return fail(MOSAIC_ERR_CAPACITY, "ctx_lens[%d] = %d > max_tokens %d", s, L, c->cap[s]);
        maxL = std::max(maxL, L);
        any_tail |= (L % SEG) != 0;
    }
    if (seq_stride < maxL || seq_stride < 1) return fail(MOSAIC_ERR_INVALID, "seq_stride %lld < longest context %d",
                                                         (long long)seq_stride, maxL);
    if (ws) {
        const size_t need = (size_t)c->npairs * c->max_desc * ((size_t)c->slot_tok + c->slot_sc);
        if (ws_bytes < need) return fail(MOSAIC_ERR_INVALID, "compress workspace %zu bytes < %zu required", ws_bytes, need);
        if ((uintptr_t)ws % 16) return fail(MOSAIC_ERR_INVALID, "compress workspace not 16-byte aligned");
    }
    hipStream_t s = (hipStream_t)stream;
    const Geom g = c->geom();
    int32_t *ctx_dev = (int32_t *)(c->arena + c->ctx_off);
    hipError_t e = launch_ctx_copy(ctx_dev, ctx_lens_host, c->num_seqs, s);
    if (e != hipSuccess) return hip_fail(e, "copy of context lengths");
    if ((e = launch_pairs_copy((uint64_t *)(c->arena + c->lay.pairs_off), c->pairs.data(), c->npairs, s)) != hipSuccess)
        return hip_fail(e, "copy of the pair table");
    if (c->rotated && (e = launch_copy_rot(g, rot_k, rot_v, c->nw_src, s)) != hipSuccess) return hip_fail(e, "rotation copy");
    e = launch_compress(g, (const uint16_t *)k, (const uint16_t *)v, seq_stride, ctx_dev, maxL / SEG, any_tail,
                        (uint8_t *)ws, c->slot_tok, c->slot_sc, s);
    if (e != hipSuccess) return hip_fail(e, "compress launch");
    for (int q = 0; q < c->num_seqs; ++q) c->L[q] = ctx_lens_host[q];
    if (c->dyn)
        for (int p = 0; p < c->npairs; ++p) {
            c->nwin[p] = std::min((c->L[p / c->P.num_kv_heads] / SEG) / (c->P.rot_window / SEG) + 1, c->nw);
            c->pend[p] = -1;
        }
    c->poll_due = false;
    c->compressed = true;
    return ok();
}

mosaic_status mosaic_append(mosaic_cache *c, const void *k_new, const void *v_new, void *stream) {
    if (!c) return fail(MOSAIC_ERR_INVALID, "NULL cache");
    if (!c->arena || !c->compressed) return fail(MOSAIC_ERR_STATE, "append before compress");
    if (!k_new || !v_new) return fail(MOSAIC_ERR_INVALID, "NULL k_new or v_new");
    if (((uintptr_t)k_new | (uintptr_t)v_new) % 4) return fail(MOSAIC_ERR_INVALID, "k_new/v_new must be 4-byte aligned");
    int due = 0;                            // MAINT_FLUSH / MAINT_FINALIZE of some sequence
    for (int q = 0; q < c->num_seqs; ++q) {
        if (c->L[q] + 1 > c->cap[q]) return fail(MOSAIC_ERR_CAPACITY, "sequence %d is full (%d tokens)", q, c->L[q]);
        if ((c->L[q] + 1) % UBUF == 0) {
            due |= ((c->L[q] + 1) % SEG == 0) ? MAINT_FINALIZE : MAINT_FLUSH;
            if (c->dyn && c->poll_due)
                return fail(MOSAIC_ERR_STATE, "a segment completed since the last mosaic_window_poll: poll (and close "
                                              "what it reports) before the buffer of sequence %d is compressed", q);
            if (c->dyn)
                for (int h = 0; h < c->P.num_kv_heads; ++h)
                    if (c->pend[q * c->P.num_kv_heads + h] >= 0)
                        return fail(MOSAIC_ERR_STATE, "sequence %d kv head %d: a closed window awaits its rotation "
                                                      "(mosaic_window_close)", q, h);
        }
    }
    hipStream_t s = (hipStream_t)stream;
    const Geom g = c->geom();
    hipError_t e = launch_append(g, (const uint16_t *)k_new, (const uint16_t *)v_new, s);
    if (e != hipSuccess) return hip_fail(e, "append launch");
    if (due && (e = launch_maintain(g, MAINT_APPEND, due, s)) != hipSuccess) return hip_fail(e, "flush/finalize launch");
    for (int q = 0; q < c->num_seqs; ++q) c->L[q] += 1;
    if (c->dyn && (due & MAINT_FINALIZE)) c->poll_due = true;
    return ok();
}

mosaic_status mosaic_decode_attention(mosaic_cache *c, const void *q, float *out, float sm_scale, void *ws,
                                      size_t ws_bytes, void *stream) {
    if (!c) return fail(MOSAIC_ERR_INVALID, "NULL cache");
    if (!c->arena || !c->compressed) return fail(MOSAIC_ERR_STATE, "decode before compress");
    if (!q || !out || !ws) return fail(MOSAIC_ERR_INVALID, "NULL q, out or workspace");
    if (ws_bytes < c->wsl.total) return fail(MOSAIC_ERR_INVALID, "workspace %zu bytes < %llu required", ws_bytes,
                                             (unsigned long long)c->wsl.total);
    if ((uintptr_t)ws % 256) return fail(MOSAIC_ERR_INVALID, "workspace not 256-byte aligned");
    if (((uintptr_t)q % 4) || ((uintptr_t)out % 4)) return fail(MOSAIC_ERR_INVALID, "q/out misaligned");
    if (!std::isfinite(sm_scale)) return fail(MOSAIC_ERR_INVALID, "sm_scale not finite");
    int max_desc = 0, maxL = 0;
    for (int q2 = 0; q2 < c->num_seqs; ++q2) {
        const int L = c->L[q2];
        max_desc = std::max(max_desc, L / SEG + ((L % SEG) >= UBUF ? 1 : 0));
        maxL = std::max(maxL, L);
    }
    int nwu = std::max(1, std::min(c->nw, (maxL + c->P.rot_window - 1) / c->P.rot_window));
    Geom g = c->geom();
    if (c->dyn) {
        // the windows in use as of the last poll: a window closed since then
        // is still empty (nothing is compressed before the poll), so it adds
        // nothing; the decode works on that many windows
        nwu = 1;
        for (int p = 0; p < c->npairs; ++p) nwu = std::max(nwu, c->nwin[p]);
        g.nw = nwu;
    }
    hipError_t e = launch_decode(g, c->wsgeom(ws), (const uint16_t *)q, out, sm_scale, max_desc, nwu,
                                 (hipStream_t)stream, c->timing ? c->ev : nullptr);
    if (e != hipSuccess) return hip_fail(e, "decode launch");
    if (c->timing) c->timed_once = true;
    return ok();
}

mosaic_status mosaic_decode_attention_noalloc(mosaic_cache *c, const void *q, float *out, float sm_scale, void *stream) {
    if (!c) return fail(MOSAIC_ERR_INVALID, "NULL cache");
    if (c->wsl.total > (uint64_t)MOSAIC_NOALLOC_SCRATCH_BYTES)
        return fail(MOSAIC_ERR_UNSUPPORTED, "decode workspace of %llu bytes exceeds the %llu-byte fixed buffer",
                    (unsigned long long)c->wsl.total, (unsigned long long)MOSAIC_NOALLOC_SCRATCH_BYTES);
    void *ws = nullptr;
    const mosaic_status st = scratch_of_current_device(&ws);
    if (st != MOSAIC_OK) return st;
    return mosaic_decode_attention(c, q, out, sm_scale, ws, (size_t)MOSAIC_NOALLOC_SCRATCH_BYTES, stream);
}

mosaic_status mosaic_dense_workspace_bytes(int32_t num_seqs, int32_t num_kv_heads, int32_t group_size,
                                           int32_t max_ctx, size_t *bytes) {
    if (!bytes) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (num_seqs < 1 || num_kv_heads < 1 || group_size < 1 || group_size > 8 || max_ctx < 0)
        return fail(MOSAIC_ERR_INVALID, "bad shape");
    *bytes = dense_part_bytes(num_seqs * num_kv_heads, group_size, max_ctx);
    return ok();
}

mosaic_status mosaic_dense_decode_attention(const void *q, const void *k, const void *v, float *out, int32_t num_seqs,
                                            int32_t num_kv_heads, int32_t group_size, int32_t head_dim, int32_t dtype,
                                            int64_t seq_stride, int32_t max_ctx, const int32_t *ctx_lens,
                                            float sm_scale, void *ws, size_t ws_bytes, void *stream) {
    if (!q || !k || !v || !out || !ctx_lens || !ws) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (head_dim != 128) return fail(MOSAIC_ERR_UNSUPPORTED, "head_dim %d", head_dim);
    if (dtype != MOSAIC_FP16 && dtype != MOSAIC_BF16) return fail(MOSAIC_ERR_INVALID, "dtype %d", dtype);
    if (num_seqs < 1 || num_kv_heads < 1 || group_size < 1 || group_size > 8) return fail(MOSAIC_ERR_INVALID, "bad shape");
    if (max_ctx < 0 || seq_stride < max_ctx) return fail(MOSAIC_ERR_INVALID, "seq_stride %lld < max_ctx %d",
                                                         (long long)seq_stride, max_ctx);
    if (((uintptr_t)k | (uintptr_t)v) % 16) return fail(MOSAIC_ERR_INVALID, "k/v must be 16-byte aligned");
    const size_t need = dense_part_bytes(num_seqs * num_kv_heads, group_size, max_ctx);
    if (ws_bytes < need) return fail(MOSAIC_ERR_INVALID, "workspace %zu < %zu", ws_bytes, need);
    hipError_t e = launch_dense((const uint16_t *)q, (const uint16_t *)k, (const uint16_t *)v, out, num_seqs,
                                num_kv_heads, group_size, dtype, seq_stride, max_ctx, ctx_lens, sm_scale, (float *)ws, 0,
                                (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "dense launch");
    return ok();
}

static mosaic_status rotation_shape(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens, int &nw) {
    if (!params) return fail(MOSAIC_ERR_INVALID, "NULL params");
    if (params->head_dim != 128) return fail(MOSAIC_ERR_UNSUPPORTED, "head_dim %d", params->head_dim);
    if (params->num_kv_heads < 1 || num_seqs < 1 || max_tokens < 1)
        return fail(MOSAIC_ERR_INVALID, "num_seqs %d, num_kv_heads %d, max_tokens %d", num_seqs, params->num_kv_heads,
                    max_tokens);
    if (params->rot_window < SEG || params->rot_window % SEG)
        return fail(MOSAIC_ERR_INVALID, "rot_window %d: a positive multiple of %d", params->rot_window, SEG);
    nw = (max_tokens + params->rot_window - 1) / params->rot_window;
    return MOSAIC_OK;
}

mosaic_status mosaic_rotation_workspace_bytes(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                              size_t *bytes) {
    int nw = 0;
    if (!bytes) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    const mosaic_status st = rotation_shape(params, num_seqs, max_tokens, nw);
    if (st != MOSAIC_OK) return st;
    *bytes = rotation_ws_bytes(num_seqs, params->num_kv_heads, nw, params->rot_window);
    return ok();
}

mosaic_status mosaic_compute_rotations(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                       const void *k, const void *v, int64_t seq_stride,
                                       const int32_t *ctx_lens_host, float *rot_k, float *rot_v, float *evals_k,
                                       float *evals_v, void *ws, size_t ws_bytes, void *stream) {
    int nw = 0;
    const mosaic_status st = rotation_shape(params, num_seqs, max_tokens, nw);
    if (st != MOSAIC_OK) return st;
    if (!k || !v || !ctx_lens_host || !rot_k || !rot_v || !ws) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (params->dtype != MOSAIC_FP16 && params->dtype != MOSAIC_BF16) return fail(MOSAIC_ERR_INVALID, "dtype %d", params->dtype);
    if (((uintptr_t)k | (uintptr_t)v | (uintptr_t)rot_k | (uintptr_t)rot_v | (uintptr_t)ws) % 16)
        return fail(MOSAIC_ERR_INVALID, "k, v, rot_k, rot_v and ws must be 16-byte aligned");
    if ((evals_k == nullptr) != (evals_v == nullptr)) return fail(MOSAIC_ERR_INVALID, "evals_k and evals_v: both or neither");
    int maxL = 0;
    for (int s = 0; s < num_seqs; ++s) {
        const int L = ctx_lens_host[s];
        if (L < 0) return fail(MOSAIC_ERR_INVALID, "ctx_lens[%d] = %d < 0", s, L);
        if (L > max_tokens) return fail(MOSAIC_ERR_CAPACITY, "ctx_lens[%d] = %d > max_tokens %d", s, L, max_tokens);
        maxL = std::max(maxL, L);
    }
    if (seq_stride < maxL || seq_stride < 1) return fail(MOSAIC_ERR_INVALID, "seq_stride %lld < longest context %d",
                                                         (long long)seq_stride, maxL);
    const size_t need = rotation_ws_bytes(num_seqs, params->num_kv_heads, nw, params->rot_window);
    if (ws_bytes < need) return fail(MOSAIC_ERR_INVALID, "workspace %zu < %zu", ws_bytes, need);
    hipStream_t s = (hipStream_t)stream;
    int32_t *ctx_dev = (int32_t *)ws;
    hipError_t e = hipMemcpyAsync(ctx_dev, ctx_lens_host, sizeof(int32_t) * num_seqs, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "copy of context lengths");
    e = launch_rotations((const uint16_t *)k, (const uint16_t *)v, seq_stride, num_seqs, params->num_kv_heads,
                         params->dtype, ctx_dev, params->rot_window, nw, rot_k, rot_v, evals_k, evals_v,
                         (float *)((uint8_t *)ws + rotation_ctx_bytes(num_seqs)), s);
    if (e != hipSuccess) return hip_fail(e, "rotation launch");
    return ok();
}

mosaic_status mosaic_reorder_workspace_bytes(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                             size_t *bytes) {
    int nw = 0;
    if (!bytes) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    const mosaic_status st = rotation_shape(params, num_seqs, max_tokens, nw);
    if (st != MOSAIC_OK) return st;
    *bytes = reorder_ws_bytes(num_seqs, params->num_kv_heads, nw, std::min(params->rot_window, max_tokens));
    return ok();
}

mosaic_status mosaic_reorder_rotations(const mosaic_params *params, int32_t num_seqs, int32_t max_tokens,
                                       const void *k, const void *v, int64_t seq_stride,
                                       const int32_t *ctx_lens_host, float *rot_k, float *rot_v, void *ws,
                                       size_t ws_bytes, void *stream) {
    int nw = 0;
    const mosaic_status st = rotation_shape(params, num_seqs, max_tokens, nw);
    if (st != MOSAIC_OK) return st;
    if (!k || !v || !ctx_lens_host || !rot_k || !rot_v || !ws) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (params->dtype != MOSAIC_FP16 && params->dtype != MOSAIC_BF16) return fail(MOSAIC_ERR_INVALID, "dtype %d", params->dtype);
    if (params->default_keep < 1 || params->default_keep > D)
        return fail(MOSAIC_ERR_INVALID, "default_keep %d: 1..128", params->default_keep);
    if (((uintptr_t)k | (uintptr_t)v | (uintptr_t)rot_k | (uintptr_t)rot_v) % 16 || (uintptr_t)ws % 256)
        return fail(MOSAIC_ERR_INVALID, "k, v, rot_k and rot_v must be 16-byte aligned, ws 256-byte aligned");
    int maxL = 0;
    for (int s = 0; s < num_seqs; ++s) {
        const int L = ctx_lens_host[s];
        if (L < 0) return fail(MOSAIC_ERR_INVALID, "ctx_lens[%d] = %d < 0", s, L);
        if (L > max_tokens) return fail(MOSAIC_ERR_CAPACITY, "ctx_lens[%d] = %d > max_tokens %d", s, L, max_tokens);
        maxL = std::max(maxL, L);
    }
    if (seq_stride < maxL || seq_stride < 1) return fail(MOSAIC_ERR_INVALID, "seq_stride %lld < longest context %d",
                                                         (long long)seq_stride, maxL);
    const int wtok = std::min(params->rot_window, max_tokens);          // tokens of a window at most
    const size_t need = reorder_ws_bytes(num_seqs, params->num_kv_heads, nw, wtok);
    if (ws_bytes < need) return fail(MOSAIC_ERR_INVALID, "workspace %zu < %zu", ws_bytes, need);
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = hipMemcpyAsync(ws, ctx_lens_host, sizeof(int32_t) * num_seqs, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "copy of context lengths");
    e = launch_reorder((const uint16_t *)k, (const uint16_t *)v, seq_stride, num_seqs, params->num_kv_heads,
                       params->dtype, (const int32_t *)ws, params->rot_window, nw, wtok, params->default_keep, rot_k,
                       rot_v, (uint8_t *)ws, s);
    if (e != hipSuccess) return hip_fail(e, "reorder launch");
    return ok();
}

mosaic_status mosaic_cache_stats(const mosaic_cache *c, mosaic_stats *out, void *stream) {
    if (!c || !out) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (!c->arena || !c->compressed) return fail(MOSAIC_ERR_STATE, "stats before compress");
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "stream synchronize");
    std::memset(out, 0, sizeof(*out));
    std::vector<PairMeta> meta(c->npairs);
    std::vector<Desc> desc((size_t)c->max_desc);
    for (int p = 0; p < c->npairs; ++p) {
        e = hipMemcpy(&meta[p], c->arena + c->lay.meta_off + (uint64_t)p * c->lay.meta_stride, sizeof(PairMeta),
                      hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "meta copy");
    }
    const int hkv = c->P.num_kv_heads;
    for (int p = 0; p < c->npairs; ++p) {
        const int L = meta[p].L, nf = L / SEG, rem = L % SEG, prov = rem >= UBUF, nbuf = rem - (prov ? UBUF : 0);
        const int nd = nf + prov;
        if (nd > 0) {
            e = hipMemcpy(desc.data(), c->arena + c->lay.desc_off + c->pairs[4 * p], sizeof(Desc) * nd,
                          hipMemcpyDeviceToHost);
            if (e != hipSuccess) return hip_fail(e, "descriptor copy");
        }
        int64_t used = (int64_t)meta[p].tok_tail + meta[p].sc_tail + 16ll * nd + (int64_t)nbuf * 2 * D * 2;
        if (prov) {
            const Desc &d = desc[nf];
            const int rec = tok_vec_bytes(d.r, d.log2g, c->P.trunc_channels, c->P.value_fp8);
            const int srec = vec_bytes(d.r, d.log2g, c->P.trunc_channels);
            used += (int64_t)UBUF * 2 * rec + (int64_t)(UBUF >> d.log2b) * srec;
        }
        out->used_bytes += used;
        out->tokens += (p % hkv == 0) ? L : 0;
        out->segments += nf;
        for (int s = 0; s < nf; ++s) {
            int ri = -1, gi = -1, bi = -1;
            for (int i = 0; i < 3; ++i) {
                if (c->P.keep_cand[i] == desc[s].r && ri < 0) ri = i;
                if (c->P.group_cand[i] == (1 << desc[s].log2g) && gi < 0) gi = i;
                if (c->P.block_cand[i] == (1 << desc[s].log2b) && bi < 0) bi = i;
            }
            if (ri >= 0 && gi >= 0 && bi >= 0) out->strategy_hist[ri][gi][bi]++;
        }
        if (c->rotated)
            out->rotation_bytes += (int64_t)(c->dyn ? meta[p].nwin : (L + c->P.rot_window - 1) / c->P.rot_window) * 2 * D * D * 4;
    }
    out->dense_bytes = out->tokens * 2 * D * 2 * hkv;
    return ok();
}

mosaic_status mosaic_window_poll(mosaic_cache *c, int32_t *out_host, int32_t *n_closed_host, void *stream) {
    if (!c || !out_host || !n_closed_host) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (!c->dyn) return fail(MOSAIC_ERR_INVALID, "the cache was created without dynamic windows");
    if (!c->arena || !c->compressed) return fail(MOSAIC_ERR_STATE, "poll before compress");
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "stream synchronize");
    std::vector<uint8_t> meta((size_t)c->npairs * c->lay.meta_stride);
    e = hipMemcpy(meta.data(), c->arena + c->lay.meta_off, meta.size(), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "meta copy");
    int n = 0;
    for (int p = 0; p < c->npairs; ++p) {
        const uint8_t *m = meta.data() + (size_t)p * c->lay.meta_stride;
        PairMeta pm;
        std::memcpy(&pm, m, sizeof(pm));
        const int32_t *wt = (const int32_t *)(m + sizeof(PairMeta));
        if (pm.nwin < 1 || pm.nwin > c->nw || pm.pend < -1 || pm.pend >= pm.nwin - 1)
            return fail(MOSAIC_ERR_STATE, "pair %d: window state out of range (%d windows, pending %d)", p, pm.nwin, pm.pend);
        c->nwin[p] = pm.nwin;
        c->pend[p] = pm.pend;
        c->pend_len[p] = pm.pend >= 0 ? (wt[pm.pend + 1] - wt[pm.pend]) * SEG : 0;
        out_host[3 * p] = pm.pend;
        out_host[3 * p + 1] = pm.pend >= 0 ? wt[pm.pend] * SEG : 0;
        out_host[3 * p + 2] = pm.pend >= 0 ? (wt[pm.pend + 1] - wt[pm.pend]) * SEG : 0;
        n += pm.pend >= 0;
    }
    c->poll_due = false;
    *n_closed_host = n;
    return ok();
}

mosaic_status mosaic_window_rotations(mosaic_cache *c, float *rot_k, float *rot_v, void *ws, size_t ws_bytes,
                                      void *stream) {
    if (!c) return fail(MOSAIC_ERR_INVALID, "NULL cache");
    if (!c->dyn) return fail(MOSAIC_ERR_INVALID, "the cache was created without dynamic windows");
    if (!c->arena || !c->compressed) return fail(MOSAIC_ERR_STATE, "rotations before compress");
    if (c->poll_due) return fail(MOSAIC_ERR_STATE, "a segment completed since the last mosaic_window_poll");
    if (!rot_k || !rot_v || !ws) return fail(MOSAIC_ERR_INVALID, "NULL rot_k, rot_v or ws");
    if (((uintptr_t)rot_k | (uintptr_t)rot_v) % 16 || (uintptr_t)ws % 256)
        return fail(MOSAIC_ERR_INVALID, "rot_k and rot_v must be 16-byte aligned, ws 256-byte aligned");
    if (ws_bytes < window_rot_ws_bytes(c->npairs))
        return fail(MOSAIC_ERR_INVALID, "workspace %zu bytes < %zu required", ws_bytes, window_rot_ws_bytes(c->npairs));
    float *part = (float *)((uint8_t *)ws + align256((uint64_t)c->npairs * 4));
    hipError_t e = launch_window_rotations(c->geom(), rot_k, rot_v, part, (int32_t *)ws, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "window rotation launch");
    return ok();
}

mosaic_status mosaic_window_close(mosaic_cache *c, const float *rot_k, const float *rot_v, const void *k, const void *v,
                                  int64_t seq_stride, void *stream) {
    if (!c) return fail(MOSAIC_ERR_INVALID, "NULL cache");
    if (!c->dyn) return fail(MOSAIC_ERR_INVALID, "the cache was created without dynamic windows");
    if (!c->arena || !c->compressed) return fail(MOSAIC_ERR_STATE, "close before compress");
    if (c->poll_due) return fail(MOSAIC_ERR_STATE, "a segment completed since the last mosaic_window_poll");
    if (!rot_k || !rot_v || !k || !v) return fail(MOSAIC_ERR_INVALID, "NULL rot_k, rot_v, k or v");
    if (((uintptr_t)rot_k | (uintptr_t)rot_v | (uintptr_t)k | (uintptr_t)v) % 16)
        return fail(MOSAIC_ERR_INVALID, "rot_k, rot_v, k and v must be 16-byte aligned");
    int max_tok = 0, n = 0;
    for (int p = 0; p < c->npairs; ++p) {
        if (c->pend[p] < 0) continue;
        ++n;
        max_tok = std::max(max_tok, c->pend_len[p]);
    }
    if (n == 0) return ok();
    if (seq_stride < max_tok)
        return fail(MOSAIC_ERR_INVALID, "seq_stride %lld < longest closed window %d", (long long)seq_stride, max_tok);
    const int max_segs = max_tok / SEG;
    hipError_t e = launch_close(c->geom(), rot_k, rot_v, (const uint16_t *)k, (const uint16_t *)v, seq_stride, max_segs,
                                (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "close launch");
    for (int p = 0; p < c->npairs; ++p) { c->pend[p] = -1; c->pend_len[p] = 0; }
    return ok();
}

mosaic_status mosaic_set_timing(mosaic_cache *c, int32_t enable) {
    if (!c) return fail(MOSAIC_ERR_INVALID, "NULL cache");
    if (enable && !c->ev[0]) {
        for (auto &e : c->ev) {
            hipError_t r = hipEventCreate(&e);
            if (r != hipSuccess) return hip_fail(r, "event create");
        }
    }
    c->timing = enable != 0;
    c->timed_once = false;
    return ok();
}

mosaic_status mosaic_decode_timing(mosaic_cache *c, float *ms) {
    if (!c || !ms) return fail(MOSAIC_ERR_INVALID, "NULL argument");
    if (!c->timing || !c->timed_once) return fail(MOSAIC_ERR_STATE, "no timed decode");
    hipError_t e = hipEventSynchronize(c->ev[5]);
    if (e != hipSuccess) return hip_fail(e, "event synchronize");
    for (int i = 0; i < 5; ++i) {
        e = hipEventElapsedTime(&ms[i], c->ev[i], c->ev[i + 1]);
        if (e != hipSuccess) return hip_fail(e, "event elapsed");
    }
    return ok();
}

const char *mosaic_last_error(void) { return g_err.c_str(); }

}  // extern "C"
