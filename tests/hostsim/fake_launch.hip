// Test double of the library's launch layer: every launch function the host
// library calls records what it was asked to launch instead of launching, so
// that the host bookkeeping (validation, the append schedule, launch
// planning) runs and can be checked on a machine without a GPU.  Linked with
// the real csrc/api.hip into a separate test library; the product library
// never contains it.
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>
#include "../../paper_2607_00760_amd/csrc/mosaic_internal.h"

namespace {
std::vector<std::string> g_log;
void rec(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void rec(const char *fmt, ...) {
    char buf[256];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_log.emplace_back(buf);
}
}  // namespace

extern "C" int fake_log_count() { return (int)g_log.size(); }
extern "C" const char *fake_log_entry(int i) { return (i >= 0 && i < (int)g_log.size()) ? g_log[i].c_str() : ""; }
extern "C" void fake_log_clear() { g_log.clear(); }

namespace mosaic {
hipError_t launch_ctx_copy(int32_t *, const int32_t *src_host, int n, hipStream_t) {
    std::string s = "ctx_copy";
    for (int i = 0; i < n; ++i) s += " " + std::to_string(src_host[i]);
    rec("%s", s.c_str());
    return hipSuccess;
}
hipError_t launch_pairs_copy(uint64_t *, const uint64_t *src_host, int npairs, hipStream_t) {
    std::string s = "pairs_copy npairs=" + std::to_string(npairs) + " tok";
    for (int i = 0; i < npairs && i < 16; ++i) s += " " + std::to_string((unsigned long long)src_host[4 * i + 2]);
    rec("%s", s.c_str());
    return hipSuccess;
}
hipError_t launch_copy_rot(const Geom &g, const float *, const float *, int nw_src, hipStream_t) {
    rec("copy_rot npairs=%d nw=%d src=%d", g.npairs, g.nw, nw_src);
    return hipSuccess;
}
hipError_t launch_window_rotations(const Geom &g, float *, float *, float *, int32_t *, hipStream_t) {
    rec("window_rotations npairs=%d", g.npairs);
    return hipSuccess;
}
hipError_t launch_close(const Geom &g, const float *, const float *, const uint16_t *, const uint16_t *,
                        int64_t seq_stride, int max_segs, hipStream_t) {
    rec("close npairs=%d stride=%lld segs=%d", g.npairs, (long long)seq_stride, max_segs);
    return hipSuccess;
}
hipError_t launch_compress(const Geom &g, const uint16_t *, const uint16_t *, int64_t seq_stride, const int32_t *,
                           int full_segs, int any_tail, uint8_t *ws, uint32_t, uint32_t, hipStream_t) {
    rec("compress npairs=%d stride=%lld segs=%d tail=%d%s", g.npairs, (long long)seq_stride, full_segs, any_tail,
        ws ? " single-pass" : "");
    return hipSuccess;
}
hipError_t launch_set_meta(const Geom &g, const int32_t *, hipStream_t) {
    rec("set_meta npairs=%d", g.npairs);
    return hipSuccess;
}
hipError_t launch_append(const Geom &g, const uint16_t *, const uint16_t *, hipStream_t) {
    rec("append npairs=%d", g.npairs);
    return hipSuccess;
}
hipError_t launch_maintain(const Geom &g, int mode, int what, hipStream_t) {
    rec("maintain mode=%d flush=%d finalize=%d", mode, (what & MAINT_FLUSH) ? 1 : 0, (what & MAINT_FINALIZE) ? 1 : 0);
    (void)g;
    return hipSuccess;
}
hipError_t launch_decode(const Geom &g, const WsGeom &, const uint16_t *, float *, float scale, int max_desc_used,
                         int max_windows_used, hipStream_t, hipEvent_t *) {
    rec("decode npairs=%d desc=%d windows=%d scale=%.6f", g.npairs, max_desc_used, max_windows_used, scale);
    return hipSuccess;
}
hipError_t launch_dense(const uint16_t *, const uint16_t *, const uint16_t *, float *, int nseq, int hkv, int G,
                        int, int64_t, int, const int32_t *, float, float *, int, hipStream_t) {
    rec("dense nseq=%d hkv=%d G=%d", nseq, hkv, G);
    return hipSuccess;
}
hipError_t launch_reorder(const uint16_t *, const uint16_t *, int64_t, int, int, int, const int32_t *, int, int, int,
                          int, float *, float *, uint8_t *, hipStream_t) {
    rec("reorder");
    return hipSuccess;
}
hipError_t launch_rotations(const uint16_t *, const uint16_t *, int64_t, int, int, int, const int32_t *, int, int,
                            float *, float *, float *, float *, float *, hipStream_t) {
    rec("rotations");
    return hipSuccess;
}
// workspace sizes of the rotation, reorder and dense paths (not exercised here)
size_t dense_part_bytes(int, int, int) { return 256; }
size_t reorder_ws_bytes(int, int, int, int) { return 256; }
size_t rotation_ws_bytes(int, int, int, int) { return 256; }
size_t rotation_ctx_bytes(int) { return 256; }
}  // namespace mosaic
