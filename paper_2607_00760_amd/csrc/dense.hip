// dense.hip -- uncompressed split-K decode attention (the "Full" baseline of
// Sec. 6.1) on the same K/V layout the compression pass reads.
//
// One workgroup per (pair, 1024-token chunk).  Lane per token for q . k (the
// token's 256-byte key row, G heads at once), online softmax in fp32, lane per
// channel pair for P . V (coalesced 256-byte value rows), then a log-sum-exp
// merge of the chunks.
#include "mosaic_internal.h"

namespace mosaic {

namespace {

constexpr int DCHUNK = 1024;

template <int GP>
__global__ void __launch_bounds__(256) k_dense_split(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                                                     int hkv, int G, int dtype, int64_t seq_stride,
                                                     const int32_t *ctx, float scale, float *part, int max_splits) {
    __shared__ float qs[D * GP];
    __shared__ float ps[4][64][GP];
    __shared__ float mrg[4][GP][D + 2];
    const int p = blockIdx.y, s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int L = ctx[p / hkv];
    const int t0 = s * DCHUNK;
    if (t0 >= L) return;
    const int t1 = min(L, t0 + DCHUNK);
    for (int i = tid; i < D * GP; i += 256) {
        const int c = i / GP, h = i % GP;
        qs[i] = (h < G) ? h2f(q[((uint64_t)p * G + h) * D + c], dtype) : 0.0f;
    }
    __syncthreads();
    const uint16_t *kp = k + (uint64_t)p * seq_stride * D;
    const uint16_t *vp = v + (uint64_t)p * seq_stride * D;
    float m_run[GP], l_run[GP], acc[GP][2];
#pragma unroll
    for (int h = 0; h < GP; ++h) { m_run[h] = -INFINITY; l_run[h] = 0.0f; acc[h][0] = acc[h][1] = 0.0f; }
    for (int base = t0; base < t1; base += 256) {            // uniform across waves
        const int cb = base + wave * 64;
        const int t = cb + lane;
        const bool valid = t < t1;
        float z[GP];
#pragma unroll
        for (int h = 0; h < GP; ++h) z[h] = 0.0f;
        if (valid) {
            const uint4 *row = (const uint4 *)(kp + (uint64_t)t * D);
#pragma unroll 4
            for (int x = 0; x < D / 8; ++x) {
                const uint4 u = row[x];
                const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float k0 = h2f((uint16_t)(w4[e] & 0xffffu), dtype), k1 = h2f((uint16_t)(w4[e] >> 16), dtype);
                    const float *q0 = qs + (x * 8 + 2 * e) * GP;
#pragma unroll
                    for (int h = 0; h < GP; ++h) { z[h] = fmaf(q0[h], k0, z[h]); z[h] = fmaf(q0[GP + h], k1, z[h]); }
                }
            }
        }
        const bool any = cb < t1;
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
            ps[wave][lane][h] = pv;
        }
        __syncthreads();
        const int tmax = any ? min(64, t1 - cb) : 0;
#pragma unroll 8
        for (int tt = 0; tt < tmax; ++tt) {
            const uint32_t w2 = *(const uint32_t *)(vp + (uint64_t)(cb + tt) * D + 2 * lane);
            const float v0 = h2f((uint16_t)(w2 & 0xffffu), dtype), v1 = h2f((uint16_t)(w2 >> 16), dtype);
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                const float pv = ps[wave][tt][h];
                acc[h][0] = fmaf(pv, v0, acc[h][0]);
                acc[h][1] = fmaf(pv, v1, acc[h][1]);
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int h = 0; h < GP; ++h) {
        if (lane == 0) { mrg[wave][h][0] = m_run[h]; mrg[wave][h][1] = l_run[h]; }
        mrg[wave][h][2 + 2 * lane] = acc[h][0];
        mrg[wave][h][3 + 2 * lane] = acc[h][1];
    }
    __syncthreads();
    float *out = part + ((uint64_t)p * max_splits + s) * GP * (D + 2);
    for (int i = tid; i < GP * D; i += 256) {
        const int h = i / D, c = i % D;
        float M = -INFINITY;
        for (int x = 0; x < 4; ++x) M = fmaxf(M, mrg[x][h][0]);
        float A = 0.0f, Ls = 0.0f;
        for (int x = 0; x < 4; ++x) {
            const float f = (mrg[x][h][0] == -INFINITY) ? 0.0f : __expf(mrg[x][h][0] - M);
            A += mrg[x][h][2 + c] * f;
            Ls += mrg[x][h][1] * f;
        }
        out[2 * GP + h * D + c] = A;
        if (c == 0) { out[h] = M; out[GP + h] = Ls; }
    }
}

// grid (pairs, GP * D / 256): one output per thread; the loads of 32 chunks
// are issued together, then merged by online log-sum-exp
template <int GP>
__global__ void __launch_bounds__(256) k_dense_reduce(int hkv, int G, const int32_t *ctx, const float *part,
                                                      int max_splits, float *outp) {
    constexpr int CB = 32;
    const int p = blockIdx.x, i = blockIdx.y * 256 + threadIdx.x, h = i / D;
    const int L = ctx[p / hkv];
    const int ns = (L + DCHUNK - 1) / DCHUNK;
    float M = -INFINITY, Ls = 0.0f, A = 0.0f;
    for (int s0 = 0; s0 < ns; s0 += CB) {
        float m[CB], l[CB], a[CB];
#pragma unroll
        for (int e = 0; e < CB; ++e) {
            if (s0 + e < ns) {
                const float *ps = part + ((uint64_t)p * max_splits + s0 + e) * GP * (D + 2);
                m[e] = ps[h];
                l[e] = ps[GP + h];
                a[e] = ps[2 * GP + i];
            }
        }
#pragma unroll
        for (int e = 0; e < CB; ++e) {
            if (s0 + e < ns && m[e] != -INFINITY) {
                const float mn = fmaxf(M, m[e]);
                const float x = (M == -INFINITY) ? 0.0f : __expf(M - mn), y = __expf(m[e] - mn);
                A = A * x + a[e] * y;
                Ls = Ls * x + l[e] * y;
                M = mn;
            }
        }
    }
    if (h < G) outp[(uint64_t)p * G * D + i] = (Ls > 0.0f) ? A / Ls : 0.0f;
}

}  // namespace

size_t dense_part_bytes(int npairs, int G, int max_ctx) {
    const int GP = G <= 4 ? 4 : 8;
    const int ms = max(1, (max_ctx + DCHUNK - 1) / DCHUNK);
    return (size_t)npairs * ms * GP * (D + 2) * sizeof(float);
}

hipError_t launch_dense(const uint16_t *q, const uint16_t *k, const uint16_t *v, float *out, int nseq, int hkv, int G,
                        int dtype, int64_t seq_stride, int max_ctx, const int32_t *ctx, float scale, float *part,
                        int max_splits_unused, hipStream_t s) {
    (void)max_splits_unused;
    const int npairs = nseq * hkv;
    const int ms = max(1, (max_ctx + DCHUNK - 1) / DCHUNK);
    if (G <= 4) {
        hipLaunchKernelGGL(k_dense_split<4>, dim3(ms, npairs), dim3(256), 0, s, q, k, v, hkv, G, dtype, seq_stride, ctx,
                           scale, part, ms);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_dense_reduce<4>, dim3(npairs, 4 * D / 256), dim3(256), 0, s, hkv, G, ctx, part, ms, out);
    } else {
        hipLaunchKernelGGL(k_dense_split<8>, dim3(ms, npairs), dim3(256), 0, s, q, k, v, hkv, G, dtype, seq_stride, ctx,
                           scale, part, ms);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_dense_reduce<8>, dim3(npairs, 8 * D / 256), dim3(256), 0, s, hkv, G, ctx, part, ms, out);
    }
    return hipGetLastError();
}

}  // namespace mosaic
