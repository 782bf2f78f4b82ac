// rotation.hip -- gfx950 kernels that compute each window's rotation matrix
// from the cache itself (Sec. 2.3; Sec. 5.2: once the KV cache exists, the
// SVD rotation of its K and of its V matrix is computed, then every vector is
// rotated by it).  The rows of R are the right singular vectors of the
// window's matrix X, i.e. the eigenvectors of X^T X by descending eigenvalue.
//
//   k_cov    : uncentered covariance X^T X on the matrix cores (16x16x32,
//              16-bit operands: every product is exact, fp32 accumulation)
//              over 4096-token slices; the solver sums the slices in slice
//              order, so the result does not depend on scheduling.
//   k_jacobi : one 1024-thread workgroup per matrix: A and the accumulated rotations V in
//              LDS (rows padded to 129 floats), cyclic Jacobi with the
//              round-robin ordering that pairs all 128 indices into 64
//              disjoint rotations per step (127 steps per sweep), A updated
//              one 2 x 2 block (rows of one pair, columns of another) per
//              thread and V by columns in the same pass, sweeps until the
//              off-diagonal energy is below 1e-12 of the diagonal's (at most
//              30).  Then the
//              eigenvalues are ranked (descending, index ascending on ties)
//              and each eigenvector is written as row rank of R, normalized
//              and signed so that its largest-magnitude component is
//              positive.
//
// A window past a sequence's last token repeats the last window that has
// one (its workgroup solves that window again: identical input, identical
// result); a sequence with no token gets the identity.
#include "mosaic_internal.h"

namespace mosaic {

namespace {

constexpr int COV_SLICE = 4096;   // tokens per covariance workgroup
constexpr int COV_TILE = 64;      // tokens staged per round
constexpr int JP = D + 1;         // padded LDS row of the solver
constexpr int JACOBI_MAX_SWEEPS = 30;

typedef float cov_f4 __attribute__((ext_vector_type(4)));

template <int DT> struct CovMma;
template <> struct CovMma<1> {
    typedef __bf16 v8 __attribute__((ext_vector_type(8)));
    static __device__ __forceinline__ cov_f4 run(v8 a, v8 b, cov_f4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};
template <> struct CovMma<0> {
    typedef _Float16 v8 __attribute__((ext_vector_type(8)));
    static __device__ __forceinline__ cov_f4 run(v8 a, v8 b, cov_f4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};

// grid (slices, windows, pairs * 2); z = 2 * pair + (0: K, 1: V).  C = X^T X
// on the matrix cores: both operands are "8 consecutive tokens of one
// channel", so each 64-token tile is staged channel-major in LDS (the lanes
// of a store write 64 consecutive tokens of one channel; rows padded to 72
// elements so that the 16 lanes of an operand read spread over the banks).
// Wave w owns output rows 32 w .. 32 w + 31 (2 x 8 tiles of 16 x 16).
template <int DT>
__global__ void __launch_bounds__(256) k_cov(const uint16_t *k, const uint16_t *v, int64_t seq_stride, int hkv,
                                             const int32_t *ctx, int W, int nslices, float *part) {
    using M8 = typename CovMma<DT>::v8;
    constexpr int XS = COV_TILE + 8;                       // elements per staged channel row
    __shared__ __align__(16) uint16_t xt[D * XS];
    const int sl = blockIdx.x, w = blockIdx.y, z = blockIdx.z, p = z >> 1, kv = z & 1;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l16 = lane & 15, q4 = lane >> 4;
    const int L = ctx[p / hkv];
    const int64_t a = (int64_t)w * W + (int64_t)sl * COV_SLICE;
    const int64_t b = min(min((int64_t)(w + 1) * W, (int64_t)L), a + COV_SLICE);
    const uint16_t *src = (kv ? v : k) + (uint64_t)p * (uint64_t)seq_stride * D;
    cov_f4 acc[2][8];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[r][c] = cov_f4{0.0f, 0.0f, 0.0f, 0.0f};
    const uint32_t xa = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint16_t *)xt;
    for (int64_t t0 = a; t0 < b; t0 += COV_TILE) {
        const int n = (int)min((int64_t)COV_TILE, b - t0);
        __syncthreads();                                   // previous tile consumed
        {
            const int t = lane;                            // token of this lane; octets wave, wave + 4, ...
            uint4 val[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const int o = wave + 4 * kk;
                val[kk] = (t < n) ? *(const uint4 *)(src + (uint64_t)(t0 + t) * D + 8 * o) : make_uint4(0u, 0u, 0u, 0u);
            }
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const int o = wave + 4 * kk;
                const uint32_t wv[4] = {val[kk].x, val[kk].y, val[kk].z, val[kk].w};
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    xt[(8 * o + e) * XS + t] = (uint16_t)((e & 1) ? (wv[e >> 1] >> 16) : wv[e >> 1]);
            }
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < COV_TILE / 32; ++ks) {
            M8 bo[8];
#pragma unroll
            for (int c = 0; c < 8; ++c)
                bo[c] = __builtin_bit_cast(M8, *(const __attribute__((address_space(3))) uint4 *)(uintptr_t)(
                                                   xa + (uint32_t)(((16 * c + l16) * XS + 32 * ks + 8 * q4) * 2)));
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const M8 ao = __builtin_bit_cast(M8, *(const __attribute__((address_space(3))) uint4 *)(uintptr_t)(
                                                         xa + (uint32_t)(((16 * (2 * wave + r) + l16) * XS + 32 * ks + 8 * q4) * 2)));
#pragma unroll
                for (int c = 0; c < 8; ++c) acc[r][c] = CovMma<DT>::run(ao, bo[c], acc[r][c]);
            }
        }
    }
    // accumulator layout: element e of tile (r, c) is row 4 q4 + e, column l16
    float *out = part + ((((uint64_t)z * gridDim.y + w) * nslices + sl) * D * D);
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int c = 0; c < 8; ++c)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                out[(uint64_t)(16 * (2 * wave + r) + 4 * q4 + e) * D + 16 * c + l16] = acc[r][c][e];
}

// position i of step s of the round-robin tournament over 128 indices
__device__ __forceinline__ int rr_index(int i, int s) { return i == 0 ? 0 : 1 + (i - 1 + s) % (D - 1); }

constexpr int JT = 1024;          // threads of a solver workgroup

// sum over the JT threads of the block (fixed order); red: JT / 64 floats of LDS
__device__ __forceinline__ float block_sum_jt(float x, float *red) {
    x = tree64(x);                                         // the wave's tree (every lane holds it)
    const int tid = threadIdx.x;
    __syncthreads();
    if ((tid & 63) == 0) red[tid >> 6] = x;
    __syncthreads();
    float t = 0.0f;
#pragma unroll
    for (int i = 0; i < JT / 64; ++i) t += red[i];
    return t;
}

// grid (windows, pairs * 2); dynamic LDS: A and V [D][JP] floats
__global__ void __launch_bounds__(JT) k_jacobi(const int32_t *ctx, int hkv, int W, int nw, int nslices,
                                                const float *part, float *rot_k, float *rot_v, float *ev_k,
                                                float *ev_v) {
    extern __shared__ __align__(16) float jsm[];
    float *A = jsm, *V = jsm + D * JP;
    __shared__ float rc[64], rs[64], red[JT / 64];
    __shared__ int rp[64], rq[64];
    __shared__ int s_done;
    const int w = blockIdx.x, z = blockIdx.y, p = z >> 1, kv = z & 1, tid = threadIdx.x;
    const int L = ctx[p / hkv];
    const int nwt = (int)min((int64_t)nw, ((int64_t)L + W - 1) / W);     // windows with tokens
    float *R = (kv ? rot_v : rot_k) + ((uint64_t)p * nw + w) * D * D;
    float *ev = (kv ? ev_v : ev_k);
    if (ev) ev += ((uint64_t)p * nw + w) * D;
    if (nwt == 0) {                                        // no token: the identity
        for (int i = tid; i < D * D; i += JT) R[i] = (i / D == i % D) ? 1.0f : 0.0f;
        if (ev)
            for (int i = tid; i < D; i += JT) ev[i] = 0.0f;
        return;
    }
    const int ws = min(w, nwt - 1);                        // the window solved here
    const float *src = part + (((uint64_t)z * nw + ws) * nslices) * D * D;
    for (int i = tid; i < D * D; i += JT) {
        // the matrix-core products round C[i][j] and C[j][i] separately: both
        // halves take the upper triangle's value, so A is exactly symmetric
        const int r = i / D, c = i % D, u = min(r, c) * D + max(r, c);
        float x = 0.0f;
        for (int sl = 0; sl < nslices; ++sl) x += src[(uint64_t)sl * D * D + u];
        A[r * JP + c] = x;
        V[(i / D) * JP + i % D] = (i / D == i % D) ? 1.0f : 0.0f;
    }
    __syncthreads();
    for (int sweep = 0; sweep < JACOBI_MAX_SWEEPS; ++sweep) {
        // convergence: off-diagonal energy against the diagonal's
        float off = 0.0f, dia = 0.0f;
        for (int i = tid; i < D * D; i += JT) {
            const int r = i / D, c = i % D;
            const float x = A[r * JP + c];
            if (r == c) dia = fmaf(x, x, dia);
            else off = fmaf(x, x, off);
        }
        off = block_sum_jt(off, red);
        dia = block_sum_jt(dia, red);
        if (tid == 0) s_done = !(off > 1e-12f * dia);
        __syncthreads();
        if (s_done) break;
        for (int st = 0; st < D - 1; ++st) {
            if (tid < 64) {
                int pp = rr_index(tid, st), qq = rr_index(D - 1 - tid, st);
                if (pp > qq) { const int t = pp; pp = qq; qq = t; }
                const float app = A[pp * JP + pp], aqq = A[qq * JP + qq], apq = A[pp * JP + qq];
                float c = 1.0f, s = 0.0f;
                if (apq != 0.0f) {
                    const float tau = (aqq - app) / (2.0f * apq);
                    const float at = fabsf(tau);
                    const float t = (at > 1e15f) ? 0.5f / tau : copysignf(1.0f, tau) / (at + sqrtf(fmaf(tau, tau, 1.0f)));
                    c = 1.0f / sqrtf(fmaf(t, t, 1.0f));
                    s = t * c;
                }
                rp[tid] = pp; rq[tid] = qq; rc[tid] = c; rs[tid] = s;
            }
            __syncthreads();
            // A <- J^T A J one 2 x 2 block (rows of pair kk, columns of pair mm)
            // at a time: the block's new value depends on the block only, so
            // one pass suffices (rows first, then columns, per element)
            for (int u = tid; u < 64 * 64; u += JT) {
                const int kk = u >> 6, mm = u & 63;
                const float ck = rc[kk], sk = rs[kk], cm = rc[mm], sm = rs[mm];
                const int pk = rp[kk], qk = rq[kk], pm = rp[mm], qm = rq[mm];
                const float bpp = A[pk * JP + pm], bpq = A[pk * JP + qm], bqp = A[qk * JP + pm], bqq = A[qk * JP + qm];
                const float tpp = ck * bpp - sk * bqp, tpq = ck * bpq - sk * bqq;
                const float tqp = sk * bpp + ck * bqp, tqq = sk * bpq + ck * bqq;
                A[pk * JP + pm] = cm * tpp - sm * tpq;
                A[qk * JP + qm] = sm * tqp + cm * tqq;
                if (kk == mm) {                            // the rotated pair is zero by construction
                    A[pk * JP + qm] = 0.0f;
                    A[qk * JP + pm] = 0.0f;
                } else {
                    A[pk * JP + qm] = sm * tpp + cm * tpq;
                    A[qk * JP + pm] = cm * tqp - sm * tqq;
                }
            }
            // V <- V J
            for (int u = tid; u < 64 * D; u += JT) {
                const int mm = u & 63, i = u >> 6;
                const float cm = rc[mm], sm = rs[mm];
                float *vr = V + i * JP;
                const float x = vr[rp[mm]], y = vr[rq[mm]];
                vr[rp[mm]] = cm * x - sm * y;
                vr[rq[mm]] = sm * x + cm * y;
            }
            __syncthreads();
        }
    }
    // rank the eigenvalues (descending, index ascending on ties); eigenvector
    // i is column i of V
    if (tid < D) {
        const int i = tid;
        const float li = A[i * JP + i];
        int rank = 0;
        for (int j = 0; j < D; ++j) {
            const float lj = A[j * JP + j];
            rank += (lj > li || (lj == li && j < i)) ? 1 : 0;
        }
        int am = 0;
        float best = -1.0f;
        for (int j = 0; j < D; ++j) {
            const float m = fabsf(V[j * JP + i]);
            if (m > best) { best = m; am = j; }
        }
        // the accumulated rotations drift from unit length by about one
        // rounding per step: the eigenvector is normalized on the way out
        float nn = 0.0f;
        for (int j = 0; j < D; ++j) nn = fmaf(V[j * JP + i], V[j * JP + i], nn);
        const float sg = (V[am * JP + i] < 0.0f ? -1.0f : 1.0f) / sqrtf(nn);
        float *row = R + (uint64_t)rank * D;
        for (int j = 0; j < D; ++j) row[j] = sg * V[j * JP + i];
        if (ev) ev[rank] = li;
    }
}

// grid (pairs * 2), 256 threads: the incremental covariance of each pair's
// window awaiting its rotation (K for z even, V for z odd), cast to fp32 and
// symmetrized from the upper triangle as the solver expects, into the
// solver's partials (one window, one slice); one_tok[pair] = 1 if the pair has
// such a window (the solver then treats it as one window with a token), else
// 0 (the solver writes the identity)
__global__ void __launch_bounds__(256) k_cov_gather(Geom g, float *part, int32_t *one_tok) {
    const int z = blockIdx.x, p = z >> 1, kv = z & 1, tid = threadIdx.x;
    const int pw = g.meta_of(p)->pend;
    if (tid == 0 && kv == 0) one_tok[p] = pw >= 0 ? 1 : 0;
    if (pw < 0) return;
    const double *C = g.cov_of(p, pw, kv);
    float *dst = part + (uint64_t)z * D * D;
    for (int i = tid; i < D * D; i += 256) {
        const int r = i / D, c = i % D;
        dst[i] = (float)C[min(r, c) * D + max(r, c)];
    }
}

}  // namespace

hipError_t launch_window_rotations(const Geom &g, float *rot_k, float *rot_v, float *part, int32_t *one_tok,
                                   hipStream_t s) {
    hipLaunchKernelGGL(k_cov_gather, dim3(g.npairs * 2), dim3(256), 0, s, g, part, one_tok);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t smem = (size_t)2 * D * JP * sizeof(float);
    // one "sequence" per pair, one window of one token when a window awaits
    hipLaunchKernelGGL(k_jacobi, dim3(1, g.npairs * 2), dim3(JT), smem, s, (const int32_t *)one_tok, 1, 1, 1, 1,
                       (const float *)part, rot_k, rot_v, (float *)nullptr, (float *)nullptr);
    return hipGetLastError();
}

// workspace: the context lengths (int32 [num_seqs], padded to 256 bytes), then
// the covariance partials [pairs][K, V][windows][slices][D][D] fp32
size_t rotation_ctx_bytes(int num_seqs) { return ((size_t)num_seqs * sizeof(int32_t) + 255) / 256 * 256; }

size_t rotation_ws_bytes(int num_seqs, int hkv, int nw, int W) {
    const int nslices = (W + COV_SLICE - 1) / COV_SLICE;
    return rotation_ctx_bytes(num_seqs) + (size_t)num_seqs * hkv * 2 * nw * nslices * D * D * sizeof(float);
}

hipError_t launch_rotations(const uint16_t *k, const uint16_t *v, int64_t seq_stride, int num_seqs, int hkv,
                            int dtype, const int32_t *ctx_dev, int W, int nw, float *rot_k, float *rot_v, float *ev_k,
                            float *ev_v, float *part, hipStream_t s) {
    const int npairs = num_seqs * hkv;
    const int nslices = (W + COV_SLICE - 1) / COV_SLICE;
    if (dtype == 1)
        hipLaunchKernelGGL(k_cov<1>, dim3(nslices, nw, npairs * 2), dim3(256), 0, s, k, v, seq_stride, hkv, ctx_dev, W,
                           nslices, part);
    else
        hipLaunchKernelGGL(k_cov<0>, dim3(nslices, nw, npairs * 2), dim3(256), 0, s, k, v, seq_stride, hkv, ctx_dev, W,
                           nslices, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t smem = (size_t)2 * D * JP * sizeof(float);
    hipLaunchKernelGGL(k_jacobi, dim3(nw, npairs * 2), dim3(JT), smem, s, ctx_dev, hkv, W, nw, nslices, part, rot_k,
                       rot_v, ev_k, ev_v);
    return hipGetLastError();
}

}  // namespace mosaic
