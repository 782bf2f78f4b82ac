// rotation.hip -- gfx950 kernels that compute each window's rotation matrix
// from the cache itself (Sec. 2.3; Sec. 5.2: once the KV cache exists, the
// SVD rotation of its K and of its V matrix is computed, then every vector is
// rotated by it).  The rows of R are the right singular vectors of the
// window's matrix X, i.e. the eigenvectors of X^T X by descending eigenvalue.
//
//   k_cov    : uncentered covariance X^T X in fp32.  The 16-bit inputs make
//              every product exact in fp32; each element is one fused chain in
//              token order over a 4096-token slice, and the slices are summed
//              in slice order by the solver, so the result does not depend on
//              scheduling.  A workgroup stages 64 tokens at a time in LDS and
//              thread (ti, tj) owns the 8 x 8 tile of rows 8 ti.. and columns
//              8 tj.. (64 FMAs per four 16-byte LDS reads).
//   k_jacobi : one workgroup per matrix: A and the accumulated rotations V in
//              LDS (rows padded to 129 floats), cyclic Jacobi with the
//              round-robin ordering that pairs all 128 indices into 64
//              disjoint rotations per step (127 steps per sweep), rows of A,
//              then columns of A and V, sweeps until the off-diagonal energy
//              is below 1e-14 of the diagonal's (at most 40).  Then the
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
constexpr int JACOBI_MAX_SWEEPS = 40;

// grid (slices, windows, pairs * 2); z = 2 * pair + (0: K, 1: V)
__global__ void __launch_bounds__(256) k_cov(const uint16_t *k, const uint16_t *v, int64_t seq_stride, int hkv,
                                             int dtype, const int32_t *ctx, int W, int nslices, float *part) {
    __shared__ __align__(16) float xs[COV_TILE][D];
    const int sl = blockIdx.x, w = blockIdx.y, z = blockIdx.z, p = z >> 1, kv = z & 1;
    const int tid = threadIdx.x, ti = tid >> 4, tj = tid & 15;
    const int L = ctx[p / hkv];
    const int64_t a = (int64_t)w * W + (int64_t)sl * COV_SLICE;
    const int64_t b = min(min((int64_t)(w + 1) * W, (int64_t)L), a + COV_SLICE);
    const uint16_t *src = (kv ? v : k) + (uint64_t)p * (uint64_t)seq_stride * D;
    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = 0.0f;
    for (int64_t t0 = a; t0 < b; t0 += COV_TILE) {
        const int n = (int)min((int64_t)COV_TILE, b - t0);
        __syncthreads();                                   // previous tile consumed
        for (int i = tid; i < COV_TILE * D; i += 256) {
            const int t = i / D, c = i % D;
            xs[t][c] = (t < n) ? h2f(src[(uint64_t)(t0 + t) * D + c], dtype) : 0.0f;
        }
        __syncthreads();
        for (int t = 0; t < n; ++t) {
            const float4 r0 = *(const float4 *)&xs[t][8 * ti], r1 = *(const float4 *)&xs[t][8 * ti + 4];
            const float4 c0 = *(const float4 *)&xs[t][8 * tj], c1 = *(const float4 *)&xs[t][8 * tj + 4];
            const float r[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
            const float c[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(r[i], c[j], acc[i][j]);
        }
    }
    float *out = part + ((((uint64_t)z * gridDim.y + w) * nslices + sl) * D * D);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float4 *o = (float4 *)(out + (uint64_t)(8 * ti + i) * D + 8 * tj);
        o[0] = make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
        o[1] = make_float4(acc[i][4], acc[i][5], acc[i][6], acc[i][7]);
    }
}

// position i of step s of the round-robin tournament over 128 indices
__device__ __forceinline__ int rr_index(int i, int s) { return i == 0 ? 0 : 1 + (i - 1 + s) % (D - 1); }

// sum over the 256 threads of the block; red: 4 floats of LDS
__device__ __forceinline__ float block_sum_256(float x, float *red) {
    x = tree64(x);                                         // lane 63's tree over the wave (broadcast)
    const int tid = threadIdx.x;
    __syncthreads();
    if ((tid & 63) == 0) red[tid >> 6] = x;
    __syncthreads();
    return (red[0] + red[1]) + (red[2] + red[3]);
}

// grid (windows, pairs * 2); dynamic LDS: A and V [D][JP] floats
__global__ void __launch_bounds__(256) k_jacobi(const int32_t *ctx, int hkv, int W, int nw, int nslices,
                                                const float *part, float *rot_k, float *rot_v, float *ev_k,
                                                float *ev_v) {
    extern __shared__ __align__(16) float jsm[];
    float *A = jsm, *V = jsm + D * JP;
    __shared__ float rc[64], rs[64], red[4];
    __shared__ int rp[64], rq[64];
    __shared__ int s_done;
    const int w = blockIdx.x, z = blockIdx.y, p = z >> 1, kv = z & 1, tid = threadIdx.x;
    const int L = ctx[p / hkv];
    const int nwt = (int)min((int64_t)nw, ((int64_t)L + W - 1) / W);     // windows with tokens
    float *R = (kv ? rot_v : rot_k) + ((uint64_t)p * nw + w) * D * D;
    float *ev = (kv ? ev_v : ev_k);
    if (ev) ev += ((uint64_t)p * nw + w) * D;
    if (nwt == 0) {                                        // no token: the identity
        for (int i = tid; i < D * D; i += 256) R[i] = (i / D == i % D) ? 1.0f : 0.0f;
        if (ev)
            for (int i = tid; i < D; i += 256) ev[i] = 0.0f;
        return;
    }
    const int ws = min(w, nwt - 1);                        // the window solved here
    const float *src = part + (((uint64_t)z * nw + ws) * nslices) * D * D;
    for (int i = tid; i < D * D; i += 256) {
        float x = 0.0f;
        for (int sl = 0; sl < nslices; ++sl) x += src[(uint64_t)sl * D * D + i];
        A[(i / D) * JP + i % D] = x;
        V[(i / D) * JP + i % D] = (i / D == i % D) ? 1.0f : 0.0f;
    }
    __syncthreads();
    for (int sweep = 0; sweep < JACOBI_MAX_SWEEPS; ++sweep) {
        // convergence: off-diagonal energy against the diagonal's
        float off = 0.0f, dia = 0.0f;
        for (int i = tid; i < D * D; i += 256) {
            const int r = i / D, c = i % D;
            const float x = A[r * JP + c];
            if (r == c) dia = fmaf(x, x, dia);
            else off = fmaf(x, x, off);
        }
        off = block_sum_256(off, red);
        dia = block_sum_256(dia, red);
        if (tid == 0) s_done = !(off > 1e-14f * dia);
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
            // rows: A <- J^T A
            for (int u = tid; u < 64 * D; u += 256) {
                const int kk = u / D, j = u % D;
                const float c = rc[kk], s = rs[kk];
                float *ap = A + rp[kk] * JP, *aq = A + rq[kk] * JP;
                const float x = ap[j], y = aq[j];
                ap[j] = c * x - s * y;
                aq[j] = s * x + c * y;
            }
            __syncthreads();
            // columns: A <- A J, V <- V J
            for (int u = tid; u < 64 * D; u += 256) {
                const int kk = u % 64, i = u / 64;
                const float c = rc[kk], s = rs[kk];
                const int pp = rp[kk], qq = rq[kk];
                float *ar = A + i * JP, *vr = V + i * JP;
                const float x = ar[pp], y = ar[qq];
                ar[pp] = c * x - s * y;
                ar[qq] = s * x + c * y;
                const float vx = vr[pp], vy = vr[qq];
                vr[pp] = c * vx - s * vy;
                vr[qq] = s * vx + c * vy;
            }
            __syncthreads();
            if (tid < 64) {                                // the rotated pair is zero by construction
                A[rp[tid] * JP + rq[tid]] = 0.0f;
                A[rq[tid] * JP + rp[tid]] = 0.0f;
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

}  // namespace

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
    hipLaunchKernelGGL(k_cov, dim3(nslices, nw, npairs * 2), dim3(256), 0, s, k, v, seq_stride, hkv, dtype, ctx_dev,
                       W, nslices, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t smem = (size_t)2 * D * JP * sizeof(float);
    hipLaunchKernelGGL(k_jacobi, dim3(nw, npairs * 2), dim3(256), smem, s, ctx_dev, hkv, W, nw, nslices, part, rot_k,
                       rot_v, ev_k, ev_v);
    return hipGetLastError();
}

}  // namespace mosaic
