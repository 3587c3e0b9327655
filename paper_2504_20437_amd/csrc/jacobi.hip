// Small SVD of the projected matrix B = Q^T A (k x l) in the randomized SVD
// (Halko et al. 2011, direct SVD of the small matrix; paper §4.1.2).
//
// The left singular vectors of B are the eigenvectors of B B^T = Z^T Z with
// Z = A^T Q = B^T. The host factors that Gram in fp64 as R^T R (Cholesky), so
// they are also the right singular vectors of the k x k factor R. They are
// found by one-sided (Hestenes) Jacobi on the columns of X = R, accumulating
// the rotations in V (X V = U Sigma, V = left singular vectors of B).
//
// Blocked for the GPU: the k columns form blocks of 16; a round-robin
// tournament pairs the blocks so that every step is a set of disjoint pairs,
// one workgroup per (pair, matrix). A workgroup forms the 32 x 32 fp64 Gram of
// its two blocks, skips the pair if every column pair is already orthogonal to
// the tolerance, otherwise diagonalises the small Gram with cyclic two-sided
// Jacobi in LDS and applies the resulting rotation to its columns of X and V.
// A sweep is nb - 1 steps; the matrix has converged when a whole sweep
// rotates nothing (rotation counts per sweep live in device memory, so no
// host synchronisation is needed). X and V are stored transposed (column c
// contiguous) so that a block of columns is a contiguous slab.
#include "common.hpp"

namespace galore {
namespace {

constexpr int JB = kJacobiBlock;   // columns per block
constexpr int JW = 2 * JB;         // columns per pair
constexpr int JT = 256;            // threads
constexpr int JR = 64;             // rows per staged chunk

__device__ __forceinline__ int ring_slot(int pos, int step, int n) {
    // circle method: slot 0 fixed, the others rotate by one per step
    if (pos == 0) return 0;
    int v = (pos - 1 - step) % (n - 1);
    if (v < 0) v += n - 1;
    return 1 + v;
}

__global__ __launch_bounds__(256) void jacobi_prepare_kernel(const double* Rb, int k,
                                                             int64_t strideR, float* Xtb,
                                                             float* Vtb, int64_t strideX, int* rotb,
                                                             int max_sweeps) {
    const int b = blockIdx.y;
    const double* R = Rb + static_cast<int64_t>(b) * strideR;
    float* Xt = Xtb + static_cast<int64_t>(b) * strideX;
    float* Vt = Vtb + static_cast<int64_t>(b) * strideX;
    if (blockIdx.x == 0 && threadIdx.x < static_cast<unsigned>(max_sweeps))
        rotb[static_cast<int64_t>(b) * max_sweeps + threadIdx.x] = 0;
    const int64_t total = static_cast<int64_t>(k) * k;
    for (int64_t pos = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; pos < total;
         pos += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int c = static_cast<int>(pos / k);
        const int i = static_cast<int>(pos - static_cast<int64_t>(c) * k);
        Xt[pos] = (i <= c) ? static_cast<float>(R[static_cast<int64_t>(i) * k + c]) : 0.0f;
        Vt[pos] = (i == c) ? 1.0f : 0.0f;
    }
}

__global__ __launch_bounds__(JT) void jacobi_step_kernel(float* Xtb, float* Vtb, int k,
                                                         int64_t strideX, int nb, int step,
                                                         int sweep, int* rotb, int max_sweeps,
                                                         double tol) {
    const int b = blockIdx.y;
    int* rot = rotb + static_cast<int64_t>(b) * max_sweeps;
    if (sweep > 0 && rot[sweep - 1] == 0) return;     // converged in an earlier sweep
    const int tid = threadIdx.x;
    const int h = blockIdx.x;
    const int bi = ring_slot(h, step, nb);
    const int bj = ring_slot(nb - 1 - h, step, nb);

    float* Xt = Xtb + static_cast<int64_t>(b) * strideX;
    float* Vt = Vtb + static_cast<int64_t>(b) * strideX;

    __shared__ double Xs[JW][JR + 1];
    __shared__ double Gs[JW][JW + 1];
    __shared__ double Th[JW][JW + 1];
    __shared__ int col[JW];
    __shared__ double red[JT / 64];
    __shared__ double cs[JW / 2], sn[JW / 2];
    __shared__ int pp[JW / 2], qq[JW / 2];
    __shared__ int any_rot;

    if (tid < JW) {
        const int blk = (tid < JB) ? bi : bj;
        const int c = blk * JB + (tid & (JB - 1));
        col[tid] = (c < k) ? c : -1;
    }
    __syncthreads();

    // ---- Gram of the pair's columns (fp64) ---------------------------------
    const int gp = tid >> 3;
    const int gq0 = (tid & 7) * 4;
    double g[4] = {0.0, 0.0, 0.0, 0.0};
    for (int r0 = 0; r0 < k; r0 += JR) {
        const int rc = min(JR, k - r0);
        for (int idx = tid; idx < JW * JR; idx += JT) {
            const int w = idx / JR, rr = idx % JR;
            const int c = col[w];
            Xs[w][rr] = (c >= 0 && rr < rc) ? static_cast<double>(Xt[static_cast<int64_t>(c) * k + r0 + rr])
                                            : 0.0;
        }
        __syncthreads();
        for (int rr = 0; rr < rc; ++rr) {
            const double xp = Xs[gp][rr];
#pragma unroll
            for (int e = 0; e < 4; ++e) g[e] += xp * Xs[gq0 + e][rr];
        }
        __syncthreads();
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) Gs[gp][gq0 + e] = g[e];
    __syncthreads();

    // ---- convergence test: largest relative off-diagonal -------------------
    double off = 0.0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int q = gq0 + e;
        if (q > gp) {
            const double dd = Gs[gp][gp] * Gs[q][q];
            if (dd > 0.0) {
                const double rel = fabs(Gs[gp][q]) / sqrt(dd);
                off = (rel > off || rel != rel) ? rel : off;
            }
        }
    }
    for (int o = 32; o > 0; o >>= 1) {
        const double other = __shfl_xor(off, o);
        off = (other > off || other != other) ? other : off;
    }
    if ((tid & 63) == 0) red[tid >> 6] = off;
    __syncthreads();
    if (tid == 0) {
        double m = red[0];
        for (int w = 1; w < JT / 64; ++w) m = (red[w] > m || red[w] != red[w]) ? red[w] : m;
        red[0] = m;
    }
    __syncthreads();
    const double off_all = red[0];
    if (!(off_all > tol) && off_all == off_all) return;   // already orthogonal
    if (tid == 0) atomicAdd(&rot[sweep], 1);

    // ---- diagonalise the 32 x 32 Gram: cyclic parallel-order Jacobi --------
    for (int idx = tid; idx < JW * JW; idx += JT) {
        const int i = idx / JW, j = idx % JW;
        Th[i][j] = (i == j) ? 1.0 : 0.0;
    }
    __syncthreads();
    for (int isw = 0; isw < 16; ++isw) {
        if (tid == 0) any_rot = 0;
        __syncthreads();
        for (int st = 0; st < JW - 1; ++st) {
            if (tid < JW / 2) {
                int p = ring_slot(tid, st, JW);
                int q = ring_slot(JW - 1 - tid, st, JW);
                if (p > q) { const int tmp = p; p = q; q = tmp; }
                const double a = Gs[p][p], bb = Gs[q][q], gm = Gs[p][q];
                double c = 1.0, s = 0.0;
                if (fabs(gm) > 1e-14 * sqrt(a * bb)) {
                    const double zeta = (bb - a) / (2.0 * gm);
                    const double sg = (zeta >= 0.0) ? 1.0 : -1.0;
                    const double tt = sg / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
                    c = 1.0 / sqrt(1.0 + tt * tt);
                    s = c * tt;
                    any_rot = 1;
                }
                cs[tid] = c;
                sn[tid] = s;
                pp[tid] = p;
                qq[tid] = q;
            }
            __syncthreads();
            // columns p, q of G and of Theta: x_p' = c x_p - s x_q, x_q' = s x_p + c x_q
            for (int idx = tid; idx < (JW / 2) * JW; idx += JT) {
                const int hh = idx / JW, row = idx % JW;
                const int p = pp[hh], q = qq[hh];
                const double c = cs[hh], s = sn[hh];
                const double gpv = Gs[row][p], gqv = Gs[row][q];
                Gs[row][p] = c * gpv - s * gqv;
                Gs[row][q] = s * gpv + c * gqv;
                const double tp = Th[row][p], tq = Th[row][q];
                Th[row][p] = c * tp - s * tq;
                Th[row][q] = s * tp + c * tq;
            }
            __syncthreads();
            // rows p, q of G
            for (int idx = tid; idx < (JW / 2) * JW; idx += JT) {
                const int hh = idx / JW, cc = idx % JW;
                const int p = pp[hh], q = qq[hh];
                const double c = cs[hh], s = sn[hh];
                const double gpv = Gs[p][cc], gqv = Gs[q][cc];
                Gs[p][cc] = c * gpv - s * gqv;
                Gs[q][cc] = s * gpv + c * gqv;
            }
            __syncthreads();
        }
        const int done = (any_rot == 0);
        __syncthreads();
        if (done) break;
    }

    // ---- apply Theta to the pair's columns of X and V ----------------------
    const int ar = tid & (JR - 1);
    const int acg = tid >> 6;          // 4 groups of 8 output columns
    for (int pass = 0; pass < 2; ++pass) {
        float* M = (pass == 0) ? Xt : Vt;
        for (int r0 = 0; r0 < k; r0 += JR) {
            const int rc = min(JR, k - r0);
            for (int idx = tid; idx < JW * JR; idx += JT) {
                const int w = idx / JR, rr = idx % JR;
                const int c = col[w];
                Xs[w][rr] = (c >= 0 && rr < rc) ? static_cast<double>(M[static_cast<int64_t>(c) * k + r0 + rr])
                                                : 0.0;
            }
            __syncthreads();
            if (ar < rc) {
                double out[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) out[e] = 0.0;
#pragma unroll 2
                for (int p = 0; p < JW; ++p) {
                    const double xv = Xs[p][ar];
#pragma unroll
                    for (int e = 0; e < 8; ++e) out[e] += xv * Th[p][acg * 8 + e];
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int c = col[acg * 8 + e];
                    if (c >= 0) M[static_cast<int64_t>(c) * k + r0 + ar] = static_cast<float>(out[e]);
                }
            }
            __syncthreads();
        }
    }
}

__global__ __launch_bounds__(256) void jacobi_finalize_kernel(const float* Xtb, const float* Vtb,
                                                              int k, int64_t strideX, int r,
                                                              float* Urb, int64_t strideUr,
                                                              float* sigma, int64_t stride_sigma,
                                                              const int* rotb, int max_sweeps,
                                                              int* info) {
    extern __shared__ unsigned char smem[];
    double* sig = reinterpret_cast<double*>(smem);
    int* perm = reinterpret_cast<int*>(sig + k);
    const int b = blockIdx.x;
    const float* Xt = Xtb + static_cast<int64_t>(b) * strideX;
    const float* Vt = Vtb + static_cast<int64_t>(b) * strideX;
    float* Ur = Urb + static_cast<int64_t>(b) * strideUr;
    const int tid = threadIdx.x;
    for (int c = tid; c < k; c += blockDim.x) {
        double s = 0.0;
        const float* x = Xt + static_cast<int64_t>(c) * k;
        for (int i = 0; i < k; ++i) s += static_cast<double>(x[i]) * static_cast<double>(x[i]);
        sig[c] = sqrt(s);
    }
    __syncthreads();
    // descending by value, ties by index; NaN sorts last
    for (int c = tid; c < k; c += blockDim.x) {
        const double vc = (sig[c] == sig[c]) ? sig[c] : -1.0;
        int rank = 0;
        for (int c2 = 0; c2 < k; ++c2) {
            const double v2 = (sig[c2] == sig[c2]) ? sig[c2] : -1.0;
            rank += (v2 > vc) || (v2 == vc && c2 < c);
        }
        perm[rank] = c;
    }
    __syncthreads();
    if (sigma != nullptr) {
        for (int j = tid; j < r; j += blockDim.x)
            sigma[static_cast<int64_t>(b) * stride_sigma + j] = static_cast<float>(sig[perm[j]]);
    }
    const int64_t total = static_cast<int64_t>(k) * r;
    for (int64_t pos = tid; pos < total; pos += blockDim.x) {
        const int i = static_cast<int>(pos / r);
        const int j = static_cast<int>(pos - static_cast<int64_t>(i) * r);
        Ur[pos] = Vt[static_cast<int64_t>(perm[j]) * k + i];
    }
    if (tid == 0 && info != nullptr) {
        const int* rot = rotb + static_cast<int64_t>(b) * max_sweeps;
        int result = max_sweeps;
        for (int w = 0; w < max_sweeps; ++w) {
            if (rot[w] == 0) { result = 0; break; }
        }
        info[b] = result;
    }
}

}  // namespace

hipError_t launch_jacobi_prepare(const double* R, int k, int64_t strideR, float* Xt, float* Vt,
                                 int64_t strideX, int* rot, int max_sweeps, int batch,
                                 hipStream_t stream) {
    int64_t blocks = (static_cast<int64_t>(k) * k + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(jacobi_prepare_kernel, dim3(static_cast<unsigned>(blocks), batch), dim3(256),
                       0, stream, R, k, strideR, Xt, Vt, strideX, rot, max_sweeps);
    return hipGetLastError();
}

hipError_t launch_jacobi_step(float* Xt, float* Vt, int k, int64_t strideX, int nblocks, int step,
                              int sweep, int* rot, int max_sweeps, double tol, int batch,
                              hipStream_t stream) {
    hipLaunchKernelGGL(jacobi_step_kernel, dim3(nblocks / 2, batch), dim3(JT), 0, stream, Xt, Vt, k,
                       strideX, nblocks, step, sweep, rot, max_sweeps, tol);
    return hipGetLastError();
}

hipError_t launch_jacobi_finalize(const float* Xt, const float* Vt, int k, int64_t strideX, int r,
                                  float* Ur, int64_t strideUr, float* sigma, int64_t stride_sigma,
                                  const int* rot, int max_sweeps, int* info, int batch,
                                  hipStream_t stream) {
    const size_t shmem = static_cast<size_t>(k) * (sizeof(double) + sizeof(int));
    hipLaunchKernelGGL(jacobi_finalize_kernel, dim3(batch), dim3(256), shmem, stream, Xt, Vt, k,
                       strideX, r, Ur, strideUr, sigma, stride_sigma, rot, max_sweeps, info);
    return hipGetLastError();
}

}  // namespace galore
