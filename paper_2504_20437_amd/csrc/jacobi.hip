// Small SVD of the projected matrix B = Q^T A (k x l) in the randomized SVD
// (Halko et al. 2011, direct SVD of the small matrix; paper §4.1.2).
//
// The left singular vectors of B are the eigenvectors of B B^T = Z^T Z with
// Z = A^T Q = B^T. The host factors that Gram in fp64 as R^T R (Cholesky), so
// they are also the right singular vectors of the k x k factor R. They are
// found by one-sided (Hestenes) Jacobi on the columns of X = R, accumulating
// the rotations in V (X V = U Sigma, V = left singular vectors of B).
//
// Blocked for the GPU: the k columns form blocks of 32; a round-robin
// tournament pairs the blocks so that every step is a set of disjoint pairs,
// one workgroup per (pair, matrix). A workgroup
//   1. forms the 64 x 64 fp64 Gram of its two blocks on the fp64 matrix cores
//      (v_mfma_f64_16x16x4f64) from row chunks staged in LDS;
//   2. skips the pair if every column pair is already orthogonal to the
//      tolerance (relative off-diagonal), otherwise
//   3. reduces the small Gram with cyclic two-sided Jacobi in LDS (fp64,
//      parallel ordering: 63 rounds of 32 disjoint rotations per inner sweep,
//      each round one read-modify-write of the Gram and of the accumulated
//      rotation Theta), and
//   4. applies Theta to its 64 columns of X and of V on the fp32 matrix cores
//      (v_mfma_f32_32x32x2f32), 64-row chunks staged through LDS.
// A sweep is nb - 1 steps; the matrix has converged when a whole sweep
// rotates nothing (rotation counts per sweep live in device memory, so no
// host synchronisation is needed). X and V are stored transposed (column c
// contiguous) so that a block of columns is a contiguous slab.
#include "common.hpp"

namespace galore {
namespace {

constexpr int JB = kJacobiBlock;   // columns per block
constexpr int JW = 2 * JB;         // columns per pair (64)
constexpr int JT = 256;            // threads (4 waves)
constexpr int GR = 32;             // rows per Gram chunk
constexpr int AR = 64;             // rows per apply chunk
constexpr int PD = JW + 1;         // padded LDS row
constexpr int kInnerSweeps = 1;    // inner sweeps over the 64 x 64 Gram per step

static_assert(JW == 64, "the pair kernels assume 64 columns per pair");

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

// LDS plan (two 64 x 65 fp64 regions, 66.6 KB, two workgroups per CU):
//   region A: Gram G (phases 1-3), then fp32 Theta + fp32 X chunk (phase 4)
//   region B: fp64 row chunks for the Gram (phase 1), then Theta (phase 3)
__global__ __launch_bounds__(JT, 2) void jacobi_step_kernel(float* Xtb, float* Vtb, int k,
                                                            int64_t strideX, int nb, int step,
                                                            int sweep, int* rotb, int max_sweeps,
                                                            double tol) {
    const int b = blockIdx.y;
    int* rot = rotb + static_cast<int64_t>(b) * max_sweeps;
    if (sweep > 0 && rot[sweep - 1] == 0) return;     // converged in an earlier sweep
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = blockIdx.x;
    const int bi = ring_slot(h, step, nb);
    const int bj = ring_slot(nb - 1 - h, step, nb);

    float* Xt = Xtb + static_cast<int64_t>(b) * strideX;
    float* Vt = Vtb + static_cast<int64_t>(b) * strideX;

    __shared__ double regA[JW][PD];
    __shared__ double regB[JW][PD];
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

    // ---- 1. Gram of the pair's 64 columns on the fp64 matrix cores ---------
    double (*G)[PD] = regA;
    double (*Xs)[PD] = regB;            // Xs[t][w], t < GR
    {
        // waves 0, 1, 2 own the quadrants (0,0), (0,1), (1,1) of the 64 x 64 Gram
        const int qa = (wave == 2) ? 1 : 0;
        const int qb = (wave == 0) ? 0 : 1;
        f64x4 acc[2][2];
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) acc[x][y] = f64x4{0.0, 0.0, 0.0, 0.0};
        const int l16 = lane & 15;
        const int lk = lane >> 4;
        for (int r0 = 0; r0 < k; r0 += GR) {
            const int rc = min(GR, k - r0);
            for (int idx = tid; idx < JW * GR; idx += JT) {
                const int w = idx / GR, t = idx % GR;
                const int c = col[w];
                Xs[t][w] = (c >= 0 && t < rc) ? static_cast<double>(Xt[static_cast<int64_t>(c) * k + r0 + t]) : 0.0;
            }
            __syncthreads();
            if (wave < 3) {
#pragma unroll
                for (int kk = 0; kk < GR; kk += 4) {
                    const double a0 = Xs[kk + lk][32 * qa + l16];
                    const double a1 = Xs[kk + lk][32 * qa + 16 + l16];
                    const double b0 = Xs[kk + lk][32 * qb + l16];
                    const double b1 = Xs[kk + lk][32 * qb + 16 + l16];
                    acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc[0][0], 0, 0, 0);
                    acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc[0][1], 0, 0, 0);
                    acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc[1][0], 0, 0, 0);
                    acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc[1][1], 0, 0, 0);
                }
            }
            __syncthreads();
        }
        // fp64 16x16 block layout: lane holds column (lane & 15); accumulator
        // register v holds row 4 v + (lane >> 4).
        if (wave < 3) {
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int i = 32 * qa + 16 * x + 4 * v + lk;
                        const int j = 32 * qb + 16 * y + l16;
                        G[i][j] = acc[x][y][v];
                        if (qa != qb) G[j][i] = acc[x][y][v];
                    }
        }
        __syncthreads();
    }

    // ---- 2. convergence test: largest relative off-diagonal ----------------
    {
        double off = 0.0;
        for (int idx = tid; idx < JW * JW; idx += JT) {
            const int p = idx / JW, q = idx % JW;
            if (q > p) {
                const double dd = G[p][p] * G[q][q];
                if (dd > 0.0) {
                    const double rel = fabs(G[p][q]) / sqrt(dd);
                    off = (rel > off || rel != rel) ? rel : off;
                }
            }
        }
        for (int o = 32; o > 0; o >>= 1) {
            const double other = __shfl_xor(off, o);
            off = (other > off || other != other) ? other : off;
        }
        if (lane == 0) red[wave] = off;
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
    }

    // ---- 3. reduce the 64 x 64 Gram: cyclic two-sided Jacobi ---------------
    double (*Th)[PD] = regB;
    for (int idx = tid; idx < JW * JW; idx += JT) {
        const int i = idx / JW, j = idx % JW;
        Th[i][j] = (i == j) ? 1.0 : 0.0;
    }
    __syncthreads();
    for (int isw = 0; isw < kInnerSweeps; ++isw) {
        if (tid == 0) any_rot = 0;
        __syncthreads();
        for (int st = 0; st < JW - 1; ++st) {
            if (tid < JW / 2) {
                int p = ring_slot(tid, st, JW);
                int q = ring_slot(JW - 1 - tid, st, JW);
                if (p > q) { const int tmp = p; p = q; q = tmp; }
                const double a = G[p][p], bb = G[q][q], gm = G[p][q];
                double c = 1.0, s = 0.0;
                if (fabs(gm) > 1e-15 * sqrt(a * bb)) {
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
            // G <- J^T G J by 2 x 2 blocks (row pair ha, column pair hb);
            // column p' = c p - s q, column q' = s p + c q
            for (int idx = tid; idx < (JW / 2) * (JW / 2); idx += JT) {
                const int ha = idx / (JW / 2), hb = idx % (JW / 2);
                const int pa = pp[ha], qa2 = qq[ha], pb = pp[hb], qb2 = qq[hb];
                const double ca = cs[ha], sa = sn[ha], cb = cs[hb], sb = sn[hb];
                const double g00 = G[pa][pb], g01 = G[pa][qb2], g10 = G[qa2][pb], g11 = G[qa2][qb2];
                const double r00 = ca * g00 - sa * g10, r01 = ca * g01 - sa * g11;
                const double r10 = sa * g00 + ca * g10, r11 = sa * g01 + ca * g11;
                G[pa][pb] = cb * r00 - sb * r01;
                G[pa][qb2] = sb * r00 + cb * r01;
                G[qa2][pb] = cb * r10 - sb * r11;
                G[qa2][qb2] = sb * r10 + cb * r11;
            }
            // Theta <- Theta J
            for (int idx = tid; idx < (JW / 2) * JW; idx += JT) {
                const int hh = idx / JW, row = idx % JW;
                const int p = pp[hh], q = qq[hh];
                const double c = cs[hh], s = sn[hh];
                const double tp = Th[row][p], tq = Th[row][q];
                Th[row][p] = c * tp - s * tq;
                Th[row][q] = s * tp + c * tq;
            }
            __syncthreads();
        }
        const int done = (any_rot == 0);
        __syncthreads();
        if (done) break;
    }

    // ---- 4. X_P <- X_P Theta, V_P <- V_P Theta on the fp32 matrix cores ----
    float (*Tf)[PD] = reinterpret_cast<float (*)[PD]>(&regA[0][0]);            // 64 x 65 fp32
    float (*Xc)[PD] = reinterpret_cast<float (*)[PD]>(&regA[0][0]) + JW;       // 64 x 65 fp32
    for (int idx = tid; idx < JW * JW; idx += JT) {
        const int i = idx / JW, j = idx % JW;
        Tf[i][j] = static_cast<float>(Th[i][j]);
    }
    __syncthreads();
    const int tm = wave >> 1, tn = wave & 1;
    const int l32 = lane & 31, lk2 = lane >> 5;
    for (int pass = 0; pass < 2; ++pass) {
        float* M = (pass == 0) ? Xt : Vt;
        for (int r0 = 0; r0 < k; r0 += AR) {
            const int rc = min(AR, k - r0);
            for (int idx = tid; idx < JW * AR; idx += JT) {
                const int w = idx / AR, t = idx % AR;
                const int c = col[w];
                Xc[w][t] = (c >= 0 && t < rc) ? M[static_cast<int64_t>(c) * k + r0 + t] : 0.0f;
            }
            __syncthreads();
            f32x16 acc;
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll 8
            for (int kk = 0; kk < JW; kk += 2) {
                const float a = Xc[kk + lk2][32 * tm + l32];   // A[t][w] = X[t][w]
                const float bv = Tf[kk + lk2][32 * tn + l32];  // B[w][c] = Theta[w][c]
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv, acc, 0, 0, 0);
            }
            __syncthreads();
            // 32x32 block layout: lane holds column (lane & 31) and rows
            // (v & 3) + 8 (v >> 2) + 4 (lane >> 5) for accumulator register v.
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int t = 32 * tm + (v & 3) + 8 * (v >> 2) + 4 * lk2;
                Xc[32 * tn + l32][t] = acc[v];
            }
            __syncthreads();
            for (int idx = tid; idx < JW * AR; idx += JT) {
                const int w = idx / AR, t = idx % AR;
                const int c = col[w];
                if (c >= 0 && t < rc) M[static_cast<int64_t>(c) * k + r0 + t] = Xc[w][t];
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
