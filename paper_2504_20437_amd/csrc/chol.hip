// Cholesky factorisation of the k x k fp64 Gram matrices and the inverse of the
// factor, for the Cholesky-based orthonormalisation (Q = Y R^-1 with
// R^T R = Y^T Y) that keeps the sketch well conditioned between the products
// of the randomized subspace iteration (Halko et al. 2011, §4.5 re-orthonormal-
// ises after every application of A or A^T), and for the square factor the
// small SVD works on.
//
// Right-looking, blocked by CB = 64 rows; every launch covers all matrices of
// the batch (grid z / y = matrix), so the chip is filled by (tiles x batch)
// workgroups rather than one workgroup per matrix:
//   for each block row J:
//     diag     factor the 64 x 64 diagonal block in LDS (unblocked, fp64) and
//              invert it (D_J = R'_JJ^-1, kept in the fp64 inverse buffer);
//     panel    R_JT = D_J^T C_JT for every block column T > J;
//     trailing C_T1T2 -= R_JT1^T R_JT2 on the upper tiles T1 <= T2 right of J.
//   inverse  X = R'^-1 by levels d = T - I: X_IT = -D_I sum_{I<U<=T} R_IU X_UT,
//            written in fp64 and as fp32 (lower triangle zero) for the GEMM
//            that applies it.
// R overwrites the upper triangle of C; the lower triangle is not used.
//
// Semi-definite inputs: a pivot d <= tau_rel * (original diagonal) marks the
// column as numerically dependent on the previous ones. Its row of R is set to
// zero (R^T R still reproduces the Gram), and for the inverse that row is
// replaced by the unit row so that R' stays invertible; the caller replaces the
// corresponding column of Q by a generic unit vector (fill_deficient).
#include "common.hpp"

namespace galore {
namespace {

constexpr int CB = 64;     // block size
constexpr int CT = 256;    // threads per workgroup (16 x 16, 4 x 4 outputs each)
constexpr int LP = CB + 1; // padded LDS row

// acc[i][j] += sum_t As[t][ty + 16 i] * Bs[t][tx + 16 j], t < kk
__device__ __forceinline__ void tile_tn(double (*As)[LP], double (*Bs)[LP], int kk, double acc[4][4],
                                        int ty, int tx) {
    for (int t = 0; t < kk; ++t) {
        double a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = As[t][ty + 16 * i];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = Bs[t][tx + 16 * j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
    }
}

// S[r][c] = M[(r0 + r) * ld + c0 + c] for r < nr, c < nc; zero elsewhere
__device__ __forceinline__ void load_tile(double (*S)[LP], const double* M, int64_t ld, int r0, int c0,
                                          int nr, int nc) {
    for (int idx = threadIdx.x; idx < CB * CB; idx += CT) {
        const int r = idx / CB, c = idx % CB;
        S[r][c] = (r < nr && c < nc) ? M[static_cast<int64_t>(r0 + r) * ld + c0 + c] : 0.0;
    }
}

// S[c][r] = M[(r0 + r) * ld + c0 + c] (transposed load)
__device__ __forceinline__ void load_tile_t(double (*S)[LP], const double* M, int64_t ld, int r0, int c0,
                                            int nr, int nc) {
    for (int idx = threadIdx.x; idx < CB * CB; idx += CT) {
        const int r = idx / CB, c = idx % CB;
        S[c][r] = (r < nr && c < nc) ? M[static_cast<int64_t>(r0 + r) * ld + c0 + c] : 0.0;
    }
}

__global__ __launch_bounds__(CT) void chol_diag_kernel(double* Cb, int k, int64_t strideC, int J,
                                                       double* diag0b, int* deficB, double* Xb,
                                                       float* Rib, int64_t strideInv, double tau_rel) {
    const int b = blockIdx.x;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    double* diag0 = diag0b + static_cast<int64_t>(b) * k;
    int* defic = deficB + static_cast<int64_t>(b) * k;
    double* X = Xb + static_cast<int64_t>(b) * strideInv;
    const int tid = threadIdx.x;
    const int j0 = J * CB;
    const int jb = min(CB, k - j0);
    __shared__ double S[CB][LP];
    __shared__ double T[CB][LP];
    __shared__ int dfl[CB];
    __shared__ double corig[CB];

    if (J == 0) {
        for (int i = tid; i < k; i += CT) diag0[i] = C[static_cast<int64_t>(i) * k + i];
    }
    load_tile(S, C, k, j0, j0, jb, jb);
    // the original diagonal of this block, staged once (the pivot loop below
    // is serial and must not wait on global memory)
    if (tid < jb) corig[tid] = (J == 0) ? C[static_cast<int64_t>(j0 + tid) * k + j0 + tid] : diag0[j0 + tid];
    __syncthreads();
    // one barrier per column: every thread derives the pivot itself, the
    // trailing update reads row i unscaled and scales it on the fly, and row i
    // is rescaled in place after the barrier (no later column reads it)
    const int tx = tid & 15, ty = tid >> 4;
    for (int i = 0; i < jb; ++i) {
        const double d = S[i][i];
        const bool def = (d <= tau_rel * corig[i]);   // NaN compares false
        const double rii = def ? 0.0 : sqrt(d);
        const double pv = def ? 0.0 : 1.0 / rii;
        // rank-1 update of the trailing upper triangle, 16 x 16 threads
        // striding over it (no division by the runtime extent)
        for (int a = i + 1 + ty; a < jb; a += 16) {
            const double sa = S[i][a] * pv;
            for (int c = i + 1 + tx; c < jb; c += 16)
                if (c >= a) S[a][c] -= sa * (S[i][c] * pv);
        }
        __syncthreads();
        if (tid > i && tid < jb) S[i][tid] *= pv;
        if (tid == 0) {
            S[i][i] = rii;
            dfl[i] = def ? 1 : 0;
        }
    }
    __syncthreads();
    for (int idx = tid; idx < CB * CB; idx += CT) {
        const int r = idx / CB, c = idx % CB;
        if (r < jb && c < jb && c >= r) C[static_cast<int64_t>(j0 + r) * k + j0 + c] = S[r][c];
    }
    if (tid < jb) defic[j0 + tid] = dfl[tid];
    // D = R'^-1 of the block (unit rows for deficient pivots), upper
    // triangular, by rows from the bottom: lane c of the first wave owns column
    // c and forms D[i][c] from the entries D[t][c], t > i, it wrote before
    // (D[t][c] = 0 for t > c, so every lane runs the same loop).
    if (tid < CB) {
        const int c = tid;
        for (int t = 0; t < CB; ++t) T[t][c] = 0.0;
        for (int i = jb - 1; i >= 0; --i) {
            // four partial sums, eight independent LDS reads in flight
            double acc4[4] = {0.0, 0.0, 0.0, 0.0};
            int t = i + 1;
            for (; t + 8 <= jb; t += 8) {
                double sv[8], tv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    sv[e] = S[i][t + e];
                    tv[e] = T[t + e][c];
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) acc4[e & 3] = fma(sv[e], tv[e], acc4[e & 3]);
            }
            for (; t < jb; ++t) acc4[0] = fma(S[i][t], T[t][c], acc4[0]);
            const double acc = (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
            double v;
            if (dfl[i]) v = (c == i) ? 1.0 : 0.0;                     // unit row: x_i = delta_ic
            else v = (c < i) ? 0.0 : (((c == i) ? 1.0 : 0.0) - acc) / S[i][i];
            if (c < jb) T[i][c] = v;
        }
    }
    __syncthreads();
    for (int idx = tid; idx < CB * CB; idx += CT) {
        const int r = idx / CB, c = idx % CB;
        if (r < jb && c < jb) {
            const double v = (c >= r) ? T[r][c] : 0.0;
            X[static_cast<int64_t>(j0 + r) * k + j0 + c] = v;
            if (Rib != nullptr) Rib[static_cast<int64_t>(b) * strideInv + static_cast<int64_t>(j0 + r) * k + j0 + c] =
                static_cast<float>(v);
        }
    }
}

// R_JT = D_J^T C_JT (deficient rows zero), in place in C, for T = J + 1 + blockIdx.x
__global__ __launch_bounds__(CT) void chol_panel_kernel(double* Cb, int k, int64_t strideC, int J,
                                                        const int* deficB, const double* Xb,
                                                        int64_t strideInv) {
    const int b = blockIdx.y;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    const int* defic = deficB + static_cast<int64_t>(b) * k;
    const double* X = Xb + static_cast<int64_t>(b) * strideInv;
    const int j0 = J * CB;
    const int jb = min(CB, k - j0);
    const int c0 = (J + 1 + blockIdx.x) * CB;
    const int cb = min(CB, k - c0);
    __shared__ double As[CB][LP];
    __shared__ double Bs[CB][LP];
    load_tile(As, X, k, j0, j0, jb, jb);   // As[t][i] = D[t][i]
    load_tile(Bs, C, k, j0, c0, jb, cb);   // Bs[t][c] = C_JT[t][c]
    __syncthreads();
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    double acc[4][4] = {};
    tile_tn(As, Bs, jb, acc, ty, tx);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = ty + 16 * i;
        if (r >= jb) continue;
        const bool def = defic[j0 + r] != 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = tx + 16 * j;
            if (c < cb) C[static_cast<int64_t>(j0 + r) * k + c0 + c] = def ? 0.0 : acc[i][j];
        }
    }
}

// C_T1T2 -= R_JT1^T R_JT2 for J < T1 <= T2; blockIdx.x enumerates the upper tiles
__global__ __launch_bounds__(CT) void chol_trailing_kernel(double* Cb, int k, int64_t strideC, int J,
                                                           int nb) {
    const int b = blockIdx.y;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    const int n = nb - J - 1;
    // blockIdx.x -> (u, v) with 0 <= u <= v < n, row-major over the upper triangle
    int idx = blockIdx.x, u = 0;
    while (idx >= n - u) {
        idx -= n - u;
        ++u;
    }
    const int v = u + idx;
    const int j0 = J * CB;
    const int jb = min(CB, k - j0);
    const int r0 = (J + 1 + u) * CB, rb = min(CB, k - r0);
    const int c0 = (J + 1 + v) * CB, cb = min(CB, k - c0);
    __shared__ double As[CB][LP];
    __shared__ double Bs[CB][LP];
    load_tile(As, C, k, j0, r0, jb, rb);
    load_tile(Bs, C, k, j0, c0, jb, cb);
    __syncthreads();
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    double acc[4][4] = {};
    tile_tn(As, Bs, jb, acc, ty, tx);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = ty + 16 * i;
        if (r >= rb) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = tx + 16 * j;
            if (c < cb && (u != v || c >= r)) C[static_cast<int64_t>(r0 + r) * k + c0 + c] -= acc[i][j];
        }
    }
}

// Level d of the inverse: tile (I, I + d) for I = blockIdx.x.
__global__ __launch_bounds__(CT) void chol_inverse_level_kernel(const double* Cb, int k, int64_t strideC,
                                                                int d, double* Xb, float* Rib,
                                                                int64_t strideInv) {
    const int b = blockIdx.y;
    const double* C = Cb + static_cast<int64_t>(b) * strideC;
    double* X = Xb + static_cast<int64_t>(b) * strideInv;
    float* Ri = Rib + static_cast<int64_t>(b) * strideInv;
    const int I = blockIdx.x, Jc = I + d;
    const int i0 = I * CB, ib = min(CB, k - i0);
    const int c0 = Jc * CB, cb = min(CB, k - c0);
    __shared__ double As[CB][LP];
    __shared__ double Bs[CB][LP];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    // S = sum_{U = I+1 .. Jc} R_IU X_UJc
    double acc[4][4] = {};
    for (int U = I + 1; U <= Jc; ++U) {
        const int u0 = U * CB, ub = min(CB, k - u0);
        load_tile_t(As, C, k, i0, u0, ib, ub);   // As[t][a] = R_IU[a][t]
        load_tile(Bs, X, k, u0, c0, ub, cb);     // Bs[t][c] = X_UJc[t][c]
        __syncthreads();
        tile_tn(As, Bs, ub, acc, ty, tx);
        __syncthreads();
    }
    // X_IJc = -D_I S
    load_tile_t(As, X, k, i0, i0, ib, ib);       // As[t][a] = D_I[a][t]
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) Bs[ty + 16 * i][tx + 16 * j] = acc[i][j];
    __syncthreads();
    double out[4][4] = {};
    tile_tn(As, Bs, ib, out, ty, tx);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = ty + 16 * i;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = tx + 16 * j;
            if (r < ib && c < cb) {
                const double v = -out[i][j];
                X[static_cast<int64_t>(i0 + r) * k + c0 + c] = v;
                if (Rib != nullptr) {
                    Ri[static_cast<int64_t>(i0 + r) * k + c0 + c] = static_cast<float>(v);
                }
            }
            // the mirrored (lower) tile of the fp32 inverse is zero
            if (Rib != nullptr && r < cb && c < ib) Ri[static_cast<int64_t>(c0 + r) * k + i0 + c] = 0.0f;
        }
    }
}

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    // splitmix64 finaliser (Steele, Lea, Flood 2014)
    z += 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void fill_deficient_kernel(float* Qb, int rows, int k,
                                                             int64_t strideQ, const int* deficB) {
    const int b = blockIdx.y;
    const int j = blockIdx.x;
    if (!deficB[static_cast<int64_t>(b) * k + j]) return;
    float* Q = Qb + static_cast<int64_t>(b) * strideQ;
    const float scale = 1.0f / sqrtf(static_cast<float>(rows));
    for (int i = threadIdx.x; i < rows; i += blockDim.x) {
        const uint64_t h = mix64((static_cast<uint64_t>(j) << 32) | static_cast<uint32_t>(i));
        Q[static_cast<int64_t>(i) * k + j] = (h & 1ULL) ? scale : -scale;
    }
}

}  // namespace

hipError_t launch_cholesky(double* C, int k, int64_t strideC, float* rinv32, double* xinv,
                           int64_t strideInv, int* defic, double* diag0, double tau_rel, int batch,
                           hipStream_t stream) {
    const int nb = (k + CB - 1) / CB;
    for (int J = 0; J < nb; ++J) {
        hipLaunchKernelGGL(chol_diag_kernel, dim3(batch), dim3(CT), 0, stream, C, k, strideC, J, diag0,
                           defic, xinv, rinv32, strideInv, tau_rel);
        const int n = nb - J - 1;
        if (n > 0) {
            hipLaunchKernelGGL(chol_panel_kernel, dim3(n, batch), dim3(CT), 0, stream, C, k, strideC, J,
                               defic, xinv, strideInv);
            hipLaunchKernelGGL(chol_trailing_kernel, dim3(n * (n + 1) / 2, batch), dim3(CT), 0, stream, C,
                               k, strideC, J, nb);
        }
    }
    if (rinv32 != nullptr) {
        for (int d = 1; d < nb; ++d)
            hipLaunchKernelGGL(chol_inverse_level_kernel, dim3(nb - d, batch), dim3(CT), 0, stream, C, k,
                               strideC, d, xinv, rinv32, strideInv);
    }
    return hipGetLastError();
}

hipError_t launch_fill_deficient(float* Q, int rows, int k, int64_t strideQ, const int* defic,
                                 int batch, hipStream_t stream) {
    hipLaunchKernelGGL(fill_deficient_kernel, dim3(k, batch), dim3(256), 0, stream, Q, rows, k,
                       strideQ, defic);
    return hipGetLastError();
}

}  // namespace galore
