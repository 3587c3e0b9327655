// fp64 refinement of the small SVD's singular vectors (Ogita & Aishima 2018,
// "Iterative refinement for symmetric eigenvalue decomposition", Japan J.
// Indust. Appl. Math. 35: one Newton-type correction built from matrix
// products only).
//
// The left singular vectors of B (paper §4.1.2: the direct SVD of the small
// projected matrix of Halko et al. 2011) are the eigenvectors of
// H = B B^T = R^T R, with R the fp64 Cholesky factor of the exact Gram. The
// block Jacobi (jacobi.hip) produces them in fp32: its columns live in fp32 and
// each of the ~330 rotations a column takes adds fp32 rounding, so two
// singular vectors whose singular values differ by a relative 3e-4 (the gap at
// r of a spectrum whose tail is in the noise bulk) stay mixed at the 1e-3
// level. Each refinement step, with X the current vectors (columns, fp32):
//   T = R X                         (fp64)
//   S = T^T T = X^T H X,  G = X^T X (fp64, symmetric)
//   lambda_i = S_ii / G_ii
//   E_ij = (S_ij + lambda_j (delta_ij - G_ij)) / (lambda_j - lambda_i)   i != j
//        = (delta_ij - G_ij) / 2                                          otherwise
//   X <- X + X E
// where "otherwise" is the diagonal and every pair whose correction would
// exceed 0.1 (a pair of near-equal eigenvalues, whose individual vectors are
// not determined by H at this accuracy: it is only re-orthogonalised). The
// step leaves the span of the r leading vectors accurate to second order in
// the error before it (1e-3 -> about 1e-6), but their basis only orthonormal to
// first order (the corrections of near-equal pairs are large); so the r vectors
// of largest lambda are then re-orthonormalised among themselves, which keeps
// their span: X_r <- X_r (I - D / 2), D = X_r^T X_r - I, first-order Lowdin
// (orthonormal to O(|D|^2)).
//
// Layouts (per matrix, k x k, ld = k): X is stored by columns (Xt: column c
// contiguous, i.e. X^T row-major, as the Jacobi stores its columns); R is the
// row-major upper triangle left by the Cholesky (the lower triangle holds
// stale data and is masked); T is stored as T^T; S and G are full symmetric;
// E is stored transposed (Et[j][i] = E_ij).
// T, S and G are formed on the fp64 matrix cores (v_mfma_f64_16x16x4f64), the
// two updates' small correction sums on the fp32 ones (v_mfma_f32_16x16x4f32,
// see refine_update_kernel), all in 96 x 96 output tiles staged through LDS
// (below).
#include <float.h>

#include "common.hpp"

namespace galore {
namespace {

constexpr double kEmax = 0.1;

typedef double f64x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// ---- 96 x 96 tiles through LDS ------------------------------------------------
// A workgroup of four waves computes a 96 x 96 output tile (wave (wm, wn): rows
// 48 wm .. + 47, columns 48 wn .. + 47, as 3 x 3 blocks of 16 x 16 on the fp64
// matrix cores). Per 32-deep chunk of the contraction both operands are staged
// in LDS as [t][m] / [t][n] (fp64, rows of 112 doubles: the four 16-lane
// groups of an operand read fall on two disjoint halves of the 64 banks), the
// next chunk is loaded into registers while the current one is multiplied.
// 96 divides the sketch width 1056 of the 4096 x 11008 workload.
constexpr int QT = 96;              // output tile
constexpr int QK = 32;              // contraction chunk
constexpr int QP = 112;             // LDS row pitch (doubles)

// chunk item e (0..2) of thread tid: 96 rows x 8 groups of 4 contraction indices
__device__ __forceinline__ void q_item(int tid, int e, int& row, int& tq) {
    const int q = tid + 256 * e;
    tq = q / QT;
    row = q - tq * QT;
}

// 4 consecutive values M[row * ld + t .. t + 3] in fp64, zero outside row < nr, t < nt
template <typename T>
__device__ __forceinline__ f64x4 quad_at(const T* M, int64_t ld, int row, int t, int nr, int nt, bool vec) {
    f64x4 p = {0.0, 0.0, 0.0, 0.0};
    if (row < nr) {
        const T* q = M + static_cast<int64_t>(row) * ld + t;
        if (vec && t + 3 < nt) {
            if constexpr (sizeof(T) == 8) {
                const f64x2 a = *reinterpret_cast<const f64x2*>(q), b = *reinterpret_cast<const f64x2*>(q + 2);
                p = f64x4{a[0], a[1], b[0], b[1]};
            } else {
                const f32x4 f = *reinterpret_cast<const f32x4*>(q);
                p = f64x4{f[0], f[1], f[2], f[3]};
            }
        } else {
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (t + v < nt) p[v] = static_cast<double>(q[v]);
        }
    }
    return p;
}

// acc[x][y] += sum over the chunk in LDS (As[t][m], Bs[t][n]); fp64 or fp32
// matrix cores by the element type
template <typename T, typename V>
__device__ __forceinline__ void q_mma(const T* As, const T* Bs, V acc[3][3], int wm, int wn, int lane) {
    const int l16 = lane & 15, g = lane >> 4;
#pragma unroll
    for (int s = 0; s < QK / 4; ++s) {
        const int t = 4 * s + g;
        T a[3], b[3];
#pragma unroll
        for (int x = 0; x < 3; ++x) {
            a[x] = As[t * QP + 48 * wm + 16 * x + l16];
            b[x] = Bs[t * QP + 48 * wn + 16 * x + l16];
        }
#pragma unroll
        for (int x = 0; x < 3; ++x)
#pragma unroll
            for (int y = 0; y < 3; ++y) {
                if constexpr (sizeof(T) == 8)
                    acc[x][y] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[x], b[y], acc[x][y], 0, 0, 0);
                else
                    acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[x], b[y], acc[x][y], 0, 0, 0);
            }
    }
}

// C[m][n] = sum_{t < kc} A[m][t] B[n][t] for m, n < nn (both operands row-major
// with the contraction index contiguous, row pitch ld; C row pitch ldc). TRI: B
// is upper triangular (B[n][t] = 0 for t < n; the stored lower part is
// ignored). SYM: A == B, only the upper tiles are computed and each off-diagonal
// tile is also stored mirrored, so C is full and symmetric. Every matrix whose
// flag is 0 is skipped. grid: (tiles, batch).
template <typename TA, typename TB, bool TRI, bool SYM>
__global__ __launch_bounds__(256) void refine_nt_kernel(const TA* Ab, int64_t strideA, const TB* Bb, int64_t strideB,
                                                        double* Cb, int64_t strideC, int nn, int kc, int64_t ld,
                                                        int64_t ldc, const int* flags) {
    const int b = blockIdx.y;
    if (flags[b] == 0) return;
    const int nt = (nn + QT - 1) / QT;
    int tm, tn;
    if (SYM) {
        int idx = blockIdx.x, u = 0;
        while (idx >= nt - u) {
            idx -= nt - u;
            ++u;
        }
        tm = u;
        tn = u + idx;
    } else {
        tm = blockIdx.x / nt;
        tn = blockIdx.x % nt;
    }
    __shared__ __attribute__((aligned(16))) double As[QK * QP];
    __shared__ __attribute__((aligned(16))) double Bs[QK * QP];
    const TA* A = Ab + static_cast<int64_t>(b) * strideA;
    const TB* B = Bb + static_cast<int64_t>(b) * strideB;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    const int m0 = QT * tm, n0 = QT * tn;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const bool vec = (ld & 3) == 0;
    // B[n][t] = 0 for t < n: the tile needs t >= n0 only (a multiple of 4)
    const int tlo = TRI ? n0 : 0;
    f64x4 ra[3], rb[3];
    auto fetch = [&](int t0) {
#pragma unroll
        for (int e = 0; e < 3; ++e) {
            int row, tq;
            q_item(tid, e, row, tq);
            const int t = t0 + 4 * tq;
            ra[e] = quad_at(A, ld, m0 + row, t, nn, kc, vec);
            f64x4 q = quad_at(B, ld, n0 + row, t, nn, kc, vec);
            if (TRI) {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (t + v < n0 + row) q[v] = 0.0;
            }
            rb[e] = q;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int e = 0; e < 3; ++e) {
            int row, tq;
            q_item(tid, e, row, tq);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                As[(4 * tq + v) * QP + row] = ra[e][v];
                Bs[(4 * tq + v) * QP + row] = rb[e][v];
            }
        }
    };
    f64x4 acc[3][3];
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y) acc[x][y] = f64x4{0.0, 0.0, 0.0, 0.0};
    fetch(tlo);
    for (int t0 = tlo; t0 < kc; t0 += QK) {
        stash();
        __syncthreads();
        if (t0 + QK < kc) fetch(t0 + QK);
        q_mma(As, Bs, acc, wm, wn, lane);
        __syncthreads();
    }
    // accumulator register v of block (x, y): row 48 wm + 16 x + 4 v + g, column 48 wn + 16 y + l16
    const int l16 = lane & 15, g = lane >> 4;
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = m0 + 48 * wm + 16 * x + 4 * v + g;
                const int col = n0 + 48 * wn + 16 * y + l16;
                if (row < nn && col < nn) {
                    C[static_cast<int64_t>(row) * ldc + col] = acc[x][y][v];
                    if (SYM && tm != tn) C[static_cast<int64_t>(col) * ldc + row] = acc[x][y][v];
                }
            }
}

// lambda_i = S_ii / G_ii; grid (batch), flags as above
__global__ __launch_bounds__(256) void refine_lambda_kernel(const double* Sb, const double* Gb, int64_t strideKK,
                                                            double* lamb, int k, const int* flags) {
    const int b = blockIdx.x;
    if (flags[b] == 0) return;
    const double* S = Sb + static_cast<int64_t>(b) * strideKK;
    const double* G = Gb + static_cast<int64_t>(b) * strideKK;
    double* lam = lamb + static_cast<int64_t>(b) * k;
    for (int i = threadIdx.x; i < k; i += blockDim.x) {
        const int64_t d = static_cast<int64_t>(i) * k + i;
        lam[i] = S[d] / G[d];
    }
}

// Et[j][i] = E_ij (see the file comment); grid (ceil(k*k / 256), batch)
__global__ __launch_bounds__(256) void refine_e_kernel(const double* Sb, const double* Gb, int64_t strideKK,
                                                       const double* lamb, double* Etb, int k, const int* flags) {
    const int b = blockIdx.y;
    if (flags[b] == 0) return;
    const int64_t pos = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (pos >= static_cast<int64_t>(k) * k) return;
    const int j = static_cast<int>(pos / k);
    const int i = static_cast<int>(pos - static_cast<int64_t>(j) * k);
    const double* S = Sb + static_cast<int64_t>(b) * strideKK;
    const double* G = Gb + static_cast<int64_t>(b) * strideKK;
    const double* lam = lamb + static_cast<int64_t>(b) * k;
    // S and G are symmetric: row j, column i holds S_ij and G_ij
    const double rr = ((i == j) ? 1.0 : 0.0) - G[pos];
    double e = 0.5 * rr;
    if (i != j) {
        const double lj = lam[j], li = lam[i];
        const double num = S[pos] + lj * rr;
        const double dl = lj - li;
        if (dl != 0.0 && fabs(num) <= kEmax * fabs(dl)) e = num / dl;
    }
    Etb[static_cast<int64_t>(b) * strideKK + pos] = e;
}

// Xn[j][a] = X[j][a] + alpha sum_{i < nn} (M[j][i] - shift delta_ji) X[i][a] for
// j < nn, a < kc: rows of X are vectors (row pitch ld), M is nn x nn fp64 (row
// pitch ldm). With Ur != nullptr the result is written transposed,
// Ur[a][j] (row pitch ldu), instead of into Xn. 96 x 96 tiles as above: A = M
// (contraction index contiguous), B = X (rows of the contraction index).
// P = float: the correction sum runs on the fp32 matrix cores (twice the fp64
// rate). M - shift I is formed in fp64 and then rounded to fp32; both updates
// of a step apply a small correction (entries of E are at most 0.1 and of
// order 1e-5 outside near-equal pairs; D - I is the orthogonality error), so
// the fp32 sum's error, of order 2^-24 sum_i |M - shift I|_ji |X_ia|, stays far
// under the fp32 rounding of X itself, to which the sum is added once, in
// fp64, before the result is rounded to fp32.
template <typename P>
__global__ __launch_bounds__(256) void refine_update_kernel(const double* Mb, int64_t strideM, int64_t ldm,
                                                            const float* Xb, int64_t strideX, float* Xnb, int nn,
                                                            int kc, int64_t ld, double alpha, double shift,
                                                            float* Urb, int64_t strideUr, int64_t ldu,
                                                            const int* flags) {
    const int b = blockIdx.y;
    if (flags[b] == 0) return;
    const int ntm = (nn + QT - 1) / QT, ntn = (kc + QT - 1) / QT;
    const int tm = blockIdx.x / ntn, tn = blockIdx.x % ntn;
    if (tm >= ntm) return;
    __shared__ __attribute__((aligned(16))) P As[QK * QP];
    __shared__ __attribute__((aligned(16))) P Bs[QK * QP];
    const double* M = Mb + static_cast<int64_t>(b) * strideM;
    const float* X = Xb + static_cast<int64_t>(b) * strideX;
    const int m0 = QT * tm, n0 = QT * tn;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const bool vecm = (ldm & 3) == 0, vecx = (ld & 3) == 0;
    f64x4 ra[3], rb[3];
    // B items: 32 contraction rows x 24 groups of 4 columns
    auto fetch = [&](int t0) {
#pragma unroll
        for (int e = 0; e < 3; ++e) {
            int row, tq;
            q_item(tid, e, row, tq);
            const int t = t0 + 4 * tq;
            f64x4 p = quad_at(M, ldm, m0 + row, t, nn, nn, vecm);
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (t + v == m0 + row) p[v] -= shift;
            ra[e] = p;
            const int q = tid + 256 * e;
            const int bt = q / (QT / 4), bg = q - bt * (QT / 4);
            rb[e] = quad_at(X, ld, t0 + bt, n0 + 4 * bg, nn, kc, vecx);
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int e = 0; e < 3; ++e) {
            int row, tq;
            q_item(tid, e, row, tq);
#pragma unroll
            for (int v = 0; v < 4; ++v) As[(4 * tq + v) * QP + row] = static_cast<P>(ra[e][v]);
            const int q = tid + 256 * e;
            const int bt = q / (QT / 4), bg = q - bt * (QT / 4);
            if constexpr (sizeof(P) == 8) {
                *reinterpret_cast<f64x2*>(&Bs[bt * QP + 4 * bg]) = f64x2{rb[e][0], rb[e][1]};
                *reinterpret_cast<f64x2*>(&Bs[bt * QP + 4 * bg + 2]) = f64x2{rb[e][2], rb[e][3]};
            } else {
                *reinterpret_cast<f32x4*>(&Bs[bt * QP + 4 * bg]) =
                    f32x4{static_cast<float>(rb[e][0]), static_cast<float>(rb[e][1]), static_cast<float>(rb[e][2]),
                          static_cast<float>(rb[e][3])};
            }
        }
    };
    typedef P pv4 __attribute__((ext_vector_type(4)));
    pv4 acc[3][3];
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y) acc[x][y] = pv4{P(0), P(0), P(0), P(0)};
    fetch(0);
    for (int t0 = 0; t0 < nn; t0 += QK) {
        stash();
        __syncthreads();
        if (t0 + QK < nn) fetch(t0 + QK);
        q_mma(As, Bs, acc, wm, wn, lane);
        __syncthreads();
    }
    const int l16 = lane & 15, g = lane >> 4;
    // register v of a 16 x 16 block: row 4 v + g (fp64), 4 g + v (fp32)
    auto out_row = [&](int x, int v) { return m0 + 48 * wm + 16 * x + ((sizeof(P) == 8) ? 4 * v + g : 4 * g + v); };
    auto out_col = [&](int y) { return n0 + 48 * wn + 16 * y + l16; };
    // the lane's 36 values of X read together before any store (one memory
    // latency, not one per value); outside the nn x kc block they read its
    // last row or column, whose values are not stored
    float xo[3][3][4];
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                xo[x][y][v] = X[static_cast<int64_t>(min(out_row(x, v), nn - 1)) * ld + min(out_col(y), kc - 1)];
    // a tile inside the block stores without per-value branches (the two
    // choices below are uniform): at the joins of such branches the compiler
    // waits for every memory operation in flight again
    auto value = [&](int x, int y, int v) {
        return static_cast<float>(static_cast<double>(xo[x][y][v]) + alpha * static_cast<double>(acc[x][y][v]));
    };
    float* Ur = (Urb != nullptr) ? Urb + static_cast<int64_t>(b) * strideUr : nullptr;
    float* Xn = (Urb != nullptr) ? nullptr : Xnb + static_cast<int64_t>(b) * strideX;
    if (m0 + QT <= nn && n0 + QT <= kc) {
        if (Ur != nullptr) {
#pragma unroll
            for (int x = 0; x < 3; ++x)
#pragma unroll
                for (int y = 0; y < 3; ++y)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        Ur[static_cast<int64_t>(out_col(y)) * ldu + out_row(x, v)] = value(x, y, v);
        } else {
#pragma unroll
            for (int x = 0; x < 3; ++x)
#pragma unroll
                for (int y = 0; y < 3; ++y)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        Xn[static_cast<int64_t>(out_row(x, v)) * ld + out_col(y)] = value(x, y, v);
        }
        return;
    }
#pragma unroll
    for (int x = 0; x < 3; ++x)
#pragma unroll
        for (int y = 0; y < 3; ++y)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = out_row(x, v), col = out_col(y);
                if (row < nn && col < kc) {
                    if (Ur != nullptr)
                        Ur[static_cast<int64_t>(col) * ldu + row] = value(x, y, v);
                    else
                        Xn[static_cast<int64_t>(row) * ld + col] = value(x, y, v);
                }
            }
}

// Order the refined vectors by lambda (descending, ties by index; a NaN last):
// permb[b][j] = index of the j-th, sigma_j = sqrt(lambda). One thread per
// vector, its rank the number of vectors ahead of it; grid (ceil(k / 256),
// batch), each workgroup with the matrix's lambdas in LDS (dynamic: k doubles).
__global__ __launch_bounds__(256) void refine_rank_kernel(const double* lamb, int k, int r, int* permb, float* sigma,
                                                          int64_t stride_sigma, const int* flags) {
    const int b = blockIdx.y;
    if (flags[b] == 0) return;
    extern __shared__ unsigned char smem[];
    double* lam = reinterpret_cast<double*>(smem);
    for (int i = threadIdx.x; i < k; i += blockDim.x) {
        const double v = lamb[static_cast<int64_t>(b) * k + i];
        lam[i] = (v == v) ? v : -DBL_MAX;
    }
    __syncthreads();
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= k) return;
    const double vc = lam[c];
    int rank = 0;
    for (int c2 = 0; c2 < k; ++c2) rank += (lam[c2] > vc) || (lam[c2] == vc && c2 < c);
    permb[static_cast<int64_t>(b) * k + rank] = c;
    if (sigma != nullptr && rank < r)
        sigma[static_cast<int64_t>(b) * stride_sigma + rank] = static_cast<float>(sqrt(fmax(vc, 0.0)));
}

// Xs[j][:] = Xt[perm[j]][:] for the r leading vectors; grid (r, batch)
__global__ __launch_bounds__(256) void refine_gather_kernel(const float* Xtb, int64_t strideX, const int* permb, int k,
                                                            float* Xsb, const int* flags) {
    const int b = blockIdx.y;
    if (flags[b] == 0) return;
    const int j = blockIdx.x;
    const int c = permb[static_cast<int64_t>(b) * k + j];
    const float* x = Xtb + static_cast<int64_t>(b) * strideX + static_cast<int64_t>(c) * k;
    float* y = Xsb + static_cast<int64_t>(b) * strideX + static_cast<int64_t>(j) * k;
    for (int i = threadIdx.x; i < k; i += blockDim.x) y[i] = x[i];
}

}  // namespace

hipError_t launch_refine(const double* R, int64_t strideR, float* Xa, float* Xb, int64_t strideX, double* T,
                         double* S, double* G, int64_t strideKK, double* lam, int* perm, int k, int r, float* Ur,
                         int64_t strideUr, float* sigma, int64_t stride_sigma, const int* flags, int batch,
                         hipStream_t stream) {
    const int nt = (k + QT - 1) / QT, ntr = (r + QT - 1) / QT;
    const dim3 full(nt * nt, batch), upper(nt * (nt + 1) / 2, batch);
    // one step: T^T = X^T R^T (C[c][a] = sum_t Xa[c][t] R[a][t], R upper triangular)
    hipLaunchKernelGGL((refine_nt_kernel<float, double, true, false>), full, dim3(256), 0, stream, Xa, strideX, R,
                       strideR, T, strideKK, k, k, static_cast<int64_t>(k), static_cast<int64_t>(k), flags);
    // S = T^T T and G = X^T X, both full symmetric
    hipLaunchKernelGGL((refine_nt_kernel<double, double, false, true>), upper, dim3(256), 0, stream, T, strideKK, T,
                       strideKK, S, strideKK, k, k, static_cast<int64_t>(k), static_cast<int64_t>(k), flags);
    hipLaunchKernelGGL((refine_nt_kernel<float, float, false, true>), upper, dim3(256), 0, stream, Xa, strideX, Xa,
                       strideX, G, strideKK, k, k, static_cast<int64_t>(k), static_cast<int64_t>(k), flags);
    hipLaunchKernelGGL(refine_lambda_kernel, dim3(batch), dim3(256), 0, stream, S, G, strideKK, lam, k, flags);
    // E^T into T's buffer (T is no longer needed), then Xb = Xa + Xa E
    const int64_t kk = static_cast<int64_t>(k) * k;
    hipLaunchKernelGGL(refine_e_kernel, dim3(static_cast<unsigned>((kk + 255) / 256), batch), dim3(256), 0, stream, S,
                       G, strideKK, lam, T, k, flags);
    hipLaunchKernelGGL(refine_update_kernel<float>, full, dim3(256), 0, stream, T, strideKK, static_cast<int64_t>(k),
                       Xa, strideX, Xb, k, k, static_cast<int64_t>(k), 1.0, 0.0, static_cast<float*>(nullptr),
                       static_cast<int64_t>(0), static_cast<int64_t>(0), flags);
    // the r vectors of largest lambda, in order, into the rows of Xa
    hipLaunchKernelGGL(refine_rank_kernel, dim3((k + 255) / 256, batch), dim3(256), static_cast<size_t>(k) * sizeof(double),
                       stream, lam, k, r, perm, sigma, stride_sigma, flags);
    hipLaunchKernelGGL(refine_gather_kernel, dim3(r, batch), dim3(256), 0, stream, Xb, strideX, perm, k, Xa, flags);
    // their Gram D = X_r^T X_r (into S), then Ur = (X_r (I - (D - I) / 2))^T
    const dim3 upper_r(ntr * (ntr + 1) / 2, batch), full_r(ntr * nt, batch);
    hipLaunchKernelGGL((refine_nt_kernel<float, float, false, true>), upper_r, dim3(256), 0, stream, Xa, strideX, Xa,
                       strideX, S, strideKK, r, k, static_cast<int64_t>(k), static_cast<int64_t>(r), flags);
    hipLaunchKernelGGL(refine_update_kernel<float>, full_r, dim3(256), 0, stream, S, strideKK,
                       static_cast<int64_t>(r), Xa, strideX, static_cast<float*>(nullptr), r, k,
                       static_cast<int64_t>(k), -0.5, 1.0, Ur, strideUr, static_cast<int64_t>(r), flags);
    return hipGetLastError();
}

}  // namespace galore
