// Cholesky factorisation of the k x k fp64 Gram matrices and the inverse of the
// factor, for the Cholesky-based orthonormalisation (Q = Y R^-1 with
// R^T R = Y^T Y) that keeps the sketch well conditioned between the products
// of the randomized subspace iteration (Halko et al. 2011, §4.5 re-orthonormal-
// ises after every application of A or A^T), and for the square factor the
// small SVD works on.
//
// One workgroup (512 threads) per matrix; matrices of a batch run side by side.
// Left-looking by blocks of 16 rows: each thread owns one column c of the
// current block row, accumulates the 16 inner products against the rows above
// (their 16-wide slice staged in LDS), the 16 x 16 diagonal block is factored
// in LDS, then each thread finishes its column by forward substitution.
//
// Semi-definite inputs: a pivot d <= tau_rel * (original diagonal) marks the
// column as numerically dependent on the previous ones. Its row of R is set to
// zero (R^T R still reproduces the Gram), and for the inverse that row is
// replaced by the unit row so that R' stays invertible; the caller replaces the
// corresponding column of Q by a generic unit vector (fill_deficient).
#include "common.hpp"

namespace galore {
namespace {

constexpr int CB = 16;    // block rows
constexpr int CT = 512;   // threads
constexpr int CH = 64;    // staged rows per chunk

__global__ __launch_bounds__(CT) void cholesky_kernel(double* Cb, int k, int64_t strideC,
                                                      float* rinvB, double* xinvB,
                                                      int64_t strideInv, int* deficB,
                                                      double tau_rel) {
    const int b = blockIdx.x;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    int* defic = deficB + static_cast<int64_t>(b) * k;
    const int tid = threadIdx.x;
    __shared__ double Rs[CH][CB + 1];
    __shared__ double Sd[CB][CB + 1];
    __shared__ double pinv;
    __shared__ int dfl[CB];

    // ------------------------------------------------------------ factor
    for (int J = 0; J < k; J += CB) {
        const int jb = min(CB, k - J);
        for (int cg = 0; cg < k - J; cg += CT) {
            const int c = J + cg + tid;
            const bool active = c < k;
            double acc[CB];
#pragma unroll
            for (int i = 0; i < CB; ++i) acc[i] = 0.0;
            for (int t0 = 0; t0 < J; t0 += CH) {
                const int tc = min(CH, J - t0);
                for (int idx = tid; idx < CH * CB; idx += CT) {
                    const int tt = idx / CB, i = idx % CB;
                    Rs[tt][i] = (tt < tc && i < jb)
                                    ? C[static_cast<int64_t>(t0 + tt) * k + J + i] : 0.0;
                }
                __syncthreads();
                if (active) {
                    for (int tt = 0; tt < tc; ++tt) {
                        const double rv = C[static_cast<int64_t>(t0 + tt) * k + c];
#pragma unroll
                        for (int i = 0; i < CB; ++i) acc[i] += Rs[tt][i] * rv;
                    }
                }
                __syncthreads();
            }
            if (active) {
#pragma unroll
                for (int i = 0; i < CB; ++i)
                    if (i < jb) acc[i] = C[static_cast<int64_t>(J + i) * k + c] - acc[i];
            }
            if (cg == 0) {
                if (tid < jb) {
#pragma unroll
                    for (int i = 0; i < CB; ++i)
                        if (i < jb) Sd[i][tid] = acc[i];
                }
                __syncthreads();
                for (int i = 0; i < jb; ++i) {
                    if (tid == 0) {
                        const double d = Sd[i][i];
                        const double corig = C[static_cast<int64_t>(J + i) * k + J + i];
                        const bool def = (d <= tau_rel * corig);   // NaN compares false
                        dfl[i] = def ? 1 : 0;
                        const double rii = def ? 0.0 : sqrt(d);
                        Sd[i][i] = rii;
                        pinv = def ? 0.0 : 1.0 / rii;
                    }
                    __syncthreads();
                    if (tid > i && tid < jb) Sd[i][tid] *= pinv;
                    __syncthreads();
                    if (tid < CB * CB) {
                        const int i2 = i + 1 + tid / CB;
                        const int c2 = tid % CB;
                        if (i2 < jb && c2 >= i2 && c2 < jb) Sd[i2][c2] -= Sd[i][i2] * Sd[i][c2];
                    }
                    __syncthreads();
                }
            }
            if (active) {
                if (c < J + jb) {
                    const int cc = c - J;
#pragma unroll
                    for (int i = 0; i < CB; ++i)
                        if (i <= cc) C[static_cast<int64_t>(J + i) * k + c] = Sd[i][cc];
                } else {
#pragma unroll
                    for (int i = 0; i < CB; ++i) {
                        if (i < jb) {
                            double x = acc[i];
#pragma unroll
                            for (int tt = 0; tt < CB; ++tt)
                                if (tt < i) x -= Sd[tt][i] * acc[tt];
                            acc[i] = dfl[i] ? 0.0 : x / Sd[i][i];
                            C[static_cast<int64_t>(J + i) * k + c] = acc[i];
                        }
                    }
                }
            }
            __syncthreads();
        }
        if (tid < jb) defic[J + tid] = dfl[tid];
        __syncthreads();
    }

    if (rinvB == nullptr) return;

    // ------------------------------------------------------------ inverse of R'
    double* X = xinvB + static_cast<int64_t>(b) * strideInv;
    float* Ri = rinvB + static_cast<int64_t>(b) * strideInv;
    const int nblk = (k + CB - 1) / CB;
    for (int bi = nblk - 1; bi >= 0; --bi) {
        const int I = bi * CB;
        const int ib = min(CB, k - I);
        for (int idx = tid; idx < CB * CB; idx += CT) {
            const int i = idx / CB, c2 = idx % CB;
            double v = 0.0;
            if (i < ib && c2 < ib && c2 >= i) {
                if (defic[I + i]) v = (i == c2) ? 1.0 : 0.0;
                else v = C[static_cast<int64_t>(I + i) * k + I + c2];
            }
            Sd[i][c2] = v;
        }
        __syncthreads();
        for (int cg = 0; cg < k; cg += CT) {
            const int c = cg + tid;
            const bool active = c < k;
            double acc[CB];
#pragma unroll
            for (int i = 0; i < CB; ++i) acc[i] = 0.0;
            for (int t0 = I + ib; t0 < k; t0 += CH) {
                const int tc = min(CH, k - t0);
                for (int idx = tid; idx < CH * CB; idx += CT) {
                    const int tt = idx / CB, i = idx % CB;
                    Rs[tt][i] = (tt < tc && i < ib && !defic[I + i])
                                    ? C[static_cast<int64_t>(I + i) * k + t0 + tt] : 0.0;
                }
                __syncthreads();
                if (active && c >= I) {
                    for (int tt = 0; tt < tc; ++tt) {
                        const int t = t0 + tt;
                        if (t > c) break;
                        const double xv = X[static_cast<int64_t>(t) * k + c];
#pragma unroll
                        for (int i = 0; i < CB; ++i) acc[i] += Rs[tt][i] * xv;
                    }
                }
                __syncthreads();
            }
            if (active) {
                if (c < I) {
#pragma unroll
                    for (int i = 0; i < CB; ++i)
                        if (i < ib) Ri[static_cast<int64_t>(I + i) * k + c] = 0.0f;
                } else {
                    double x[CB];
#pragma unroll
                    for (int i = CB - 1; i >= 0; --i) {
                        x[i] = 0.0;
                        if (i < ib) {
                            double v = ((I + i) == c ? 1.0 : 0.0) - acc[i];
#pragma unroll
                            for (int t2 = 0; t2 < CB; ++t2)
                                if (t2 > i && t2 < ib) v -= Sd[i][t2] * x[t2];
                            x[i] = v / Sd[i][i];
                        }
                    }
#pragma unroll
                    for (int i = 0; i < CB; ++i) {
                        if (i < ib) {
                            X[static_cast<int64_t>(I + i) * k + c] = x[i];
                            Ri[static_cast<int64_t>(I + i) * k + c] = static_cast<float>(x[i]);
                        }
                    }
                }
            }
            __syncthreads();
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
                           int64_t strideInv, int* defic, double tau_rel, int batch,
                           hipStream_t stream) {
    hipLaunchKernelGGL(cholesky_kernel, dim3(batch), dim3(CT), 0, stream, C, k, strideC, rinv32,
                       xinv, strideInv, defic, tau_rel);
    return hipGetLastError();
}

hipError_t launch_fill_deficient(float* Q, int rows, int k, int64_t strideQ, const int* defic,
                                 int batch, hipStream_t stream) {
    hipLaunchKernelGGL(fill_deficient_kernel, dim3(k, batch), dim3(256), 0, stream, Q, rows, k,
                       strideQ, defic);
    return hipGetLastError();
}

}  // namespace galore
