// Memory-bound kernels of the hot path.
//
//  * sign_fix: canonical sign of each projector column (paper §4.1.3 and its
//    footnote: singular vectors are defined up to sign; the entry of largest
//    magnitude, lowest row on exact ties, is made positive).
//  * lowrank_adam: the low-rank Adam update (paper §3 moment equations and the
//    bias correction of paper Alg. 1) streaming R, M, V in and M, V, N out:
//    24 bytes per element, one pass over HBM, 16-byte vector accesses.
//  * align: the subspace switch's column-sign matching of a new projector to
//    the previous one (paper §4.1.3 sign indeterminacy).
//  * copy_rows: batched strided copy (the previous projector and first moment
//    kept for the switch inside the scheduled step).
#include "common.hpp"

namespace galore {
namespace {

constexpr int SF_COLS = 64;
constexpr int SF_GROUPS = 4;

// A workgroup owns 64 columns of one matrix: thread t scans column quad
// t & 15 (four columns, one 16-byte load per row when the rows are aligned) over
// the rows t >> 4, t >> 4 + 16, ... in increasing order, four rows in flight;
// the 16 row groups are reduced through LDS (larger magnitude, then lower
// row), and the columns whose chosen entry is negative are negated in a
// second pass with the same access pattern.
constexpr int SF_QUADS = SF_COLS / 4;                 // 16 column quads
constexpr int SF_RGROUPS = SF_COLS * SF_GROUPS / SF_QUADS;   // 16 row groups

__global__ __launch_bounds__(SF_COLS* SF_GROUPS) void sign_fix_kernel(float* Pb, int rows, int r,
                                                                      int64_t ldp, int64_t strideP, int vec) {
    const int b = blockIdx.y;
    float* P = Pb + static_cast<int64_t>(b) * strideP;
    const int cq = threadIdx.x % SF_QUADS, rg = threadIdx.x / SF_QUADS;
    const int c0 = blockIdx.x * SF_COLS + 4 * cq;
    __shared__ float best_abs[SF_RGROUPS][SF_COLS];
    __shared__ int best_row[SF_RGROUPS][SF_COLS];
    __shared__ float flip[SF_COLS];
    const bool full = vec && c0 + 4 <= r;
    auto quad = [&](int i) {
        const float* q = P + static_cast<int64_t>(i) * ldp + c0;
        f32x4 x;
        if (full) {
            x = *reinterpret_cast<const f32x4*>(q);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] = (c0 + e < r) ? q[e] : 0.0f;
        }
        return x;
    };
    float ba[4] = {-1.0f, -1.0f, -1.0f, -1.0f};
    int br[4] = {0x7fffffff, 0x7fffffff, 0x7fffffff, 0x7fffffff};
    if (c0 < r) {
        int i = rg;
        for (; i + 3 * SF_RGROUPS < rows; i += 4 * SF_RGROUPS) {
            f32x4 x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = quad(i + u * SF_RGROUPS);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = fabsf(x[u][e]);
                    if (a > ba[e]) { ba[e] = a; br[e] = i + u * SF_RGROUPS; }   // rows in increasing order
                }
        }
        for (; i < rows; i += SF_RGROUPS) {
            const f32x4 x = quad(i);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float a = fabsf(x[e]);
                if (a > ba[e]) { ba[e] = a; br[e] = i; }
            }
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        best_abs[rg][4 * cq + e] = ba[e];
        best_row[rg][4 * cq + e] = br[e];
    }
    __syncthreads();
    if (threadIdx.x < SF_COLS) {
        const int tc = threadIdx.x, c = blockIdx.x * SF_COLS + tc;
        float a = best_abs[0][tc];
        int rr = best_row[0][tc];
        for (int g = 1; g < SF_RGROUPS; ++g) {
            const float a2 = best_abs[g][tc];
            const int r2 = best_row[g][tc];
            if (a2 > a || (a2 == a && r2 < rr)) { a = a2; rr = r2; }
        }
        float f = 1.0f;
        if (c < r && rr < rows && P[static_cast<int64_t>(rr) * ldp + c] < 0.0f) f = -1.0f;
        flip[tc] = f;
    }
    __syncthreads();
    if (c0 >= r) return;
    const float f[4] = {flip[4 * cq], flip[4 * cq + 1], flip[4 * cq + 2], flip[4 * cq + 3]};
    if (f[0] > 0.0f && f[1] > 0.0f && f[2] > 0.0f && f[3] > 0.0f) return;
    for (int i = rg; i < rows; i += SF_RGROUPS) {
        float* q = P + static_cast<int64_t>(i) * ldp + c0;
        if (full) {
            f32x4 x = *reinterpret_cast<const f32x4*>(q);
#pragma unroll
            for (int e = 0; e < 4; ++e) x[e] *= f[e];
            *reinterpret_cast<f32x4*>(q) = x;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (c0 + e < r && f[e] < 0.0f) q[e] = -q[e];
        }
    }
}

// Subspace switch: a workgroup owns 64 columns of one matrix (4 row groups);
// the overlap <p_old_j, p_new_j> is summed in fp64 from the exact fp32
// products, and column j of the new projector is negated in place when it is
// negative (zero or NaN keeps the sign; paper §4.1.3 sign indeterminacy).
__global__ __launch_bounds__(SF_COLS* SF_GROUPS) void align_kernel(const float* Pob, int64_t ldo, int64_t strideO,
                                                                   float* Pnb, int64_t ldn, int64_t strideN,
                                                                   int rows, int r, int* flipsb) {
    const int b = blockIdx.y;
    const float* Po = Pob + static_cast<int64_t>(b) * strideO;
    float* Pn = Pnb + static_cast<int64_t>(b) * strideN;
    const int tc = threadIdx.x & (SF_COLS - 1);
    const int grp = threadIdx.x / SF_COLS;
    const int c = blockIdx.x * SF_COLS + tc;
    __shared__ double part[SF_GROUPS][SF_COLS];
    __shared__ float flip[SF_COLS];
    double acc = 0.0;
    if (c < r) {
#pragma unroll 8
        for (int i = grp; i < rows; i += SF_GROUPS)
            acc += static_cast<double>(Po[static_cast<int64_t>(i) * ldo + c]) *
                   static_cast<double>(Pn[static_cast<int64_t>(i) * ldn + c]);
    }
    part[grp][tc] = acc;
    __syncthreads();
    if (grp == 0) {
        double ov = part[0][tc];
        for (int g = 1; g < SF_GROUPS; ++g) ov += part[g][tc];
        const int f = (ov < 0.0) ? 1 : 0;
        flip[tc] = f ? -1.0f : 1.0f;
        if (c < r && flipsb != nullptr) flipsb[static_cast<int64_t>(b) * r + c] = f;
    }
    __syncthreads();
    if (c < r && flip[tc] < 0.0f) {
        for (int i = grp; i < rows; i += SF_GROUPS) {
            float* q = Pn + static_cast<int64_t>(i) * ldn + c;
            *q = -*q;
        }
    }
}

__device__ __forceinline__ void adam_elem(float g, float& m, float& v, float& n, float beta1,
                                          float beta2, float om1, float om2, float bc1, float bc2,
                                          float eps) {
    m = beta1 * m + om1 * g;
    v = beta2 * v + om2 * (g * g);
    const float mhat = m / bc1;
    const float vhat = v / bc2;
    n = mhat / (sqrtf(vhat) + eps);
}

// Contiguous state: flat index over batch * rows * cols, 16-byte vectors.
__global__ __launch_bounds__(256) void adam_flat_kernel(const float* R, float* M, float* V, float* N,
                                                       int64_t total, float beta1, float beta2,
                                                       float eps, float bc1, float bc2) {
    const float om1 = 1.0f - beta1;
    const float om2 = 1.0f - beta2;
    const int64_t nvec = total / 4;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    const f32x4* R4 = reinterpret_cast<const f32x4*>(R);
    f32x4* M4 = reinterpret_cast<f32x4*>(M);
    f32x4* V4 = reinterpret_cast<f32x4*>(V);
    f32x4* N4 = reinterpret_cast<f32x4*>(N);
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < nvec; i += stride) {
        const f32x4 g = __builtin_nontemporal_load(R4 + i);
        f32x4 m = __builtin_nontemporal_load(M4 + i);
        f32x4 v = __builtin_nontemporal_load(V4 + i);
        f32x4 n;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float me = m[e], ve = v[e], ne;
            adam_elem(g[e], me, ve, ne, beta1, beta2, om1, om2, bc1, bc2, eps);
            m[e] = me;
            v[e] = ve;
            n[e] = ne;
        }
        __builtin_nontemporal_store(m, M4 + i);
        __builtin_nontemporal_store(v, V4 + i);
        __builtin_nontemporal_store(n, N4 + i);
    }
    // tail (total % 4 elements)
    const int64_t tail0 = nvec * 4;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (gid < total - tail0) {
        const int64_t i = tail0 + gid;
        float m = M[i], v = V[i], n;
        adam_elem(R[i], m, v, n, beta1, beta2, om1, om2, bc1, bc2, eps);
        M[i] = m;
        V[i] = v;
        N[i] = n;
    }
}

// Strided state (ld > cols or padded batch stride); R and N share one layout,
// M and V another.
__global__ __launch_bounds__(256) void adam_strided_kernel(const float* R, float* N, int64_t ldrn, int64_t srn,
                                                          float* M, float* V, int64_t ldmv, int64_t smv,
                                                          int64_t rows, int64_t cols, float beta1, float beta2,
                                                          float eps, float bc1, float bc2) {
    const float om1 = 1.0f - beta1;
    const float om2 = 1.0f - beta2;
    const int64_t b = blockIdx.y;
    const int64_t per = rows * cols;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < per;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = e / cols;
        const int64_t j = e - i * cols;
        const int64_t o = b * srn + i * ldrn + j;
        const int64_t om = b * smv + i * ldmv + j;
        float m = M[om], v = V[om], n;
        adam_elem(R[o], m, v, n, beta1, beta2, om1, om2, bc1, bc2, eps);
        M[om] = m;
        V[om] = v;
        N[o] = n;
    }
}

// Batched row copy: rows x cols of each matrix from (lds, strideS) to (ldd, strideD).
__global__ __launch_bounds__(256) void copy_rows_kernel(const float* src, int64_t lds, int64_t strideS, float* dst,
                                                       int64_t ldd, int64_t strideD, int rows, int cols) {
    const int64_t b = blockIdx.y;
    for (int i = blockIdx.x; i < rows; i += gridDim.x) {
        const float* s = src + b * strideS + static_cast<int64_t>(i) * lds;
        float* d = dst + b * strideD + static_cast<int64_t>(i) * ldd;
        for (int j = threadIdx.x; j < cols; j += blockDim.x) d[j] = s[j];
    }
}

}  // namespace

hipError_t launch_sign_fix(float* P, int rows, int r, int64_t ldp, int64_t strideP, int batch,
                           hipStream_t stream) {
    dim3 grid((r + SF_COLS - 1) / SF_COLS, batch);
    const int vec = (ldp % 4 == 0) && (batch == 1 || strideP % 4 == 0) && (reinterpret_cast<uintptr_t>(P) % 16 == 0);
    hipLaunchKernelGGL(sign_fix_kernel, grid, dim3(SF_COLS * SF_GROUPS), 0, stream, P, rows, r, ldp,
                       strideP, vec);
    return hipGetLastError();
}

hipError_t launch_align(const float* P_old, int64_t ldo, int64_t strideO, float* P_new, int64_t ldn, int64_t strideN,
                        int rows, int r, int* flips, int batch, hipStream_t stream) {
    dim3 grid((r + SF_COLS - 1) / SF_COLS, batch);
    hipLaunchKernelGGL(align_kernel, grid, dim3(SF_COLS * SF_GROUPS), 0, stream, P_old, ldo, strideO, P_new, ldn,
                       strideN, rows, r, flips);
    return hipGetLastError();
}

hipError_t launch_copy_rows(const float* src, int64_t lds, int64_t strideS, float* dst, int64_t ldd,
                            int64_t strideD, int rows, int cols, int batch, hipStream_t stream) {
    const int blocks = rows < 65536 ? rows : 65536;
    hipLaunchKernelGGL(copy_rows_kernel, dim3(blocks, batch), dim3(256), 0, stream, src, lds, strideS, dst, ldd,
                       strideD, rows, cols);
    return hipGetLastError();
}

hipError_t launch_adam(const float* R, float* M, float* V, float* N, int64_t rows, int64_t cols,
                       int64_t ld, int64_t stride, int batch, float beta1, float beta2, float eps,
                       float bc1, float bc2, hipStream_t stream) {
    return launch_adam2(R, N, ld, stride, M, V, ld, stride, rows, cols, batch, beta1, beta2, eps, bc1, bc2, stream);
}

hipError_t launch_adam2(const float* R, float* N, int64_t ldrn, int64_t srn, float* M, float* V, int64_t ldmv,
                        int64_t smv, int64_t rows, int64_t cols, int batch, float beta1, float beta2, float eps,
                        float bc1, float bc2, hipStream_t stream) {
    const bool contiguous = (ldrn == cols) && (ldmv == cols) && (srn == rows * cols) && (smv == rows * cols);
    const bool aligned = ((reinterpret_cast<uintptr_t>(R) | reinterpret_cast<uintptr_t>(M) |
                           reinterpret_cast<uintptr_t>(V) | reinterpret_cast<uintptr_t>(N)) & 15) == 0;
    if (contiguous && aligned) {
        const int64_t total = rows * cols * batch;
        // One 16-byte vector per thread and a grid that covers the whole array: a
        // capped grid-stride launch (65536 workgroups) streams about 11% slower
        // at 64 x 1024 x 11008 (5.19 vs 5.83 TB/s measured).
        int64_t blocks = (total / 4 + 255) / 256;
        if (blocks < 1) blocks = 1;
        if (blocks > 0x7fffffff) blocks = 0x7fffffff;
        hipLaunchKernelGGL(adam_flat_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                           R, M, V, N, total, beta1, beta2, eps, bc1, bc2);
    } else {
        int64_t blocks = (rows * cols + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        hipLaunchKernelGGL(adam_strided_kernel, dim3(static_cast<unsigned>(blocks), batch), dim3(256),
                           0, stream, R, N, ldrn, srn, M, V, ldmv, smv, rows, cols, beta1, beta2, eps, bc1, bc2);
    }
    return hipGetLastError();
}

}  // namespace galore
