// Cholesky factorisation of the k x k Gram matrices (fp64) and the inverse of the
// factor, for the Cholesky-based orthonormalisation (Q = Y R^-1 with
// R^T R = Y^T Y) that keeps the sketch well conditioned between the products
// of the randomized subspace iteration (Halko et al. 2011, §4.5 re-orthonormal-
// ises after every application of A or A^T), and for the square factor the
// small SVD works on.
//
// Right-looking, blocked by CB = 64 rows; every launch covers all matrices of
// the batch (grid y = matrix), so the chip is filled by (tiles x batch)
// workgroups rather than one workgroup per matrix. The inverse X = R'^-1 is
// built alongside, column block by column block (X R' = I gives
// X_IJ = -(sum_{U<J} X_IU R_UJ) D_J), its partial sums P_IJ accumulated by the
// trailing launches in X's own upper blocks, so no separate inverse phase runs:
//   diag 0   factor the 64 x 64 diagonal block 0 in registers (unblocked,
//            fp64) and invert it (D_0 = R'_00^-1, kept in X's diagonal block);
//   for each block row J:
//     panel+X  R_JT = D_J^T C_JT for every block column T > J, and block column J
//              of the inverse, X_IJ = -P_IJ D_J for I < J (fp64 and fp32, the
//              fp32 copy's lower tiles zero for the GEMM that applies it);
//     trailing C_T1T2 -= R_JT1^T R_JT2 on the upper tiles J < T1 <= T2, and
//              P_IT (+)= X_IJ R_JT for I <= J < T; the workgroup of tile
//              (J + 1, J + 1) then factors and inverts that diagonal block
//              (step J + 1's diagonal), whose last update it just made.
// The panel, inverse, trailing and partial-sum tiles are 64 x 64 x 64 products
// on the fp64 matrix cores, operands loaded from memory straight into
// registers. Two launches per block row (with the factor's inverse or without).
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
constexpr int CT = 256;    // threads per workgroup (4 waves)

__device__ __forceinline__ void zero_acc(f64x4 acc[2][2]) {
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = f64x4{0.0, 0.0, 0.0, 0.0};
}

typedef double f64x2 __attribute__((ext_vector_type(2)));

// (M[row * ld + col], M[row * ld + col + 1]) with zeros outside row < nr,
// col < nc; one 16-byte load when vec (even ld and offsets)
__device__ __forceinline__ f64x2 ld_pair(const double* M, int64_t ld, int row, int col, int nr, int nc,
                                         bool vec) {
    f64x2 p = {0.0, 0.0};
    if (row < nr) {
        const double* q = M + static_cast<int64_t>(row) * ld + col;
        if (vec && col + 1 < nc) {
            p = *reinterpret_cast<const f64x2*>(q);
        } else {
            if (col < nc) p[0] = q[0];
            if (col + 1 < nc) p[1] = q[1];
        }
    }
    return p;
}

// Register-direct 64 x 64 x 64 product for the tile kernels: wave (wm, wn)
// owns output rows 32 wm + 2 i + bi and columns 32 wn + 2 j + bj (i, j < 16,
// bi, bj < 2), so each lane's A (B) operands for the two row (column) blocks
// are one 16-byte pair; step s of the contraction takes rows 4 s + (lane >> 4)
// of the two row-major operand panels Ap (t x rows) and Bp (t x cols).
// Accumulator register v of block (bi, bj) holds row 32 wm + 2 (4 v + (lane >> 4)) + bi,
// column 32 wn + 2 (lane & 15) + bj.
__device__ __forceinline__ void mma64_pairs(const double* Ap, const double* Bp, int64_t ld, int nt, int na,
                                            int nbc, bool vec, f64x4 acc[2][2], int wm, int wn, int lane) {
    const int l16 = lane & 15, lk = lane >> 4;
    // four groups of four steps, the next group's operands in flight while the
    // current one is multiplied (keeps the kernels within 128 registers)
    f64x2 av[2][4], bv[2][4];
    auto load = [&](int g, int buf) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int t = 4 * (4 * g + i) + lk;
            av[buf][i] = ld_pair(Ap, ld, t, 32 * wm + 2 * l16, nt, na, vec);
            bv[buf][i] = ld_pair(Bp, ld, t, 32 * wn + 2 * l16, nt, nbc, vec);
        }
    };
    load(0, 0);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        if (g + 1 < 4) load(g + 1, (g + 1) & 1);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                for (int bj = 0; bj < 2; ++bj)
                    acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[g & 1][i][bi], bv[g & 1][i][bj],
                                                                       acc[bi][bj], 0, 0, 0);
    }
}

// Factor the diagonal block J and invert its factor, one workgroup per matrix.
// The 64 x 64 block lives in registers, thread (ty, tx) holding the entries
// (ty + 16 q, tx + 16 w); each pivot step broadcasts one row (and, for the
// inverse, one column) through a ping-pong LDS buffer, so a step costs one
// barrier and no LDS read-modify-write.
//  * factor (right-looking): pivot d = S_ii; d <= tau_rel * (original diagonal)
//    marks a dependent column, whose row of R is zero; otherwise
//    R_ii = sqrt(d), R_ic = S_ic / R_ii and S_ac -= R_ia R_ic for a, c > i.
//  * inverse D = R'^-1 (R' = R with unit rows for the dependent pivots), by
//    columns from the last: row i of D is final once rows t > i are
//    eliminated from it, D_i = X_i / R'_ii, then X_a -= R_ai D_i for a < i.
// (the body of one matrix's diagonal step; every thread of the workgroup calls it)
__device__ __forceinline__ void diag_block(double* C, int k, int J, double* diag0, int* defic, double* X, float* Ri,
                                           double tau_rel) {
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int j0 = J * CB;
    const int jb = min(CB, k - j0);
    __shared__ double rowb[2][CB];
    __shared__ double colb[2][CB];
    __shared__ double piv[CB];
    __shared__ int dfl[CB];
    __shared__ double corig[CB];

    if (J == 0) {
        for (int i = tid; i < k; i += CT) diag0[i] = C[static_cast<int64_t>(i) * k + i];
    }
    // the original diagonal of this block, staged once (the pivot loop below
    // is serial and must not wait on global memory)
    if (tid < jb) corig[tid] = (J == 0) ? C[static_cast<int64_t>(j0 + tid) * k + j0 + tid] : diag0[j0 + tid];
    // only the upper triangle (c >= a) is live; the lower one is loaded as it
    // stands and never read
    double s[4][4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const int a = ty + 16 * q, c = tx + 16 * w;
            s[q][w] = (a < jb && c < jb) ? C[static_cast<int64_t>(j0 + a) * k + j0 + c] : 0.0;
        }
    __syncthreads();

#pragma unroll
    for (int ib = 0; ib < 4; ++ib) {
        for (int i16 = 0; i16 < 16; ++i16) {
            const int i = 16 * ib + i16;
            if (i >= jb) break;
            const int buf = i & 1;
            if (ty == i16) {
#pragma unroll
                for (int w = 0; w < 4; ++w) rowb[buf][tx + 16 * w] = s[ib][w];
            }
            __syncthreads();
            const double d = rowb[buf][i];
            const bool def = (d <= tau_rel * corig[i]);   // NaN compares false
            const double rii = def ? 0.0 : sqrt(d);
            const double pv = def ? 0.0 : 1.0 / rii;
            double ra[4], rc[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                ra[q] = rowb[buf][ty + 16 * q] * pv;
                rc[q] = rowb[buf][tx + 16 * q] * pv;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int w = 0; w < 4; ++w)
                    if (ty + 16 * q > i && tx + 16 * w > i) s[q][w] = fma(-ra[q], rc[w], s[q][w]);
            if (ty == i16) {
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const int c = tx + 16 * w;
                    if (c > i) s[ib][w] *= pv;
                    else if (c == i) s[ib][w] = rii;
                }
            }
            if (tid == 0) {
                piv[i] = def ? 1.0 : rii;
                dfl[i] = def ? 1 : 0;
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const int a = ty + 16 * q, c = tx + 16 * w;
            if (a < jb && c < jb && c >= a) C[static_cast<int64_t>(j0 + a) * k + j0 + c] = s[q][w];
        }
    if (tid < jb) defic[j0 + tid] = dfl[tid];

    double x[4][4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int w = 0; w < 4; ++w) x[q][w] = (ty + 16 * q == tx + 16 * w) ? 1.0 : 0.0;
#pragma unroll
    for (int ib = 3; ib >= 0; --ib) {
        for (int i16 = 15; i16 >= 0; --i16) {
            const int i = 16 * ib + i16;
            if (i >= jb) continue;
            const int buf = i & 1;
            if (ty == i16) {
                const double inv = 1.0 / piv[i];
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    x[ib][w] *= inv;
                    rowb[buf][tx + 16 * w] = x[ib][w];
                }
            }
            if (tx == i16) {
#pragma unroll
                for (int q = 0; q < 4; ++q) colb[buf][ty + 16 * q] = s[q][ib];   // R_ai, a < i
            }
            __syncthreads();
            double xi[4], ra[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                xi[q] = rowb[buf][tx + 16 * q];
                ra[q] = colb[buf][ty + 16 * q];
            }
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int w = 0; w < 4; ++w)
                    if (ty + 16 * q < i) x[q][w] = fma(-ra[q], xi[w], x[q][w]);
        }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const int r = ty + 16 * q, c = tx + 16 * w;
            if (r < jb && c < jb) {
                const double v = (c >= r) ? x[q][w] : 0.0;
                X[static_cast<int64_t>(j0 + r) * k + j0 + c] = v;
                if (Ri != nullptr) Ri[static_cast<int64_t>(j0 + r) * k + j0 + c] = static_cast<float>(v);
            }
        }
}

__global__ __launch_bounds__(CT) void chol_diag_kernel(double* Cb, int k, int64_t strideC, int J,
                                                       double* diag0b, int* deficB, double* Xb,
                                                       float* Rib, int64_t strideInv, double tau_rel) {
    const int b = blockIdx.x;
    diag_block(Cb + static_cast<int64_t>(b) * strideC, k, J, diag0b + static_cast<int64_t>(b) * k,
               deficB + static_cast<int64_t>(b) * k, Xb + static_cast<int64_t>(b) * strideInv,
               Rib != nullptr ? Rib + static_cast<int64_t>(b) * strideInv : nullptr, tau_rel);
}

// acc += A B for one 64 x 64 x 64 tile with A given by rows (A[i * ld + t], t
// contiguous) and B by contraction rows (B[t * ld + c]), operands straight from
// global memory into registers: contraction step s takes t = 8 (s / 2) +
// 2 (lane >> 4) + s % 2, so a lane's A entries A[i][t], A[i][t + 1] are one
// 16-byte pair. The result lands in the pair layout of mma64_pairs (row
// 32 wm + 2 (4 v + (lane >> 4)) + bi, column 32 wn + 2 (lane & 15) + bj).
__device__ __forceinline__ void mma64_rowA(const double* Ap, const double* Bp, int64_t ld, int nar, int nt, int nbc,
                                           bool vec, f64x4 acc[2][2], int wm, int wn, int lane) {
    const int l16 = lane & 15, lk = lane >> 4;
    // four groups of four steps (two A pairs per row block), double-buffered as
    // in mma64_pairs
    f64x2 a2[2][2][2], b2[2][4];
    auto load = [&](int g, int buf) {
#pragma unroll
        for (int mm = 0; mm < 2; ++mm)
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
                a2[buf][mm][bi] = ld_pair(Ap, ld, 32 * wm + 2 * l16 + bi, 8 * (2 * g + mm) + 2 * lk, nar, nt, vec);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int s = 4 * g + i;
            b2[buf][i] = ld_pair(Bp, ld, 8 * (s >> 1) + 2 * lk + (s & 1), 32 * wn + 2 * l16, nt, nbc, vec);
        }
    };
    load(0, 0);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        if (g + 1 < 4) load(g + 1, (g + 1) & 1);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                for (int bj = 0; bj < 2; ++bj)
                    acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(a2[g & 1][i >> 1][bi][i & 1], b2[g & 1][i][bj],
                                                                       acc[bi][bj], 0, 0, 0);
    }
}

// Step J, after the diagonal block J (factor R_JJ and D_J = R'_JJ^-1):
//  * blockIdx.x < n (n = nb - J - 1): the panel tile T = J + 1 + blockIdx.x,
//    R_JT = D_J^T C_JT (deficient rows zero), in place in C;
//  * with the inverse, blockIdx.x = n + I (I < J): block column J of the
//    inverse X = R'^-1, X_IJ = -P_IJ D_J, where P_IJ (held in X's block (I, J))
//    is the sum over U < J of X_IU R_UJ that the trailing steps accumulated;
//    written in fp64 and as fp32, whose mirrored (lower) tile is set to zero.
__global__ __launch_bounds__(CT, 4) void chol_panel_x_kernel(double* Cb, int k, int64_t strideC, int J, int n,
                                                          const int* deficB, double* Xb, float* Rib,
                                                          int64_t strideInv) {
    const int b = blockIdx.y;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    const int* defic = deficB + static_cast<int64_t>(b) * k;
    double* X = Xb + static_cast<int64_t>(b) * strideInv;
    const int j0 = J * CB;
    const int jb = min(CB, k - j0);
    const bool vec = (k & 1) == 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l16 = lane & 15, lk = lane >> 4;
    f64x4 acc[2][2];
    zero_acc(acc);
    if (static_cast<int>(blockIdx.x) < n) {
        const int c0 = (J + 1 + blockIdx.x) * CB;
        const int cb = min(CB, k - c0);
        // A[i][t] = D[t][i] (rows j0 + t of the block inverse), B[t][c] = C_JT[t][c]
        mma64_pairs(X + static_cast<int64_t>(j0) * k + j0, C + static_cast<int64_t>(j0) * k + c0, k, jb, jb, cb,
                    vec, acc, wm, wn, lane);
        // the deficiency flags of the lane's eight rows, read together
        bool dfl[2][4];
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int v = 0; v < 4; ++v) dfl[bi][v] = defic[j0 + min(32 * wm + 2 * (4 * v + lk) + bi, jb - 1)] != 0;
        __syncthreads();   // every wave has its operands before the tile is overwritten
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int r = 32 * wm + 2 * (4 * v + lk) + bi;
                if (r >= jb) continue;
                const bool def = dfl[bi][v];
                const int c = 32 * wn + 2 * l16;
                double* dst = C + static_cast<int64_t>(j0 + r) * k + c0 + c;
                const double o0 = def ? 0.0 : acc[bi][0][v], o1 = def ? 0.0 : acc[bi][1][v];
                if (vec && c + 1 < cb) {
                    *reinterpret_cast<f64x2*>(dst) = f64x2{o0, o1};
                } else {
                    if (c < cb) dst[0] = o0;
                    if (c + 1 < cb) dst[1] = o1;
                }
            }
        return;
    }
    const int I = blockIdx.x - n;
    const int i0 = I * CB;
    // A = P_IJ (rows i0.., columns j0..), B = D_J (rows j0 + t)
    mma64_rowA(X + static_cast<int64_t>(i0) * k + j0, X + static_cast<int64_t>(j0) * k + j0, k, CB, jb, jb, vec, acc,
               wm, wn, lane);
    __syncthreads();       // P_IJ is overwritten by X_IJ below
    float* Ri = Rib + static_cast<int64_t>(b) * strideInv;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int r = 32 * wm + 2 * (4 * v + lk) + bi;
                const int c = 32 * wn + 2 * l16 + bj;
                if (c < jb) {
                    const double val = -acc[bi][bj][v];
                    X[static_cast<int64_t>(i0 + r) * k + j0 + c] = val;
                    Ri[static_cast<int64_t>(i0 + r) * k + j0 + c] = static_cast<float>(val);
                }
                // the mirrored (lower) tile of the fp32 inverse is zero
                if (r < jb) Ri[static_cast<int64_t>(j0 + r) * k + i0 + c] = 0.0f;
            }
}

// Step J's updates, after the panel:
//  * blockIdx.x < n (n + 1) / 2: C_T1T2 -= R_JT1^T R_JT2 on the upper tiles
//    J < T1 <= T2; the workgroup of tile (J + 1, J + 1) then factors that
//    diagonal block (step J + 1's diagonal), whose last update this was;
//  * with the inverse, the rest: P_IT (+)= X_IJ R_JT for I <= J < T, the
//    partial sums block column T of the inverse needs (I = J starts the sum).
__global__ __launch_bounds__(CT, 4) void chol_trailing_p_kernel(double* Cb, int k, int64_t strideC, int J, int nb,
                                                             double* diag0b, int* deficB, double* Xb, float* Rib,
                                                             int64_t strideInv, double tau_rel) {
    const int b = blockIdx.y;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    double* X = Xb + static_cast<int64_t>(b) * strideInv;
    const int n = nb - J - 1;
    const int ntrail = n * (n + 1) / 2;
    const int j0 = J * CB;
    const int jb = min(CB, k - j0);
    const bool vec = (k & 1) == 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l16 = lane & 15, lk = lane >> 4;
    f64x4 acc[2][2];
    zero_acc(acc);
    if (static_cast<int>(blockIdx.x) < ntrail) {
        // blockIdx.x -> (u, vt) with 0 <= u <= vt < n, row-major over the upper triangle
        int idx = blockIdx.x, u = 0;
        while (idx >= n - u) {
            idx -= n - u;
            ++u;
        }
        const int vt = u + idx;
        const int r0 = (J + 1 + u) * CB, rb = min(CB, k - r0);
        const int c0 = (J + 1 + vt) * CB, cb = min(CB, k - c0);
        // on a diagonal tile the quadrant below the diagonal is not needed
        if (!(u == vt && wm > wn)) {
            // operands: rows j0 + t of the block row J just finished (R_JT1, R_JT2);
            // the tile updated lies in a later block row, so no wave reads what
            // another one writes
            mma64_pairs(C + static_cast<int64_t>(j0) * k + r0, C + static_cast<int64_t>(j0) * k + c0, k, jb, rb, cb,
                        vec, acc, wm, wn, lane);
            if (vec && rb == CB && cb == CB && u != vt) {
                // an interior tile off the diagonal (uniform): the lane's eight
                // pairs are read together, then written (read-modify-write one
                // pair at a time waited a memory latency per pair)
                const int c = 32 * wn + 2 * l16;
                f64x2 o[2][4];
#pragma unroll
                for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        o[bi][v] = *reinterpret_cast<const f64x2*>(
                            C + static_cast<int64_t>(r0 + 32 * wm + 2 * (4 * v + lk) + bi) * k + c0 + c);
#pragma unroll
                for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        *reinterpret_cast<f64x2*>(C + static_cast<int64_t>(r0 + 32 * wm + 2 * (4 * v + lk) + bi) * k +
                                                  c0 + c) =
                            f64x2{o[bi][v][0] - acc[bi][0][v], o[bi][v][1] - acc[bi][1][v]};
            } else {
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int r = 32 * wm + 2 * (4 * v + lk) + bi;
                    if (r >= rb) continue;
                    const int c = 32 * wn + 2 * l16;
                    const bool k0 = c < cb && (u != vt || c >= r);
                    const bool k1 = c + 1 < cb && (u != vt || c + 1 >= r);
                    double* dst = C + static_cast<int64_t>(r0 + r) * k + c0 + c;
                    if (vec && k0 && k1) {
                        f64x2 o = *reinterpret_cast<f64x2*>(dst);
                        o[0] -= acc[bi][0][v];
                        o[1] -= acc[bi][1][v];
                        *reinterpret_cast<f64x2*>(dst) = o;
                    } else {
                        if (k0) dst[0] -= acc[bi][0][v];
                        if (k1) dst[1] -= acc[bi][1][v];
                    }
                }
            }
        }
        if (blockIdx.x == 0) {
            // tile (J + 1, J + 1) is final: factor it (its updates above are
            // visible to the whole workgroup past the barrier)
            __syncthreads();
            diag_block(C, k, J + 1, diag0b + static_cast<int64_t>(b) * k, deficB + static_cast<int64_t>(b) * k, X,
                       Rib != nullptr ? Rib + static_cast<int64_t>(b) * strideInv : nullptr, tau_rel);
        }
        return;
    }
    const int p = blockIdx.x - ntrail;
    const int I = p / n, T = J + 1 + p % n;
    const int i0 = I * CB;
    const int c0 = T * CB, cb = min(CB, k - c0);
    // A = X_IJ (rows i0.., columns j0..), B = R_JT (rows j0 + t of C)
    mma64_rowA(X + static_cast<int64_t>(i0) * k + j0, C + static_cast<int64_t>(j0) * k + c0, k, CB, jb, cb, vec, acc,
               wm, wn, lane);
    const bool first = (I == J);
    if (vec && i0 + CB <= k && cb == CB) {
        // a whole tile (uniform): the lane's eight pairs read together first
        const int c = 32 * wn + 2 * l16;
        f64x2 o[2][4];
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                o[bi][v] = first ? f64x2{0.0, 0.0}
                                 : *reinterpret_cast<const f64x2*>(
                                       X + static_cast<int64_t>(i0 + 32 * wm + 2 * (4 * v + lk) + bi) * k + c0 + c);
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                *reinterpret_cast<f64x2*>(X + static_cast<int64_t>(i0 + 32 * wm + 2 * (4 * v + lk) + bi) * k + c0 + c) =
                    f64x2{o[bi][v][0] + acc[bi][0][v], o[bi][v][1] + acc[bi][1][v]};
        return;
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = 32 * wm + 2 * (4 * v + lk) + bi;
            if (i0 + r >= k) continue;
            const int c = 32 * wn + 2 * l16;
            double* dst = X + static_cast<int64_t>(i0 + r) * k + c0 + c;
            if (vec && c + 1 < cb) {
                f64x2 o = first ? f64x2{0.0, 0.0} : *reinterpret_cast<f64x2*>(dst);
                o[0] += acc[bi][0][v];
                o[1] += acc[bi][1][v];
                *reinterpret_cast<f64x2*>(dst) = o;
            } else {
                if (c < cb) dst[0] = (first ? 0.0 : dst[0]) + acc[bi][0][v];
                if (c + 1 < cb) dst[1] = (first ? 0.0 : dst[1]) + acc[bi][1][v];
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

// The same generic unit vector written as the three bf16 planes of column j
// (plane row j, transposed layout of GemmArgs::planes), for a Q that exists
// only as its planes; rows past `rows` keep the zeros the product wrote.
__global__ __launch_bounds__(256) void fill_deficient_planes_kernel(uint16_t* planesb, int64_t ldpl, int64_t planeStride,
                                                                    int64_t stridePl, int rows, int k,
                                                                    const int* deficB) {
    const int b = blockIdx.y;
    const int j = blockIdx.x;
    if (!deficB[static_cast<int64_t>(b) * k + j]) return;
    uint16_t* pl = planesb + static_cast<int64_t>(b) * stridePl + static_cast<int64_t>(j) * ldpl;
    const float scale = 1.0f / sqrtf(static_cast<float>(rows));
    for (int i = threadIdx.x; i < rows; i += blockDim.x) {
        const uint64_t h = mix64((static_cast<uint64_t>(j) << 32) | static_cast<uint32_t>(i));
        uint16_t h1, h2, h3;
        split3_rn((h & 1ULL) ? scale : -scale, h1, h2, h3);
        pl[i] = h1;
        pl[planeStride + i] = h2;
        pl[2 * planeStride + i] = h3;
    }
}

}  // namespace

hipError_t launch_cholesky(double* C, int k, int64_t strideC, float* rinv32, double* xinv,
                           int64_t strideInv, int* defic, double* diag0, double tau_rel, int batch,
                           hipStream_t stream) {
    const int nb = (k + CB - 1) / CB;
    const bool inv = rinv32 != nullptr;
    hipLaunchKernelGGL(chol_diag_kernel, dim3(batch), dim3(CT), 0, stream, C, k, strideC, 0, diag0, defic, xinv,
                       rinv32, strideInv, tau_rel);
    for (int J = 0; J < nb; ++J) {
        const int n = nb - J - 1;
        const int px = n + (inv ? J : 0);
        if (px > 0)
            hipLaunchKernelGGL(chol_panel_x_kernel, dim3(px, batch), dim3(CT), 0, stream, C, k, strideC, J, n, defic,
                               xinv, rinv32, strideInv);
        if (n > 0)
            hipLaunchKernelGGL(chol_trailing_p_kernel, dim3(n * (n + 1) / 2 + (inv ? (J + 1) * n : 0), batch),
                               dim3(CT), 0, stream, C, k, strideC, J, nb, diag0, defic, xinv, rinv32, strideInv,
                               tau_rel);
    }
    return hipGetLastError();
}

hipError_t launch_fill_deficient(float* Q, int rows, int k, int64_t strideQ, const int* defic,
                                 int batch, hipStream_t stream) {
    hipLaunchKernelGGL(fill_deficient_kernel, dim3(k, batch), dim3(256), 0, stream, Q, rows, k,
                       strideQ, defic);
    return hipGetLastError();
}

hipError_t launch_fill_deficient_planes(uint16_t* planes, int64_t ldpl, int64_t planeStride, int64_t stridePl,
                                        int rows, int k, const int* defic, int batch, hipStream_t stream) {
    hipLaunchKernelGGL(fill_deficient_planes_kernel, dim3(k, batch), dim3(256), 0, stream, planes, ldpl, planeStride,
                       stridePl, rows, k, defic);
    return hipGetLastError();
}

}  // namespace galore
