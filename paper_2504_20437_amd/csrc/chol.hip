// Cholesky factorisation of the k x k Gram matrices (fp64) and the inverse of the
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
//     diag     factor the 64 x 64 diagonal block in registers (unblocked, fp64)
//              and invert it (D_J = R'_JJ^-1, kept in the fp64 inverse buffer);
//     panel    R_JT = D_J^T C_JT for every block column T > J;
//     trailing C_T1T2 -= R_JT1^T R_JT2 on the upper tiles T1 <= T2 right of J.
//   inverse  X = R'^-1 by levels d = T - I: X_IT = -D_I sum_{I<U<=T} R_IU X_UT,
//            written in fp64 and as fp32 (lower triangle zero) for the GEMM
//            that applies it.
// The panel, trailing and inverse tiles are 64 x 64 x 64 products on the fp64
// matrix cores.
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
constexpr int LP = CB + 1; // padded LDS row

// acc[bi][bj] += sum_{t < CB} As[t][32 wm + 16 bi + i] * Bs[t][32 wn + 16 bj + j] on the
// fp64 matrix cores: wave (wm, wn) owns a 32 x 32 quadrant of the 64 x 64
// result as 2 x 2 blocks of 16 x 16. Operand layout of the 16x16x4 fp64 MFMA:
// lane l supplies A[l & 15][l >> 4] and B[l >> 4][l & 15]; accumulator
// register v of lane l holds C[4 v + (l >> 4)][l & 15]. Rows of As / Bs
// beyond the live extent are zero, so the full depth CB is always run.
__device__ __forceinline__ void mma64_tn(double (*As)[LP], double (*Bs)[LP], f64x4 acc[2][2], int wm,
                                         int wn, int lane) {
    const int l16 = lane & 15, lk = lane >> 4;
#pragma unroll 4
    for (int t = 0; t < CB; t += 4) {
        double a[2], bv[2];
#pragma unroll
        for (int bi = 0; bi < 2; ++bi) a[bi] = As[t + lk][32 * wm + 16 * bi + l16];
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) bv[bj] = Bs[t + lk][32 * wn + 16 * bj + l16];
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int bj = 0; bj < 2; ++bj)
                acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[bi], bv[bj], acc[bi][bj], 0, 0, 0);
    }
}

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
    f64x2 av[16], bv[16];
#pragma unroll
    for (int s = 0; s < 16; ++s) {
        const int t = 4 * s + lk;
        av[s] = ld_pair(Ap, ld, t, 32 * wm + 2 * l16, nt, na, vec);
        bv[s] = ld_pair(Bp, ld, t, 32 * wn + 2 * l16, nt, nbc, vec);
    }
#pragma unroll
    for (int s = 0; s < 16; ++s)
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int bj = 0; bj < 2; ++bj)
                acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[s][bi], bv[s][bj], acc[bi][bj], 0, 0, 0);
}

// S[c][r] = M[(r0 + r) * ld + c0 + c] (transposed load)
__device__ __forceinline__ void load_tile_t(double (*S)[LP], const double* M, int64_t ld, int r0, int c0,
                                            int nr, int nc) {
    for (int idx = threadIdx.x; idx < CB * CB; idx += CT) {
        const int r = idx / CB, c = idx % CB;
        S[c][r] = (r < nr && c < nc) ? M[static_cast<int64_t>(r0 + r) * ld + c0 + c] : 0.0;
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
__global__ __launch_bounds__(CT) void chol_diag_kernel(double* Cb, int k, int64_t strideC, int J,
                                                       double* diag0b, int* deficB, double* Xb,
                                                       float* Rib, int64_t strideInv, double tau_rel) {
    const int b = blockIdx.x;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    double* diag0 = diag0b + static_cast<int64_t>(b) * k;
    int* defic = deficB + static_cast<int64_t>(b) * k;
    double* X = Xb + static_cast<int64_t>(b) * strideInv;
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
                if (Rib != nullptr)
                    Rib[static_cast<int64_t>(b) * strideInv + static_cast<int64_t>(j0 + r) * k + j0 + c] =
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
    const bool vec = (k & 1) == 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l16 = lane & 15, lk = lane >> 4;
    f64x4 acc[2][2];
    zero_acc(acc);
    // A[i][t] = D[t][i] (rows j0 + t of the block inverse), B[t][c] = C_JT[t][c]
    mma64_pairs(X + static_cast<int64_t>(j0) * k + j0, C + static_cast<int64_t>(j0) * k + c0, k, jb, jb, cb,
                vec, acc, wm, wn, lane);
    __syncthreads();   // every wave has its operands before the tile is overwritten
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int r = 32 * wm + 2 * (4 * v + lk) + bi;
            if (r >= jb) continue;
            const bool def = defic[j0 + r] != 0;
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
}

// C_T1T2 -= R_JT1^T R_JT2 for J < T1 <= T2; blockIdx.x enumerates the upper tiles
__global__ __launch_bounds__(CT) void chol_trailing_kernel(double* Cb, int k, int64_t strideC, int J,
                                                           int nb) {
    const int b = blockIdx.y;
    double* C = Cb + static_cast<int64_t>(b) * strideC;
    const int n = nb - J - 1;
    // blockIdx.x -> (u, vt) with 0 <= u <= vt < n, row-major over the upper triangle
    int idx = blockIdx.x, u = 0;
    while (idx >= n - u) {
        idx -= n - u;
        ++u;
    }
    const int vt = u + idx;
    const int j0 = J * CB;
    const int jb = min(CB, k - j0);
    const int r0 = (J + 1 + u) * CB, rb = min(CB, k - r0);
    const int c0 = (J + 1 + vt) * CB, cb = min(CB, k - c0);
    const bool vec = (k & 1) == 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l16 = lane & 15, lk = lane >> 4;
    // on a diagonal tile the quadrant below the diagonal is not needed
    if (u == vt && wm > wn) return;
    f64x4 acc[2][2];
    zero_acc(acc);
    // operands: rows j0 + t of the block row J just finished (R_JT1, R_JT2);
    // the tile updated lies in a later block row, so no wave reads what
    // another one writes
    mma64_pairs(C + static_cast<int64_t>(j0) * k + r0, C + static_cast<int64_t>(j0) * k + c0, k, jb, rb, cb,
                vec, acc, wm, wn, lane);
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
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l16 = lane & 15, lk = lane >> 4;
    // S = sum_{U = I+1 .. Jc} R_IU X_UJc, operands straight from global memory:
    // contraction step s = 2 m + e takes t = 8 m + 2 (lane >> 4) + e, so a
    // lane's A entries R_IU[a][t], R_IU[a][t + 1] are one 16-byte pair; S lands
    // in the pair layout of mma64_pairs (row 32 wm + 2 (4 v + lk) + bi, column
    // 32 wn + 2 l16 + bj)
    const bool vec = (k & 1) == 0;
    f64x4 acc[2][2];
    zero_acc(acc);
    for (int U = I + 1; U <= Jc; ++U) {
        const int u0 = U * CB, ub = min(CB, k - u0);
        const double* Rp = C + static_cast<int64_t>(i0) * k + u0;
        const double* Xp = X + static_cast<int64_t>(u0) * k + c0;
        f64x2 a2[2][8], b2[16];
#pragma unroll
        for (int m = 0; m < 8; ++m)
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
                a2[bi][m] = ld_pair(Rp, k, 32 * wm + 2 * l16 + bi, 8 * m + 2 * lk, ib, ub, vec);
#pragma unroll
        for (int s = 0; s < 16; ++s)
            b2[s] = ld_pair(Xp, k, 8 * (s >> 1) + 2 * lk + (s & 1), 32 * wn + 2 * l16, ub, cb, vec);
#pragma unroll
        for (int s = 0; s < 16; ++s)
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                for (int bj = 0; bj < 2; ++bj)
                    acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(a2[bi][s >> 1][s & 1], b2[s][bj],
                                                                       acc[bi][bj], 0, 0, 0);
    }
    // X_IJc = -D_I S
    load_tile_t(As, X, k, i0, i0, ib, ib);       // As[t][a] = D_I[a][t]
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int v = 0; v < 4; ++v) Bs[32 * wm + 2 * (4 * v + lk) + bi][32 * wn + 2 * l16 + bj] = acc[bi][bj][v];
    __syncthreads();
    f64x4 out[2][2];
    zero_acc(out);
    mma64_tn(As, Bs, out, wm, wn, lane);
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int r = 32 * wm + 16 * bi + 4 * v + lk;
                const int c = 32 * wn + 16 * bj + l16;
                if (r < ib && c < cb) {
                    const double val = -out[bi][bj][v];
                    X[static_cast<int64_t>(i0 + r) * k + c0 + c] = val;
                    if (Rib != nullptr) Ri[static_cast<int64_t>(i0 + r) * k + c0 + c] = static_cast<float>(val);
                }
                // the mirrored (lower) tile of the fp32 inverse is zero
                if (Rib != nullptr && r < cb && c < ib) Ri[static_cast<int64_t>(c0 + r) * k + i0 + c] = 0.0f;
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
