// Internal helpers shared by the gfx950 kernels of the GaLore 2 library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace galore {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef double f64x4 __attribute__((ext_vector_type(4)));

struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) {
    return __uint_as_float(static_cast<uint32_t>(x.bits) << 16);
}

// bits of the bfloat16 nearest to x (ties to even; NaN stays NaN), and back
__device__ __forceinline__ uint16_t bf16_bits_rn(float x) {
    // round to nearest even (inputs here are finite or propagate NaN)
    const uint32_t u = __float_as_uint(x);
    if ((u & 0x7f800000u) == 0x7f800000u) return static_cast<uint16_t>((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// x = h1 + h2 + h3 with the three bf16 terms rounded to nearest in turn (the
// three planes of an fp32 operand of the bf16 matrix-core products)
__device__ __forceinline__ void split3_rn(float x, uint16_t& h1, uint16_t& h2, uint16_t& h3) {
    h1 = bf16_bits_rn(x);
    const float r1 = x - bf16_bits_to_f32(h1);
    h2 = bf16_bits_rn(r1);
    const float r2 = r1 - bf16_bits_to_f32(h2);
    h3 = bf16_bits_rn(r2);
}

// MI355X deals workgroups to its 8 XCDs round-robin by linear id (x fastest,
// then y, then z) and every XCD has its own L2. xcd_logical_id remaps the
// linear id so that XCD x receives the contiguous range [x * per, (x+1) * per)
// of logical ids (per = total / 8; ids past the last multiple of 8 keep their
// value): workgroups with neighbouring logical ids share an L2.
__device__ __forceinline__ int xcd_logical_id(int lin, int total) {
    constexpr int kXcd = 8;
    const int main = total - total % kXcd;
    if (lin >= main) return lin;
    const int per = main / kXcd;
    return (lin % kXcd) * per + lin / kXcd;
}

// Logical tile id -> (m, n) tile of one matrix, grouped by `group` tile rows:
// consecutive ids walk the rows of a group first, so that the tiles in flight
// on one XCD share both their A rows and their B columns.
__device__ __forceinline__ void grouped_tile(int t, int num_m, int num_n, int group, int& m, int& n) {
    const int per_group = group * num_n;
    const int g = t / per_group;
    const int first = g * group;
    const int gsize = min(group, num_m - first);
    const int r = t - g * per_group;
    m = first + r % gsize;
    n = r / gsize;
}

// Operand layouts of the GEMM kernels.
//   A operand (M x K): kKContig -> A[i*lda + kk]   kMContig -> A[kk*lda + i]
//   B operand (K x N): kNContig -> B[kk*ldb + j]   kKContigB -> B[j*ldb + kk]
enum class ALayout { kKContig, kMContig };
enum class BLayout { kNContig, kKContig };

struct GemmArgs {
    const void* A;
    int64_t lda, strideA;
    const void* B;
    int64_t ldb, strideB;
    float* C;
    int64_t ldc, strideC;
    int M, N, K;
    float alpha, beta;   // C = alpha * op(A) op(B) + beta * C  (beta == 0: C not read)
    int b_upper;         // op(B) upper triangular: column tile j0 only needs k < j0 + tile width
    // planes != nullptr (beta == 0 only): instead of C, the three bf16 planes
    // of alpha op(A) op(B) (split3_rn), transposed: plane p of matrix b holds
    // element (i, j) at planes[b * stridePl + p * planeStride + j * ldpl + i],
    // rows M <= i < rows_pad written as zero (rows_pad <= M rounded up to 128)
    uint16_t* planes;
    int64_t ldpl, planeStride, stridePl;
    int rows_pad;
};

// Exact Gram of the fixed-point image of X on the int8 matrix cores (gram_i8.hip):
// upper triangle of C (cols x cols, row-major, ld = ldc) only.
struct GramI8Args {
    const float* X;      // rows x cols, row-major
    int64_t ldx, strideX;
    int rows, cols;
    unsigned* cmax;      // per matrix: strideCM >= cols column maxima (scratch)
    int64_t strideCM;
    int8_t* D;           // per matrix: strideD >= gram_i8_digit_bytes(rows, cols) bytes (scratch)
    int64_t strideD;
    double* C;
    int64_t ldc, strideC;
    int cmax_ready;      // cmax already holds the column maxima of X (its producer wrote them)
};
int64_t gram_i8_ld(int rows);          // bytes per digit row (rows padded to 128)
int gram_i8_cols_pad(int cols);        // digit rows per plane (cols padded to 64)
inline int64_t gram_i8_digit_bytes(int rows, int cols) { return 3 * gram_i8_cols_pad(cols) * gram_i8_ld(rows); }

// Launchers (defined in the .hip files). All return hipError_t of the launch.
hipError_t launch_gram_i8(const GramI8Args& g, int batch, hipStream_t stream);
// zero n unsigned (the column-maximum buffer before a producer fills it)
hipError_t launch_fill_u32(unsigned* p, int64_t n, hipStream_t stream);
hipError_t launch_gemm(ALayout la, BLayout lb, bool a_bf16, bool b_bf16, const GemmArgs& g, int batch,
                       hipStream_t stream);

hipError_t launch_sketch(float* omega, int64_t l, int64_t k, int64_t stride, uint64_t seed,
                         uint64_t sketch_index0, int batch, hipStream_t stream);
// the sketch as the one bf16 plane of Omega^T (k rows of ldp, zero past l);
// zero_rest also zeroes the next two planes
hipError_t launch_sketch_plane(uint16_t* planes, int64_t ldp, int64_t planeStride, int64_t stride, int64_t l,
                               int64_t k, uint64_t seed, uint64_t sketch_index0, bool zero_rest, int batch,
                               hipStream_t stream);

// Cholesky of the k x k fp64 Gram (in place, upper factor R in the upper
// triangle). xinv (k x k fp64) receives the inverses of the diagonal blocks
// and, if rinv32 != nullptr, the whole inverse of R' (R with rank-deficient
// rows replaced by unit rows), also written in fp32 into rinv32 (k x k, lower
// triangle zero). defic[b*k + j] = 1 marks deficient pivots; diag0 (k fp64 per
// matrix) keeps the original diagonal for the deficiency test.
hipError_t launch_cholesky(double* C, int k, int64_t strideC, float* rinv32, double* xinv,
                           int64_t strideInv, int* defic, double* diag0, double tau_rel, int batch,
                           hipStream_t stream);
// Replace columns flagged deficient by a deterministic generic unit vector.
hipError_t launch_fill_deficient(float* Q, int rows, int k, int64_t strideQ, const int* defic,
                                 int batch, hipStream_t stream);
// the same into the three bf16 planes of Q (GemmArgs::planes layout)
hipError_t launch_fill_deficient_planes(uint16_t* planes, int64_t ldpl, int64_t planeStride, int64_t stridePl,
                                        int rows, int k, const int* defic, int batch, hipStream_t stream);
// Yt (k x k, column c contiguous) = columns of 2^e Y, Y = R^T, in fp32 from the
// fp64 factor (the row-major upper triangle of R), with the power of two e of
// each matrix (written to exps[b]) taken from the diagonal diag (k fp64 per
// matrix) of the Gram that R factors; clears the rotation counters.
hipError_t launch_jacobi_prepare(const double* R, int k, int64_t strideR, float* Yt, int64_t strideX,
                                 int* rot, int max_sweeps, const double* diag, int* exps, int batch,
                                 hipStream_t stream);
// order of the columns for sweep `sweep` (by decreasing norm) into jperm
// (k per matrix), with the column norms in norms (k per matrix); matrices
// converged in the previous sweep are skipped
hipError_t launch_jacobi_order(const float* Yt, int k, int64_t strideX, double* norms, int* jperm, const int* rot,
                               int max_sweeps, int sweep, int batch, hipStream_t stream);
hipError_t launch_jacobi_step(float* Yt, int k, int64_t strideX, int nblocks, int step, int sweep, int* rot,
                              int max_sweeps, double tol, const int* jperm, int batch, hipStream_t stream);
// scratch: at least 2 k + r doubles per matrix at stride strideScratch (doubles);
// exps: the per-matrix exponents launch_jacobi_prepare wrote (sigma = 2^-e |y|);
// norms (k fp64) and perm (k int) per matrix: scratch for the column norms and
// their order; Xa (optional, k x k fp32 per matrix at strideX, with flags):
// all k ordered unit columns (column j contiguous) for launch_refine, flags[b] =
// 1 when matrix b has them (every column norm finite and positive; Ur is then
// left to launch_refine), else 0
hipError_t launch_jacobi_finalize(const float* Yt, int k, int64_t strideX, int r, float* Ur, int64_t strideUr,
                                  float* sigma, int64_t stride_sigma, const int* rot, int max_sweeps, int nsweeps,
                                  int* info,
                                  double* scratch, int64_t strideScratch, const int* exps, double* norms, int* perm,
                                  float* Xa, int* flags, int batch, hipStream_t stream);
// fp64 refinement of the small SVD's vectors (refine.hip): one Ogita-Aishima
// step on H = R^T R (R: the row-major upper triangle of the fp64 Cholesky
// factor) from the vectors in the rows of Xa, then the r refined vectors of
// largest Rayleigh quotient re-orthonormalised among themselves and written as
// the columns of Ur (k x r) with sigma = sqrt(lambda). Xa, Xb: fp32 k x k
// (scratch afterwards); T, S, G: fp64 k x k scratch at strideKK; lam (k doubles)
// and perm (k int) per matrix: scratch. Only the matrices whose flag is set are
// touched.
hipError_t launch_refine(const double* R, int64_t strideR, float* Xa, float* Xb, int64_t strideX, double* T,
                         double* S, double* G, int64_t strideKK, double* lam, int* perm, int k, int r, float* Ur,
                         int64_t strideUr, float* sigma, int64_t stride_sigma, const int* flags, int batch,
                         hipStream_t stream);
// Subspace switch: negate the columns of P_new whose overlap with the same
// column of P_old is negative (rows x r each); flips (batch x r, may be null)
// receives 1 for a negated column.
hipError_t launch_align(const float* P_old, int64_t ldo, int64_t strideO, float* P_new, int64_t ldn, int64_t strideN,
                        int rows, int r, int* flips, int batch, hipStream_t stream);
hipError_t launch_sign_fix(float* P, int rows, int r, int64_t ldp, int64_t strideP, int batch,
                           hipStream_t stream);
hipError_t launch_adam(const float* R, float* M, float* V, float* N, int64_t rows, int64_t cols,
                       int64_t ld, int64_t stride, int batch, float beta1, float beta2, float eps,
                       float bc1, float bc2, hipStream_t stream);
// Adam with R and N in one layout (ldrn, srn) and M and V in another (ldmv, smv).
hipError_t launch_adam2(const float* R, float* N, int64_t ldrn, int64_t srn, float* M, float* V, int64_t ldmv,
                        int64_t smv, int64_t rows, int64_t cols, int batch, float beta1, float beta2, float eps,
                        float bc1, float bc2, hipStream_t stream);
// Low-bit projector (quant.hip): codes of the s x r projector, 8 bits (one
// byte each) or 4 bits (two per byte, even column in the low nibble).
hipError_t launch_quantize(const float* P, int64_t ldp, int64_t strideP, int rows, int r, int bits, uint8_t* Q,
                           int64_t ldq, int64_t strideQ, float* scales, int64_t strideS, int batch, hipStream_t stream);
// bf16 plane of the codes: rows x cols_pad (zero past r), or transposed
// r x rows_pad (zero past rows)
hipError_t launch_codes_plane(const uint8_t* Q, int64_t ldq, int64_t strideQ, int bits, int rows, int r, uint16_t* plane,
                              int64_t ldpl, int64_t stridePl, int pad, bool transpose, int batch, hipStream_t stream);
// fp32 dequantised projector code * scale (rows x r, ld ldt)
hipError_t launch_dequantize(const uint8_t* Q, int64_t ldq, int64_t strideQ, int bits, const float* scales,
                             int64_t strideS, int rows, int r, float* Pt, int64_t ldt, int64_t strideT, int batch,
                             hipStream_t stream);
// 8-bit block-wise Adam (adam8.hip): blocks of 2048 elements of the packed
// row-major state; R and N share (ld, stride)
int64_t adam8_block_count(int64_t rows, int64_t cols);
hipError_t launch_adam8(const float* R, float* N, int64_t ld, int64_t stride, uint8_t* M8, float* Ms, uint8_t* V8,
                        float* Vs, int64_t rows, int64_t cols, int batch, float beta1, float beta2, float eps,
                        float bc1, float bc2, hipStream_t stream);
// measurement helper (probe.hip): blocks x 256 threads of sustained bf16 MFMA chains
hipError_t launch_mfma_probe(int64_t iters, int blocks, float* sink, hipStream_t stream);
hipError_t launch_copy_probe(const void* src, void* dst, int64_t nvec, hipStream_t stream);
hipError_t launch_copy_rows(const float* src, int64_t lds, int64_t strideS, float* dst, int64_t ldd,
                            int64_t strideD, int rows, int cols, int batch, hipStream_t stream);

// bf16 matrix-core products with an exactly bf16 operand (bf16x3.hip)
hipError_t launch_transpose_bf16(const void* src, int64_t lds, int64_t strideS, void* dst, int64_t ldd,
                                 int64_t strideD, int rows, int cols, int batch, hipStream_t stream);
hipError_t launch_split3_transpose(const float* src, int64_t lds, int64_t strideS, void* planes, int64_t ldp,
                                   int64_t planeStride, int64_t strideP, int rows, int cols, int rows_pad,
                                   int batch, hipStream_t stream, const float* rowscale = nullptr,
                                   int64_t strideRS = 0);
// C (M x N, or its transpose when c_trans) = alpha A B + beta C with A bf16
// (rows K-contiguous, A[i * lda + kk], or M-contiguous when a_mcontig,
// A[kk * lda + i]) and B given as three bf16 planes, each N x K rows.
// M-contiguous A and transposed C need the direct-load kernel: check
// bf16x3_direct_ok first (hipErrorInvalidValue otherwise).
bool bf16x3_direct_ok(const void* A, int64_t lda, int64_t strideA, const void* Bplanes, int64_t ldb,
                      int64_t planeStride, int64_t strideB, int M, int K, int batch, int a_mcontig);
// cmax (row-major C on the direct-load kernel only, else hipErrorInvalidValue):
// per matrix strideCM unsigned, atomicMax'ed with the bits of |C| per column
// (the caller zeroes it first); null for none.
hipError_t launch_gemm_bf16x3(const void* A, int64_t lda, int64_t strideA, int a_mcontig, const void* Bplanes,
                              int64_t ldb, int64_t planeStride, int64_t strideB, float* C, int64_t ldc,
                              int64_t strideC, int c_trans, int M, int N, int K, float alpha, float beta, int batch,
                              hipStream_t stream, unsigned* cmax = nullptr, int64_t strideCM = 0, int planesB = 3,
                              const float* nscale = nullptr, int64_t strideNS = 0);

// fp32 x fp32 products on the bf16 matrix cores: both operands given as three
// bf16 planes with K-contiguous rows (A: M rows, B: N rows), six plane products
// accumulated in fp32 (error below fp32 rounding of the products). C as for
// launch_gemm_bf16x3; b_upper: B[kk][n] = 0 for kk > n (the K loop stops at
// the tile's last column). Needs bf16x6_ok (hipErrorInvalidValue otherwise).
hipError_t launch_split3_rows(const float* src, int64_t lds, int64_t strideS, void* planes, int64_t ldp,
                              int64_t planeStride, int64_t strideP, int rows, int cols, int cols_pad, int batch,
                              hipStream_t stream);
bool bf16x6_ok(const void* Aplanes, int64_t lda, int64_t planeStrideA, int64_t strideA, const void* Bplanes,
               int64_t ldb, int64_t planeStrideB, int64_t strideB, int K, int batch);
hipError_t launch_gemm_bf16x6(const void* Aplanes, int64_t lda, int64_t planeStrideA, int64_t strideA,
                              const void* Bplanes, int64_t ldb, int64_t planeStrideB, int64_t strideB, float* C,
                              int64_t ldc, int64_t strideC, int c_trans, int b_upper, int M, int N, int K,
                              float alpha, float beta, int batch, hipStream_t stream);

constexpr int kJacobiBlock = 32;     // columns per Jacobi block (pairs of 64)
constexpr int kInfoSweepLimit = 24;  // info: the small SVD's sweeps ran out before a rotation-free sweep
constexpr int kInfoNonFinite = 25;   // info: a column norm of the small SVD is NaN or Inf

}  // namespace galore
