// Gram matrices C = X^T X of the tall fp32 panels orthonormalised by
// Cholesky-QR (Halko et al. 2011, §4.5 re-orthonormalisation between the
// products of the subspace iteration), computed exactly on the int8 matrix
// cores.
//
// Cholesky-QR needs the Gram of some matrix close to X to full working
// accuracy: an unstructured Gram error E costs |E| / sigma_min(X)^2 of
// orthogonality, while the exact Gram of X + dX costs only about
// |dX| / sigma_min(X). So X is first rounded column by column to fixed point:
// column j gets the power-of-two scale 2^s_j with max_i |x_ij| * 2^s_j < 2^22
// (s_j from the column maximum), q_ij = rint(x_ij 2^s_j) is an integer of at
// most 23 bits with sign, and |dx_ij| <= 2^-23 max_i |x_ij| (normwise, below
// 2^-23 sqrt(rows) |x_j|; a dense column loses about 2^-23 * 4 of its norm).
// q is split into three balanced signed bytes, q = 2^16 d0 + 2^8 d1 + d2 with
// d1, d2 in [-128, 127] and |d0| <= 65, and
//     C_pq = 2^-(s_p + s_q) sum_{a, b} 2^(8 (4 - a - b)) (D_a^T D_b)_pq
// where every D_a^T D_b is an exact int32 sum (rows * 33024 < 2^31 for the
// five weight groups a + b = 0..4 up to 65024 rows; longer panels are summed
// in segments) and the five groups are combined in fp64 (2^-53 relative).
//
// Three launches per Gram:
//   colmax    the bit pattern of max_i |x_ij| per column (unsigned atomicMax
//             over row blocks; a NaN or Inf wins and marks the column), unless
//             the kernel that produced X already wrote them;
//   quantize  128 x 32 tiles of X -> digit planes D_a stored by columns
//             (column j of X is row j of each plane, rows padded with zeros),
//             so that the Gram reads K-contiguous 16-byte fragments;
//   gram      128 x 128 tiles of the upper triangle, 8 waves of 32 x 64, nine
//             v_mfma_i32_32x32x32_i8 per 32 x 32 block and 32 rows of X, digit
//             rows staged through LDS by direct buffer loads (32-bit lane
//             offsets), 64 rows per stage, the next stage in flight while the
//             current one is multiplied.
// Only the upper triangle of C (blocks on or above the diagonal) is written:
// the Cholesky factorisation reads nothing else.
#include "common.hpp"

namespace galore {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

constexpr int QR = 128;             // quantize tile rows
constexpr int QC = 32;              // quantize tile columns
constexpr int GT = 128;             // Gram tile (and column padding of the digit planes)

__global__ __launch_bounds__(256) void fill_u32_kernel(unsigned* p, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

// cmax[j] = max over rows of the bits of |x_ij| (non-negative floats order
// like their bit patterns; NaN and Inf compare above every finite value).
// Thread t of a workgroup takes column quad t (16-byte row loads, 8 rows in
// flight) when vec (rows 16-byte aligned, cols a multiple of 4), else single
// columns; grid (ceil(rows / rb), batch).
__global__ __launch_bounds__(256) void colmax_kernel(const float* Xb, int64_t ldx, int64_t strideX, int rows,
                                                     int cols, int rb, unsigned* cmaxb, int64_t strideCM, int vec) {
    const int b = blockIdx.y;
    const float* X = Xb + static_cast<int64_t>(b) * strideX;
    unsigned* cmax = cmaxb + static_cast<int64_t>(b) * strideCM;
    const int i0 = blockIdx.x * rb;
    const int i1 = min(rows, i0 + rb);
    if (vec) {
        for (int q = threadIdx.x; 4 * q < cols; q += blockDim.x) {
            unsigned m[4] = {0u, 0u, 0u, 0u};
            for (int i = i0; i < i1; i += 8) {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (i + e < i1) {
                        const f32x4 x = *reinterpret_cast<const f32x4*>(X + static_cast<int64_t>(i + e) * ldx + 4 * q);
#pragma unroll
                        for (int c = 0; c < 4; ++c) m[c] = max(m[c], __float_as_uint(fabsf(x[c])));
                    }
            }
#pragma unroll
            for (int c = 0; c < 4; ++c) atomicMax(cmax + 4 * q + c, m[c]);
        }
        return;
    }
    for (int j = threadIdx.x; j < cols; j += blockDim.x) {
        unsigned m[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) m[e] = 0u;
        // 16 independent loads in flight per thread
        for (int i = i0; i < i1; i += 16) {
#pragma unroll
            for (int e = 0; e < 16; ++e)
                if (i + e < i1) m[e] = max(m[e], __float_as_uint(fabsf(X[static_cast<int64_t>(i + e) * ldx + j])));
        }
#pragma unroll
        for (int e = 1; e < 16; ++e) m[0] = max(m[0], m[e]);
        atomicMax(cmax + j, m[0]);
    }
}

// scale exponent s with max |x| * 2^s < 2^22 (0 for a zero column)
__device__ __forceinline__ int col_shift(unsigned bits) {
    if (bits == 0u) return 0;
    int e;
    frexpf(__uint_as_float(bits), &e);     // max = f 2^e, f in [0.5, 1)
    return 22 - e;
}

// digit planes D_a[j][i] (int8), plane a at a * planeStride, row j at j * ldq;
// grid (ldq / QR, colsPad / QC, batch), rows >= `rows` and columns >= `cols` zero.
// No LDS: thread t of a 128-row x 32-column tile takes columns 4 (t >> 5) ..
// + 3 and rows 4 (t & 31) .. + 3 (four 16-byte row loads) and writes, per plane
// and column, its four rows' digits as one 4-byte store: the 32 threads of a
// column quad read 128 contiguous bytes of each row and fill 128 contiguous
// bytes of each plane row (measured on the headline step: 743 us per launch,
// 4.5 TB/s, against 878 us for 64 x 64 tiles and 1069 us for the LDS
// transpose it replaced).
__global__ __launch_bounds__(256) void quantize_kernel(const float* Xb, int64_t ldx, int64_t strideX, int rows,
                                                       int cols, const unsigned* cmaxb, int64_t strideCM,
                                                       int8_t* Db, int64_t ldq, int64_t planeStride,
                                                       int64_t strideD, int vload) {
    const int b = blockIdx.z;
    const float* X = Xb + static_cast<int64_t>(b) * strideX;
    const unsigned* cmax = cmaxb + static_cast<int64_t>(b) * strideCM;
    int8_t* D = Db + static_cast<int64_t>(b) * strideD;
    const int j0 = blockIdx.y * QC + 4 * (threadIdx.x >> 5);
    const int ib = blockIdx.x * QR + 4 * (threadIdx.x & 31);
    int sh[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) sh[e] = (j0 + e < cols) ? col_shift(cmax[j0 + e]) : 0;
    float xv[4][4];   // [row][column]
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int i = ib + v;
        const float* row = X + static_cast<int64_t>(i) * ldx + j0;
        if (i < rows && vload && j0 + 4 <= cols) {
            const f32x4 x = *reinterpret_cast<const f32x4*>(row);
#pragma unroll
            for (int e = 0; e < 4; ++e) xv[v][e] = x[e];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) xv[v][e] = (i < rows && j0 + e < cols) ? row[e] : 0.0f;
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        unsigned w0 = 0u, w1 = 0u, w2 = 0u;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int q = static_cast<int>(rintf(ldexpf(xv[v][e], sh[e])));
            const int d2 = static_cast<signed char>(q & 0xff);
            const int q1 = (q - d2) >> 8;
            const int d1 = static_cast<signed char>(q1 & 0xff);
            const int d0 = (q1 - d1) >> 8;
            w0 |= (static_cast<unsigned>(d0) & 0xffu) << (8 * v);
            w1 |= (static_cast<unsigned>(d1) & 0xffu) << (8 * v);
            w2 |= (static_cast<unsigned>(d2) & 0xffu) << (8 * v);
        }
        int8_t* dst = D + static_cast<int64_t>(j0 + e) * ldq + ib;
        *reinterpret_cast<unsigned*>(dst) = w0;
        *reinterpret_cast<unsigned*>(dst + planeStride) = w1;
        *reinterpret_cast<unsigned*>(dst + 2 * planeStride) = w2;
    }
}

typedef __attribute__((address_space(3))) void lds_void_t;

// one 16-byte buffer load per lane into LDS (lane i writes bytes 16 i .. of the
// wave's 1 KB); byte address voff + soff within the buffer
constexpr int kBufferDword3 = 0x00020000;   // raw buffer: 32-bit data format, no swizzle
__device__ __forceinline__ void buffer_load_lds16(__amdgpu_buffer_rsrc_t rsrc, int voff, int soff, void* lds_base) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)lds_base, 16, voff, soff, 0, 0);
}

constexpr int GK = 64;                   // rows of X (contraction) per LDS stage
constexpr int kPlaneB = GT * GK;         // one plane of one side in a stage (8 KB)
constexpr int kSideB = 3 * kPlaneB;      // three planes (24 KB)
constexpr int kStageB = 2 * kSideB;      // p side and q side (48 KB)
constexpr int kSegStages = 1016;         // stages per exact int32 segment (65024 rows)
// stages in LDS (two or three: 96 or 144 KB); measured on the headline step,
// 2466 us per launch with two against 2496 with three
#ifndef GALORE_GRAM_STAGES
#define GALORE_GRAM_STAGES 2
#endif
constexpr int kGramStages = GALORE_GRAM_STAGES;
static_assert(kGramStages == 2 || kGramStages == 3, "two or three Gram stages");

// Upper GT x GT tiles (u <= v) of C, one workgroup of 8 waves each: wave
// (wm, wn) owns rows 32 wm .. + 31 and columns 64 wn .. + 63 of the tile (two
// 32 x 32 blocks), five int32 accumulators (weight groups) per block. Each
// stage stages 64 rows of X for the tile's 128 p columns and 128 q columns
// (three digit planes each; a diagonal tile loads the p side only) through
// direct loads; a digit row's four 16-byte chunks sit at slot
// chunk ^ ((row / 4) % 4), so the 16 lanes of a fragment read hit 64 distinct
// banks. The next stage in flight while the current one is multiplied.
__global__ __launch_bounds__(512, 1) void gram_i8_kernel(const int8_t* Db, int64_t ldq, int64_t planeStride,
                                                         int64_t strideD, const unsigned* cmaxb, int64_t strideCM,
                                                         double* Cb, int64_t ldc, int64_t strideC, int cols, int nt) {
    __shared__ __attribute__((aligned(16))) int8_t sm[kGramStages * kStageB];
    const int ntiles = nt * (nt + 1) / 2;
    const int logical = xcd_logical_id(blockIdx.x + ntiles * blockIdx.y, ntiles * gridDim.y);
    const int b = logical / ntiles;
    int idx = logical - b * ntiles, u = 0;
    while (idx >= nt - u) {
        idx -= nt - u;
        ++u;
    }
    const int v = u + idx;
    const bool diag = (u == v);
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, lk = lane >> 5;
    // on a diagonal tile, a wave whose rows all lie below its columns has nothing
    // to do, nor has a wave whose rows all lie past the last column (the last
    // tile row of cols = 1056, say); ny = the wave's 32-column blocks with
    // columns before cols (the others are not stored)
    const bool idle = (diag && (wm >= 2 * wn + 2)) || GT * u + 32 * wm >= cols;
    const int qw = GT * v + 64 * wn;
    const int ny = __builtin_amdgcn_readfirstlane(qw >= cols ? 0 : (qw + 32 >= cols ? 1 : 2));
    const int8_t* D = Db + static_cast<int64_t>(b) * strideD;

    // this wave's direct loads: j = 6 wave + i -> side j / 24, plane (j / 8) % 3,
    // rows 16 (j % 8) + lane / 4 of the side, chunk slot lane % 4
    const int nload = (diag && wave >= 4) ? 0 : 6;
    // source offsets within the matrix's planes (3 planes of cpad x ldq bytes < 2^31)
    int src[6];
#pragma unroll
    for (int i = 0; i < 6; ++i) {
        const int j = 6 * wave + i;
        const int side = j / 24, pl = (j / 8) % 3, rb = j % 8;
        const int rloc = 16 * rb + (lane >> 2);
        const int row = (side ? GT * v : GT * u) + rloc;
        const int chunk = (lane & 3) ^ ((lane >> 4) & 3);          // (rloc / 4) % 4 == (lane / 16) % 4
        src[i] = static_cast<int>(pl * planeStride + static_cast<int64_t>(row) * ldq) + 16 * chunk;
    }
    // the matrix's digit planes as one buffer (strideD < 2^31 bytes): 32-bit
    // lane offsets and a scalar stage offset, so no 64-bit lane addresses are
    // kept in registers
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(D), 0, static_cast<int>(strideD), kBufferDword3);
    const int qside = diag ? 0 : kSideB;
    const int KT = static_cast<int>(ldq / GK);

    const unsigned* cmax = cmaxb + static_cast<int64_t>(b) * strideCM;
    double* C = Cb + static_cast<int64_t>(b) * strideC;

    for (int sg = 0; sg < KT; sg += kSegStages) {
        const int se = min(KT, sg + kSegStages);
        i32x16 acc[5][2];
#pragma unroll
        for (int w = 0; w < 5; ++w)
#pragma unroll
            for (int y = 0; y < 2; ++y)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[w][y][r] = 0;
        auto issue = [&](int buf, int kt) {
            int8_t* base = sm + buf * kStageB;
#pragma unroll
            for (int i = 0; i < 6; ++i) {
                const int j = 6 * wave + i;     // LDS destination: side j / 24, plane (j / 8) % 3, rows 16 (j % 8) ..
                if (i < nload)
                    buffer_load_lds16(rsrc, src[i], kt * GK,
                                      base + (j / 24) * kSideB + ((j / 8) % 3) * kPlaneB + (j % 8) * 1024);
            }
        };
        __syncthreads();                       // the previous segment's last stage is read
#pragma unroll
        for (int st = 0; st < kGramStages - 1; ++st)
            if (sg + st < se) issue(st, sg + st);
        for (int kt = sg; kt < se; ++kt) {
            // stage kt landed (a wave issues 6 or no loads per stage, so with
            // the next stage already in flight at most 6 may stay outstanding),
            // then for every wave; past the barrier every wave has also
            // finished stage kt - 1, whose buffer the next issue refills
            if (kGramStages == 3 && kt + 1 < se)
                asm volatile("s_waitcnt vmcnt(6)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
            else
                asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
            if (kt + kGramStages - 1 < se) issue((kt + kGramStages - 1 - sg) % kGramStages, kt + kGramStages - 1);
            if (idle) continue;
            const int8_t* sp = sm + ((kt - sg) % kGramStages) * kStageB;
            const int8_t* sq = sp + qside;
#pragma unroll 1
            for (int ks = 0; ks < 2; ++ks) {
                const int c = 2 * ks + lk;
                i32x4 fp[3];
                const int rp = 32 * wm + l32;
#pragma unroll
                for (int a = 0; a < 3; ++a)
                    fp[a] = *reinterpret_cast<const i32x4*>(sp + a * kPlaneB + rp * GK + 16 * (c ^ ((rp >> 2) & 3)));
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    if (y >= ny) break;
                    const int rq = 64 * wn + 32 * y + l32;
                    i32x4 fq[3];
#pragma unroll
                    for (int a = 0; a < 3; ++a)
                        fq[a] = *reinterpret_cast<const i32x4*>(sq + a * kPlaneB + rq * GK + 16 * (c ^ ((rq >> 2) & 3)));
#pragma unroll
                    for (int a = 0; a < 3; ++a)
#pragma unroll
                        for (int d = 0; d < 3; ++d)
                            acc[a + d][y] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fp[a], fq[d], acc[a + d][y], 0, 0, 0);
                }
            }
        }
        // the column maxima of the tile's p and q columns, staged in the
        // (now unused) digit stages once every wave is past the last one: the
        // epilogue reads one per stored entry, which from global memory waited
        // a latency per entry
        __syncthreads();
        unsigned* cms = reinterpret_cast<unsigned*>(sm);
        if (t < 2 * GT) cms[t] = cmax[min((t < GT ? GT * u : GT * v - GT) + t, cols - 1)];
        __syncthreads();
        if (idle) continue;
        // 32 x 32 accumulator layout: lane holds column (lane & 31), register r
        // holds row (r & 3) + 8 (r >> 2) + 4 (lane >> 5)
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const int q = GT * v + 64 * wn + 32 * y + l32;
            if (q >= cols) continue;
            const unsigned bq = cms[GT + 64 * wn + 32 * y + l32];
            const int shq = col_shift(bq);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int p = GT * u + 32 * wm + (r & 3) + 8 * (r >> 2) + 4 * lk;
                if (p >= cols) continue;
                const unsigned bp = cms[32 * wm + (r & 3) + 8 * (r >> 2) + 4 * lk];
                double* dstc = C + static_cast<int64_t>(p) * ldc + q;
                if (bp >= 0x7f800000u || bq >= 0x7f800000u) {
                    *dstc = __builtin_nan("");
                    continue;
                }
                const double sum = ldexp(static_cast<double>(acc[0][y][r]), 32) +
                                   ldexp(static_cast<double>(acc[1][y][r]), 24) +
                                   ldexp(static_cast<double>(acc[2][y][r]), 16) +
                                   ldexp(static_cast<double>(acc[3][y][r]), 8) + static_cast<double>(acc[4][y][r]);
                const double val = ldexp(sum, -(col_shift(bp) + shq));
                // the first segment stores (a select with the old value would
                // read it, and wait for it, before every store)
                if (sg == 0)
                    *dstc = val;
                else
                    *dstc += val;
            }
        }
    }
}

}  // namespace

int64_t gram_i8_ld(int rows) { return (static_cast<int64_t>(rows) + 127) / 128 * 128; }
int gram_i8_cols_pad(int cols) { return (cols + GT - 1) / GT * GT; }

hipError_t launch_fill_u32(unsigned* p, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream, p, n);
    return hipGetLastError();
}

hipError_t launch_gram_i8(const GramI8Args& g, int batch, hipStream_t stream) {
    const int64_t ldq = gram_i8_ld(g.rows);
    const int cpad = gram_i8_cols_pad(g.cols);
    const int64_t planeStride = static_cast<int64_t>(cpad) * ldq;
    const int64_t strideD = 3 * planeStride;
    // the Gram kernel addresses the digit planes with 32-bit offsets
    if (strideD > g.strideD || strideD > INT32_MAX || g.ldc < g.cols) return hipErrorInvalidValue;
    if (!g.cmax_ready) {
        const hipError_t e = launch_fill_u32(g.cmax, g.strideCM * batch, stream);
        if (e != hipSuccess) return e;
        const int rb = 128;
        dim3 grid((g.rows + rb - 1) / rb, batch);
        const int vec = (g.cols % 4 == 0) && (g.ldx % 4 == 0) && (batch == 1 || g.strideX % 4 == 0) &&
                        (reinterpret_cast<uintptr_t>(g.X) % 16 == 0);
        hipLaunchKernelGGL(colmax_kernel, grid, dim3(256), 0, stream, g.X, g.ldx, g.strideX, g.rows, g.cols, rb,
                           g.cmax, g.strideCM, vec);
    }
    {
        // 16-byte row loads where every row start of X is aligned (the digit
        // planes' rows, ldq a multiple of 128 bytes, always are for 4-byte stores)
        const int vload = (g.ldx % 4 == 0) && (batch == 1 || g.strideX % 4 == 0) &&
                          (reinterpret_cast<uintptr_t>(g.X) % 16 == 0);
        if (reinterpret_cast<uintptr_t>(g.D) % 4 != 0) return hipErrorInvalidValue;
        dim3 grid(static_cast<unsigned>(ldq / QR), cpad / QC, batch);
        hipLaunchKernelGGL(quantize_kernel, grid, dim3(256), 0, stream, g.X, g.ldx, g.strideX, g.rows, g.cols,
                           g.cmax, g.strideCM, g.D, ldq, planeStride, strideD, vload);
    }
    {
        const int nt = cpad / GT;
        dim3 grid(nt * (nt + 1) / 2, batch);
        hipLaunchKernelGGL(gram_i8_kernel, grid, dim3(512), 0, stream, g.D, ldq, planeStride, strideD, g.cmax,
                           g.strideCM, g.C, g.ldc, g.strideC, g.cols, nt);
    }
    return hipGetLastError();
}

}  // namespace galore
