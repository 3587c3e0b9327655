// Small SVD of the projected matrix B = Q^T A (k x l) in the randomized SVD
// (Halko et al. 2011, direct SVD of the small matrix; paper §4.1.2).
//
// The left singular vectors of B are the eigenvectors of B B^T = Z^T Z with
// Z = A^T Q = B^T. The host factors that Gram in fp64 as R^T R (Cholesky), so
// they are also the left singular vectors of Y = R^T (k x k). One-sided
// (Hestenes) Jacobi rotates the columns of Y until they are mutually
// orthogonal: Y W = U Sigma, so sigma_j is the norm of column j and u_j the
// column divided by it; no rotation needs to be accumulated. Y is stored by
// columns (column c contiguous), which is exactly the row-major upper
// triangle of R.
//
// Blocked for the GPU: the k columns form blocks of 32; a round-robin
// tournament pairs the blocks so that every step is a set of disjoint pairs
// (with an odd number of blocks, the pair with the padding block is not
// launched). A step is one launch, one workgroup per pair and matrix, which
//   1. forms the 64 x 64 Gram of its two blocks: 32-row chunks split exactly
//      into three bf16 planes in LDS, six plane products per tile on the bf16
//      matrix cores (v_mfma_f32_16x16x32_bf16) summed in fp32 per chunk and
//      in fp64 across chunks;
//   2. skips the pair if every column pair is already orthogonal to the
//      tolerance (relative off-diagonal), otherwise
//   3. reduces the small Gram by one sweep of two-sided Jacobi held in
//      registers (fp32 entries, fp64 diagonal and angles; odd-even ordering,
//      64 rounds of up to 32 disjoint rotations, accumulating the rotation
//      Theta), and
//   4. applies Theta to the pair's 64 columns of Y on the bf16 matrix cores,
//      Theta and the 32-row chunks of Y split into three planes as in 1.
// A sweep is nb - 1 steps; the matrix has converged when a whole sweep
// rotates nothing (rotation counts per sweep live in device memory, so no
// host synchronisation is needed).
//
// Rank deficiency: a pivot the Cholesky found dependent zeroes a row of R,
// i.e. a column of Y; zero columns are never rotated and stay exactly zero.
// If one of them is among the r leading columns, the finalize kernel replaces
// it by an orthonormal completion (unit vectors orthogonalised twice against
// the columns already kept), the singular value staying 0.
#include <float.h>

#include <type_traits>

#include "common.hpp"

namespace galore {
namespace {

constexpr int JB = kJacobiBlock;   // columns per block
constexpr int JW = 2 * JB;         // columns per pair (64)
#ifndef GALORE_JAC_INNER
#define GALORE_JAC_INNER 1
#endif
constexpr int kInnerSweeps = GALORE_JAC_INNER;   // inner sweeps of a pair's 64 x 64 Gram per visit
constexpr int JT = 256;            // threads (4 waves)
constexpr int PD = JW + 1;         // padded LDS row

static_assert(JW == 64, "the pair kernels assume 64 columns per pair");

__device__ __forceinline__ int ring_slot(int pos, int step, int n) {
    // circle method: slot 0 fixed, the others rotate by one per step
    if (pos == 0) return 0;
    int v = (pos - 1 - step) % (n - 1);
    if (v < 0) v += n - 1;
    return 1 + v;
}

// Power-of-two exponent e of each matrix with 2^e sqrt(max_j d_j) in [1/2, 1),
// d = the diagonal of the Gram Z^T Z that R factors (the squared column norms
// of B^T). Y = R^T enters the sweeps as 2^e R^T: the fp32 columns and the
// fp32 matrix-core partial sums of their Gram then neither underflow nor
// overflow whatever the gradient's scale (a gradient with singular values near
// 1e-20 would otherwise give partial products below the fp32 range and pass
// as converged), and sigma is scaled back by 2^-e, exactly. A zero or
// non-finite maximum gives e = 0.
__global__ __launch_bounds__(256) void jacobi_scale_kernel(const double* diagb, int k, int* expb) {
    const int b = blockIdx.x;
    const double* d = diagb + static_cast<int64_t>(b) * k;
    __shared__ double red[4];
    double mx = 0.0;
    for (int i = threadIdx.x; i < k; i += blockDim.x) mx = fmax(mx, d[i]);   // fmax drops NaN
    for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
        mx = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
        int e = 0;
        if (mx > 0.0 && mx <= DBL_MAX) {
            int ex;
            frexp(sqrt(mx), &ex);      // sqrt(mx) = f 2^ex, f in [1/2, 1)
            e = -ex;
        }
        expb[b] = e;
    }
}

__global__ __launch_bounds__(256) void jacobi_prepare_kernel(const double* Rb, int k,
                                                             int64_t strideR, float* Ytb,
                                                             int64_t strideX, int* rotb,
                                                             int max_sweeps, const int* expb) {
    const int b = blockIdx.y;
    const double* R = Rb + static_cast<int64_t>(b) * strideR;
    float* Yt = Ytb + static_cast<int64_t>(b) * strideX;
    const int e = expb[b];
    if (blockIdx.x == 0 && threadIdx.x < static_cast<unsigned>(max_sweeps))
        rotb[static_cast<int64_t>(b) * max_sweeps + threadIdx.x] = 0;
    const int64_t total = static_cast<int64_t>(k) * k;
    // column c of Y = R^T is row c of R
    for (int64_t pos = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; pos < total;
         pos += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int c = static_cast<int>(pos / k);
        const int i = static_cast<int>(pos - static_cast<int64_t>(c) * k);
        Yt[pos] = (i >= c) ? static_cast<float>(ldexp(R[pos], e)) : 0.0f;
    }
}

// Jacobi rotation (c, s) that zeroes the off-diagonal of [[a, g], [g, b]]
// under column p' = c p - s q, q' = s p + c q: t = tan(theta) is the smaller
// root of t^2 + 2 zeta t - 1 = 0, zeta = (b - a) / (2 g) (Rutishauser's
// form), b - a taken in fp64. The rotation is applied to fp32 entries, so
// fp32 suffices for the rest: the hardware reciprocal, square root and
// reciprocal square root (c = 1 / sqrt(1 + t^2), s = c t: c^2 + s^2 = 1 to a
// few fp32 ulp). The angle only has to be close: a residual off-diagonal is
// removed by later sweeps, and every visit recomputes the pair's Gram from the
// columns in fp64. |zeta| past the fp32 range gives t = 0.
__device__ __forceinline__ void rotation(double a, double b, float g, float& c, float& s) {
    const float zf = static_cast<float>(b - a) * 0.5f * __builtin_amdgcn_rcpf(g);
    const float az = fabsf(zf);
    float tf = __builtin_amdgcn_rcpf(az + __builtin_amdgcn_sqrtf(fmaf(az, az, 1.0f)));   // |zeta| huge: 0
    tf = (zf >= 0.0f) ? tf : -tf;                                                         // sign(0) = +1
    c = __builtin_amdgcn_rsqf(fmaf(tf, tf, 1.0f));
    s = c * tf;
}

// Cross-lane moves of an fp32 value within a wave (DPP, no LDS traffic).
// dpp_swap_pairs: lane x receives lane x ^ 1. dpp_from_next / dpp_from_prev:
// lane x receives lane x + 1 / x - 1 (whole-wave shifts); lanes without a
// source (63 / 0) read 0. A zero old value and bound_ctrl let the compiler
// fold the lane move into the multiply that uses it.
__device__ __forceinline__ float dpp_swap_pairs(float v) {
    const int i = __float_as_int(v);
    return __int_as_float(__builtin_amdgcn_update_dpp(0, i, 0xB1, 0xf, 0xf, true));
}
__device__ __forceinline__ float dpp_from_next(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x130, 0xf, 0xf, true));
}
__device__ __forceinline__ float dpp_from_prev(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x138, 0xf, 0xf, true));
}
// odd rounds: an odd lane's partner row is lane x + 1, an even lane's x - 1;
// with cn = c on odd lanes (0 on even ones) and cp the other way round, the
// partner term is fma(v[x - 1], cp, cn * v[x + 1]). Both lane moves are folded
// into the two instructions that use them (the compiler's own DPP folding
// leaves one or both as separate moves here: five instructions per value
// instead of three); lanes 0 and 63 read 0 for their missing neighbour, as
// the moves above do. The leading s_nop gives the two wait states a DPP read
// needs after a VALU write of its source (not checked by the compiler inside
// inline assembly).
__device__ __forceinline__ float rotate_odd(float v, float sg, float cn, float cp) {
    float t;
    asm("s_nop 1\n\t"
        "v_mul_f32_dpp %0, %1, %2 wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %1, %3 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
        : "=&v"(t)
        : "v"(v), "v"(cn), "v"(cp));
    return fmaf(sg, v, t);
}

// ---- bf16 planes of the pair's columns (Gram and rotation phases) ----------
// A 32-row chunk of the pair's 64 columns is held in LDS as three bf16 planes
// (h, m, l with x = h + m + l exactly: each plane takes the leading 8
// significant bits of what the previous ones left, by truncation, and an fp32
// significand has 24). Plane p of buffer s starts at s * kChunkBytes +
// p * kPlaneBytes; column c is 64 bytes (32 rows), its row octet o stored at
// 16-byte slot o ^ ((c >> 2) & 3), which keeps the 16-byte fragment reads, the
// transposing reads and the stores free of bank conflicts.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int PC = 32;                         // rows per plane chunk
constexpr int kPlaneBytes = JW * PC * 2;
constexpr int kChunkBytes = 3 * kPlaneBytes;
// plane products kept: h h, h m, m h, m m, h l, l h (the others are below
// 2^-25 of |a| |b|)
constexpr int kPlanePairs[6][2] = {{0, 0}, {0, 1}, {1, 0}, {1, 1}, {0, 2}, {2, 0}};

__device__ __forceinline__ void split8(f32x4 a, f32x4 b, bf16x8& h, bf16x8& m, bf16x8& l) {
    const float x[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    u32x4 ph, pm, pl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const unsigned u0 = __float_as_uint(x[2 * i]), u1 = __float_as_uint(x[2 * i + 1]);
        const float r0 = x[2 * i] - __uint_as_float(u0 & 0xffff0000u);
        const float r1 = x[2 * i + 1] - __uint_as_float(u1 & 0xffff0000u);
        const unsigned v0 = __float_as_uint(r0), v1 = __float_as_uint(r1);
        const float q0 = r0 - __uint_as_float(v0 & 0xffff0000u);
        const float q1 = r1 - __uint_as_float(v1 & 0xffff0000u);
        ph[i] = (u0 >> 16) | (u1 & 0xffff0000u);
        pm[i] = (v0 >> 16) | (v1 & 0xffff0000u);
        pl[i] = (__float_as_uint(q0) >> 16) | (__float_as_uint(q1) & 0xffff0000u);
    }
    h = __builtin_bit_cast(bf16x8, ph);
    m = __builtin_bit_cast(bf16x8, pm);
    l = __builtin_bit_cast(bf16x8, pl);
}

// thread t loads rows r0 + 8 (t & 3) .. + 7 of pair column t >> 2 (zeros past
// k and for padding columns)
__device__ __forceinline__ void pair_fetch(const float* X, int k, const int* col, int tid, int r0, f32x4& a,
                                           f32x4& b) {
    const int c = col[tid >> 2];
    const int rr = r0 + 8 * (tid & 3);
    const int64_t base = static_cast<int64_t>(c) * k + rr;
    if (c >= 0 && (k & 3) == 0 && rr + 8 <= k) {
        a = *reinterpret_cast<const f32x4*>(X + base);
        b = *reinterpret_cast<const f32x4*>(X + base + 4);
    } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            a[v] = (c >= 0 && rr + v < k) ? X[base + v] : 0.0f;
            b[v] = (c >= 0 && rr + 4 + v < k) ? X[base + 4 + v] : 0.0f;
        }
    }
}

__device__ __forceinline__ void pair_stash(unsigned char* lds, int s, int tid, f32x4 a, f32x4 b) {
    bf16x8 h, m, l;
    split8(a, b, h, m, l);
    const int c = tid >> 2, o = tid & 3;
    unsigned char* dst = lds + s * kChunkBytes + c * 64 + 16 * (o ^ ((c >> 2) & 3));
    *reinterpret_cast<bf16x8*>(dst) = h;
    *reinterpret_cast<bf16x8*>(dst + kPlaneBytes) = m;
    *reinterpret_cast<bf16x8*>(dst + 2 * kPlaneBytes) = l;
}

// Gram operand (A and B alike) of 16-column block blk: lane l holds column
// 16 blk + (l & 15), rows 8 (l >> 4) .. + 7 of the chunk
__device__ __forceinline__ bf16x8 gram_frag(const unsigned char* lds, int s, int p, int blk, int lane) {
    const int c = 16 * blk + (lane & 15), o = lane >> 4;
    return *reinterpret_cast<const bf16x8*>(lds + s * kChunkBytes + p * kPlaneBytes + c * 64 +
                                            16 * (o ^ ((c >> 2) & 3)));
}

// Rotation operand A (rows of Y_P): lane l holds row 16 tm + (l & 15) of the
// chunk, columns 32 ks + 8 (l >> 4) .. + 7. Two transposing reads: in each
// group of 16 lanes, lane j receives element j % 4 of the 8 bytes that lane
// 4 e + j / 4 points at (e = 0..3); lane L points at column w0 + L / 4, rows
// 16 tm + 4 (L % 4) .. + 3, so lane j gets row 16 tm + j, columns w0 .. w0 + 3.
__device__ __forceinline__ bf16x8 apply_frag(const unsigned char* lds, int s, int p, int tm, int ks, int lane) {
    const int L = lane & 15;
    const int t = 16 * tm + 4 * (L & 3);
    bf16x4 q[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int w = 32 * ks + 8 * (lane >> 4) + 4 * h + (L >> 2);
        const int off = s * kChunkBytes + p * kPlaneBytes + w * 64 + 16 * ((t >> 3) ^ ((w >> 2) & 3)) + 2 * (t & 7);
        q[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(reinterpret_cast<__attribute__((address_space(3))) bf16x4*>(
            reinterpret_cast<__attribute__((address_space(3))) unsigned char*>(reinterpret_cast<size_t>(lds)) + off));
    }
    return __builtin_shufflevector(q[0], q[1], 0, 1, 2, 3, 4, 5, 6, 7);
}

// Element type of the inner sweep's Gram and accumulated rotation. fp32: the
// rotation is applied to fp32 columns on the fp32 matrix cores anyway, the
// sweep only has to produce an orthogonal Theta that reduces the pair's
// off-diagonal; the pair Gram, the convergence test, the diagonal the sweep
// carries and the rotation angles stay fp64, so pairs are judged converged
// (and the last sweeps are steered) at fp64 accuracy.
typedef float jreal;

// Step of the block Jacobi (one workgroup per pair and matrix): Gram of the
// pair's 64 columns, convergence test, reduction of the small Gram, rotation
// of the columns, all in one 64 x 65 fp64 LDS buffer (see below).
__global__ __launch_bounds__(JT, 4) void jacobi_pair_kernel(float* Xtb, int k, int64_t strideX, int nb,
                                                            int step, int sweep, int* rotb, int max_sweeps,
                                                            double tol, int skip_dummy, const int* jpermb) {
    const int b = blockIdx.y;
    int* rot = rotb + static_cast<int64_t>(b) * max_sweeps;
    if (sweep > 0 && rot[sweep - 1] == 0) return;     // converged in an earlier sweep
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int h = blockIdx.x;
    if (skip_dummy) {
        // the padding block nb - 1 holds no columns: its pair is not launched
        // (every column pair inside a real block is still reduced by the inner
        // sweeps of that block's other pairs)
        const int pos = 1 + (step + nb - 2) % (nb - 1);
        const int hd = (pos < nb / 2) ? pos : nb - 1 - pos;
        h += (h >= hd) ? 1 : 0;
    }
    const int bi = ring_slot(h, step, nb);
    const int bj = ring_slot(nb - 1 - h, step, nb);
    const float* Xt = Xtb + static_cast<int64_t>(b) * strideX;

    // one 64 x 65 fp64 LDS buffer, reused phase by phase: the Gram's staged fp32
    // row chunks, then the Gram, then the inner sweep's exchange arrays, then the
    // fp32 Theta and row chunks of the rotation
    __shared__ double G[JW][PD];
    double (*regB)[PD] = G;
    __shared__ int col[JW];

    if (tid < JW) {
        // logical column c of the sweep's order -> stored column jperm[c]
        const int blk = (tid < JB) ? bi : bj;
        const int c = blk * JB + (tid & (JB - 1));
        col[tid] = (c < k) ? jpermb[static_cast<int64_t>(b) * k + c] : -1;
    }
    __syncthreads();

    unsigned char* lds = reinterpret_cast<unsigned char*>(&G[0][0]);
    static_assert(2 * kChunkBytes <= JW * PD * static_cast<int>(sizeof(double)), "two plane chunks fit the buffer");
    f32x4 pre0, pre1;

    // ---- 1. Gram of the pair's columns on the bf16 matrix cores: every
    //         32-row chunk of the 64 columns is split exactly into three bf16
    //         planes (x = h + m + l, 8 significant bits each, so the split of
    //         an fp32 value loses nothing) and staged in LDS, double-buffered,
    //         the next chunk in flight in registers. A 16 x 16 tile of the Gram
    //         sums the six plane products h h, h m, m h, m m, h l, l h
    //         (v_mfma_f32_16x16x32_bf16; the three left out are below 2^-25 of
    //         |y_p| |y_q|) in fp32 per chunk, each chunk's sum added into fp64.
    //         Tiles per wave: waves 0 and 1 the three upper tiles of blocks
    //         {0, 1} and {2, 3}, waves 2 and 3 the tiles (0, 2), (1, 2) and
    //         (0, 3), (1, 3), so a wave reads the fragments of at most three
    //         16-column blocks.
    {
        f64x4 acc[3];
#pragma unroll
        for (int x = 0; x < 3; ++x) acc[x] = f64x4{0.0, 0.0, 0.0, 0.0};
        const int nchunk = (k + PC - 1) / PC;
        pair_fetch(Xt, k, col, tid, 0, pre0, pre1);
        pair_stash(lds, 0, tid, pre0, pre1);
        __syncthreads();
        const bool diag = wave < 2;
        const int a0 = (wave == 1) ? 2 : 0, a1 = a0 + 1, bb = wave;     // bb: third block of waves 2, 3
        for (int ch = 0; ch < nchunk; ++ch) {
            const int s = ch & 1;
            if (ch + 1 < nchunk) pair_fetch(Xt, k, col, tid, (ch + 1) * PC, pre0, pre1);
            bf16x8 f0[3], f1[3];
#pragma unroll
            for (int p = 0; p < 3; ++p) {
                f0[p] = gram_frag(lds, s, p, a0, lane);
                f1[p] = gram_frag(lds, s, p, a1, lane);
            }
            if (diag) {
                f32x4 part[3];
#pragma unroll
                for (int x = 0; x < 3; ++x) part[x] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int q = 0; q < 6; ++q) {
                    const int pa = kPlanePairs[q][0], pb = kPlanePairs[q][1];
                    part[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f0[pa], f0[pb], part[0], 0, 0, 0);
                    part[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f0[pa], f1[pb], part[1], 0, 0, 0);
                    part[2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f1[pa], f1[pb], part[2], 0, 0, 0);
                }
#pragma unroll
                for (int x = 0; x < 3; ++x)
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[x][v] += static_cast<double>(part[x][v]);
            } else {
                bf16x8 f2[3];
#pragma unroll
                for (int p = 0; p < 3; ++p) f2[p] = gram_frag(lds, s, p, bb, lane);
                f32x4 part[2];
#pragma unroll
                for (int x = 0; x < 2; ++x) part[x] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int q = 0; q < 6; ++q) {
                    const int pa = kPlanePairs[q][0], pb = kPlanePairs[q][1];
                    part[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f0[pa], f2[pb], part[0], 0, 0, 0);
                    part[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f1[pa], f2[pb], part[1], 0, 0, 0);
                }
#pragma unroll
                for (int x = 0; x < 2; ++x)
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[x][v] += static_cast<double>(part[x][v]);
            }
            if (ch + 1 < nchunk) pair_stash(lds, s ^ 1, tid, pre0, pre1);
            __syncthreads();
        }
        // 16 x 16 block layout: lane holds column (lane & 15); accumulator
        // register v holds row 4 (lane >> 4) + v. The planes are dead: the
        // last barrier above ends every read of them.
        const int ntile = diag ? 3 : 2;
#pragma unroll
        for (int x = 0; x < 3; ++x) {
            if (x < ntile) {
                const int ti = diag ? ((x == 2) ? a1 : a0) : ((x == 0) ? a0 : a1);
                const int tj = diag ? ((x == 0) ? a0 : a1) : bb;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int i = 16 * ti + 4 * (lane >> 4) + v;
                    const int j = 16 * tj + (lane & 15);
                    G[i][j] = acc[x][v];
                    G[j][i] = acc[x][v];
                }
            }
        }
        __syncthreads();
    }

    // ---- 2. convergence test: every column pair orthogonal to the tolerance?
    //         |g_pq| <= tol sqrt(g_pp g_qq), compared squared; a pair with a
    //         zero column never counts, a pair with a NaN or Inf entry always
    //         does (non-finite input must not pass as converged: such a matrix
    //         runs every sweep and reports the sweep limit)
    {
        const double tol2 = tol * tol;
        int need = 0;
        for (int idx = tid; idx < JW * JW; idx += JT) {
            const int p = idx / JW, q = idx % JW;
            if (q > p) {
                const double dd = G[p][p] * G[q][q];
                const double gpq = G[p][q];
                if (dd != 0.0 && (!(dd <= DBL_MAX) || !(gpq * gpq <= tol2 * dd))) need = 1;
            }
        }
        need = __syncthreads_or(need);
        if (tid == 0 && need) atomicAdd(&rot[sweep], 1);
        if (!need) return;
    }

    // ---- 3. reduce the 64 x 64 Gram by one sweep of two-sided Jacobi, held
    //         in registers: lane x holds row x, wave w the columns
    //         16 w .. 16 w + 15 of it and of the accumulated rotation Theta.
    //         Odd-even ordering: round t pairs the slots (p, p + 1) with
    //         p = t mod 2, t mod 2 + 2, ...; every rotation also swaps its two
    //         slots, so that after 64 rounds every pair of columns has met once
    //         and the slot order is reversed. Row exchanges are lane shuffles,
    //         column exchanges register moves; the columns at a wave's slab
    //         edges come from its neighbours (halo copies) in odd rounds. The
    //         pair's diagonal entries are carried along exactly (2 x 2 formulas),
    //         its off-diagonal entry is read back from the holder each round.
    {
        double* Dv = &regB[0][0];                  // [2][64]: diagonal, ping-pong by round
        jreal* CSw = reinterpret_cast<jreal*>(Dv + 2 * JW);   // [4 waves][64][2]: (c, s) by first slot, wave-private
        jreal* Band = CSw + 4 * JW * 2;            // [2][4][16][16]: rows whose (x, x+1) entry a wave holds
        jreal* Halo = Band + 2 * 4 * 16 * 16;      // [4 waves][4][64]: edge columns (G left/right, Theta left/right)
        const int x = lane;
        const int c0 = 16 * wave;
        jreal gv[16], tv[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            gv[j] = static_cast<jreal>(G[x][c0 + j]);
            tv[j] = (x == c0 + j) ? jreal(1) : jreal(0);
        }
        const double dxx = G[x][x];
        const jreal exx = (x & 1) ? jreal(0) : static_cast<jreal>(G[x][x + 1]);
        __syncthreads();                       // the exchange arrays overwrite the Gram
        if (wave == 0) Dv[x] = dxx;
        // round 0 reads (x, x+1) for even x: stage it in Band[0]
        {
            const int jj = x + 1 - c0;
            if (!(x & 1) && jj >= 0 && jj < 16) {
                jreal* row = Band + ((0 * 4 + wave) * 16 + jj) * 16;
                row[jj] = exx;
            }
        }
        __syncthreads();
        jreal hgL = 0, hgR = 0, htL = 0, htR = 0;
        // rounds in (even, odd) pairs: the parity is a compile-time constant of
        // each half, so the parity branches vanish and the loop-carried
        // registers need no copies between rounds
        auto round = [&](auto parc) {
            constexpr int par = decltype(parc)::value;
            const double* Dc = Dv + par * JW;
            double* Dn = Dv + (par ^ 1) * JW;
            const jreal* Bc = Band + par * (4 * 16 * 16);
            jreal* Bn = Band + (par ^ 1) * (4 * 16 * 16);
            if (par) {
                // halo columns 16 w - 1 and 16 w + 16 as the neighbours left them
                if (wave > 0) {
                    hgL = Halo[((wave - 1) * 4 + 1) * JW + x];
                    htL = Halo[((wave - 1) * 4 + 3) * JW + x];
                }
                if (wave < 3) {
                    hgR = Halo[((wave + 1) * 4 + 0) * JW + x];
                    htR = Halo[((wave + 1) * 4 + 2) * JW + x];
                }
            }
            // the pair of row x and its rotation (every lane computes its own)
            const int p = par ? ((x & 1) ? x : x - 1) : (x & ~1);
            const bool idle = par && (x == 0 || x == JW - 1);
            jreal c = 0, sg = 1;               // idle rows stay as they are
            if (!idle) {
                const int q = p + 1;
                const int wq = q >> 4, jq = q & 15;
                const double a = Dc[p], b = Dc[q];
                const jreal gf = Bc[(wq * 16 + jq) * 16 + jq];
                const double g = static_cast<double>(gf);
                jreal cf = 1.0f, sf = 0.0f;
                if (g * g > 1e-30 * (a * b)) rotation(a, b, gf, cf, sf);
                // rotated slot p' = c p - s q goes to slot q, q' = s p + c q to slot p
                if (x == p) {
                    if ((p >> 4) == wave) {
                        const double cr = cf, sr = sf;
                        const double cs2 = 2.0 * cr * sr * g;
                        Dn[p] = sr * sr * a + cs2 + cr * cr * b;
                        Dn[q] = cr * cr * a - cs2 + sr * sr * b;
                    }
                    CSw[(wave * JW + p) * 2 + 0] = cf;
                    CSw[(wave * JW + p) * 2 + 1] = sf;
                }
                c = cf;
                sg = (x == p) ? sf : -sf;
            } else if ((x >> 4) == wave) {
                Dn[x] = Dc[x];
            }
            // rows: new row p = s row_p + c row_q, new row q = c row_p - s row_q;
            // the partner row is lane x ^ 1 (even rounds) or x -/+ 1 (odd rounds)
            if (!par) {
#pragma unroll
                for (int j = 0; j < 16; ++j) gv[j] = sg * gv[j] + c * dpp_swap_pairs(gv[j]);
            } else {
                const bool odd = (x & 1) != 0;
                const jreal cn = odd ? c : jreal(0), cp = odd ? jreal(0) : c;
#pragma unroll
                for (int j = 0; j < 16; ++j) gv[j] = rotate_odd(gv[j], sg, cn, cp);
                hgL = rotate_odd(hgL, sg, cn, cp);
                hgR = rotate_odd(hgR, sg, cn, cp);
            }
            // (c, s) of this wave's column pairs, published by their first rows
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const jreal* cw = CSw + wave * JW * 2;
            // columns: new col p = s col_p + c col_q, new col q = c col_p - s col_q
            if (!par) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const jreal cc = cw[(c0 + 2 * i) * 2 + 0], ss = cw[(c0 + 2 * i) * 2 + 1];
                    const jreal g0 = gv[2 * i], g1 = gv[2 * i + 1];
                    gv[2 * i] = ss * g0 + cc * g1;
                    gv[2 * i + 1] = cc * g0 - ss * g1;
                    const jreal t0 = tv[2 * i], t1 = tv[2 * i + 1];
                    tv[2 * i] = ss * t0 + cc * t1;
                    tv[2 * i + 1] = cc * t0 - ss * t1;
                }
            } else {
#pragma unroll
                for (int i = 0; i < 7; ++i) {
                    const jreal cc = cw[(c0 + 2 * i + 1) * 2 + 0], ss = cw[(c0 + 2 * i + 1) * 2 + 1];
                    const jreal g0 = gv[2 * i + 1], g1 = gv[2 * i + 2];
                    gv[2 * i + 1] = ss * g0 + cc * g1;
                    gv[2 * i + 2] = cc * g0 - ss * g1;
                    const jreal t0 = tv[2 * i + 1], t1 = tv[2 * i + 2];
                    tv[2 * i + 1] = ss * t0 + cc * t1;
                    tv[2 * i + 2] = cc * t0 - ss * t1;
                }
                if (wave > 0) {      // pair (16 w - 1, 16 w): this wave keeps the second slot
                    const jreal cc = cw[(c0 - 1) * 2 + 0], ss = cw[(c0 - 1) * 2 + 1];
                    gv[0] = cc * hgL - ss * gv[0];
                    tv[0] = cc * htL - ss * tv[0];
                }
                if (wave < 3) {      // pair (16 w + 15, 16 w + 16): this wave keeps the first slot
                    const jreal cc = cw[(c0 + 15) * 2 + 0], ss = cw[(c0 + 15) * 2 + 1];
                    gv[15] = ss * gv[15] + cc * hgR;
                    tv[15] = ss * tv[15] + cc * htR;
                }
            }
            // publish for the next round: the rows whose (x, x+1) entry lies in
            // this wave's slab, and after an even round the slab's edge columns
            {
                const int jj = x + 1 - c0;
                const int np = (par ^ 1) ? ((x & 1) ? x : -1) : ((x & 1) ? -1 : x);   // x first of a next pair?
                if (np >= 0 && x + 1 < JW && jj >= 0 && jj < 16) {
                    jreal* row = Bn + (wave * 16 + jj) * 16;
#pragma unroll
                    for (int j = 0; j < 16; ++j) row[j] = gv[j];
                }
                if (!par) {
                    Halo[(wave * 4 + 0) * JW + x] = gv[0];
                    Halo[(wave * 4 + 1) * JW + x] = gv[15];
                    Halo[(wave * 4 + 2) * JW + x] = tv[0];
                    Halo[(wave * 4 + 3) * JW + x] = tv[15];
                }
            }
            __syncthreads();
                };
        for (int isw = 0; isw < kInnerSweeps; ++isw)
            for (int t = 0; t < JW; t += 2) {
                round(std::integral_constant<int, 0>());
                round(std::integral_constant<int, 1>());
            }
        // ---- Theta to LDS in fp32 for the matrix cores; a sweep reverses the
        //      slot order, so after an odd number of sweeps output column j is
        //      slot 63 - j (a pair whose rotations are all small keeps its
        //      columns in place)
        float (*Tf0)[PD] = reinterpret_cast<float (*)[PD]>(&G[0][0]);
#pragma unroll
        for (int j = 0; j < 16; ++j)
            Tf0[x][(kInnerSweeps & 1) ? JW - 1 - (c0 + j) : c0 + j] = static_cast<float>(tv[j]);
        __syncthreads();
    }
    // ---- 4. Y_P <- Y_P Theta on the bf16 matrix cores: Theta split into
    //         three planes once (the wave's B fragments stay in registers),
    //         32-row chunks of Y_P split and staged as in the Gram, the A
    //         fragments (8 consecutive columns of one row) read with the
    //         transposing LDS read; six plane products per output, as in the
    //         Gram. Wave (tm, tn) writes rows 16 tm .. 16 tm + 15 of each chunk,
    //         columns 32 tn .. 32 tn + 31 (two 16 x 16 tiles), a lane four
    //         consecutive rows of one column per tile.
    {
        const int tm = wave >> 1, tn = wave & 1;
        const float (*Tf)[PD] = reinterpret_cast<const float (*)[PD]>(&G[0][0]);   // Theta[w][c], fp32
        bf16x8 bq[2][2][3];   // [column tile][K step of 32][plane]
#pragma unroll
        for (int ct = 0; ct < 2; ++ct)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const int c = 32 * tn + 16 * ct + (lane & 15);
                const int w0 = 32 * ks + 8 * (lane >> 4);
                f32x4 t0, t1;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    t0[v] = Tf[w0 + v][c];
                    t1[v] = Tf[w0 + 4 + v][c];
                }
                split8(t0, t1, bq[ct][ks][0], bq[ct][ks][1], bq[ct][ks][2]);
            }
        __syncthreads();                       // the Y_P planes overwrite Theta
        float* Y = Xtb + static_cast<int64_t>(b) * strideX;
        const int nch = (k + PC - 1) / PC;
        pair_fetch(Y, k, col, tid, 0, pre0, pre1);
        pair_stash(lds, 0, tid, pre0, pre1);
        __syncthreads();
        const int cst[2] = {col[32 * tn + (lane & 15)], col[32 * tn + 16 + (lane & 15)]};
        const bool vec4 = (k & 3) == 0;
        for (int ch = 0; ch < nch; ++ch) {
            const int s = ch & 1;
            const int r0 = ch * PC;
            if (ch + 1 < nch) pair_fetch(Y, k, col, tid, r0 + PC, pre0, pre1);
            f32x4 acc[2] = {f32x4{0.0f, 0.0f, 0.0f, 0.0f}, f32x4{0.0f, 0.0f, 0.0f, 0.0f}};
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                bf16x8 af[3];
#pragma unroll
                for (int p = 0; p < 3; ++p) af[p] = apply_frag(lds, s, p, tm, ks, lane);
#pragma unroll
                for (int q = 0; q < 6; ++q)
#pragma unroll
                    for (int ct = 0; ct < 2; ++ct)
                        acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[kPlanePairs[q][0]],
                                                                          bq[ct][ks][kPlanePairs[q][1]], acc[ct], 0,
                                                                          0, 0);
            }
            // rows r0 + 16 tm + 4 (lane >> 4) + v of column cst[ct]
            const int rr = r0 + 16 * tm + 4 * (lane >> 4);
#pragma unroll
            for (int ct = 0; ct < 2; ++ct) {
                const int c = cst[ct];
                if (c >= 0) {
                    float* dst = Y + static_cast<int64_t>(c) * k + rr;
                    if (vec4 && rr + 4 <= k) {
                        *reinterpret_cast<f32x4*>(dst) = acc[ct];
                    } else {
#pragma unroll
                        for (int v = 0; v < 4; ++v)
                            if (rr + v < k) dst[v] = acc[ct][v];
                    }
                }
            }
            if (ch + 1 < nch) pair_stash(lds, s ^ 1, tid, pre0, pre1);
            __syncthreads();
        }
    }
}

// norms[b][c] = |y_c| in fp64, one wave per column (coalesced over the
// column's k contiguous entries); grid (ceil(k / 4), batch). Between sweeps
// (rotb != NULL) a matrix whose previous sweep rotated nothing is skipped.
__global__ __launch_bounds__(256) void jacobi_norms_kernel(const float* Ytb, int k, int64_t strideX,
                                                           double* normsb, const int* rotb, int max_sweeps,
                                                           int sweep) {
    const int b = blockIdx.y;
    if (rotb != nullptr && sweep > 0 && rotb[static_cast<int64_t>(b) * max_sweeps + sweep - 1] == 0) return;
    const int c = 4 * blockIdx.x + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (c >= k) return;
    const float* y = Ytb + static_cast<int64_t>(b) * strideX + static_cast<int64_t>(c) * k;
    double s = 0.0;
    for (int i = lane; i < k; i += 64) s += static_cast<double>(y[i]) * static_cast<double>(y[i]);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) normsb[static_cast<int64_t>(b) * k + c] = sqrt(s);
}

// The order of the columns for the coming sweep: by decreasing norm (ties
// by index; a NaN norm counts as -1, last), jperm[b][rank] = column. Sweeping
// the blocks of a norm-ordered matrix pairs columns of like size first and
// cuts the rotations the later sweeps need (about 17% fewer pair rotations
// and one sweep fewer on the 4096 x 11008 workload in a CPU model of these
// sweeps). The rank of column c is the number of columns ahead of it; one
// thread per column, (k / 256) workgroups per matrix, each with the matrix's
// norms in LDS (one workgroup of 1024 threads per matrix took 63-124 us a
// sweep); converged matrices are skipped.
__global__ __launch_bounds__(256) void jacobi_order_kernel(const double* normsb, int k, int* jpermb,
                                                           const int* rotb, int max_sweeps, int sweep) {
    const int b = blockIdx.y;
    if (sweep > 0 && rotb[static_cast<int64_t>(b) * max_sweeps + sweep - 1] == 0) return;
    extern __shared__ unsigned char smem[];
    double* nv = reinterpret_cast<double*>(smem);
    for (int c = threadIdx.x; c < k; c += blockDim.x) {
        const double v = normsb[static_cast<int64_t>(b) * k + c];
        nv[c] = (v == v) ? v : -1.0;
    }
    __syncthreads();
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= k) return;
    const double vc = nv[c];
    int rank = 0;
    for (int c2 = 0; c2 < k; ++c2) {
        const double v2 = nv[c2];
        rank += (v2 > vc) || (v2 == vc && c2 < c);
    }
    jpermb[static_cast<int64_t>(b) * k + rank] = c;
}

// Xa[j][:] = y_perm(j) / sigma_perm(j) (row j of the result contiguous) for the
// matrices finalize marked refinable; one workgroup per row j; grid (k, batch)
__global__ __launch_bounds__(256) void jacobi_gather_kernel(const float* Ytb, int k, int64_t strideX,
                                                            const double* normsb, const int* permb,
                                                            const int* flags, float* Xab) {
    const int b = blockIdx.y;
    if (flags[b] == 0) return;
    const int j = blockIdx.x;
    const int c = permb[static_cast<int64_t>(b) * k + j];
    const double inv = 1.0 / normsb[static_cast<int64_t>(b) * k + c];
    const float* y = Ytb + static_cast<int64_t>(b) * strideX + static_cast<int64_t>(c) * k;
    float* x = Xab + static_cast<int64_t>(b) * strideX + static_cast<int64_t>(j) * k;
    for (int i = threadIdx.x; i < k; i += blockDim.x) x[i] = static_cast<float>(static_cast<double>(y[i]) * inv);
}

// sigma_j = |y_j| (fp64), order descending (ties by index, NaN last);
// Ur[:, j] = y_perm(j) / sigma_perm(j) for the r leading columns, zero columns
// completed orthonormally. scratch: 2 k + r doubles per matrix.
__global__ __launch_bounds__(256) void jacobi_finalize_kernel(const float* Ytb, int k, int64_t strideX,
                                                              int r, float* Urb, int64_t strideUr,
                                                              float* sigma, int64_t stride_sigma,
                                                              const int* rotb, int max_sweeps, int nsweeps, int* info,
                                                              double* scratchb, int64_t strideScratch,
                                                              const int* expb, const double* normsb, const int* permb,
                                                              int* flags) {
    extern __shared__ unsigned char smem[];
    double* sig = reinterpret_cast<double*>(smem);
    int* perm = reinterpret_cast<int*>(sig + k);
    __shared__ double red[4];
    __shared__ int nkeep_s;
    const int b = blockIdx.x;
    const float* Yt = Ytb + static_cast<int64_t>(b) * strideX;
    float* Ur = Urb + static_cast<int64_t>(b) * strideUr;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // the descending order of the norms (ties by index, NaN last), ranked by
    // jacobi_order_kernel into permb before this kernel
    for (int c = tid; c < k; c += blockDim.x) {
        sig[c] = normsb[static_cast<int64_t>(b) * k + c];
        perm[c] = permb[static_cast<int64_t>(b) * k + c];
    }
    __syncthreads();
    if (tid == 0) {
        int nk = 0;
        while (nk < r && sig[perm[nk]] > 0.0) ++nk;      // NaN and zero columns end the run
        nkeep_s = nk;
    }
    if (sigma != nullptr) {
        for (int j = tid; j < r; j += blockDim.x) {
            const double v = ldexp(sig[perm[j]], -expb[b]);     // undo the sweeps' scaling
            sigma[static_cast<int64_t>(b) * stride_sigma + j] = (v > 0.0 || v != v) ? static_cast<float>(v) : 0.0f;
        }
    }
    __syncthreads();
    const int nkeep = nkeep_s;
    // refinable: every column norm finite and positive; those matrices get all
    // k ordered columns (jacobi_gather_kernel, from permb) and their Ur from the
    // fp64 refinement; the others (rank-deficient, non-finite) keep the vectors
    // written here
    const bool refinable = flags != nullptr && (nkeep == r) && sig[perm[k - 1]] > 0.0 && sig[perm[0]] <= DBL_MAX;
    if (flags != nullptr && tid == 0) flags[b] = refinable ? 1 : 0;
    if (!refinable) {
        const int64_t total = static_cast<int64_t>(k) * nkeep;
        for (int64_t pos = tid; pos < total; pos += blockDim.x) {
            const int i = static_cast<int>(pos / nkeep);
            const int j = static_cast<int>(pos - static_cast<int64_t>(i) * nkeep);
            const int c = perm[j];
            Ur[static_cast<int64_t>(i) * r + j] =
                static_cast<float>(static_cast<double>(Yt[static_cast<int64_t>(c) * k + i]) / sig[c]);
        }
    }
    if (tid == 0 && info != nullptr) {
        // 0: converged; kInfoSweepLimit: none of the nsweeps sweeps run came
        // out rotation-free; kInfoNonFinite: a column norm is NaN or Inf
        // (non-finite input)
        const int* rot = rotb + static_cast<int64_t>(b) * max_sweeps;
        int result = kInfoSweepLimit;
        for (int w = 0; w < nsweeps; ++w) {
            if (rot[w] == 0) { result = 0; break; }
        }
        for (int c = 0; c < k; ++c)
            if (!(sig[c] <= DBL_MAX)) result = kInfoNonFinite;
        info[b] = result;
    }
    if (nkeep >= r) return;
    // ---- orthonormal completion of columns nkeep .. r-1 (rank-deficient B) ----
    // Each new column starts from the unit vector e_i least covered by the
    // columns kept so far (smallest squared row norm rn2[i], so its residual
    // 1 - rn2[i] is the largest, at least (k - j) / k), is orthogonalised twice
    // against them (classical Gram-Schmidt) and normalised.
    __syncthreads();
    double* v = scratchb + static_cast<int64_t>(b) * strideScratch;   // k
    double* dots = v + k;                                              // r
    double* rn2 = dots + r;                                            // k
    __shared__ double bestv[4];
    __shared__ int besti[4];
    for (int i = tid; i < k; i += blockDim.x) {
        double a = 0.0;
        for (int m = 0; m < nkeep; ++m) {
            const double u = Ur[static_cast<int64_t>(i) * r + m];
            a += u * u;
        }
        rn2[i] = a;
    }
    __syncthreads();
    for (int j = nkeep; j < r; ++j) {
        // argmin of rn2 (lowest index on ties)
        double bv = 1e300;
        int bi = k;
        for (int i = tid; i < k; i += blockDim.x)
            if (rn2[i] < bv) { bv = rn2[i]; bi = i; }
        for (int o = 32; o > 0; o >>= 1) {
            const double ov = __shfl_xor(bv, o);
            const int oi = __shfl_xor(bi, o);
            if (ov < bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
        }
        if (lane == 0) { bestv[wave] = bv; besti[wave] = bi; }
        __syncthreads();
        int cand = besti[0];
        double cv = bestv[0];
        for (int w = 1; w < 4; ++w)
            if (bestv[w] < cv || (bestv[w] == cv && besti[w] < cand)) { cv = bestv[w]; cand = besti[w]; }
        for (int i = tid; i < k; i += blockDim.x) v[i] = (i == cand) ? 1.0 : 0.0;
        __syncthreads();
        for (int pass = 0; pass < 2; ++pass) {
            for (int m = tid; m < j; m += blockDim.x) {
                double d = 0.0;
                for (int i = 0; i < k; ++i) d += static_cast<double>(Ur[static_cast<int64_t>(i) * r + m]) * v[i];
                dots[m] = d;
            }
            __syncthreads();
            for (int i = tid; i < k; i += blockDim.x) {
                double x = v[i];
                for (int m = 0; m < j; ++m) x -= dots[m] * static_cast<double>(Ur[static_cast<int64_t>(i) * r + m]);
                v[i] = x;
            }
            __syncthreads();
        }
        double nn = 0.0;
        for (int i = tid; i < k; i += blockDim.x) nn += v[i] * v[i];
        for (int o = 32; o > 0; o >>= 1) nn += __shfl_xor(nn, o);
        if (lane == 0) red[wave] = nn;
        __syncthreads();
        const double norm = sqrt(red[0] + red[1] + red[2] + red[3]);
        const double inv = (norm > 0.0) ? 1.0 / norm : 0.0;
        for (int i = tid; i < k; i += blockDim.x) {
            const double u = v[i] * inv;
            Ur[static_cast<int64_t>(i) * r + j] = static_cast<float>(u);
            rn2[i] += u * u;
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_jacobi_prepare(const double* R, int k, int64_t strideR, float* Yt, int64_t strideX,
                                 int* rot, int max_sweeps, const double* diag, int* exps, int batch,
                                 hipStream_t stream) {
    hipLaunchKernelGGL(jacobi_scale_kernel, dim3(batch), dim3(256), 0, stream, diag, k, exps);
    int64_t blocks = (static_cast<int64_t>(k) * k + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(jacobi_prepare_kernel, dim3(static_cast<unsigned>(blocks), batch), dim3(256),
                       0, stream, R, k, strideR, Yt, strideX, rot, max_sweeps, exps);
    return hipGetLastError();
}

hipError_t launch_jacobi_order(const float* Yt, int k, int64_t strideX, double* norms, int* jperm, const int* rot,
                               int max_sweeps, int sweep, int batch, hipStream_t stream) {
    hipLaunchKernelGGL(jacobi_norms_kernel, dim3((k + 3) / 4, batch), dim3(256), 0, stream, Yt, k, strideX, norms, rot,
                       max_sweeps, sweep);
    hipLaunchKernelGGL(jacobi_order_kernel, dim3((k + 255) / 256, batch), dim3(256), static_cast<size_t>(k) * sizeof(double),
                       stream, norms, k, jperm, rot, max_sweeps, sweep);
    return hipGetLastError();
}

hipError_t launch_jacobi_step(float* Yt, int k, int64_t strideX, int nblocks, int step, int sweep, int* rot,
                              int max_sweeps, double tol, const int* jperm, int batch, hipStream_t stream) {
    // an odd number of real blocks (at least 3) leaves one padding block
    const int nreal = (k + JB - 1) / JB;
    const int skip_dummy = (nblocks > nreal && nreal >= 3) ? 1 : 0;
    hipLaunchKernelGGL(jacobi_pair_kernel, dim3(nblocks / 2 - skip_dummy, batch), dim3(JT), 0, stream, Yt, k,
                       strideX, nblocks, step, sweep, rot, max_sweeps, tol, skip_dummy, jperm);
    return hipGetLastError();
}

hipError_t launch_jacobi_finalize(const float* Yt, int k, int64_t strideX, int r, float* Ur, int64_t strideUr,
                                  float* sigma, int64_t stride_sigma, const int* rot, int max_sweeps, int nsweeps,
                                  int* info,
                                  double* scratch, int64_t strideScratch, const int* exps, double* norms,
                                  int* perm, float* Xa, int* flags, int batch, hipStream_t stream) {
    hipLaunchKernelGGL(jacobi_norms_kernel, dim3((k + 3) / 4, batch), dim3(256), 0, stream, Yt, k, strideX, norms,
                       static_cast<const int*>(nullptr), 0, 0);
    // their descending order into perm (sweep 0: no convergence check)
    hipLaunchKernelGGL(jacobi_order_kernel, dim3((k + 255) / 256, batch), dim3(256), static_cast<size_t>(k) * sizeof(double),
                       stream, norms, k, perm, static_cast<const int*>(nullptr), 0, 0);
    const size_t shmem = static_cast<size_t>(k) * (sizeof(double) + sizeof(int));
    hipLaunchKernelGGL(jacobi_finalize_kernel, dim3(batch), dim3(256), shmem, stream, Yt, k, strideX, r, Ur,
                       strideUr, sigma, stride_sigma, rot, max_sweeps, nsweeps, info, scratch, strideScratch, exps,
                       norms,
                       perm, flags);
    if (Xa != nullptr)
        hipLaunchKernelGGL(jacobi_gather_kernel, dim3(k, batch), dim3(256), 0, stream, Yt, k, strideX, norms, perm,
                           flags, Xa);
    return hipGetLastError();
}

}  // namespace galore
