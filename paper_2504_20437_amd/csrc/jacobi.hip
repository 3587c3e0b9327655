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
//   1. forms the 64 x 64 Gram of its two blocks in fp64 from fp32 matrix-core
//      partial sums of 8 products (v_mfma_f32_16x16x4f32), row chunks staged
//      in LDS;
//   2. skips the pair if every column pair is already orthogonal to the
//      tolerance (relative off-diagonal), otherwise
//   3. reduces the small Gram by one sweep of two-sided Jacobi held in
//      registers (fp32 entries, fp64 diagonal and angles; odd-even ordering,
//      64 rounds of up to 32 disjoint rotations, accumulating the rotation
//      Theta), and
//   4. applies Theta to the pair's 64 columns of Y on the fp32 matrix cores
//      (v_mfma_f32_32x32x2f32), 64-row chunks staged through LDS.
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
constexpr int GR = 64;             // rows per Gram chunk (two fp32 chunks fill the LDS buffer)
constexpr int AR = 64;             // rows per apply chunk
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
// form). The angle only has to be close (a residual off-diagonal is removed
// by later sweeps), so zeta and t use the hardware fp64 reciprocal and fp32
// square root; the rotation itself must be orthogonal to fp64 rounding, so
// c = 1 / sqrt(1 + t^2) is refined by two Newton steps from v_rsq_f64 and
// s = c t, giving c^2 + s^2 = 1 to within a few ulp.
__device__ __forceinline__ void rotation(double a, double b, double g, double& c, double& s) {
    const double zeta = (b - a) * 0.5 * __builtin_amdgcn_rcp(g);
    const float zf = static_cast<float>(zeta);
    const float az = fabsf(zf);
    float tf = __builtin_amdgcn_rcpf(az + __builtin_amdgcn_sqrtf(fmaf(az, az, 1.0f)));   // |zeta| huge: 0
    tf = (zf >= 0.0f) ? tf : -tf;                                                         // sign(0) = +1
    const double t = static_cast<double>(tf);
    const double x = fma(t, t, 1.0);
    double y = __builtin_amdgcn_rsq(x);
    y = y * fma(-0.5 * x * y, y, 1.5);
    y = y * fma(-0.5 * x * y, y, 1.5);
    c = y;
    s = y * t;
}

// Cross-lane moves of an fp32 value within a wave (DPP, no LDS traffic).
// dpp_swap_pairs: lane x receives lane x ^ 1. dpp_odd_partner: an odd lane x
// receives lane x + 1, an even lane x - 1. Lanes without a source (0 and 63 in
// the odd pattern) read 0, which only idle lanes consume; a zero old value and
// bound_ctrl let the compiler fold the lane move into the multiply that uses it
__device__ __forceinline__ float dpp_swap_pairs(float v) {
    const int i = __float_as_int(v);
    return __int_as_float(__builtin_amdgcn_update_dpp(0, i, 0xB1, 0xf, 0xf, true));
}
__device__ __forceinline__ float dpp_odd_partner(float v, bool odd) {
    const int i = __float_as_int(v);
    const int l = __builtin_amdgcn_update_dpp(0, i, 0x130, 0xf, 0xf, true);
    const int r = __builtin_amdgcn_update_dpp(0, i, 0x138, 0xf, 0xf, true);
    return __int_as_float(odd ? l : r);
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
                                                            double tol, int skip_dummy) {
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
        const int blk = (tid < JB) ? bi : bj;
        const int c = blk * JB + (tid & (JB - 1));
        col[tid] = (c < k) ? c : -1;
    }
    __syncthreads();

    // ---- 1. Gram of the pair's columns: the 10 upper 16 x 16 tiles of the
    //         64 x 64 result spread over the 4 waves, row chunks of GR rows
    //         double-buffered in LDS (fp32, as stored) with the next chunk
    //         prefetched in registers. Products on the fp32 matrix cores, two
    //         4-term MFMAs per partial sum, each partial sum added into fp64:
    //         an entry's error stays below about 8 fp32 ulps of
    //         sum_t |y_tp y_tq| <= |y_p| |y_q|, far under the tolerance the
    //         test and the rotations work to.
    {
        float (*Xs0)[PD] = reinterpret_cast<float (*)[PD]>(&regB[0][0]);   // rows 0 .. GR-1
        float (*Xs1)[PD] = Xs0 + GR;                                      // rows GR .. 2GR-1
        // tiles (ti, tj), ti <= tj, per wave; -1 = none
        const int tiles[4][3][2] = {{{0, 0}, {0, 1}, {0, 2}}, {{0, 3}, {1, 1}, {1, 2}},
                                    {{1, 3}, {2, 2}, {-1, -1}}, {{2, 3}, {3, 3}, {-1, -1}}};
        f64x4 acc[3];
#pragma unroll
        for (int x = 0; x < 3; ++x) acc[x] = f64x4{0.0, 0.0, 0.0, 0.0};
        const int l16 = lane & 15;
        const int lk = lane >> 4;
        // loader: thread t moves rows 4 q .. 4 q + 3 (q = t % 16) of columns
        // t / 16 + 16 e, e < 4, as 16-byte vectors (lanes of a column read
        // 256 contiguous bytes; the LDS writes hit 64 distinct banks)
        const bool vec4 = (k & 3) == 0;
        f32x4 pre[4];
        auto fetch = [&](int r0) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int w = (tid >> 4) + 16 * e, q = tid & 15;
                const int c = col[w];
                const int rr = r0 + 4 * q;
                const int64_t base = static_cast<int64_t>(c) * k + rr;
                if (c >= 0 && vec4 && rr + 4 <= k) {
                    pre[e] = *reinterpret_cast<const f32x4*>(Xt + base);
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v) pre[e][v] = (c >= 0 && rr + v < k) ? Xt[base + v] : 0.0f;
                }
            }
        };
        auto stash = [&](float (*Xs)[PD]) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int w = (tid >> 4) + 16 * e, q = tid & 15;
#pragma unroll
                for (int v = 0; v < 4; ++v) Xs[4 * q + v][w] = pre[e][v];
            }
        };
        const int nchunk = (k + GR - 1) / GR;
        fetch(0);
        stash(Xs0);
        __syncthreads();
        for (int ch = 0; ch < nchunk; ++ch) {
            float (*cur)[PD] = (ch & 1) ? Xs1 : Xs0;
            float (*nxt)[PD] = (ch & 1) ? Xs0 : Xs1;
            if (ch + 1 < nchunk) fetch((ch + 1) * GR);
#pragma unroll
            for (int x = 0; x < 3; ++x) {
                const int ti = tiles[wave][x][0], tj = tiles[wave][x][1];
                if (ti >= 0) {
#pragma unroll
                    for (int kk = 0; kk < GR; kk += 8) {
                        f32x4 part = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            cur[kk + lk][16 * ti + l16], cur[kk + lk][16 * tj + l16], f32x4{0.0f, 0.0f, 0.0f, 0.0f},
                            0, 0, 0);
                        part = __builtin_amdgcn_mfma_f32_16x16x4f32(cur[kk + 4 + lk][16 * ti + l16],
                                                                    cur[kk + 4 + lk][16 * tj + l16], part, 0, 0, 0);
#pragma unroll
                        for (int v = 0; v < 4; ++v) acc[x][v] += static_cast<double>(part[v]);
                    }
                }
            }
            if (ch + 1 < nchunk) stash(nxt);
            __syncthreads();
        }
        // fp32 16x16 block layout: lane holds column (lane & 15); accumulator
        // register v holds row 4 (lane >> 4) + v.
#pragma unroll
        for (int x = 0; x < 3; ++x) {
            const int ti = tiles[wave][x][0], tj = tiles[wave][x][1];
            if (ti >= 0) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int i = 16 * ti + 4 * lk + v;
                    const int j = 16 * tj + l16;
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
                const double g = static_cast<double>(Bc[(wq * 16 + jq) * 16 + jq]);
                double cr = 1.0, sr = 0.0;
                if (g * g > 1e-30 * (a * b)) rotation(a, b, g, cr, sr);
                // rotated slot p' = c p - s q goes to slot q, q' = s p + c q to slot p
                if (x == p) {
                    if ((p >> 4) == wave) {
                        const double cs2 = 2.0 * cr * sr * g;
                        Dn[p] = sr * sr * a + cs2 + cr * cr * b;
                        Dn[q] = cr * cr * a - cs2 + sr * sr * b;
                    }
                    CSw[(wave * JW + p) * 2 + 0] = static_cast<jreal>(cr);
                    CSw[(wave * JW + p) * 2 + 1] = static_cast<jreal>(sr);
                }
                c = static_cast<jreal>(cr);
                sg = static_cast<jreal>((x == p) ? sr : -sr);
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
#pragma unroll
                for (int j = 0; j < 16; ++j) gv[j] = sg * gv[j] + c * dpp_odd_partner(gv[j], odd);
                hgL = sg * hgL + c * dpp_odd_partner(hgL, odd);
                hgR = sg * hgR + c * dpp_odd_partner(hgR, odd);
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
    // ---- 4. Y_P <- Y_P Theta on the fp32 matrix cores: 64-row chunks through
    //         LDS (the next chunk in flight in registers), results stored from
    //         the accumulators (a lane writes four consecutive rows of a column)
    float (*Tf)[PD] = reinterpret_cast<float (*)[PD]>(&G[0][0]);          // 64 x 65 fp32
    float (*Xc)[PD] = reinterpret_cast<float (*)[PD]>(&G[0][0]) + JW;     // Xc[w][t]: column w, row t
    float* Y = Xtb + static_cast<int64_t>(b) * strideX;
    const bool vec4 = (k & 3) == 0;
    // loader: thread t moves rows 4 (t % 16) .. +3 of columns t / 16 + 16 e, e < 4
    const int aq = tid & 15, aw = tid >> 4;
    f32x4 pre[4];
    auto fetch = [&](int r0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int w = aw + 16 * e;
            const int c = col[w];
            const int rr = r0 + 4 * aq;
            const int64_t base = static_cast<int64_t>(c) * k + rr;
            if (c >= 0 && vec4 && rr + 4 <= k) {
                pre[e] = *reinterpret_cast<const f32x4*>(Y + base);
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v) pre[e][v] = (c >= 0 && rr + v < k) ? Y[base + v] : 0.0f;
            }
        }
    };
    const int tm = wave >> 1, tn = wave & 1;
    const int l32 = lane & 31, lk2 = lane >> 5;
    const int nch = (k + AR - 1) / AR;
    fetch(0);
    for (int ch = 0; ch < nch; ++ch) {
        const int r0 = ch * AR;
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int v = 0; v < 4; ++v) Xc[aw + 16 * e][4 * aq + v] = pre[e][v];
        __syncthreads();
        if (ch + 1 < nch) fetch(r0 + AR);
        f32x16 acc;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
#pragma unroll 8
        for (int kk = 0; kk < JW; kk += 2) {
            const float a = Xc[kk + lk2][32 * tm + l32];   // A[t][w] = Y[t][w]
            const float bv = Tf[kk + lk2][32 * tn + l32];  // B[w][c] = Theta[w][c]
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bv, acc, 0, 0, 0);
        }
        // 32x32 block layout: lane holds column (lane & 31) and rows
        // (v & 3) + 8 (v >> 2) + 4 (lane >> 5) for accumulator register v.
        const int c = col[32 * tn + l32];
        if (c >= 0) {
            float* dst = Y + static_cast<int64_t>(c) * k + r0;
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                const int t0 = 32 * tm + 8 * g4 + 4 * lk2;
                if (vec4 && r0 + t0 + 4 <= k) {
                    *reinterpret_cast<f32x4*>(dst + t0) =
                        f32x4{acc[4 * g4 + 0], acc[4 * g4 + 1], acc[4 * g4 + 2], acc[4 * g4 + 3]};
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (r0 + t0 + v < k) dst[t0 + v] = acc[4 * g4 + v];
                }
            }
        }
        __syncthreads();
    }
}

// norms[b][c] = |y_c| in fp64, one wave per column (coalesced over the
// column's k contiguous entries); grid (ceil(k / 4), batch)
__global__ __launch_bounds__(256) void jacobi_norms_kernel(const float* Ytb, int k, int64_t strideX,
                                                           double* normsb) {
    const int b = blockIdx.y;
    const int c = 4 * blockIdx.x + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (c >= k) return;
    const float* y = Ytb + static_cast<int64_t>(b) * strideX + static_cast<int64_t>(c) * k;
    double s = 0.0;
    for (int i = lane; i < k; i += 64) s += static_cast<double>(y[i]) * static_cast<double>(y[i]);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) normsb[static_cast<int64_t>(b) * k + c] = sqrt(s);
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
                                                              const int* rotb, int max_sweeps, int* info,
                                                              double* scratchb, int64_t strideScratch,
                                                              const int* expb, const double* normsb, int* permb,
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
    for (int c = tid; c < k; c += blockDim.x) sig[c] = normsb[static_cast<int64_t>(b) * k + c];
    __syncthreads();
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
    if (flags != nullptr) {
        if (tid == 0) flags[b] = refinable ? 1 : 0;
        for (int j = tid; j < k; j += blockDim.x) permb[static_cast<int64_t>(b) * k + j] = perm[j];
    }
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
        // 0: converged; max_sweeps: no sweep came out rotation-free;
        // max_sweeps + 1: a column norm is NaN or Inf (non-finite input)
        const int* rot = rotb + static_cast<int64_t>(b) * max_sweeps;
        int result = max_sweeps;
        for (int w = 0; w < max_sweeps; ++w) {
            if (rot[w] == 0) { result = 0; break; }
        }
        for (int c = 0; c < k; ++c)
            if (!(sig[c] <= DBL_MAX)) result = max_sweeps + 1;
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

hipError_t launch_jacobi_step(float* Yt, int k, int64_t strideX, int nblocks, int step, int sweep, int* rot,
                              int max_sweeps, double tol, int batch, hipStream_t stream) {
    // an odd number of real blocks (at least 3) leaves one padding block
    const int nreal = (k + JB - 1) / JB;
    const int skip_dummy = (nblocks > nreal && nreal >= 3) ? 1 : 0;
    hipLaunchKernelGGL(jacobi_pair_kernel, dim3(nblocks / 2 - skip_dummy, batch), dim3(JT), 0, stream, Yt, k,
                       strideX, nblocks, step, sweep, rot, max_sweeps, tol, skip_dummy);
    return hipGetLastError();
}

hipError_t launch_jacobi_finalize(const float* Yt, int k, int64_t strideX, int r, float* Ur, int64_t strideUr,
                                  float* sigma, int64_t stride_sigma, const int* rot, int max_sweeps, int* info,
                                  double* scratch, int64_t strideScratch, const int* exps, double* norms,
                                  int* perm, float* Xa, int* flags, int batch, hipStream_t stream) {
    hipLaunchKernelGGL(jacobi_norms_kernel, dim3((k + 3) / 4, batch), dim3(256), 0, stream, Yt, k, strideX, norms);
    const size_t shmem = static_cast<size_t>(k) * (sizeof(double) + sizeof(int));
    hipLaunchKernelGGL(jacobi_finalize_kernel, dim3(batch), dim3(256), shmem, stream, Yt, k, strideX, r, Ur,
                       strideUr, sigma, stride_sigma, rot, max_sweeps, info, scratch, strideScratch, exps, norms,
                       perm, flags);
    if (Xa != nullptr)
        hipLaunchKernelGGL(jacobi_gather_kernel, dim3(k, batch), dim3(256), 0, stream, Yt, k, strideX, norms, perm,
                           flags, Xa);
    return hipGetLastError();
}

}  // namespace galore
