// Products with a bf16-stored gradient on the bf16 matrix cores, exact to
// fp32 accumulation.
//
// When G is stored in bf16, every product A X (or A^T Q) of the subspace
// update has one operand that is exactly bf16. The fp32 operand X is split
// into three bf16 terms, X = X1 + X2 + X3 (X1 = bf16(X), X2 = bf16(X - X1),
// X3 = bf16(X - X1 - X2): 3 x 8 significand bits cover the 24 of fp32), so
//   A X = A X1 + A X2 + A X3
// is three v_mfma_f32_32x32x16_bf16 products with exact bf16 x bf16 partial
// products accumulated in fp32: the same arithmetic class as an fp32 GEMM, on
// a unit with 16x the fp32 matrix rate.
//
// Operand layouts (both with the reduction index contiguous, so that a lane's
// eight consecutive k values are one 16-byte LDS read):
//   A: bf16, M x K rows (G itself, or its transposed copy made by
//      transpose_bf16 for the products with A^T);
//   B: three bf16 planes, each N x K rows (made by split3_transpose from the
//      fp32 K x N operand).
// C = alpha * A B + beta * C in fp32, M x N row-major.
//
// Tile 128 x 128 x 64, four wave64s each owning 64 x 64 (2 x 2 blocks of
// 32 x 32), LDS rows padded to 72 bf16 (144 bytes: the 16 lanes of a 16-byte
// read fall on distinct banks), next tile prefetched in registers, XCD-aware
// row-grouped tile order.
#include <type_traits>

#include "common.hpp"

namespace galore {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int XM = 128;
constexpr int XN = 128;
constexpr int XK = 64;
constexpr int XKP = XK + 8;     // padded LDS row (bf16): 144 bytes, 16-byte lane reads conflict-free
constexpr int XT = 256;


// --------------------------------------------------------------------------
// dst (cols x rows, ld ldd) = src^T (src rows x cols, ld lds), bf16, 64 x 64 tiles
// --------------------------------------------------------------------------
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* srcb, int64_t lds, int64_t strideS,
                                                             uint16_t* dstb, int64_t ldd, int64_t strideD, int rows,
                                                             int cols) {
    __shared__ uint16_t tile[64][66];
    const int b = blockIdx.z;
    const uint16_t* src = srcb + static_cast<int64_t>(b) * strideS;
    uint16_t* dst = dstb + static_cast<int64_t>(b) * strideD;
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int r = r0 + i, c = c0 + tx;
        tile[i][tx] = (r < rows && c < cols) ? src[static_cast<int64_t>(r) * lds + c] : 0;
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int c = c0 + i, r = r0 + tx;
        if (c < cols && r < rows) dst[static_cast<int64_t>(c) * ldd + r] = tile[tx][i];
    }
}

// --------------------------------------------------------------------------
// plane_p (cols x rows, ld ldp) = split_p(src)^T, src fp32 rows x cols (ld lds);
// planes at planeStride elements from each other; rows..rows_pad-1 zero-filled.
// No LDS: in a 64 x 64 tile, thread t takes the 4 x 4 block of columns
// 4 (t >> 4) .. + 3 and rows 4 (t & 15) .. + 3 (four 16-byte row loads) and
// writes, per plane and column, its four rows as one 8-byte store, so that the
// 16 threads of a column quad fill 128 contiguous bytes of each plane row
// (measured: 911 us per launch of the headline step's mix against 982 us for
// 128-row x 32-column tiles and 1076 us for the LDS transpose it replaced).
// --------------------------------------------------------------------------
__global__ __launch_bounds__(256) void split3_transpose_kernel(const float* srcb, int64_t lds, int64_t strideS,
                                                               uint16_t* planesb, int64_t ldp, int64_t planeStride,
                                                               int64_t strideP, int rows, int cols, int rows_pad,
                                                               const float* rowscaleb, int64_t strideRS, int vload,
                                                               int vstore) {
    const int b = blockIdx.z;
    const float* src = srcb + static_cast<int64_t>(b) * strideS;
    uint16_t* planes = planesb + static_cast<int64_t>(b) * strideP;
    const float* rowscale = rowscaleb ? rowscaleb + static_cast<int64_t>(b) * strideRS : nullptr;
    const int c0 = blockIdx.x * 64 + 4 * (threadIdx.x >> 4);
    const int rb = blockIdx.y * 64 + 4 * (threadIdx.x & 15);
    if (c0 >= cols || rb >= rows_pad) return;
    float x[4][4];   // [row][column]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = rb + i;
        const float* row = src + static_cast<int64_t>(r) * lds + c0;
        if (r < rows && vload && c0 + 4 <= cols) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(row);
#pragma unroll
            for (int e = 0; e < 4; ++e) x[i][e] = v[e];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) x[i][e] = (r < rows && c0 + e < cols) ? row[e] : 0.0f;
        }
        if (rowscale && r < rows) {
            const float sc = rowscale[r];   // one fp32 rounding, then an exact split
#pragma unroll
            for (int e = 0; e < 4; ++e) x[i][e] *= sc;
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int c = c0 + e;
        if (c >= cols) break;
        uint16_t h[3][4];
#pragma unroll
        for (int i = 0; i < 4; ++i) split3_rn(x[i][e], h[0][i], h[1][i], h[2][i]);
        uint16_t* dst = planes + static_cast<int64_t>(c) * ldp + rb;
        if (vstore && rb + 4 <= rows_pad) {
#pragma unroll
            for (int p = 0; p < 3; ++p)
                *reinterpret_cast<uint2*>(dst + p * planeStride) =
                    make_uint2(h[p][0] | (static_cast<uint32_t>(h[p][1]) << 16),
                               h[p][2] | (static_cast<uint32_t>(h[p][3]) << 16));
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (rb + i < rows_pad) {
#pragma unroll
                    for (int p = 0; p < 3; ++p) dst[p * planeStride + i] = h[p][i];
                }
        }
    }
}

// --------------------------------------------------------------------------
// plane_p (rows x ldp) = split_p(src), src fp32 rows x cols (ld lds), columns
// cols..cols_pad-1 zero-filled; four consecutive columns per thread (one
// 16-byte load, one 8-byte store per plane when aligned)
// --------------------------------------------------------------------------
__global__ __launch_bounds__(256) void split3_rows_kernel(const float* srcb, int64_t lds, int64_t strideS,
                                                          uint16_t* planesb, int64_t ldp, int64_t planeStride,
                                                          int64_t strideP, int rows, int cols, int cols_pad,
                                                          int vec) {
    const int b = blockIdx.z;
    const float* src = srcb + static_cast<int64_t>(b) * strideS;
    uint16_t* planes = planesb + static_cast<int64_t>(b) * strideP;
    const int r = blockIdx.y;
    const int c0 = 4 * (blockIdx.x * blockDim.x + threadIdx.x);
    if (r >= rows || c0 >= cols_pad) return;
    const float* srow = src + static_cast<int64_t>(r) * lds;
    float x[4];
    if (vec && c0 + 4 <= cols) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(srow + c0);
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = v[e];
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = (c0 + e < cols) ? srow[c0 + e] : 0.0f;
    }
    uint16_t h[3][4];
#pragma unroll
    for (int e = 0; e < 4; ++e) split3_rn(x[e], h[0][e], h[1][e], h[2][e]);
    const int64_t o = static_cast<int64_t>(r) * ldp + c0;
#pragma unroll
    for (int p = 0; p < 3; ++p) {
        uint16_t* dst = planes + o + p * planeStride;
        if (vec && c0 + 4 <= cols_pad) {
            *reinterpret_cast<uint2*>(dst) = make_uint2(h[p][0] | (uint32_t(h[p][1]) << 16),
                                                        h[p][2] | (uint32_t(h[p][3]) << 16));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (c0 + e < cols_pad) dst[e] = h[p][e];
        }
    }
}

// --------------------------------------------------------------------------
// C (M x N) = alpha * A (M x K bf16 rows) * B^T (3 planes, N x K bf16 rows) + beta * C
// --------------------------------------------------------------------------
struct Bx3Args {
    const uint16_t* A;
    int64_t lda, strideA;
    const uint16_t* B;          // plane 0; planes p at B + p * planeStride
    int64_t ldb, planeStride, strideB;
    float* C;
    int64_t ldc, strideC;
    int M, N, K;
    float alpha, beta;
    int c_trans;                // direct kernel only: store C^T (C[n * ldc + m])
    int64_t planeStrideA;       // direct kernel with three A planes: plane p at A + p * planeStrideA
    int b_upper;                // direct kernel: B upper triangular (B[kk][n] = 0 for kk > n)
    unsigned* cmax;             // direct kernel, row-major C: per-column max of |C| (bits; atomicMax), or null
    int64_t strideCM;
    const float* nscale;        // direct kernel: C(m, n) scaled by nscale[n] (per matrix at strideNS), or null
    int64_t strideNS;
};

__global__ __launch_bounds__(XT, 2) void gemm_bf16x3_kernel(Bx3Args g, int vec) {
    __shared__ __attribute__((aligned(16))) uint16_t As[XM][XKP];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[3][XN][XKP];

    const int num_n = gridDim.x, num_m = gridDim.y;
    const int tiles = num_n * num_m;
    const int lin = blockIdx.x + num_n * (blockIdx.y + num_m * blockIdx.z);
    const int logical = xcd_logical_id(lin, tiles * gridDim.z);
    const int bz = logical / tiles;
    int tm, tn;
    grouped_tile(logical - bz * tiles, num_m, num_n, 8, tm, tn);
    const uint16_t* A = g.A + static_cast<int64_t>(bz) * g.strideA;
    const uint16_t* B = g.B + static_cast<int64_t>(bz) * g.strideB;
    float* C = g.C + static_cast<int64_t>(bz) * g.strideC;
    const int M = g.M, N = g.N, K = g.K;
    const int row0 = tm * XM, col0 = tn * XN;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // loader: a 128 x 64 bf16 tile is 1024 segments of 8 (16 bytes); thread t
    // moves segments t + 256 e, e < 4 (row seg / 8, k offset 8 (seg % 8))
    constexpr int SEGS = XM * XK / 8 / XT;
    constexpr int SPR = XK / 8;     // segments per row
    uint4 ra[SEGS], rb[3][SEGS];
    const bool a_in = vec && row0 + XM <= M;
    const bool b_in = vec && col0 + XN <= N;
    auto load_rows = [&](const uint16_t* base, int64_t ld, int r0, int R, int k0, bool fast, uint4* out) {
#pragma unroll
        for (int e = 0; e < SEGS; ++e) {
            const int seg = t + XT * e;
            const int rr = r0 + seg / SPR, kk = k0 + 8 * (seg % SPR);
            const uint16_t* src = base + static_cast<int64_t>(rr) * ld + kk;
            if (fast && kk + 8 <= K) {
                out[e] = *reinterpret_cast<const uint4*>(src);
            } else {
                uint16_t v[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) v[q] = (rr < R && kk + q < K) ? src[q] : 0;
                out[e] = make_uint4(v[0] | (uint32_t(v[1]) << 16), v[2] | (uint32_t(v[3]) << 16),
                                    v[4] | (uint32_t(v[5]) << 16), v[6] | (uint32_t(v[7]) << 16));
            }
        }
    };
    auto fetch = [&](int k0) {
        load_rows(A, g.lda, row0, M, k0, a_in, ra);
#pragma unroll
        for (int p = 0; p < 3; ++p) load_rows(B + p * g.planeStride, g.ldb, col0, N, k0, b_in, rb[p]);
    };
    auto stash = [&]() {
#pragma unroll
        for (int e = 0; e < SEGS; ++e) {
            const int seg = t + XT * e;
            *reinterpret_cast<uint4*>(&As[seg / SPR][8 * (seg % SPR)]) = ra[e];
#pragma unroll
            for (int p = 0; p < 3; ++p) *reinterpret_cast<uint4*>(&Bs[p][seg / SPR][8 * (seg % SPR)]) = rb[p][e];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

    const int KT = (K + XK - 1) / XK;
    const int l32 = lane & 31, lk = lane >> 5;
    fetch(0);
    for (int kt = 0; kt < KT; ++kt) {
        stash();
        __syncthreads();
        if (kt + 1 < KT) fetch((kt + 1) * XK);
#pragma unroll
        for (int ks = 0; ks < XK; ks += 16) {
            bf16x8 a[2], bq[3][2];
#pragma unroll
            for (int x = 0; x < 2; ++x)
                a[x] = *reinterpret_cast<const bf16x8*>(&As[wm * 64 + 32 * x + l32][ks + 8 * lk]);
#pragma unroll
            for (int p = 0; p < 3; ++p)
#pragma unroll
                for (int y = 0; y < 2; ++y)
                    bq[p][y] = *reinterpret_cast<const bf16x8*>(&Bs[p][wn * 64 + 32 * y + l32][ks + 8 * lk]);
#pragma unroll
            for (int p = 0; p < 3; ++p)
#pragma unroll
                for (int x = 0; x < 2; ++x)
#pragma unroll
                    for (int y = 0; y < 2; ++y)
                        acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[x], bq[p][y], acc[x][y], 0, 0, 0);
        }
        __syncthreads();
    }

    // 32x32 block layout: lane holds column (lane & 31) and rows
    // (v & 3) + 8 (v >> 2) + 4 (lane >> 5) for accumulator register v.
    const float alpha = g.alpha, beta = g.beta;
#pragma unroll
    for (int x = 0; x < 2; ++x) {
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const int c = col0 + wn * 64 + 32 * y + l32;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r = row0 + wm * 64 + 32 * x + (v & 3) + 8 * (v >> 2) + 4 * lk;
                if (r < M && c < N) {
                    float* dst = C + static_cast<int64_t>(r) * g.ldc + c;
                    float val = alpha * acc[x][y][v];
                    if (beta != 0.0f) val += beta * (*dst);
                    *dst = val;
                }
            }
        }
    }
}

// --------------------------------------------------------------------------
// Same product, pipelined through LDS by direct loads (K a multiple of 32,
// 16-byte aligned rows): tile 256 x 128 x 32, four wave64s each owning
// 128 x 64 (4 x 2 blocks of 32 x 32, times three planes: 24 MFMAs per 16-deep
// step against 10 fragment reads). Global memory goes straight to LDS
// (global_load_lds_dwordx4: lane i of an instruction fills bytes 16 i .. 16 i
// + 15 after the instruction's base), two stages of 40 KB in flight, so no
// registers stage the operands and two workgroups share a CU's 160 KB. In a
// stage a row holds four 16-byte chunks, chunk c of row r at slot
// c ^ ((r >> 2) & 3): the 16 lanes of a fragment read (16 rows, one chunk)
// fall on distinct banks of the 64-bank LDS. Rows past M (or N) load row
// M - 1 (N - 1) instead and are never stored.
// --------------------------------------------------------------------------
constexpr int YM = 256;
constexpr int YN = 128;
constexpr int YT = 256;
// tile order (measured on 64 x 4096x11008: XCD-contiguous ids 55 ms per
// product launch set vs 68 without; groups of 8 or 16 tile rows equal, 1-4 slower)
#ifndef GALORE_BX3_GROUP
#define GALORE_BX3_GROUP 8
#endif
#ifndef GALORE_BX3_XCD
#define GALORE_BX3_XCD 1
#endif
constexpr int kDirectGroup = GALORE_BX3_GROUP;   // tile rows per group of the tile order
constexpr bool kDirectXcd = GALORE_BX3_XCD != 0;  // XCD-contiguous logical tile ids


typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

__device__ __forceinline__ void load_lds16(const void* src, void* lds_base) {
    __builtin_amdgcn_global_load_lds((glb_void_t*)src, (lds_void_t*)lds_base, 16, 0, 0);
}

// wait until at most n direct loads of this wave are outstanding
template <int n>
__device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n) : "memory");
}
template <int L, int S>
__device__ __forceinline__ void wait_stages(int ahead) {
    // ahead = stages issued after the one needed now (0 .. S - 1)
    if constexpr (S >= 4) { if (ahead >= 3) { wait_vm<3 * L>(); return; } }
    if constexpr (S >= 3) { if (ahead == 2) { wait_vm<2 * L>(); return; } }
    if (ahead >= 1) { wait_vm<L>(); return; }
    wait_vm<0>();
}

// PA = 1: A is exactly bf16 and B holds three planes (three products).
// PA = 3: both operands hold three planes (fp32 x fp32): the six products
// A_i B_j with i + j <= 4 (planes counted from 1); the three left out are below
// 2^-26 of |A||B| in size, under fp32 rounding.
template <int YK, int S, bool AT, int PA, int PB = 3, int WN = 2>
__global__ __launch_bounds__(128 * WN, (S * (PA * YM + PB * 64 * WN) * YK * 2 <= 81920) ? 2 : 1) void gemm_bf16x3_direct_kernel(Bx3Args g) {
    static_assert(!AT || YK == 32, "the M-contiguous A stage assumes 32-deep stages");
    static_assert(PA == 1 || (PA == 3 && !AT), "three A planes are K-contiguous");
    static_assert(PB == 3 || (PB == 1 && PA == 1), "one B plane pairs with one A plane");
    static_assert(WN == 2 || (WN == 4 && !AT), "four waves across N: K-contiguous A only");
    // WN waves across the tile's columns (64 each), two down its rows (128 each)
    constexpr int YN = 64 * WN;
    constexpr int YT = 128 * WN;
    // the stage's two steps read and multiplied in order, the next stage's
    // loads issued after the reads (see the main loop): needed with the
    // transposing reads, and faster for three B planes either way
    constexpr bool kSplit = AT || (PA == 1 && PB == 3 && YK == 32);
    // the one-plane product reads both steps' fragments, then issues the next
    // stage's loads, then runs its MFMAs (7.97 against 8.20 ms per launch of
    // 64 with the loads first; the same order slows the three-plane A X, 18.4
    // against 16.9 ms)
    constexpr bool kReadFirst = !AT && YK == 32 && PB == 1;
    constexpr int kFragBufs = (kSplit || kReadFirst) ? 2 : 1;   // fragment register buffers
    constexpr int CPR = YK / 8;                          // 16-byte chunks per row
    constexpr int RB = YK * 2;                           // bytes per row
    constexpr int kStageA = PA * YM * RB;
    constexpr int kStageB = PB * YN * RB;
    constexpr int kStage = kStageA + kStageB;
    constexpr int LA = kStageA / 1024 / (YT / 64);       // direct loads per wave per stage (1 KB each)
    constexpr int LB = kStageB / 1024 / (YT / 64);
    static_assert(kStageA % (1024 * (YT / 64)) == 0 && kStageB % (1024 * (YT / 64)) == 0, "whole direct loads per wave");
    constexpr int RPI = 64 / CPR;                        // rows per direct load
    constexpr int RPB = 256 / RB;                        // rows per 256 bytes (one sweep of the 64 banks)
    __shared__ __attribute__((aligned(16))) unsigned char ysm[S * kStage];

    const int num_n = gridDim.x, num_m = gridDim.y;
    const int tiles = num_n * num_m;
    const int lin = blockIdx.x + num_n * (blockIdx.y + num_m * blockIdx.z);
    const int logical = kDirectXcd ? xcd_logical_id(lin, tiles * gridDim.z) : lin;
    const int bz = logical / tiles;
    int tm, tn;
    grouped_tile(logical - bz * tiles, num_m, num_n, kDirectGroup, tm, tn);
    const uint16_t* A = g.A + static_cast<int64_t>(bz) * g.strideA;
    const uint16_t* B = g.B + static_cast<int64_t>(bz) * g.strideB;
    float* C = g.C + static_cast<int64_t>(bz) * g.strideC;
    const int M = g.M, N = g.N, K = g.K;
    const int row0 = tm * YM, col0 = tn * YN;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // chunk c of stage row r sits at slot c ^ ((r / RPB) % CPR). A direct load
    // fills RPI rows; lane i -> (row RPI j + i / CPR, slot i % CPR), so it
    // fetches the chunk whose slot that is
    const int lrow = lane / CPR;
    const uint16_t* srcA[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int j = wave * LA + i;
        if constexpr (AT) {
            // M-contiguous A (A[kk * lda + i]): a stage row is one kk, 256 m
            // (32 chunks, 512 bytes), chunk c at slot c ^ (4 (kk % 4)); a direct
            // load fills 2 rows; chunks past M load the last chunk (M % 8 == 0)
            const int sr = 2 * j + (lane >> 5);
            const int slot = lane & 31;
            const int m = min(row0 + 8 * (slot ^ (4 * (sr & 3))), M - 8);
            srcA[i] = A + static_cast<int64_t>(sr) * g.lda + m;
        } else {
            const int pl = j / (YM / RPI), jb = j % (YM / RPI);   // plane, block of RPI rows
            const int sr = RPI * jb + lrow;              // row within the plane's stage
            const int r = min(row0 + sr, M - 1);
            srcA[i] = A + pl * g.planeStrideA + static_cast<int64_t>(r) * g.lda +
                      8 * ((lane % CPR) ^ ((sr / RPB) % CPR));
        }
    }
    const int64_t kstepA = AT ? static_cast<int64_t>(YK) * g.lda : YK;   // A advance per stage
    const uint16_t* srcB[LB];
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int q = wave * LB + i;                     // plane q / (YN / RPI), block q % (YN / RPI)
        const int pl = q / (YN / RPI), j = q % (YN / RPI);
        const int sr = RPI * j + lrow;
        const int r = min(col0 + sr, N - 1);
        srcB[i] = B + pl * g.planeStride + static_cast<int64_t>(r) * g.ldb + 8 * ((lane % CPR) ^ ((sr / RPB) % CPR));
    }
    auto issue = [&](int stage, int k0) {
        unsigned char* base = ysm + stage * kStage;
        const int64_t offA = (k0 / YK) * kstepA;
#pragma unroll
        for (int i = 0; i < LA; ++i) load_lds16(srcA[i] + offA, base + (wave * LA + i) * 1024);
#pragma unroll
        for (int i = 0; i < LB; ++i) load_lds16(srcB[i] + k0, base + kStageA + (wave * LB + i) * 1024);
    };

    f32x16 acc[4][2];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[x][y][v] = 0.0f;

    const int l32 = lane & 31, lk = lane >> 5;
    const int KT = (g.b_upper ? min(K, col0 + YN) : K) / YK;
#pragma unroll
    for (int st = 0; st < S - 1; ++st)
        if (st < KT) issue(st, st * YK);
    // NB = this wave's 32-column blocks that lie inside N (the last tile of a
    // 1056-wide product holds 32 valid columns): the fragment reads and MFMAs
    // of the blocks past N are skipped, the wave still issues its loads
    auto kloop = [&](auto nbc) {
    constexpr int NB = decltype(nbc)::value;
    for (int kt = 0; kt < KT; ++kt) {
        // stage kt landed for this wave, then for every wave; past the barrier
        // every wave has also finished iteration kt - 1, so its stage is refilled
        wait_stages<LA + LB, S>(min(S - 2, KT - 1 - kt));
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        const unsigned char* sa = ysm + (kt % S) * kStage;
        const unsigned char* sb = sa + kStageA;
        // fragments of 16-deep step ks into register buffer fb
        bf16x8 a[kFragBufs][PA][4], bq[kFragBufs][PB][2];
        auto fetch = [&](int fb, int ks) {
            const int c = 2 * ks + lk;
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                if constexpr (AT) {
                    // transposing LDS reads: in each group of 16 lanes, lane j
                    // receives element j % 4 of lanes 4 e + j / 4 (e = 0..3). Lane
                    // L of the group points at row kk = kb + L / 4, m = mb + 4 (L % 4),
                    // so lane j gets A[mb + j][kb .. kb + 3]
                    const int L = lane & 15;
                    const int m = wm * 128 + 32 * x + 16 * ((lane >> 4) & 1) + 4 * (L & 3);
                    bf16x4 h2[2];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int kk = 16 * ks + 8 * lk + 4 * h + (L >> 2);
                        const int off = kk * 512 + 16 * ((m >> 3) ^ (4 * (kk & 3))) + 2 * (m & 7);
                        h2[h] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                            reinterpret_cast<__attribute__((address_space(3))) bf16x4*>(
                                reinterpret_cast<__attribute__((address_space(3))) unsigned char*>(
                                    reinterpret_cast<size_t>(sa)) + off));
                    }
                    a[fb][0][x] = __builtin_shufflevector(h2[0], h2[1], 0, 1, 2, 3, 4, 5, 6, 7);
                } else {
                    const int r = wm * 128 + 32 * x + l32;
#pragma unroll
                    for (int pa = 0; pa < PA; ++pa)
                        a[fb][pa][x] = *reinterpret_cast<const bf16x8*>(sa + pa * (YM * RB) + r * RB +
                                                                        16 * (c ^ ((r / RPB) % CPR)));
                }
            }
#pragma unroll
            for (int p = 0; p < PB; ++p)
#pragma unroll
                for (int y = 0; y < NB; ++y) {
                    const int r = wn * 64 + 32 * y + l32;
                    bq[fb][p][y] = *reinterpret_cast<const bf16x8*>(sb + p * (YN * RB) + r * RB +
                                                                    16 * (c ^ ((r / RPB) % CPR)));
                }
        };
        auto multiply = [&](int fb) {
            if constexpr (PA == 1) {
#pragma unroll
                for (int p = 0; p < PB; ++p)
#pragma unroll
                    for (int x = 0; x < 4; ++x)
#pragma unroll
                        for (int y = 0; y < NB; ++y)
                            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[fb][0][x], bq[fb][p][y], acc[x][y],
                                                                                 0, 0, 0);
            } else {
                constexpr int pairs[6][2] = {{0, 0}, {0, 1}, {1, 0}, {0, 2}, {1, 1}, {2, 0}};
#pragma unroll
                for (int q = 0; q < 6; ++q)
#pragma unroll
                    for (int x = 0; x < 4; ++x)
#pragma unroll
                        for (int y = 0; y < NB; ++y)
                            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                a[fb][pairs[q][0]][x], bq[fb][pairs[q][1]][y], acc[x][y], 0, 0, 0);
            }
        };
        if constexpr (kReadFirst) {
            fetch(0, 0);
            fetch(kFragBufs - 1, 1);
            __builtin_amdgcn_sched_barrier(0);
            if (kt + S - 1 < KT) issue((kt + S - 1) % S, (kt + S - 1) * YK);
            __builtin_amdgcn_sched_barrier(0);
            multiply(0);
            multiply(kFragBufs - 1);
        } else if constexpr (kSplit) {
            // the compiler cannot tell the transposing LDS reads from the LDS
            // that the direct loads in flight may write, and before any such
            // read issued after those loads it waits for all of them (a whole
            // memory latency per stage). So the stage's two steps are read
            // before the next stage's loads are issued: step 0's fragments,
            // its MFMAs, step 1's fragments while they run, then the loads,
            // then step 1's MFMAs (measured per launch of 64 products: A^T Q
            // 15.9 against 17.9 ms with the loads first and 16.6 with all reads
            // before any MFMA; A X 16.9 against 17.8 ms with the compiler's
            // interleaving; the one-plane sketch product is faster with the
            // latter, 8.2 against 9.1 ms, and keeps it).
            fetch(0, 0);
            __builtin_amdgcn_sched_barrier(0);
            multiply(0);
            __builtin_amdgcn_sched_barrier(0);
            fetch(1, 1);
            __builtin_amdgcn_sched_barrier(0);
            if (kt + S - 1 < KT) issue((kt + S - 1) % S, (kt + S - 1) * YK);
            __builtin_amdgcn_sched_barrier(0);
            multiply(1);
        } else if constexpr (PA == 3 && YK == 16) {
            // the six-plane product (one 16-deep step per stage, three stages):
            // the next loads issued after the stage's fragment reads, so that
            // their LDS writes do not meet those reads (29.96 against 30.7 ms
            // per launch of 64 with the loads first; they still land two
            // stages ahead)
            fetch(0, 0);
            __builtin_amdgcn_sched_barrier(0);
            if (kt + S - 1 < KT) issue((kt + S - 1) % S, (kt + S - 1) * YK);
            __builtin_amdgcn_sched_barrier(0);
            multiply(0);
        } else {
            if (kt + S - 1 < KT) issue((kt + S - 1) % S, (kt + S - 1) * YK);
#pragma unroll
            for (int ks = 0; ks < YK / 16; ++ks) {
                fetch(0, ks);
                multiply(0);
            }
        }
    }
    };
    // (the six-plane kernel keeps one loop: its launches here have N a
    // multiple of the tile width, and the extra loops measured 0.6% slower)
    const int nb = PA == 3 ? 2 : __builtin_amdgcn_readfirstlane(min(2, max(0, (N - col0 - wn * 64 + 31) / 32)));
    if (PA == 3 || nb >= 2) kloop(std::integral_constant<int, 2>());
    else if (nb == 1) kloop(std::integral_constant<int, 1>());
    else kloop(std::integral_constant<int, 0>());

    const float alpha = g.alpha, beta = g.beta;
    unsigned mx[2] = {0u, 0u};   // bits of the largest |C| of this lane's two columns
    if constexpr (PA == 3) {
        // the back-projection's read-modify-write of C (W += -lr alpha P N):
        // each block's reads of C are issued together before its stores, and
        // a tile that lies inside C (uniform) stores without per-element
        // bounds branches, at whose joins the compiler would wait for the
        // reads again before every store (38.1 -> 36.4 ms per launch). The
        // other variants keep the plain epilogue: the longer code measured
        // slower for them (the sketch product 8.2 against 8.7 ms).
        const bool full_tile = beta != 0.0f && row0 + YM <= M && col0 + YN <= N;
        if (g.c_trans) {
            // C^T: a lane's registers v = 4 q .. 4 q + 3 hold four consecutive m of
            // one n, i.e. four consecutive entries of row n of the stored matrix
            const bool v4 = (g.ldc % 4) == 0 && (reinterpret_cast<uintptr_t>(C) % 16) == 0;
#pragma unroll
            for (int x = 0; x < 4; ++x) {
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    const int c = col0 + wn * 64 + 32 * y + l32;
                    if (c >= N) continue;
                    const float al = g.nscale ? alpha * g.nscale[static_cast<int64_t>(bz) * g.strideNS + c] : alpha;
                    // with beta != 0 the block's four reads of C are issued
                    // together before any store (one memory latency per block,
                    // not one per read); past the last row they read row M - 1,
                    // whose value is not stored
                    f32x4 old[4];
                    if (beta != 0.0f) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int r = row0 + wm * 128 + 32 * x + 8 * q + 4 * lk;
                            const float* src = C + static_cast<int64_t>(c) * g.ldc;
                            if (v4 && (full_tile || r + 4 <= M)) {
                                old[q] = *reinterpret_cast<const f32x4*>(src + r);
                            } else {
#pragma unroll
                                for (int e = 0; e < 4; ++e) old[q][e] = src[min(r + e, M - 1)];
                            }
                        }
                    }
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int r = row0 + wm * 128 + 32 * x + 8 * q + 4 * lk;
                        float* dst = C + static_cast<int64_t>(c) * g.ldc + r;
                        f32x4 val = {al * acc[x][y][4 * q], al * acc[x][y][4 * q + 1], al * acc[x][y][4 * q + 2],
                                     al * acc[x][y][4 * q + 3]};
                        if (beta != 0.0f) {
#pragma unroll
                            for (int e = 0; e < 4; ++e) val[e] += beta * old[q][e];
                        }
                        if (v4 && (full_tile || r + 4 <= M)) {
                            *reinterpret_cast<f32x4*>(dst) = val;
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (r + e < M) dst[e] = val[e];
                        }
                    }
                }
            }
            return;
        }
#pragma unroll
        for (int x = 0; x < 4; ++x) {
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int c = col0 + wn * 64 + 32 * y + l32;
                const float al = (g.nscale && c < N) ? alpha * g.nscale[static_cast<int64_t>(bz) * g.strideNS + c] : alpha;
                // with beta != 0 the block's sixteen reads of C first, together;
                // rows and columns past the matrix read its last row or column,
                // whose values are not stored
                float old[16];
                if (beta != 0.0f) {
                    const int cc = min(c, N - 1);
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int r = row0 + wm * 128 + 32 * x + (v & 3) + 8 * (v >> 2) + 4 * lk;
                        old[v] = C[static_cast<int64_t>(min(r, M - 1)) * g.ldc + cc];
                    }
                }
                if (full_tile) {
                    // no per-element bounds branches: at their joins the compiler
                    // would wait again for the reads above before every store
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int r = row0 + wm * 128 + 32 * x + (v & 3) + 8 * (v >> 2) + 4 * lk;
                        float val = al * acc[x][y][v];
                        if (beta != 0.0f) val += beta * old[v];
                        C[static_cast<int64_t>(r) * g.ldc + c] = val;
                        mx[y] = max(mx[y], __float_as_uint(fabsf(val)));
                    }
                } else {
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int r = row0 + wm * 128 + 32 * x + (v & 3) + 8 * (v >> 2) + 4 * lk;
                        if (r < M && c < N) {
                            float* dst = C + static_cast<int64_t>(r) * g.ldc + c;
                            float val = al * acc[x][y][v];
                            if (beta != 0.0f) val += beta * old[v];
                            *dst = val;
                            mx[y] = max(mx[y], __float_as_uint(fabsf(val)));
                        }
                    }
                }
            }
        }
    } else {
        if (g.c_trans) {
            // C^T: a lane's registers v = 4 q .. 4 q + 3 hold four consecutive m of
            // one n, i.e. four consecutive entries of row n of the stored matrix
            const bool v4 = (g.ldc % 4) == 0 && (reinterpret_cast<uintptr_t>(C) % 16) == 0;
#pragma unroll
            for (int x = 0; x < 4; ++x) {
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    const int c = col0 + wn * 64 + 32 * y + l32;
                    if (c >= N) continue;
                    const float al = g.nscale ? alpha * g.nscale[static_cast<int64_t>(bz) * g.strideNS + c] : alpha;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int r = row0 + wm * 128 + 32 * x + 8 * q + 4 * lk;
                        float* dst = C + static_cast<int64_t>(c) * g.ldc + r;
                        f32x4 val = {al * acc[x][y][4 * q], al * acc[x][y][4 * q + 1], al * acc[x][y][4 * q + 2],
                                     al * acc[x][y][4 * q + 3]};
                        if (v4 && r + 4 <= M) {
                            if (beta != 0.0f) {
                                const f32x4 old = *reinterpret_cast<const f32x4*>(dst);
#pragma unroll
                                for (int e = 0; e < 4; ++e) val[e] += beta * old[e];
                            }
                            *reinterpret_cast<f32x4*>(dst) = val;
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (r + e < M) dst[e] = (beta != 0.0f) ? val[e] + beta * dst[e] : val[e];
                        }
                    }
                }
            }
            return;
        }
#pragma unroll
        for (int x = 0; x < 4; ++x) {
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int c = col0 + wn * 64 + 32 * y + l32;
                const float al = (g.nscale && c < N) ? alpha * g.nscale[static_cast<int64_t>(bz) * g.strideNS + c] : alpha;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int r = row0 + wm * 128 + 32 * x + (v & 3) + 8 * (v >> 2) + 4 * lk;
                    if (r < M && c < N) {
                        float* dst = C + static_cast<int64_t>(r) * g.ldc + c;
                        float val = al * acc[x][y][v];
                        if (beta != 0.0f) val += beta * (*dst);
                        *dst = val;
                        mx[y] = max(mx[y], __float_as_uint(fabsf(val)));
                    }
                }
            }
        }
    }
    if (g.cmax != nullptr) {
        // column maxima for the exact Gram of C (non-negative floats order like
        // their bit patterns; NaN/Inf win): the two lane halves hold the same
        // columns, one atomic per column and wave
        unsigned* cm = g.cmax + static_cast<int64_t>(bz) * g.strideCM;
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const unsigned m = max(mx[y], static_cast<unsigned>(__shfl_xor(static_cast<int>(mx[y]), 32)));
            const int c = col0 + wn * 64 + 32 * y + l32;
            if (lk == 0 && c < N) atomicMax(cm + c, m);
        }
    }
}

#ifndef GALORE_BX3_K
#define GALORE_BX3_K 32
#endif
#ifndef GALORE_BX3_S
#define GALORE_BX3_S 2
#endif
constexpr int kDirectK = GALORE_BX3_K;     // K depth of a stage
constexpr int kDirectS = GALORE_BX3_S;     // stages in LDS
#ifndef GALORE_BX3T_S
#define GALORE_BX3T_S 2
#endif
constexpr int kDirectST = GALORE_BX3T_S;   // stages of the M-contiguous-A kernel (32 deep each)
// Three A planes (the back-projection): 256 x 256 tiles of eight waves (four
// across N), three 48 KB stages of K = 16, one workgroup per CU. Measured on
// 64 x 4096x11008, r = 1024, per launch: 30.8 ms against 35.2-37.4 ms with
// 256 x 128 tiles of four waves and two 36 KB stages (two workgroups per CU),
// 31.3 ms with the wide tile and two stages: with two stages each stage's
// loads had one stage of matrix-core time to land, and a tile that waited on
// a miss held its workgroup at the barrier.
#ifndef GALORE_BX6_K
#define GALORE_BX6_K 16
#endif
#ifndef GALORE_BX6_S
#define GALORE_BX6_S 3
#endif
#ifndef GALORE_BX6_WN
#define GALORE_BX6_WN 4
#endif
constexpr int kX6K = GALORE_BX6_K;         // K depth of a stage
constexpr int kX6S = GALORE_BX6_S;         // stages in LDS
constexpr int kX6WN = GALORE_BX6_WN;       // waves across N (tile 256 x 64 WN)

}  // namespace

hipError_t launch_transpose_bf16(const void* src, int64_t lds, int64_t strideS, void* dst, int64_t ldd,
                                 int64_t strideD, int rows, int cols, int batch, hipStream_t stream) {
    dim3 grid((cols + 63) / 64, (rows + 63) / 64, batch);
    hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(src), lds,
                       strideS, static_cast<uint16_t*>(dst), ldd, strideD, rows, cols);
    return hipGetLastError();
}

hipError_t launch_split3_transpose(const float* src, int64_t lds, int64_t strideS, void* planes, int64_t ldp,
                                   int64_t planeStride, int64_t strideP, int rows, int cols, int rows_pad,
                                   int batch, hipStream_t stream, const float* rowscale, int64_t strideRS) {
    if (rows <= 0 || cols <= 0 || rows_pad <= 0 || batch <= 0) return hipSuccess;
    // 16-byte row loads and 8-byte plane stores where every row start is aligned
    const int vload = (lds % 4 == 0) && (batch == 1 || strideS % 4 == 0) &&
                      (reinterpret_cast<uintptr_t>(src) % 16 == 0);
    const int vstore = (ldp % 4 == 0) && (planeStride % 4 == 0) && (batch == 1 || strideP % 4 == 0) &&
                       (reinterpret_cast<uintptr_t>(planes) % 8 == 0);
    dim3 grid((cols + 63) / 64, (rows_pad + 63) / 64, batch);
    hipLaunchKernelGGL(split3_transpose_kernel, grid, dim3(256), 0, stream, src, lds, strideS,
                       static_cast<uint16_t*>(planes), ldp, planeStride, strideP, rows, cols, rows_pad, rowscale,
                       strideRS, vload, vstore);
    return hipGetLastError();
}

bool bf16x3_direct_ok(const void* A, int64_t lda, int64_t strideA, const void* Bplanes, int64_t ldb,
                      int64_t planeStride, int64_t strideB, int M, int K, int batch, int a_mcontig) {
    // 16-byte direct loads need 16-byte aligned rows in A and in every plane
    const bool vec = (lda % 8 == 0) && (ldb % 8 == 0) && (planeStride % 8 == 0) &&
                     (batch == 1 || (strideA % 8 == 0 && strideB % 8 == 0)) &&
                     (reinterpret_cast<uintptr_t>(A) % 16 == 0) && (reinterpret_cast<uintptr_t>(Bplanes) % 16 == 0);
    const bool mc = !a_mcontig || (M >= 8 && M % 8 == 0);
    return vec && mc && K > 0 && K % (a_mcontig ? 32 : kDirectK) == 0;
}

hipError_t launch_gemm_bf16x3(const void* A, int64_t lda, int64_t strideA, int a_mcontig, const void* Bplanes,
                              int64_t ldb, int64_t planeStride, int64_t strideB, float* C, int64_t ldc,
                              int64_t strideC, int c_trans, int M, int N, int K, float alpha, float beta, int batch,
                              hipStream_t stream, unsigned* cmax, int64_t strideCM, int planesB, const float* nscale,
                              int64_t strideNS) {
    if (M <= 0 || N <= 0 || batch <= 0) return hipSuccess;
    if (planesB != 1 && planesB != 3) return hipErrorInvalidValue;
    Bx3Args g{};
    g.A = static_cast<const uint16_t*>(A);
    g.lda = lda;
    g.strideA = strideA;
    g.B = static_cast<const uint16_t*>(Bplanes);
    g.ldb = ldb;
    g.planeStride = planeStride;
    g.strideB = strideB;
    g.C = C;
    g.ldc = ldc;
    g.strideC = strideC;
    g.M = M;
    g.N = N;
    g.K = K;
    g.alpha = alpha;
    g.beta = beta;
    g.c_trans = c_trans;
    g.planeStrideA = 0;
    g.b_upper = 0;
    g.cmax = c_trans ? nullptr : cmax;
    g.strideCM = strideCM;
    g.nscale = nscale;
    g.strideNS = strideNS;
    if (bf16x3_direct_ok(A, lda, strideA, Bplanes, ldb, planeStride, strideB, M, K, batch, a_mcontig)) {
        dim3 grid((N + YN - 1) / YN, (M + YM - 1) / YM, batch);
        if (planesB == 1) {
            if (a_mcontig)
                hipLaunchKernelGGL((gemm_bf16x3_direct_kernel<32, kDirectST, true, 1, 1>), grid, dim3(YT), 0, stream, g);
            else
                hipLaunchKernelGGL((gemm_bf16x3_direct_kernel<kDirectK, kDirectS, false, 1, 1>), grid, dim3(YT), 0,
                                   stream, g);
        } else if (a_mcontig) {
            hipLaunchKernelGGL((gemm_bf16x3_direct_kernel<32, kDirectST, true, 1>), grid, dim3(YT), 0, stream, g);
        } else {
            hipLaunchKernelGGL((gemm_bf16x3_direct_kernel<kDirectK, kDirectS, false, 1>), grid, dim3(YT), 0, stream, g);
        }
        return hipGetLastError();
    }
    // the register-staged kernel: K-contiguous A, three B planes, row-major C only,
    // no column maxima or scales
    if (a_mcontig || c_trans || cmax != nullptr || planesB != 3 || nscale != nullptr) return hipErrorInvalidValue;
    const int vec = (lda % 8 == 0) && (ldb % 8 == 0) && (planeStride % 8 == 0) &&
                    (batch == 1 || (strideA % 8 == 0 && strideB % 8 == 0)) &&
                    (reinterpret_cast<uintptr_t>(A) % 16 == 0) && (reinterpret_cast<uintptr_t>(Bplanes) % 16 == 0);
    dim3 grid((N + XN - 1) / XN, (M + XM - 1) / XM, batch);
    hipLaunchKernelGGL(gemm_bf16x3_kernel, grid, dim3(XT), 0, stream, g, vec);
    return hipGetLastError();
}

hipError_t launch_split3_rows(const float* src, int64_t lds, int64_t strideS, void* planes, int64_t ldp,
                              int64_t planeStride, int64_t strideP, int rows, int cols, int cols_pad, int batch,
                              hipStream_t stream) {
    if (rows <= 0 || cols_pad <= 0 || batch <= 0) return hipSuccess;
    // 16-byte source rows and 8-byte plane rows
    const int vec = (lds % 4 == 0) && (batch == 1 || strideS % 4 == 0) && (reinterpret_cast<uintptr_t>(src) % 16 == 0) &&
                    (ldp % 4 == 0) && (planeStride % 4 == 0) && (batch == 1 || strideP % 4 == 0) &&
                    (reinterpret_cast<uintptr_t>(planes) % 8 == 0);
    dim3 grid((cols_pad + 1023) / 1024, rows, batch);
    hipLaunchKernelGGL(split3_rows_kernel, grid, dim3(256), 0, stream, src, lds, strideS,
                       static_cast<uint16_t*>(planes), ldp, planeStride, strideP, rows, cols, cols_pad, vec);
    return hipGetLastError();
}

bool bf16x6_ok(const void* Aplanes, int64_t lda, int64_t planeStrideA, int64_t strideA, const void* Bplanes,
               int64_t ldb, int64_t planeStrideB, int64_t strideB, int K, int batch) {
    return (lda % 8 == 0) && (planeStrideA % 8 == 0) && (ldb % 8 == 0) && (planeStrideB % 8 == 0) &&
           (batch == 1 || (strideA % 8 == 0 && strideB % 8 == 0)) &&
           (reinterpret_cast<uintptr_t>(Aplanes) % 16 == 0) && (reinterpret_cast<uintptr_t>(Bplanes) % 16 == 0) &&
           K > 0 && K % kX6K == 0;
}

hipError_t launch_gemm_bf16x6(const void* Aplanes, int64_t lda, int64_t planeStrideA, int64_t strideA,
                              const void* Bplanes, int64_t ldb, int64_t planeStrideB, int64_t strideB, float* C,
                              int64_t ldc, int64_t strideC, int c_trans, int b_upper, int M, int N, int K,
                              float alpha, float beta, int batch, hipStream_t stream) {
    if (M <= 0 || N <= 0 || batch <= 0) return hipSuccess;
    if (!bf16x6_ok(Aplanes, lda, planeStrideA, strideA, Bplanes, ldb, planeStrideB, strideB, K, batch))
        return hipErrorInvalidValue;
    Bx3Args g{};
    g.A = static_cast<const uint16_t*>(Aplanes);
    g.lda = lda;
    g.strideA = strideA;
    g.B = static_cast<const uint16_t*>(Bplanes);
    g.ldb = ldb;
    g.planeStride = planeStrideB;
    g.strideB = strideB;
    g.C = C;
    g.ldc = ldc;
    g.strideC = strideC;
    g.M = M;
    g.N = N;
    g.K = K;
    g.alpha = alpha;
    g.beta = beta;
    g.c_trans = c_trans;
    g.planeStrideA = planeStrideA;
    g.b_upper = b_upper;
    g.cmax = nullptr;
    g.strideCM = 0;
    dim3 grid((N + 64 * kX6WN - 1) / (64 * kX6WN), (M + YM - 1) / YM, batch);
    hipLaunchKernelGGL((gemm_bf16x3_direct_kernel<kX6K, kX6S, false, 3, 3, kX6WN>), grid, dim3(128 * kX6WN), 0, stream,
                       g);
    return hipGetLastError();
}

}  // namespace galore
