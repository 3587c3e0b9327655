// Dense contractions of the subspace update and the projection steps, on the
// CDNA4 matrix cores.
//
//  * gemm_f32: C = alpha * op(A) op(B) + beta * C in fp32 with
//    v_mfma_f32_32x32x2_f32. gfx950 has no TF32 matrix path, so fp32 MFMA is
//    the precision the method is computed in. bf16-stored gradients are
//    widened exactly to fp32 while staging into LDS.
//    Workgroup tile 128 x 128 x 32, four wave64s in a 2 x 2 arrangement, each
//    wave owning a 64 x 64 sub-tile (2 x 2 MFMA 32x32 blocks). LDS holds A^T
//    and B tiles in M-/N-contiguous order so that the per-lane MFMA operand
//    reads are consecutive addresses; double-buffered with one barrier per
//    K step, the next tile's global loads in flight during the MFMAs.
#include <type_traits>

#include "common.hpp"

namespace galore {
namespace {

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BK = 32;
constexpr int NT = 256;

template <typename T>
__device__ __forceinline__ float load_elem(const T* base, int64_t idx) {
    return to_f32(base[idx]);
}

// Four (fp32) or eight (bf16) consecutive elements from one 16-byte load.
__device__ __forceinline__ void load_vec16(const float* src, float* out) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(src);
    out[0] = x[0];
    out[1] = x[1];
    out[2] = x[2];
    out[3] = x[3];
}
__device__ __forceinline__ void load_vec16(const bf16_t* src, float* out) {
    const uint4 x = *reinterpret_cast<const uint4*>(src);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        out[2 * e + 0] = __uint_as_float(w[e] << 16);
        out[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
}

// A BK x 128 operand tile v(kk, c) = base[(k0 + kk) * ld + c0 + c] whose
// second index runs along memory (A stored M-contiguous, B N-contiguous):
// each thread moves E rows of one 16-byte vector.
template <typename T>
struct ContigTile {
    static constexpr int V = 16 / static_cast<int>(sizeof(T));   // elements per vector
    static constexpr int CQ = 128 / V;                           // vectors per tile row
    static constexpr int KR = NT / CQ;                           // rows per pass
    static constexpr int E = BK / KR;                            // passes (V * E == 16)
    __device__ static void load(const T* base, int64_t ld, int k0, int K, int c0, int C, bool vec, int t,
                                float* r) {
        const int cq = t % CQ, kr = t / CQ;
        const int c = c0 + V * cq;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int gk = k0 + kr + KR * e;
            const T* src = base + static_cast<int64_t>(gk) * ld + c;
            if (gk < K && vec && c + V <= C) {
                load_vec16(src, r + V * e);
            } else {
#pragma unroll
                for (int v = 0; v < V; ++v) r[V * e + v] = (gk < K && c + v < C) ? to_f32(src[v]) : 0.0f;
            }
        }
    }
    // whole tile in range and 16-byte aligned rows: unconditional vector loads
    __device__ static void load_fast(const T* base, int64_t ld, int k0, int c0, int t, float* r) {
        const int cq = t % CQ, kr = t / CQ;
        const T* src = base + static_cast<int64_t>(k0 + kr) * ld + c0 + V * cq;
#pragma unroll
        for (int e = 0; e < E; ++e) load_vec16(src + static_cast<int64_t>(KR * e) * ld, r + V * e);
    }
    __device__ static void store(float (*S)[128], int t, const float* r) {
        const int cq = t % CQ, kr = t / CQ;
#pragma unroll
        for (int e = 0; e < E; ++e)
#pragma unroll
            for (int v = 0; v < V; ++v) S[kr + KR * e][V * cq + v] = r[V * e + v];
    }
};

// A BK x 128 operand tile v(kk, c) = base[(c0 + c) * ld + k0 + kk] whose
// first (reduction) index runs along memory (A stored K-contiguous, B stored
// K-contiguous): each thread moves 16 consecutive k of one row.
template <typename T>
struct KContigTile {
    static constexpr int V = 16 / static_cast<int>(sizeof(T));
    __device__ static void load(const T* base, int64_t ld, int k0, int K, int c0, int C, bool vec, int t,
                                float* r) {
        const int c = c0 + (t >> 1);
        const int gk = k0 + (t & 1) * 16;
        const T* src = base + static_cast<int64_t>(c) * ld + gk;
        if (c < C && gk + 16 <= K && vec) {
#pragma unroll
            for (int q = 0; q < 16 / V; ++q) load_vec16(src + V * q, r + V * q);
        } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) r[e] = (c < C && gk + e < K) ? to_f32(src[e]) : 0.0f;
        }
    }
    __device__ static void load_fast(const T* base, int64_t ld, int k0, int c0, int t, float* r) {
        const T* src = base + static_cast<int64_t>(c0 + (t >> 1)) * ld + k0 + (t & 1) * 16;
#pragma unroll
        for (int q = 0; q < 16 / V; ++q) load_vec16(src + V * q, r + V * q);
    }
    __device__ static void store(float (*S)[128], int t, const float* r) {
        const int c = t >> 1;
        const int kk0 = (t & 1) * 16;
#pragma unroll
        for (int e = 0; e < 16; ++e) S[kk0 + e][c] = r[e];
    }
};

template <ALayout LA, BLayout LB, typename TA, typename TB, bool PLANES = false, bool TRIL = false>
__global__ __launch_bounds__(NT, 2) void gemm_f32_kernel(GemmArgs g, int a_vec, int b_vec) {
    // the two operand stages; the plane epilogue reuses the same 64 KB
    __shared__ __attribute__((aligned(16))) float smem[2 * BK * BM + 2 * BK * BN];
    float (*As)[BK][BM] = reinterpret_cast<float (*)[BK][BM]>(smem);
    float (*Bs)[BK][BN] = reinterpret_cast<float (*)[BK][BN]>(smem + 2 * BK * BM);

    // XCD-aware, row-grouped tile order (grid = n tiles x m tiles x batch)
    const int num_n = gridDim.x, num_m = gridDim.y;
    const int tiles = num_n * num_m;
    const int lin = blockIdx.x + num_n * (blockIdx.y + num_m * blockIdx.z);
    const int logical = xcd_logical_id(lin, tiles * gridDim.z);
    const int bz = logical / tiles;
    int tm, tn;
    grouped_tile(logical - bz * tiles, num_m, num_n, 8, tm, tn);
    // with an upper-triangular op(B) a tile's K range grows with its column
    // (the K loop stops at its last column): each group takes its longest
    // tiles first, so that the launch ends on short ones (Y R^-1 at k = 1056:
    // 33.7 -> 33.0 ms per step)
    if (g.b_upper) tn = num_n - 1 - tn;
    const TA* A = static_cast<const TA*>(g.A) + static_cast<int64_t>(bz) * g.strideA;
    const TB* B = static_cast<const TB*>(g.B) + static_cast<int64_t>(bz) * g.strideB;
    float* C = g.C + static_cast<int64_t>(bz) * g.strideC;
    const int M = g.M, N = g.N, K = g.K;
    const int row0 = tm * BM;
    const int col0 = tn * BN;
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = t >> 6;
    const int wm = wave >> 1;
    const int wn = wave & 1;

    // A tile: rows i of op(A), B tile: columns j of op(B), both BK deep
    using TileA = typename std::conditional<LA == ALayout::kKContig, KContigTile<TA>, ContigTile<TA>>::type;
    using TileB = typename std::conditional<LB == BLayout::kKContig, KContigTile<TB>, ContigTile<TB>>::type;

    float ra[16];
    float rb[16];
    // interior tiles (uniform per workgroup) take the unconditional vector path
    const bool a_full = a_vec && row0 + BM <= M;
    const bool b_full = b_vec && col0 + BN <= N;
    auto load_a = [&](int k0) {
        if (a_full && k0 + BK <= K) TileA::load_fast(A, g.lda, k0, row0, t, ra);
        else TileA::load(A, g.lda, k0, K, row0, M, a_vec != 0, t, ra);
    };
    auto load_b = [&](int k0) {
        if (b_full && k0 + BK <= K) TileB::load_fast(B, g.ldb, k0, col0, t, rb);
        else TileB::load(B, g.ldb, k0, K, col0, N, b_vec != 0, t, rb);
    };
    auto store_a = [&](int buf) { TileA::store(As[buf], t, ra); };
    auto store_b = [&](int buf) { TileB::store(Bs[buf], t, rb); };

    // wave layout: 2 x 2 waves of 64 x 64 (two 32-row and two 32-column blocks
    // each), or, for an upper-triangular op(B) (TRIL), 4 x 1 waves of 32 rows
    // by all 128 columns: in a tile's last K stages every wave then drops the
    // same column blocks, where the 2 x 2 layout left the waves of the first
    // 64 columns idle at the stage barriers
    constexpr int WMB = TRIL ? 1 : 2;            // 32-row blocks per wave
    constexpr int WNB = TRIL ? 4 : 2;            // 32-column blocks per wave
    const int wr = TRIL ? 32 * wave : 64 * wm;   // the wave's first row in the tile
    const int wc = TRIL ? 0 : 64 * wn;           // the wave's first column in the tile
    f32x16 acc[WMB][WNB];
#pragma unroll
    for (int mi = 0; mi < WMB; ++mi)
#pragma unroll
        for (int ni = 0; ni < WNB; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mi][ni][v] = 0.0f;

    const int Keff = g.b_upper ? min(K, col0 + BN) : K;   // rows of op(B) that can be nonzero
    const int KT = (Keff + BK - 1) / BK;
    load_a(0);
    load_b(0);
    store_a(0);
    store_b(0);
    __syncthreads();

    const int lrow = lane & 31;
    const int lk = lane >> 5;
    const int cw = col0 + wc;   // the wave's first column
    // one stage's MFMAs for the column blocks in MASK (bit ni: block ni),
    // the operands of step kk + 2 read while step kk's MFMAs run (two register
    // sets): the matrix pipe does not wait for the LDS between steps
    auto kstep = [&](int cur, auto maskc) {
        constexpr int MASK = decltype(maskc)::value;
        float fa[2][WMB], fb[2][WNB];
        auto read_step = [&](int fbuf, int kk) {
#pragma unroll
            for (int mi = 0; mi < WMB; ++mi) fa[fbuf][mi] = As[cur][kk + lk][wr + 32 * mi + lrow];
#pragma unroll
            for (int ni = 0; ni < WNB; ++ni)
                if ((MASK >> ni) & 1) fb[fbuf][ni] = Bs[cur][kk + lk][wc + 32 * ni + lrow];
        };
        read_step(0, 0);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 2) {
            const int fbuf = (kk >> 1) & 1;
            if (kk + 2 < BK) read_step(fbuf ^ 1, kk + 2);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int ni = 0; ni < WNB; ++ni)
                if ((MASK >> ni) & 1) {
#pragma unroll
                    for (int mi = 0; mi < WMB; ++mi)
                        acc[mi][ni] =
                            __builtin_amdgcn_mfma_f32_32x32x2f32(fa[fbuf][mi], fb[fbuf][ni], acc[mi][ni], 0, 0, 0);
                }
        }
    };
    // NB = the wave's 32-column blocks that hold columns below N (wave-uniform):
    // a block past N (the last tile column of N = 1056, say) takes no MFMAs.
    // With an upper-triangular op(B) (b_upper) a block needs only the rows up
    // to its last column: in the tile's last K stages the blocks whose columns
    // all lie before the stage's rows skip their MFMAs (zero B operands).
    auto kloop = [&](auto nbc) {
        constexpr int NB = decltype(nbc)::value;
        constexpr int FULL = (1 << NB) - 1;
        for (int kt = 0; kt < KT; ++kt) {
            const int cur = kt & 1;
            const bool more = (kt + 1 < KT);
            if (more) {
                load_a((kt + 1) * BK);
                load_b((kt + 1) * BK);
            }
            if constexpr (NB > 0) {
                const int k0 = kt * BK;
                if (!g.b_upper || k0 < cw + 32) {
                    kstep(cur, std::integral_constant<int, FULL>());
                } else if constexpr (TRIL) {
                    // blocks d .. of the wave's four (k0 = cw + 32 d, d = 1 .. 3)
                    const int d = (k0 - cw) >> 5;
                    if (d == 1) {
                        if constexpr ((FULL & 0xE) != 0) kstep(cur, std::integral_constant<int, FULL & 0xE>());
                    } else if (d == 2) {
                        if constexpr ((FULL & 0xC) != 0) kstep(cur, std::integral_constant<int, FULL & 0xC>());
                    } else if (d == 3) {
                        if constexpr ((FULL & 0x8) != 0) kstep(cur, std::integral_constant<int, FULL & 0x8>());
                    }
                } else if (NB > 1 && k0 < cw + 64) {
                    kstep(cur, std::integral_constant<int, (NB > 1) ? 2 : 0>());
                }
            }
            if (more) {
                store_a(cur ^ 1);
                store_b(cur ^ 1);
            }
            __syncthreads();
        }
    };
    if constexpr (TRIL) {
        const int nv = (N - cw + 31) / 32;
        if (nv >= 4) kloop(std::integral_constant<int, 4>());
        else if (nv == 3) kloop(std::integral_constant<int, 3>());
        else if (nv == 2) kloop(std::integral_constant<int, 2>());
        else if (nv == 1) kloop(std::integral_constant<int, 1>());
        else kloop(std::integral_constant<int, 0>());
    } else {
        if (cw + 32 < N) kloop(std::integral_constant<int, 2>());
        else if (cw < N) kloop(std::integral_constant<int, 1>());
        else kloop(std::integral_constant<int, 0>());
    }

    // ---- epilogue: 32x32 block layout, lane holds column (lane & 31) and rows
    //      (v & 3) + 8 (v >> 2) + 4 (lane >> 5) for accumulator register v.
    const float alpha = g.alpha, beta = g.beta;
    if constexpr (PLANES) {
        // the three bf16 planes of the result, transposed (plane row c holds
        // column c), through LDS so that each column's 128 rows go out as
        // whole 16-byte pieces: per half of the tile's columns, the waves that
        // hold them write T[c][r] (fp32, row pitch TP), then thread t splits
        // rows 32 (t & 3) .. + 31 of column t >> 2 and stores 64 bytes per plane
        constexpr int TP = BM + 1;
        static_assert(64 * TP <= 2 * BK * BM + 2 * BK * BN, "plane staging exceeds the operand stages");
        float* T = smem;
        uint16_t* pl = g.planes + static_cast<int64_t>(bz) * g.stridePl;
        const bool v16 = (g.ldpl % 8) == 0 && (g.planeStride % 8) == 0 && (g.stridePl % 8) == 0 &&
                         (reinterpret_cast<uintptr_t>(g.planes) % 16) == 0;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
            for (int ni = 0; ni < WNB; ++ni) {
                const int cl = wc + 32 * ni;           // the block's first column in the tile
                if ((cl >> 6) != half) continue;
#pragma unroll
                for (int mi = 0; mi < WMB; ++mi)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int rl = wr + mi * 32 + (v & 3) + 8 * (v >> 2) + 4 * lk;
                        T[(cl - 64 * half + lrow) * TP + rl] = (row0 + rl < M) ? alpha * acc[mi][ni][v] : 0.0f;
                    }
            }
            __syncthreads();
            const int cl = t >> 2, seg = t & 3;
            const int c = col0 + half * 64 + cl;
            const int r = row0 + 32 * seg;
            if (c < N && r < g.rows_pad) {
                uint16_t* dst = pl + static_cast<int64_t>(c) * g.ldpl + r;
                const float* src = T + cl * TP + 32 * seg;
                if (v16 && r + 32 <= g.rows_pad) {
#pragma unroll
                    for (int e8 = 0; e8 < 4; ++e8) {
                        uint16_t h[3][8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) split3_rn(src[8 * e8 + e], h[0][e], h[1][e], h[2][e]);
#pragma unroll
                        for (int p = 0; p < 3; ++p)
                            *reinterpret_cast<uint4*>(dst + p * g.planeStride + 8 * e8) =
                                make_uint4(h[p][0] | (static_cast<uint32_t>(h[p][1]) << 16),
                                           h[p][2] | (static_cast<uint32_t>(h[p][3]) << 16),
                                           h[p][4] | (static_cast<uint32_t>(h[p][5]) << 16),
                                           h[p][6] | (static_cast<uint32_t>(h[p][7]) << 16));
                    }
                } else {
                    for (int e = 0; e < 32 && r + e < g.rows_pad; ++e) {
                        uint16_t h1, h2, h3;
                        split3_rn(src[e], h1, h2, h3);
                        dst[e] = h1;
                        dst[g.planeStride + e] = h2;
                        dst[2 * g.planeStride + e] = h3;
                    }
                }
            }
            __syncthreads();
        }
        return;
    }
#pragma unroll
    for (int mi = 0; mi < WMB; ++mi) {
#pragma unroll
        for (int ni = 0; ni < WNB; ++ni) {
            const int c = col0 + wc + ni * 32 + lrow;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int r = row0 + wr + mi * 32 + (v & 3) + 8 * (v >> 2) + 4 * lk;
                if (r < M && c < N) {
                    float* dst = C + static_cast<int64_t>(r) * g.ldc + c;
                    float val = alpha * acc[mi][ni][v];
                    if (beta != 0.0f) val += beta * (*dst);
                    *dst = val;
                }
            }
        }
    }
}

template <ALayout LA, BLayout LB, typename TA, typename TB, bool PLANES = false, bool TRIL = false>
hipError_t launch_one(const GemmArgs& g, int batch, hipStream_t stream) {
    dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, batch);
    // 16-byte vector loads need every row start 16-byte aligned
    const int amul = (sizeof(TA) == 4) ? 4 : 8;   // elements per 16-byte vector
    const int bmul = (sizeof(TB) == 4) ? 4 : 8;
    const int a_vec = (g.lda % amul == 0) && (batch == 1 || g.strideA % amul == 0) &&
                      (reinterpret_cast<uintptr_t>(g.A) % 16 == 0);
    const int b_vec = (g.ldb % bmul == 0) && (batch == 1 || g.strideB % bmul == 0) &&
                      (reinterpret_cast<uintptr_t>(g.B) % 16 == 0);
    hipLaunchKernelGGL((gemm_f32_kernel<LA, LB, TA, TB, PLANES, TRIL>), grid, dim3(NT), 0, stream, g, a_vec, b_vec);
    return hipGetLastError();
}

template <ALayout LA, BLayout LB>
hipError_t dispatch_types(bool a_bf16, bool b_bf16, const GemmArgs& g, int batch, hipStream_t s) {
    if (a_bf16 && b_bf16) return hipErrorInvalidValue;
    if (a_bf16) return launch_one<LA, LB, bf16_t, float>(g, batch, s);
    if (b_bf16) return launch_one<LA, LB, float, bf16_t>(g, batch, s);
    return launch_one<LA, LB, float, float>(g, batch, s);
}

}  // namespace

hipError_t launch_gemm(ALayout la, BLayout lb, bool a_bf16, bool b_bf16, const GemmArgs& g, int batch,
                       hipStream_t stream) {
    if (g.M <= 0 || g.N <= 0 || batch <= 0) return hipSuccess;
    if (g.planes != nullptr) {
        // plane output: fp32 operands, A K-contiguous and B N-contiguous only
        // (the product Y R^-1 of the orthonormalisation)
        if (la != ALayout::kKContig || lb != BLayout::kNContig || a_bf16 || b_bf16 || g.beta != 0.0f ||
            g.rows_pad < g.M || g.rows_pad > (g.M + BM - 1) / BM * BM || g.ldpl < g.rows_pad ||
            g.planeStride < g.ldpl * g.N || (batch > 1 && g.stridePl < 3 * g.planeStride))
            return hipErrorInvalidValue;
        return g.b_upper ? launch_one<ALayout::kKContig, BLayout::kNContig, float, float, true, true>(g, batch, stream)
                         : launch_one<ALayout::kKContig, BLayout::kNContig, float, float, true>(g, batch, stream);
    }
    // an upper-triangular op(B) (Y R^-1): the 4 x 1 wave layout
    if (g.b_upper && la == ALayout::kKContig && lb == BLayout::kNContig && !a_bf16 && !b_bf16)
        return launch_one<ALayout::kKContig, BLayout::kNContig, float, float, false, true>(g, batch, stream);
    if (la == ALayout::kKContig && lb == BLayout::kNContig)
        return dispatch_types<ALayout::kKContig, BLayout::kNContig>(a_bf16, b_bf16, g, batch, stream);
    if (la == ALayout::kMContig && lb == BLayout::kNContig)
        return dispatch_types<ALayout::kMContig, BLayout::kNContig>(a_bf16, b_bf16, g, batch, stream);
    if (la == ALayout::kKContig && lb == BLayout::kKContig)
        return dispatch_types<ALayout::kKContig, BLayout::kKContig>(a_bf16, b_bf16, g, batch, stream);
    return dispatch_types<ALayout::kMContig, BLayout::kKContig>(a_bf16, b_bf16, g, batch, stream);
}

}  // namespace galore
