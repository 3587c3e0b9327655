// Gaussian sketch for the randomized range finder (Halko, Martinsson & Tropp
// 2011, §4), adopted for the subspace update in paper §4.1.2.
//
// Counter-based: entries (4 i4 + t, j), t = 0..3, of the l x k sketch are a
// pure function of (seed, sketch index, j * ceil(l/4) + i4), so any thread can
// produce any group, batches of matrices get independent sketches through the
// second counter word, and a column does not depend on k.
//   Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011): key (seed, 0),
//   counter (j * ceil(l/4) + i4, sketch_index, 0, 0); output words 0, 1 give
//   the Box-Muller pair of rows 4 i4 and 4 i4 + 1, words 2, 3 that of rows
//   4 i4 + 2 and 4 i4 + 3.
//   Box-Muller (1958) in fp64 on the top 53 bits: u1 in (0, 1], u2 in [0, 1),
//   radius sqrt(-2 ln u1) times cos and sin of 2 pi u2; each entry is rounded
//   once to the nearest bfloat16 (ties to even).
// The sketch is written either as fp32 values (row-major l x k), or, for the
// bf16 matrix cores, directly as the one bf16 plane of its transpose (k rows
// of ldp, zero past l): with a bf16-valued sketch the first range sample A
// Omega is a single exact bf16 product.
#include "common.hpp"

namespace galore {
namespace {

struct u64x4 {
    uint64_t v[4];
};

__device__ __forceinline__ u64x4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                               uint64_t k0, uint64_t k1) {
    constexpr uint64_t kMul0 = 0xD2E7470EE14C6C93ULL;
    constexpr uint64_t kMul1 = 0xCA5A826395121157ULL;
    constexpr uint64_t kWeyl0 = 0x9E3779B97F4A7C15ULL;
    constexpr uint64_t kWeyl1 = 0xBB67AE8584CAA73BULL;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t hi0 = __umul64hi(kMul0, c0);
        const uint64_t lo0 = kMul0 * c0;
        const uint64_t hi1 = __umul64hi(kMul1, c2);
        const uint64_t lo1 = kMul1 * c2;
        const uint64_t n0 = hi1 ^ c1 ^ k0;
        const uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += kWeyl0;
        k1 += kWeyl1;
    }
    u64x4 out;
    out.v[0] = c0;
    out.v[1] = c1;
    out.v[2] = c2;
    out.v[3] = c3;
    return out;
}

__device__ __forceinline__ void normal_pair(uint64_t x0, uint64_t x1, double& z0, double& z1) {
    const double two_pow_m53 = 1.0 / 9007199254740992.0;
    const double two_pi = 6.283185307179586;
    const double u1 = static_cast<double>((x0 >> 11) + 1) * two_pow_m53;
    const double u2 = static_cast<double>(x1 >> 11) * two_pow_m53;
    const double rad = sqrt(-2.0 * log(u1));
    double sn, cs;
    sincos(two_pi * u2, &sn, &cs);
    z0 = rad * cs;
    z1 = rad * sn;
}

// bits of the bfloat16 nearest to z (ties to even), rounded once from fp64
__device__ __forceinline__ uint32_t bf16_bits(double z) {
    if (z == 0.0) return signbit(z) ? 0x8000u : 0u;
    int e;
    const double m = frexp(z, &e);
    const double r = ldexp(rint(ldexp(m, 8)), e - 8);   // 8 significant bits: exact in fp32
    return __float_as_uint(static_cast<float>(r)) >> 16;
}

// the four entries of group (i4, j) as bf16 bits (rows past l are not drawn)
__device__ __forceinline__ void group4(int64_t l, int64_t l4, int64_t i4, int64_t j, uint64_t sidx, uint64_t seed,
                                       uint32_t* h) {
    const u64x4 w = philox4x64_10(static_cast<uint64_t>(j * l4 + i4), sidx, 0, 0, seed, 0);
    double z0, z1, z2, z3;
    normal_pair(w.v[0], w.v[1], z0, z1);
    h[0] = bf16_bits(z0);
    h[1] = bf16_bits(z1);
    if (4 * i4 + 2 < l) {
        normal_pair(w.v[2], w.v[3], z2, z3);
        h[2] = bf16_bits(z2);
        h[3] = bf16_bits(z3);
    } else {
        h[2] = h[3] = 0u;
    }
}

// fp32 values, row-major l x k; one thread per group of four rows and column
__global__ __launch_bounds__(256) void sketch_kernel(float* omega, int64_t l, int64_t k, int64_t stride, uint64_t seed,
                                                     uint64_t sketch_index0) {
    const int b = blockIdx.y;
    float* out = omega + static_cast<int64_t>(b) * stride;
    const uint64_t sidx = sketch_index0 + static_cast<uint64_t>(b);
    const int64_t l4 = (l + 3) / 4;
    const int64_t total = l4 * k;
    for (int64_t pos = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; pos < total;
         pos += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i4 = pos / k;
        const int64_t j = pos - i4 * k;
        uint32_t h[4];
        group4(l, l4, i4, j, sidx, seed, h);
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (4 * i4 + t < l) out[(4 * i4 + t) * k + j] = __uint_as_float(h[t] << 16);
    }
}

// the bf16 plane of Omega^T: plane[j][i] = Omega[i][j] (k rows of ldp, zero for
// l <= i < ldp); with zero_rest the next two planes (at planeStride) are zeroed
__global__ __launch_bounds__(256) void sketch_plane_kernel(uint16_t* planes, int64_t ldp, int64_t planeStride,
                                                           int64_t stride, int64_t l, int64_t k, uint64_t seed,
                                                           uint64_t sketch_index0, int zero_rest) {
    const int b = blockIdx.y;
    uint16_t* pl = planes + static_cast<int64_t>(b) * stride;
    const uint64_t sidx = sketch_index0 + static_cast<uint64_t>(b);
    const int64_t l4 = (l + 3) / 4;
    const int64_t quarter = ldp / 4;        // ldp is a multiple of 4
    const int64_t total = k * quarter;
    for (int64_t pos = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; pos < total;
         pos += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t j = pos / quarter;
        const int64_t i4 = pos - j * quarter;
        uint2 v = make_uint2(0u, 0u);
        if (4 * i4 < l) {
            uint32_t h[4];
            group4(l, l4, i4, j, sidx, seed, h);
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if (4 * i4 + t >= l) h[t] = 0u;
            v = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
        }
        const int64_t o = j * ldp + 4 * i4;
        *reinterpret_cast<uint2*>(pl + o) = v;
        if (zero_rest) {
            *reinterpret_cast<uint2*>(pl + planeStride + o) = make_uint2(0u, 0u);
            *reinterpret_cast<uint2*>(pl + 2 * planeStride + o) = make_uint2(0u, 0u);
        }
    }
}

}  // namespace

hipError_t launch_sketch_plane(uint16_t* planes, int64_t ldp, int64_t planeStride, int64_t stride, int64_t l,
                               int64_t k, uint64_t seed, uint64_t sketch_index0, bool zero_rest, int batch,
                               hipStream_t stream) {
    if (ldp % 4 != 0 || ldp < l || planeStride % 4 != 0 || stride % 4 != 0 ||
        reinterpret_cast<uintptr_t>(planes) % 8 != 0)
        return hipErrorInvalidValue;
    const int64_t total = k * (ldp / 4);
    int64_t blocks = (total + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    dim3 grid(static_cast<unsigned>(blocks), batch);
    hipLaunchKernelGGL(sketch_plane_kernel, grid, dim3(256), 0, stream, planes, ldp, planeStride, stride, l, k, seed,
                       sketch_index0, zero_rest ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_sketch(float* omega, int64_t l, int64_t k, int64_t stride, uint64_t seed,
                         uint64_t sketch_index0, int batch, hipStream_t stream) {
    const int64_t total = (l + 3) / 4 * k;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    dim3 grid(static_cast<unsigned>(blocks), batch);
    hipLaunchKernelGGL(sketch_kernel, grid, dim3(256), 0, stream, omega, l, k, stride, seed,
                       sketch_index0);
    return hipGetLastError();
}

}  // namespace galore
