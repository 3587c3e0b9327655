// Gaussian sketch for the randomized range finder (Halko, Martinsson & Tropp
// 2011, §4), adopted for the subspace update in paper §4.1.2.
//
// Counter-based: entry (i, j) of the l x k sketch is a pure function of
// (seed, sketch index, j*l + i), so any thread can produce any entry, batches
// of matrices get independent sketches through the second counter word, and a
// column does not depend on k.
//   Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011): key (seed, 0),
//   counter (j*l + i, sketch_index, 0, 0); output words 0 and 1.
//   Box-Muller (1958) in fp64 on the top 53 bits: u1 in (0, 1], u2 in [0, 1),
//   z = sqrt(-2 ln u1) cos(2 pi u2); the entry is z rounded to fp32.
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

__global__ __launch_bounds__(256) void sketch_kernel(float* omega, int64_t l, int64_t k,
                                                     int64_t stride, uint64_t seed,
                                                     uint64_t sketch_index0) {
    const int b = blockIdx.y;
    float* out = omega + static_cast<int64_t>(b) * stride;
    const uint64_t sidx = sketch_index0 + static_cast<uint64_t>(b);
    const int64_t total = l * k;
    const double two_pow_m53 = 1.0 / 9007199254740992.0;
    const double two_pi = 6.283185307179586;
    for (int64_t pos = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; pos < total;
         pos += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = pos / k;
        const int64_t j = pos - i * k;
        const uint64_t e = static_cast<uint64_t>(j * l + i);
        const u64x4 w = philox4x64_10(e, sidx, 0, 0, seed, 0);
        const double u1 = static_cast<double>((w.v[0] >> 11) + 1) * two_pow_m53;
        const double u2 = static_cast<double>(w.v[1] >> 11) * two_pow_m53;
        const double z = sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
        out[pos] = static_cast<float>(z);
    }
}

}  // namespace

hipError_t launch_sketch(float* omega, int64_t l, int64_t k, int64_t stride, uint64_t seed,
                         uint64_t sketch_index0, int batch, hipStream_t stream) {
    const int64_t total = l * k;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    dim3 grid(static_cast<unsigned>(blocks), batch);
    hipLaunchKernelGGL(sketch_kernel, grid, dim3(256), 0, stream, omega, l, k, stride, seed,
                       sketch_index0);
    return hipGetLastError();
}

}  // namespace galore
