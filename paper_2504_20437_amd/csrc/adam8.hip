// 8-bit block-wise low-rank Adam (paper §4.2: GaLore 2 uses the 8-bit Adam
// optimizer of bitsandbytes, after Dettmers et al.). The moments of each
// matrix live in blocks of 2048 consecutive elements of the row-major r x l
// state: M as OCP FP8 E4M3 codes of M / scale_M, V as E5M2 codes of V /
// scale_V, one binary32 scale per block (block max of |value| over the
// format's largest finite value; 0 for an all-zero block).
//
// One workgroup owns one block (256 threads x 8 consecutive elements): it
// decodes the moments, runs the Adam step in fp32 (N from the fresh moments),
// reduces the new block maxima, and re-encodes with the new scales. One pass
// over HBM: R and N 4 bytes each, the two codes 1 byte each in and out, so 12
// bytes per element against 24 for fp32 moments. The FP8 conversions are done
// in software (round half to even, saturating at the largest finite value,
// subnormals kept) so that they follow the OCP definition exactly.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "common.hpp"

namespace galore {
namespace {

constexpr int A8_BLOCK = 2048;
constexpr int A8_T = 256;
constexpr int A8_E = A8_BLOCK / A8_T;   // 8 elements per thread

// format parameters: mantissa bits, exponent bias, largest finite code
template <int MB, int BIAS, int MAXCODE>
struct Fp8 {
    static __device__ __forceinline__ float decode(unsigned c) {
        const int mag = c & 0x7F, ef = mag >> MB, m = mag & ((1 << MB) - 1);
        const float v = (ef == 0) ? ldexpf(static_cast<float>(m), 1 - BIAS - MB)
                                  : ldexpf(static_cast<float>((1 << MB) + m), ef - BIAS - MB);
        return (c & 0x80) ? -v : v;
    }
    static __device__ __forceinline__ unsigned encode(float x) {
        const unsigned bits = __float_as_uint(x);
        const unsigned sign = (bits >> 24) & 0x80u;
        const float y = fabsf(x);
        if (y == 0.0f) return sign;
        constexpr int emin = 1 - BIAS;
        int E = static_cast<int>((bits >> 23) & 0xFFu) - 127;     // y in [2^E, 2^(E+1)) for normal y
        if (E < emin) E = emin;
        if (E > 30) return sign | MAXCODE;
        float k = rintf(ldexpf(y, MB - E));                       // exact power-of-two scaling, then RNE
        if (k == static_cast<float>(2 << MB)) {
            E += 1;
            k = static_cast<float>(1 << MB);
        }
        const int ki = static_cast<int>(k);
        if (ki < (1 << MB)) return sign | static_cast<unsigned>(ki);
        int code = ((E + BIAS) << MB) | (ki - (1 << MB));
        if (code > MAXCODE) code = MAXCODE;
        return sign | static_cast<unsigned>(code);
    }
};
using E4M3 = Fp8<3, 7, 0x7E>;
using E5M2 = Fp8<2, 15, 0x7B>;

__device__ __forceinline__ float block_max(float x, float* red) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[w] = x;
    __syncthreads();
    float m = red[0];
#pragma unroll
    for (int i = 1; i < A8_T / 64; ++i) m = fmaxf(m, red[i]);
    return m;
}

__global__ __launch_bounds__(A8_T) void adam8_kernel(const float* Rb, float* Nb, int64_t ld, int64_t stride,
                                                     uint8_t* M8b, float* Msb, uint8_t* V8b, float* Vsb, int64_t cols,
                                                     int64_t count, int64_t nblk, float beta1, float beta2, float eps,
                                                     float bc1, float bc2, int vec) {
    __shared__ float red[2][A8_T / 64];
    const int64_t b = blockIdx.y;
    const int64_t blk = blockIdx.x;
    const float* R = Rb + b * stride;
    float* N = Nb + b * stride;
    uint8_t* M8 = M8b + b * count;
    uint8_t* V8 = V8b + b * count;
    float* Ms = Msb + b * nblk;
    float* Vs = Vsb + b * nblk;
    const int64_t base = blk * A8_BLOCK + static_cast<int64_t>(threadIdx.x) * A8_E;
    const float ms = Ms[blk], vs = Vs[blk];
    const float om1 = 1.0f - beta1, om2 = 1.0f - beta2;

    float g[A8_E], mf[A8_E], vf[A8_E];
    unsigned cm[A8_E], cv[A8_E];
    // the 8 elements of a thread lie in one row when cols % 8 == 0
    const bool fast = vec && base + A8_E <= count;
    if (fast) {
        const int64_t i = base / cols, j = base - i * cols;
        const f32x4* src = reinterpret_cast<const f32x4*>(R + i * ld + j);
        const f32x4 a = src[0], c = src[1];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            g[e] = a[e];
            g[4 + e] = c[e];
        }
        const uint2 qm = *reinterpret_cast<const uint2*>(M8 + base);
        const uint2 qv = *reinterpret_cast<const uint2*>(V8 + base);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            cm[e] = (qm.x >> (8 * e)) & 0xFFu;
            cm[4 + e] = (qm.y >> (8 * e)) & 0xFFu;
            cv[e] = (qv.x >> (8 * e)) & 0xFFu;
            cv[4 + e] = (qv.y >> (8 * e)) & 0xFFu;
        }
    } else {
#pragma unroll
        for (int e = 0; e < A8_E; ++e) {
            const int64_t idx = base + e;
            if (idx < count) {
                const int64_t i = idx / cols, j = idx - i * cols;
                g[e] = R[i * ld + j];
                cm[e] = M8[idx];
                cv[e] = V8[idx];
            } else {
                g[e] = 0.0f;
                cm[e] = 0u;
                cv[e] = 0u;
            }
        }
    }
    float am = 0.0f, av = 0.0f;
    float n[A8_E];
#pragma unroll
    for (int e = 0; e < A8_E; ++e) {
        const float m = E4M3::decode(cm[e]) * ms;
        const float v = E5M2::decode(cv[e]) * vs;
        const float m1 = beta1 * m + om1 * g[e];
        const float v1 = beta2 * v + om2 * (g[e] * g[e]);
        n[e] = (m1 / bc1) / (sqrtf(v1 / bc2) + eps);
        mf[e] = m1;
        vf[e] = v1;
        if (base + e < count) {
            am = fmaxf(am, fabsf(m1));
            av = fmaxf(av, fabsf(v1));
        }
    }
    // every thread has read the old scales before the first barrier
    const float bm = block_max(am, red[0]);
    const float bv = block_max(av, red[1]);
    const float sm = __fdiv_rn(bm, 448.0f), sv = __fdiv_rn(bv, 57344.0f);
    if (threadIdx.x == 0) {
        Ms[blk] = sm;
        Vs[blk] = sv;
    }
#pragma unroll
    for (int e = 0; e < A8_E; ++e) {
        cm[e] = (sm > 0.0f) ? E4M3::encode(__fdiv_rn(mf[e], sm)) : 0u;
        cv[e] = (sv > 0.0f) ? E5M2::encode(__fdiv_rn(vf[e], sv)) : 0u;
    }
    if (fast) {
        const int64_t i = base / cols, j = base - i * cols;
        f32x4* dst = reinterpret_cast<f32x4*>(N + i * ld + j);
        dst[0] = f32x4{n[0], n[1], n[2], n[3]};
        dst[1] = f32x4{n[4], n[5], n[6], n[7]};
        uint2 qm, qv;
        qm.x = cm[0] | (cm[1] << 8) | (cm[2] << 16) | (cm[3] << 24);
        qm.y = cm[4] | (cm[5] << 8) | (cm[6] << 16) | (cm[7] << 24);
        qv.x = cv[0] | (cv[1] << 8) | (cv[2] << 16) | (cv[3] << 24);
        qv.y = cv[4] | (cv[5] << 8) | (cv[6] << 16) | (cv[7] << 24);
        *reinterpret_cast<uint2*>(M8 + base) = qm;
        *reinterpret_cast<uint2*>(V8 + base) = qv;
    } else {
#pragma unroll
        for (int e = 0; e < A8_E; ++e) {
            const int64_t idx = base + e;
            if (idx < count) {
                const int64_t i = idx / cols, j = idx - i * cols;
                N[i * ld + j] = n[e];
                M8[idx] = static_cast<uint8_t>(cm[e]);
                V8[idx] = static_cast<uint8_t>(cv[e]);
            }
        }
    }
}

}  // namespace

int64_t adam8_block_count(int64_t rows, int64_t cols) { return (rows * cols + A8_BLOCK - 1) / A8_BLOCK; }

hipError_t launch_adam8(const float* R, float* N, int64_t ld, int64_t stride, uint8_t* M8, float* Ms, uint8_t* V8,
                        float* Vs, int64_t rows, int64_t cols, int batch, float beta1, float beta2, float eps,
                        float bc1, float bc2, hipStream_t stream) {
    const int64_t count = rows * cols;
    const int64_t nblk = adam8_block_count(rows, cols);
    const bool vec = (cols % 8 == 0) && (ld % 4 == 0) && (stride % 4 == 0) && (count % 8 == 0) &&
                     (reinterpret_cast<uintptr_t>(R) % 16 == 0) && (reinterpret_cast<uintptr_t>(N) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(M8) % 8 == 0) && (reinterpret_cast<uintptr_t>(V8) % 8 == 0);
    if (nblk > 0x7fffffff) return hipErrorInvalidValue;
    dim3 grid(static_cast<unsigned>(nblk), batch);
    hipLaunchKernelGGL(adam8_kernel, grid, dim3(A8_T), 0, stream, R, N, ld, stride, M8, Ms, V8, Vs, cols, count, nblk,
                       beta1, beta2, eps, bc1, bc2, vec ? 1 : 0);
    return hipGetLastError();
}

}  // namespace galore
