// 8-bit block-wise low-rank Adam (paper §4.2: GaLore 2 uses the 8-bit Adam
// optimizer of bitsandbytes, after Dettmers et al.). The moments of each
// matrix live in blocks of 2048 consecutive elements of the row-major r x l
// state: M as OCP FP8 E4M3 codes of M / scale_M, V as E5M2 codes of V /
// scale_V, one scale per block: the smallest power of two 2^k with block max
// |value| <= 2^k * (the format's largest finite value), 0 for an all-zero
// block. Power-of-two scales make encoding and decoding exact scalings, so
// only the format's own rounding decides a code.
//
// One workgroup owns one block (256 threads x 8 elements): it decodes the
// moments, runs the Adam step in fp32 (N from the fresh moments), reduces the
// new block maxima, and re-encodes with the new scales. One pass
// over HBM: R and N 4 bytes each, the two codes 1 byte each in and out, so 12
// bytes per element against 24 for fp32 moments.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "common.hpp"

namespace galore {
namespace {

constexpr int A8_BLOCK = 2048;
constexpr int A8_T = 256;
constexpr int A8_E = A8_BLOCK / A8_T;   // 8 elements per thread

// gfx950's FP8 conversions are the OCP formats: v_cvt_f32_fp8 / _bf8 decode
// E4M3 / E5M2 exactly, and v_cvt_pk_fp8_f32 / _bf8_f32 round half to even.
// With power-of-two block scales every encoded value lies within the
// format's finite range, where these conversions agree bit for bit with the
// OCP definition (compared over every binary32 value of the range and every
// code).
template <int SEL>
__device__ __forceinline__ float dec_e4m3(unsigned w) { return __builtin_amdgcn_cvt_f32_fp8(static_cast<int>(w), SEL); }
template <int SEL>
__device__ __forceinline__ float dec_e5m2(unsigned w) { return __builtin_amdgcn_cvt_f32_bf8(static_cast<int>(w), SEL); }
__device__ __forceinline__ unsigned enc4_e4m3(float a, float b, float c, float d) {
    const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
    return static_cast<unsigned>(__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true));
}
__device__ __forceinline__ unsigned enc4_e5m2(float a, float b, float c, float d) {
    const int lo = __builtin_amdgcn_cvt_pk_bf8_f32(a, b, 0, false);
    return static_cast<unsigned>(__builtin_amdgcn_cvt_pk_bf8_f32(c, d, lo, true));
}

// exponent k of the block scale: the smallest 2^k with amax <= 2^k * maxval
// (kNoScale for an all-zero block, whose scale is 0)
constexpr int kNoScale = -100000;
__device__ __forceinline__ int pow2_exponent(float amax, float maxval) {
    if (!(amax > 0.0f)) return kNoScale;
    int e, em;
    const float f = frexpf(amax, &e), fm = frexpf(maxval, &em);
    return e - em + (f > fm ? 1 : 0);
}

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

// Thread t owns elements 4 t .. 4 t + 3 and 1024 + 4 t .. 1024 + 4 t + 3 of
// its block, so each load and store instruction of a wave covers one
// contiguous span (1 KB of fp32, 256 bytes of codes).
__global__ __launch_bounds__(A8_T) void adam8_kernel(const float* Rb, float* Nb, int64_t ld, int64_t stride,
                                                     uint8_t* M8b, float* Msb, uint8_t* V8b, float* Vsb, int64_t cols,
                                                     int64_t count, int64_t nblk, float beta1, float beta2, float eps,
                                                     float ibc1, float ibc2, int vec) {
    __shared__ float red[2][A8_T / 64];
    const int64_t b = blockIdx.y;
    const int64_t blk = blockIdx.x;
    const float* R = Rb + b * stride;
    float* N = Nb + b * stride;
    uint8_t* M8 = M8b + b * count;
    uint8_t* V8 = V8b + b * count;
    float* Ms = Msb + b * nblk;
    float* Vs = Vsb + b * nblk;
    const int64_t blk0 = blk * A8_BLOCK;
    const float ms = Ms[blk], vs = Vs[blk];
    const float om1 = 1.0f - beta1, om2 = 1.0f - beta2;

    float g[A8_E], mf[A8_E], vf[A8_E];
    unsigned wm[2], wv[2];     // four codes per word, element 4 h + e in byte e of word h
    // a group of 4 lies in one row when cols % 4 == 0 (vec)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int64_t e0 = blk0 + h * (A8_BLOCK / 2) + 4 * static_cast<int64_t>(threadIdx.x);
        if (vec && e0 + 4 <= count) {
            const int64_t i = e0 / cols, j = e0 - i * cols;
            const f32x4 a = *reinterpret_cast<const f32x4*>(R + i * ld + j);
#pragma unroll
            for (int e = 0; e < 4; ++e) g[4 * h + e] = a[e];
            wm[h] = *reinterpret_cast<const unsigned*>(M8 + e0);
            wv[h] = *reinterpret_cast<const unsigned*>(V8 + e0);
        } else {
            wm[h] = 0u;
            wv[h] = 0u;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t idx = e0 + e;
                g[4 * h + e] = 0.0f;
                if (idx < count) {
                    const int64_t i = idx / cols, j = idx - i * cols;
                    g[4 * h + e] = R[i * ld + j];
                    wm[h] |= static_cast<unsigned>(M8[idx]) << (8 * e);
                    wv[h] |= static_cast<unsigned>(V8[idx]) << (8 * e);
                }
            }
        }
    }
    float m[A8_E], v[A8_E];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        m[4 * h] = dec_e4m3<0>(wm[h]);
        m[4 * h + 1] = dec_e4m3<1>(wm[h]);
        m[4 * h + 2] = dec_e4m3<2>(wm[h]);
        m[4 * h + 3] = dec_e4m3<3>(wm[h]);
        v[4 * h] = dec_e5m2<0>(wv[h]);
        v[4 * h + 1] = dec_e5m2<1>(wv[h]);
        v[4 * h + 2] = dec_e5m2<2>(wv[h]);
        v[4 * h + 3] = dec_e5m2<3>(wv[h]);
    }
    float am = 0.0f, av = 0.0f;
    float n[A8_E];
#pragma unroll
    for (int e = 0; e < A8_E; ++e) {
        const float m1 = beta1 * (m[e] * ms) + om1 * g[e];          // decoding times 2^k is exact
        const float v1 = beta2 * (v[e] * vs) + om2 * (g[e] * g[e]);
        // N = (m1 / bc1) / (sqrt(v1 / bc2) + eps) with hardware reciprocal and
        // square root (within a few ulps; the state's codes do not depend on N)
        n[e] = (m1 * ibc1) * __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(v1 * ibc2) + eps);
        mf[e] = m1;
        vf[e] = v1;
        am = fmaxf(am, fabsf(m1));     // out-of-range slots hold zeros
        av = fmaxf(av, v1);
    }
    // every thread has read the old scales before the first barrier
    const int km = pow2_exponent(block_max(am, red[0]), 448.0f);
    const int kv = pow2_exponent(block_max(av, red[1]), 57344.0f);
    if (threadIdx.x == 0) {
        Ms[blk] = (km == kNoScale) ? 0.0f : ldexpf(1.0f, km);
        Vs[blk] = (kv == kNoScale) ? 0.0f : ldexpf(1.0f, kv);
    }
    // exact scaling by 2^-k; an all-zero block gets codes 0
    const float im = (km == kNoScale) ? 0.0f : ldexpf(1.0f, -km);
    const float iv = (kv == kNoScale) ? 0.0f : ldexpf(1.0f, -kv);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        wm[h] = (km == kNoScale) ? 0u
                                 : enc4_e4m3(mf[4 * h] * im, mf[4 * h + 1] * im, mf[4 * h + 2] * im, mf[4 * h + 3] * im);
        wv[h] = (kv == kNoScale) ? 0u
                                 : enc4_e5m2(vf[4 * h] * iv, vf[4 * h + 1] * iv, vf[4 * h + 2] * iv, vf[4 * h + 3] * iv);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int64_t e0 = blk0 + h * (A8_BLOCK / 2) + 4 * static_cast<int64_t>(threadIdx.x);
        if (vec && e0 + 4 <= count) {
            const int64_t i = e0 / cols, j = e0 - i * cols;
            *reinterpret_cast<f32x4*>(N + i * ld + j) = f32x4{n[4 * h], n[4 * h + 1], n[4 * h + 2], n[4 * h + 3]};
            *reinterpret_cast<unsigned*>(M8 + e0) = wm[h];
            *reinterpret_cast<unsigned*>(V8 + e0) = wv[h];
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t idx = e0 + e;
                if (idx < count) {
                    const int64_t i = idx / cols, j = idx - i * cols;
                    N[i * ld + j] = n[4 * h + e];
                    M8[idx] = static_cast<uint8_t>(wm[h] >> (8 * e));
                    V8[idx] = static_cast<uint8_t>(wv[h] >> (8 * e));
                }
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
    const bool vec = (cols % 4 == 0) && (ld % 4 == 0) && (stride % 4 == 0) &&
                     (reinterpret_cast<uintptr_t>(R) % 16 == 0) && (reinterpret_cast<uintptr_t>(N) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(M8) % 4 == 0) && (reinterpret_cast<uintptr_t>(V8) % 4 == 0);
    if (nblk > 0x7fffffff) return hipErrorInvalidValue;
    dim3 grid(static_cast<unsigned>(nblk), batch);
    hipLaunchKernelGGL(adam8_kernel, grid, dim3(A8_T), 0, stream, R, N, ld, stride, M8, Ms, V8, Vs, cols, count, nblk,
                       beta1, beta2, eps, 1.0f / bc1, 1.0f / bc2, vec ? 1 : 0);
    return hipGetLastError();
}

}  // namespace galore
