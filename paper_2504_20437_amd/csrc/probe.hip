// Measurement helpers. The chip's sustained bf16 matrix-core rate: every wave
// runs four independent chains of v_mfma_f32_32x32x16_bf16 on register
// operands (no memory traffic inside the loop), so the launch time divided
// into the MFMA work gives the rate the matrix cores reach under sustained
// load, at whatever clock the chip holds then. The per-block results are
// stored so that the work cannot be removed. And its streaming bandwidth: a
// copy kernel with the element-wise kernels' access pattern.
#include <hip/hip_runtime.h>

#include "common.hpp"

namespace galore {
namespace {

typedef __bf16 pbf16x8 __attribute__((ext_vector_type(8)));

__global__ __launch_bounds__(256) void mfma_probe_kernel(int64_t iters, float* sink) {
    union {
        uint32_t u[4];
        pbf16x8 v;
    } a, b;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a.u[i] = 0x3f803f80u ^ (threadIdx.x & 7u);          // values near 1, lane dependent
        b.u[i] = 0x3f003f00u ^ ((threadIdx.x >> 3) & 7u);
    }
    f32x16 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.0f;
    for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, acc[j], 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) s += acc[j][v];
    sink[static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x] = s;
}

// Streaming copy: one 16-byte vector per thread over a grid covering the
// array, non-temporal loads and stores (the access pattern of the element-wise
// kernels of the path).
__global__ __launch_bounds__(256) void copy_probe_kernel(const f32x4* src, f32x4* dst, int64_t nvec) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < nvec) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

}  // namespace

hipError_t launch_copy_probe(const void* src, void* dst, int64_t nvec, hipStream_t stream) {
    const int64_t blocks = (nvec + 255) / 256;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL(copy_probe_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                       static_cast<const f32x4*>(src), static_cast<f32x4*>(dst), nvec);
    return hipGetLastError();
}

hipError_t launch_mfma_probe(int64_t iters, int blocks, float* sink, hipStream_t stream) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(256), 0, stream, iters, sink);
    return hipGetLastError();
}

}  // namespace galore
