// Low-bit projector (paper §4.2: GaLore 2 supports low-bit projection
// matrices, after Q-GaLore). Each column of the s x r projector is quantised
// symmetrically: scale_j = max_i |P_ij| / qmax and code_ij = P_ij / scale_j
// rounded half to even, clamped to [-qmax, qmax] (qmax = 127 for 8 bits, 7
// for 4 bits), every deciding step in binary32; a zero column has scale 0.
// Codes are stored row-major: 8 bits one two's-complement byte per code, 4
// bits two codes per byte (column 2c in the low nibble).
//
// The projection and back-projection consume the codes as one bf16 plane:
// |code| <= 127 is an integer that bf16 holds exactly, so code x bf16 gradient
// products are exact on the bf16 matrix cores and the per-column scale is
// applied once (in the product's epilogue, or folded into N's rows).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "common.hpp"

namespace galore {
namespace {

constexpr int QC = 64;   // columns per workgroup
constexpr int QG = 4;    // row groups (one wave each)

__device__ __forceinline__ int load_code(const uint8_t* row, int c, int bits) {
    if (bits == 8) return static_cast<int>(static_cast<int8_t>(row[c]));
    const unsigned byte = row[c >> 1];
    const int nib = static_cast<int>((c & 1) ? (byte >> 4) : (byte & 0xFu));
    return (nib ^ 8) - 8;   // 4-bit two's complement
}

// bf16 bits of a small integer (exact: |c| < 256)
__device__ __forceinline__ uint16_t int_to_bf16(int c) {
    return static_cast<uint16_t>(__float_as_uint(static_cast<float>(c)) >> 16);
}

__global__ __launch_bounds__(QC* QG) void quantize_kernel(const float* Pb, int64_t ldp, int64_t strideP, int rows,
                                                          int r, int bits, uint8_t* Qb, int64_t ldq, int64_t strideQ,
                                                          float* scb, int64_t strideS) {
    const int b = blockIdx.y;
    const float* P = Pb + static_cast<int64_t>(b) * strideP;
    uint8_t* Q = Qb + static_cast<int64_t>(b) * strideQ;
    const int tc = threadIdx.x & (QC - 1);
    const int grp = threadIdx.x / QC;
    const int c = blockIdx.x * QC + tc;
    const bool live = c < r;
    const float qmax = static_cast<float>((1 << (bits - 1)) - 1);
    __shared__ float part[QG][QC];
    __shared__ float sc[QC];
    float amax = 0.0f;
    if (live)
        for (int i = grp; i < rows; i += QG) amax = fmaxf(amax, fabsf(P[static_cast<int64_t>(i) * ldp + c]));
    part[grp][tc] = amax;
    __syncthreads();
    if (grp == 0) {
        float m = part[0][tc];
        for (int g = 1; g < QG; ++g) m = fmaxf(m, part[g][tc]);
        const float s = __fdiv_rn(m, qmax);
        sc[tc] = s;
        if (live) scb[static_cast<int64_t>(b) * strideS + c] = s;
    }
    __syncthreads();
    const float s = sc[tc];
    // every lane of a wave runs the same rows (the 4-bit store pairs lanes)
    for (int i = grp; i < rows; i += QG) {
        int code = 0;
        if (live && s > 0.0f) {
            const float q = rintf(__fdiv_rn(P[static_cast<int64_t>(i) * ldp + c], s));
            code = static_cast<int>(fminf(fmaxf(q, -qmax), qmax));
        }
        uint8_t* row = Q + static_cast<int64_t>(i) * ldq;
        if (bits == 8) {
            if (live) row[c] = static_cast<uint8_t>(code & 0xFF);
        } else {
            const int other = __shfl_xor(code, 1);
            if (live && (tc & 1) == 0) row[c >> 1] = static_cast<uint8_t>((code & 0xF) | ((other & 0xF) << 4));
        }
    }
}

// plane[i][j] = code[i][j] (j < r), 0 for r <= j < pad
__global__ __launch_bounds__(256) void codes_rows_kernel(const uint8_t* Qb, int64_t ldq, int64_t strideQ, int bits,
                                                         int rows, int r, uint16_t* plb, int64_t ldpl,
                                                         int64_t stridePl, int pad) {
    const int b = blockIdx.z;
    const int i = blockIdx.y;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= rows || j >= pad) return;
    const uint8_t* row = Qb + static_cast<int64_t>(b) * strideQ + static_cast<int64_t>(i) * ldq;
    const int code = (j < r) ? load_code(row, j, bits) : 0;
    plb[static_cast<int64_t>(b) * stridePl + static_cast<int64_t>(i) * ldpl + j] = int_to_bf16(code);
}

// plane[j][i] = code[i][j] (i < rows), 0 for rows <= i < pad; 64 x 64 tiles
__global__ __launch_bounds__(256) void codes_transpose_kernel(const uint8_t* Qb, int64_t ldq, int64_t strideQ,
                                                              int bits, int rows, int r, uint16_t* plb, int64_t ldpl,
                                                              int64_t stridePl, int pad) {
    __shared__ uint16_t tile[64][66];
    const int b = blockIdx.z;
    const uint8_t* Q = Qb + static_cast<int64_t>(b) * strideQ;
    uint16_t* pl = plb + static_cast<int64_t>(b) * stridePl;
    const int i0 = blockIdx.y * 64, j0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int ii = ty; ii < 64; ii += 4) {
        const int i = i0 + ii, j = j0 + tx;
        const int code = (i < rows && j < r) ? load_code(Q + static_cast<int64_t>(i) * ldq, j, bits) : 0;
        tile[ii][tx] = int_to_bf16(code);
    }
    __syncthreads();
    for (int jj = ty; jj < 64; jj += 4) {
        const int j = j0 + jj, i = i0 + tx;
        if (j < r && i < pad) pl[static_cast<int64_t>(j) * ldpl + i] = tile[tx][jj];
    }
}

__global__ __launch_bounds__(256) void dequantize_kernel(const uint8_t* Qb, int64_t ldq, int64_t strideQ, int bits,
                                                         const float* scb, int64_t strideS, int rows, int r,
                                                         float* Tb, int64_t ldt, int64_t strideT) {
    const int b = blockIdx.z;
    const int i = blockIdx.y;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= rows || j >= r) return;
    const uint8_t* row = Qb + static_cast<int64_t>(b) * strideQ + static_cast<int64_t>(i) * ldq;
    Tb[static_cast<int64_t>(b) * strideT + static_cast<int64_t>(i) * ldt + j] =
        static_cast<float>(load_code(row, j, bits)) * scb[static_cast<int64_t>(b) * strideS + j];
}

}  // namespace

hipError_t launch_quantize(const float* P, int64_t ldp, int64_t strideP, int rows, int r, int bits, uint8_t* Q,
                           int64_t ldq, int64_t strideQ, float* scales, int64_t strideS, int batch,
                           hipStream_t stream) {
    if (bits != 8 && bits != 4) return hipErrorInvalidValue;
    dim3 grid((r + QC - 1) / QC, batch);
    hipLaunchKernelGGL(quantize_kernel, grid, dim3(QC * QG), 0, stream, P, ldp, strideP, rows, r, bits, Q, ldq,
                       strideQ, scales, strideS);
    return hipGetLastError();
}

hipError_t launch_codes_plane(const uint8_t* Q, int64_t ldq, int64_t strideQ, int bits, int rows, int r,
                              uint16_t* plane, int64_t ldpl, int64_t stridePl, int pad, bool transpose, int batch,
                              hipStream_t stream) {
    if (bits != 8 && bits != 4) return hipErrorInvalidValue;
    if (transpose) {
        dim3 grid((r + 63) / 64, (pad + 63) / 64, batch);
        hipLaunchKernelGGL(codes_transpose_kernel, grid, dim3(256), 0, stream, Q, ldq, strideQ, bits, rows, r, plane,
                           ldpl, stridePl, pad);
    } else {
        dim3 grid((pad + 255) / 256, rows, batch);
        hipLaunchKernelGGL(codes_rows_kernel, grid, dim3(256), 0, stream, Q, ldq, strideQ, bits, rows, r, plane, ldpl,
                           stridePl, pad);
    }
    return hipGetLastError();
}

hipError_t launch_dequantize(const uint8_t* Q, int64_t ldq, int64_t strideQ, int bits, const float* scales,
                             int64_t strideS, int rows, int r, float* Pt, int64_t ldt, int64_t strideT, int batch,
                             hipStream_t stream) {
    if (bits != 8 && bits != 4) return hipErrorInvalidValue;
    dim3 grid((r + 255) / 256, rows, batch);
    hipLaunchKernelGGL(dequantize_kernel, grid, dim3(256), 0, stream, Q, ldq, strideQ, bits, scales, strideS, rows, r,
                       Pt, ldt, strideT);
    return hipGetLastError();
}

}  // namespace galore
