// Per-expert transposes of bf16 weight matrices: dst[e] = src[e]^T for n matrices of
// [rows, cols]. The backward multiplies by W2 and W13 along their output dimension; with
// transposed copies (K contiguous) those products run on the same grouped NT GEMM as the
// forward. 64 x 64 tiles staged through LDS (rows padded by two elements), 8-byte loads
// and stores along the contiguous dimension on both sides.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int TT = 64;

__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ src,
                                                         uint16_t* __restrict__ dst, int rows,
                                                         int cols) {
  __shared__ uint16_t tile[TT][TT + 2];
  const size_t mat = (size_t)rows * cols;
  const uint16_t* s = src + (size_t)blockIdx.z * mat;
  uint16_t* d = dst + (size_t)blockIdx.z * mat;
  const int r0 = blockIdx.y * TT, c0 = blockIdx.x * TT;
  const int ty = threadIdx.x >> 4, tx = threadIdx.x & 15;
  typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = ty + 16 * i;
    const u16x4 v = *(const u16x4*)(s + (size_t)(r0 + r) * cols + c0 + tx * 4);
#pragma unroll
    for (int j = 0; j < 4; ++j) tile[r][tx * 4 + j] = v[j];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = ty + 16 * i;  // row of dst = column of src
    u16x4 v;
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = tile[tx * 4 + j][c];
    *(u16x4*)(d + (size_t)(c0 + c) * rows + r0 + tx * 4) = v;
  }
}

}  // namespace

hipError_t launch_transpose(const void* src, void* dst, int n, int rows, int cols, hipStream_t s) {
  transpose_kernel<<<dim3(cols / TT, rows / TT, n), 256, 0, s>>>((const uint16_t*)src,
                                                                  (uint16_t*)dst, rows, cols);
  return hipGetLastError();
}

}  // namespace pmpe
