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

// Private rows, transposed and padded: src [rows, cols] holds the permuted rows; private
// expert p owns rows [offset[n_pub + p], offset[n_pub + p + 1]). dst [cols, P] gets
// dst[c][po_p + j] = src[offset[n_pub + p] + j][c] for j < count_p and zeros up to the next
// multiple of 64, with po_p the sum of the earlier private experts' padded counts. One
// block per 64 padded rows (x) x 64 columns (y); blocks past the last padded row do nothing.
__global__ __launch_bounds__(256) void transpose_priv_kernel(const uint16_t* __restrict__ src,
                                                              uint16_t* __restrict__ dst, int cols,
                                                              int P, const int32_t* count,
                                                              const int32_t* offset, int n_pub,
                                                              int n_priv) {
  __shared__ uint16_t tile[TT][TT + 2];
  __shared__ int s_po[PMPE_MAX_POOL + 1];
  const int tid = threadIdx.x;
  if (tid < 64) {
    int running = 0;
    for (int q0 = 0; q0 < n_priv; q0 += 64) {
      const int q = q0 + tid;
      const int v = (q < n_priv) ? (count[n_pub + q] + TT - 1) / TT * TT : 0;
      const int incl = wave_incl_scan(v);
      if (q < n_priv) s_po[q + 1] = running + incl;
      running += __shfl(incl, 63, 64);
    }
    if (tid == 0) s_po[0] = 0;
  }
  __syncthreads();
  const int j0 = blockIdx.x * TT;  // first padded row (dst column) of this block
  if (j0 >= s_po[n_priv]) return;
  int lo = 0, hi = n_priv - 1;  // last expert with s_po[q] <= j0
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_po[mid] <= j0) lo = mid; else hi = mid - 1;
  }
  const int pp = lo;
  const int jl = j0 - s_po[pp];  // first row of the block within expert pp
  const int cnt = count[n_pub + pp];
  const int src0 = offset[n_pub + pp] + jl;
  const int c0 = blockIdx.y * TT;
  const int ty = tid >> 4, tx = tid & 15;
  typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = ty + 16 * i;
    u16x4 v = u16x4{0, 0, 0, 0};
    if (jl + r < cnt) v = *(const u16x4*)(src + (size_t)(src0 + r) * cols + c0 + tx * 4);
#pragma unroll
    for (int j = 0; j < 4; ++j) tile[r][tx * 4 + j] = v[j];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = ty + 16 * i;
    u16x4 v;
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = tile[tx * 4 + j][c];
    *(u16x4*)(dst + (size_t)(c0 + c) * P + j0 + tx * 4) = v;
  }
}

}  // namespace

hipError_t launch_transpose_priv(const void* src, void* dst, int rows_max, int cols, int P,
                                 const int32_t* count, const int32_t* offset, int n_pub,
                                 int n_priv, hipStream_t s) {
  // padded private rows never exceed rows_max rounded up to 64, plus 64 per private expert
  const int ytiles = (rows_max + TT - 1) / TT + n_priv;
  transpose_priv_kernel<<<dim3(ytiles, cols / TT), 256, 0, s>>>((const uint16_t*)src, (uint16_t*)dst,
                                                                cols, P, count, offset, n_pub, n_priv);
  return hipGetLastError();
}

hipError_t launch_transpose(const void* src, void* dst, int n, int rows, int cols, hipStream_t s) {
  transpose_kernel<<<dim3(cols / TT, rows / TT, n), 256, 0, s>>>((const uint16_t*)src,
                                                                  (uint16_t*)dst, rows, cols);
  return hipGetLastError();
}

}  // namespace pmpe
