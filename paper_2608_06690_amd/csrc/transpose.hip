// Per-expert transposes of bf16 weight matrices: dst[e] = src[e]^T for n matrices of
// [rows, cols]. The backward multiplies by W2 and W13 along their output dimension; with
// transposed copies (K contiguous) those products run on the same grouped NT GEMM as the
// forward. 64 x 64 tiles staged through LDS, 16-byte loads and stores along the
// contiguous dimension on both sides.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int TT = 64;
constexpr int TP = TT + 8;  // LDS row pitch in elements (144 bytes: 16-byte aligned rows)

// One 64 x 64 tile: rows r of the source (row_ptr(r) or nullptr for a zero row, 16-byte
// aligned) to dst rows c, dst[c * ld_dst + r]. 16-byte loads and stores on both sides;
// the LDS tile is written in 16-byte rows and read down its columns.
template <class RowPtr>
__device__ __forceinline__ void tile_transpose(RowPtr row_ptr, uint16_t* __restrict__ dst,
                                               size_t ld_dst) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[TT][TP];
  const int tid = threadIdx.x;
  const int q = tid & 7;  // 16-byte chunk
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = (tid >> 3) + 32 * i;
    const uint16_t* src = row_ptr(r);
    const u32x4 v = src ? *(const u32x4*)(src + q * 8) : u32x4{0, 0, 0, 0};
    *(u32x4*)&tile[r][q * 8] = v;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = (tid >> 3) + 32 * i;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = (uint32_t)tile[q * 8 + 2 * e][c] | ((uint32_t)tile[q * 8 + 2 * e + 1][c] << 16);
    *(u32x4*)(dst + (size_t)c * ld_dst + q * 8) = u32x4{w[0], w[1], w[2], w[3]};
  }
}

__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ src,
                                                         uint16_t* __restrict__ dst, int rows,
                                                         int cols) {
  const size_t mat = (size_t)rows * cols;
  const uint16_t* s = src + (size_t)blockIdx.z * mat;
  uint16_t* d = dst + (size_t)blockIdx.z * mat;
  const int r0 = blockIdx.y * TT, c0 = blockIdx.x * TT;
  tile_transpose([&](int r) { return s + (size_t)(r0 + r) * cols + c0; }, d + (size_t)c0 * rows + r0,
                 (size_t)rows);
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
  tile_transpose([&](int r) -> const uint16_t* {
    return (jl + r < cnt) ? src + (size_t)(src0 + r) * cols + c0 : nullptr;
  }, dst + (size_t)c0 * P + j0, (size_t)P);
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
