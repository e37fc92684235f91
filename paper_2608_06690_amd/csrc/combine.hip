// K4 - combine: out[t] = sum_{j<k} gate[t,j] * y_perm[token_row[t,j]] (+ y_shared[t]).
//
// One workgroup per token; each thread owns 8 consecutive bf16 (or 4 fp32) columns,
// loaded as 16-byte vectors, so every y_perm row is read with full coalescing. The
// sum runs in fp32 in slot order j = 0..k-1 and is rounded once, which makes the
// output bitwise deterministic (no atomics). Slots with token_row = -1 (an invalid
// expert id upstream) contribute nothing.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int CB_THREADS = 256;

__global__ __launch_bounds__(CB_THREADS) void combine_bf16_kernel(CombineArgs a) {
  const int t = blockIdx.x;
  const int H = a.H;
  const uint16_t* yp = (const uint16_t*)a.y_perm;
  const uint16_t* ysh = (const uint16_t*)a.y_shared;
  uint16_t* out = (uint16_t*)a.out;
  for (int c = threadIdx.x * 8; c < H; c += CB_THREADS * 8) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int j = 0; j < a.k; ++j) {
      const int row = a.token_row[(size_t)t * a.k + j];
      if (row < 0) continue;
      const float g = a.gate[(size_t)t * a.k + j];
      const u32x4 v = *(const u32x4*)(yp + (size_t)row * H + c);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += g * bf16_to_f32(v[q] & 0xFFFFu);
        acc[2 * q + 1] += g * bf16_to_f32(v[q] >> 16);
      }
    }
    if (ysh) {
      const u32x4 v = *(const u32x4*)(ysh + (size_t)t * H + c);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += bf16_to_f32(v[q] & 0xFFFFu);
        acc[2 * q + 1] += bf16_to_f32(v[q] >> 16);
      }
    }
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = pack_bf16x2(acc[2 * q], acc[2 * q + 1]);
    *(u32x4*)(out + (size_t)t * H + c) = o;
  }
}

__global__ __launch_bounds__(CB_THREADS) void combine_f32_kernel(CombineArgs a) {
  const int t = blockIdx.x;
  const int H = a.H;
  const float* yp = (const float*)a.y_perm;
  const float* ysh = (const float*)a.y_shared;
  float* out = (float*)a.out;
  for (int c = threadIdx.x * 4; c < H; c += CB_THREADS * 4) {
    float4 acc = make_float4(0, 0, 0, 0);
    for (int j = 0; j < a.k; ++j) {
      const int row = a.token_row[(size_t)t * a.k + j];
      if (row < 0) continue;
      const float g = a.gate[(size_t)t * a.k + j];
      const float4 v = *(const float4*)(yp + (size_t)row * H + c);
      acc.x += g * v.x;
      acc.y += g * v.y;
      acc.z += g * v.z;
      acc.w += g * v.w;
    }
    if (ysh) {
      const float4 v = *(const float4*)(ysh + (size_t)t * H + c);
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
    *(float4*)(out + (size_t)t * H + c) = acc;
  }
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  if (a.act_bf16)
    hipLaunchKernelGGL(combine_bf16_kernel, dim3(a.T), dim3(CB_THREADS), 0, s, a);
  else
    hipLaunchKernelGGL(combine_f32_kernel, dim3(a.T), dim3(CB_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace pmpe
