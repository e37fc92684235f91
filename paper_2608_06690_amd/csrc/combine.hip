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

// KC > 0: top-k fixed at compile time, so the k row loads of a token are issued
// together (rows and gates first, then every slot's 16-byte vector) before the sum;
// KC == 0: any k, one slot at a time. Both add the slots in the same order.
template <int KC>
__global__ __launch_bounds__(CB_THREADS) void combine_bf16_kernel(CombineArgs a) {
  const int t = blockIdx.x;
  const int H = a.H;
  const uint16_t* yp = (const uint16_t*)a.y_perm;
  const uint16_t* ysh = (const uint16_t*)a.y_shared;
  uint16_t* out = (uint16_t*)a.out;
  int rows[KC > 0 ? KC : 1];
  float gs[KC > 0 ? KC : 1];
  if constexpr (KC > 0) {
#pragma unroll
    for (int j = 0; j < KC; ++j) {
      rows[j] = a.token_row[(size_t)t * KC + j];
      gs[j] = a.gate[(size_t)t * KC + j];
    }
  }
  for (int c = threadIdx.x * 8; c < H; c += CB_THREADS * 8) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if constexpr (KC > 0) {
      u32x4 v[KC];
#pragma unroll
      for (int j = 0; j < KC; ++j)  // a slot without a row (-1) loads row 0 and is skipped
        v[j] = *(const u32x4*)(yp + (size_t)(rows[j] < 0 ? 0 : rows[j]) * H + c);
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        if (rows[j] < 0) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[2 * q] += gs[j] * bf16_to_f32(v[j][q] & 0xFFFFu);
          acc[2 * q + 1] += gs[j] * bf16_to_f32(v[j][q] >> 16);
        }
      }
    } else {
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
  if (a.act_bf16) {
    switch (a.k) {
      case 2: hipLaunchKernelGGL(combine_bf16_kernel<2>, dim3(a.T), dim3(CB_THREADS), 0, s, a); break;
      case 6: hipLaunchKernelGGL(combine_bf16_kernel<6>, dim3(a.T), dim3(CB_THREADS), 0, s, a); break;
      case 8: hipLaunchKernelGGL(combine_bf16_kernel<8>, dim3(a.T), dim3(CB_THREADS), 0, s, a); break;
      default: hipLaunchKernelGGL(combine_bf16_kernel<0>, dim3(a.T), dim3(CB_THREADS), 0, s, a); break;
    }
  } else
    hipLaunchKernelGGL(combine_f32_kernel, dim3(a.T), dim3(CB_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace pmpe
