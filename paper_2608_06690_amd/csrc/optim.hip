// Optimizer step over the private parameters (G2 of Sec. 2.2: only private parameters
// are passed to the optimizer, frozen public ones never; Sec. 3.2 and App. C.1: AdamW).
//
// AdamW with decoupled weight decay, elementwise in fp32:
//   p <- p (1 - lr wd);  m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
//   p <- p - lr (m / c1) / (sqrt(v / c2) + eps),  c1 = 1 - b1^t, c2 = 1 - b2^t.
// A bf16 parameter keeps an fp32 master copy that takes the update and is rounded once
// (to nearest even) into the bf16 weight. HBM-bound: 28-30 bytes per element.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

template <bool BF16>
__global__ __launch_bounds__(256) void adamw_kernel(AdamwArgs a) {
  // 8 consecutive elements per thread and iteration: two 16-byte vectors of each of the
  // four input streams in flight per thread (non-temporal loads and stores measured slower)
  const uint64_t stride = (uint64_t)gridDim.x * 256 * 8;
  float* master = BF16 ? a.master : (float*)a.param;
  for (uint64_t i0 = ((uint64_t)blockIdx.x * 256 + threadIdx.x) * 8; i0 < a.n; i0 += stride) {
    const int cnt = (int)min((uint64_t)8, a.n - i0);
    float p[8], g[8], m[8], v[8];
    if (cnt == 8) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4 pv = *((const f32x4*)(master + i0) + h);
        const f32x4 gv = *((const f32x4*)(a.grad + i0) + h);
        const f32x4 mv = *((const f32x4*)(a.m + i0) + h);
        const f32x4 vv = *((const f32x4*)(a.v + i0) + h);
#pragma unroll
        for (int j = 0; j < 4; ++j) { p[4 * h + j] = pv[j]; g[4 * h + j] = gv[j]; m[4 * h + j] = mv[j]; v[4 * h + j] = vv[j]; }
      }
    } else {
      for (int j = 0; j < 8; ++j) {
        const bool in = j < cnt;
        p[j] = in ? master[i0 + j] : 0.f;
        g[j] = in ? a.grad[i0 + j] : 0.f;
        m[j] = in ? a.m[i0 + j] : 0.f;
        v[j] = in ? a.v[i0 + j] : 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      p[j] *= a.decay;
      m[j] = a.beta1 * m[j] + (1.0f - a.beta1) * g[j];
      v[j] = a.beta2 * v[j] + (1.0f - a.beta2) * g[j] * g[j];
      p[j] -= a.lr * (m[j] / a.c1) / (sqrtf(v[j] / a.c2) + a.eps);
    }
    if (cnt == 8) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        *((f32x4*)(master + i0) + h) = f32x4{p[4 * h], p[4 * h + 1], p[4 * h + 2], p[4 * h + 3]};
        *((f32x4*)(a.m + i0) + h) = f32x4{m[4 * h], m[4 * h + 1], m[4 * h + 2], m[4 * h + 3]};
        *((f32x4*)(a.v + i0) + h) = f32x4{v[4 * h], v[4 * h + 1], v[4 * h + 2], v[4 * h + 3]};
      }
      if (BF16)
        *(u32x4*)((uint16_t*)a.param + i0) = u32x4{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                                                   pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
    } else {
      for (int j = 0; j < cnt; ++j) {
        master[i0 + j] = p[j];
        a.m[i0 + j] = m[j];
        a.v[i0 + j] = v[j];
        if (BF16) ((uint16_t*)a.param)[i0 + j] = (uint16_t)f32_to_bf16_rne(p[j]);
      }
    }
  }
}

}  // namespace

hipError_t launch_adamw(const AdamwArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  const uint64_t blocks = (a.n + 2047) / 2048;
  const unsigned grid = (unsigned)(blocks < 65536 ? blocks : 65536);
  if (a.master)
    adamw_kernel<true><<<grid, 256, 0, s>>>(a);
  else
    adamw_kernel<false><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace pmpe
