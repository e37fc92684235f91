// Optimizer step over the private parameters (G2 of Sec. 2.2: only private parameters
// are passed to the optimizer, frozen public ones never; Sec. 3.2 and App. C.1: AdamW).
//
// AdamW with decoupled weight decay, one element per lane-iteration in fp32:
//   p <- p (1 - lr wd);  m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
//   p <- p - lr (m / c1) / (sqrt(v / c2) + eps),  c1 = 1 - b1^t, c2 = 1 - b2^t.
// A bf16 parameter keeps an fp32 master copy that takes the update and is rounded once
// (to nearest even) into the bf16 weight. HBM-bound: 28-30 bytes per element.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

template <bool BF16>
__global__ __launch_bounds__(256) void adamw_kernel(AdamwArgs a) {
  const uint64_t stride = (uint64_t)gridDim.x * 256 * 4;
  for (uint64_t i0 = ((uint64_t)blockIdx.x * 256 + threadIdx.x) * 4; i0 < a.n; i0 += stride) {
    const int cnt = (int)min((uint64_t)4, a.n - i0);
    float p[4], g[4], m[4], v[4];
    float* master = BF16 ? a.master : (float*)a.param;
    if (cnt == 4) {
      const f32x4 pv = *(const f32x4*)(master + i0), gv = *(const f32x4*)(a.grad + i0);
      const f32x4 mv = *(const f32x4*)(a.m + i0), vv = *(const f32x4*)(a.v + i0);
#pragma unroll
      for (int j = 0; j < 4; ++j) { p[j] = pv[j]; g[j] = gv[j]; m[j] = mv[j]; v[j] = vv[j]; }
    } else {
      for (int j = 0; j < 4; ++j) {
        const bool in = j < cnt;
        p[j] = in ? master[i0 + j] : 0.f;
        g[j] = in ? a.grad[i0 + j] : 0.f;
        m[j] = in ? a.m[i0 + j] : 0.f;
        v[j] = in ? a.v[i0 + j] : 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      p[j] *= a.decay;
      m[j] = a.beta1 * m[j] + (1.0f - a.beta1) * g[j];
      v[j] = a.beta2 * v[j] + (1.0f - a.beta2) * g[j] * g[j];
      p[j] -= a.lr * (m[j] / a.c1) / (sqrtf(v[j] / a.c2) + a.eps);
    }
    if (cnt == 4) {
      *(f32x4*)(master + i0) = f32x4{p[0], p[1], p[2], p[3]};
      *(f32x4*)(a.m + i0) = f32x4{m[0], m[1], m[2], m[3]};
      *(f32x4*)(a.v + i0) = f32x4{v[0], v[1], v[2], v[3]};
      if (BF16) {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        *(u32x2*)((uint16_t*)a.param + i0) = u32x2{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])};
      }
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
  const uint64_t blocks = (a.n + 1023) / 1024;
  const unsigned grid = (unsigned)(blocks < 65536 ? blocks : 65536);
  if (a.master)
    adamw_kernel<true><<<grid, 256, 0, s>>>(a);
  else
    adamw_kernel<false><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace pmpe
