// Request-gated LoRA control arm (Sec. 4.2 matched expert-LoRA baseline; Sec. 5.2 and
// App. F.2: the paper's request gate on such an adapter still let it execute for some
// denied requests). Rank-r adapters on every public expert's gate, up and down
// projections are added to the frozen expert, scaled by s and by the row's decision:
//   g = Wg x + tau s Bg (Ag x),  u = Wu x + tau s Bu (Au x),  h = silu(g) u,
//   y = Wd h + tau s Bd (Ad h).
// Where the decision is applied is the gate granularity, and the adapter kernels count
// every row they physically execute (per token, like the private-row audit):
//   ROW      a denied row is skipped before any adapter work;
//   TILE     a tile of 64 consecutive rows of one expert runs its adapters when any of its
//            rows allows; its denied rows are executed and their result discarded;
//   POSTHOC  every row runs the adapters; the decision only selects the result.
// The outputs are the same bits under every granularity; only the counters differ.
//
// The frozen expert runs as in pmpe_expert_ffn (GEMM1 keeping the fp32 gate and up
// projections, GEMM2 on h); lora_pre_kernel rewrites h of the rows whose adapters are
// applied, lora_post_kernel adds the down-projection adapter to their outputs. One block
// per permuted row; the adapter products run in fp32 on the vector ALUs (rank <= 128).
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int LT = 256;

// expert of permuted row r: last e with offset[e] <= r (offsets are non-decreasing)
__device__ __forceinline__ int expert_of(const int32_t* offset, int E, int r) {
  int lo = 0, hi = E - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (offset[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ bool allows(const uint32_t* words, int t) {
  return words != nullptr && words[t] == PMPE_POLICY_ALLOW;
}

// Does row r run its adapters under the gate granularity? (block-uniform)
__device__ bool runs(const LoraArgs& a, int e, int r, bool tau) {
  if (a.gate == PMPE_LORA_GATE_POSTHOC) return true;
  if (a.gate == PMPE_LORA_GATE_ROW) return tau;
  __shared__ int s_any;
  if (threadIdx.x == 0) s_any = 0;
  __syncthreads();
  const int t0 = a.offset[e] + ((r - a.offset[e]) / PMPE_LORA_TILE_ROWS) * PMPE_LORA_TILE_ROWS;
  const int t1 = min(t0 + PMPE_LORA_TILE_ROWS, a.offset[e] + a.count[e]);
  const int rr = t0 + (int)threadIdx.x;
  if (rr < t1 && allows(a.words, a.row_token[rr])) s_any = 1;
  __syncthreads();
  return s_any != 0;
}

// dot of a bf16 row (n values, 16-byte aligned) with an fp32 LDS vector, by one wave
__device__ __forceinline__ float wave_dot_bf16(const uint16_t* row, const float* v, int n) {
  const int lane = threadIdx.x & 63;
  float s = 0.f;
  for (int i = lane * 8; i < n; i += 64 * 8) {
    const u32x4 q = *(const u32x4*)(row + i);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      s += bf16_to_f32(q[j] & 0xFFFFu) * v[i + 2 * j] + bf16_to_f32(q[j] >> 16) * v[i + 2 * j + 1];
  }
  return wave_sum(s);
}

__global__ __launch_bounds__(LT) void lora_pre_kernel(LoraArgs a) {
  extern __shared__ float s_dyn[];
  float* s_x = s_dyn;            // [H]
  float* s_u = s_dyn + a.H;      // [2 r]
  const int r = blockIdx.x, E = a.n_pub + a.n_priv;
  const int e = expert_of(a.offset, E, r);
  if (e >= a.n_pub) return;  // the adapters sit on public experts only
  const int t = a.row_token[r];
  const bool tau = allows(a.words, t);
  if (!runs(a, e, r, tau)) return;
  if (threadIdx.x == 0) atomicAdd(&a.lora_rows[t], 1u);
  const int H = a.H, I = a.I, R = a.rank;
  const uint16_t* xr = a.x_perm ? (const uint16_t*)a.x_perm + (size_t)r * H
                                : (const uint16_t*)a.x + (size_t)t * H;
  for (int i = threadIdx.x; i < H; i += LT) s_x[i] = bf16_to_f32(xr[i]);
  __syncthreads();
  const uint16_t* A = a.a13 + (size_t)e * 2 * R * H;
  const int wave = threadIdx.x >> 6;
  for (int j = wave; j < 2 * R; j += LT / 64) {
    const float d = wave_dot_bf16(A + (size_t)j * H, s_x, H);
    if ((threadIdx.x & 63) == 0) s_u[j] = d;
  }
  __syncthreads();
  const uint16_t* B1 = a.b1 + (size_t)e * I * R;
  const uint16_t* B3 = a.b3 + (size_t)e * I * R;
  const float* ab = a.ab + (size_t)r * 2 * I;
  uint16_t* h = a.h + (size_t)r * I;
  for (int i = threadIdx.x; i < I; i += LT) {
    float dg = 0.f, du = 0.f;
    for (int j = 0; j < R; ++j) {
      dg += bf16_to_f32(B1[(size_t)i * R + j]) * s_u[j];
      du += bf16_to_f32(B3[(size_t)i * R + j]) * s_u[R + j];
    }
    const float g = tau ? ab[i] + a.scale * dg : ab[i];
    const float u = tau ? ab[I + i] + a.scale * du : ab[I + i];
    h[i] = (uint16_t)f32_to_bf16_rne(silu(g) * u);
  }
}

__global__ __launch_bounds__(LT) void lora_post_kernel(LoraArgs a) {
  extern __shared__ float s_dyn[];
  float* s_h = s_dyn;            // [I]
  float* s_v = s_dyn + a.I;      // [r]
  const int r = blockIdx.x, E = a.n_pub + a.n_priv;
  const int e = expert_of(a.offset, E, r);
  if (e >= a.n_pub) return;
  const int t = a.row_token[r];
  const bool tau = allows(a.words, t);
  if (!runs(a, e, r, tau)) return;
  if (threadIdx.x == 0) atomicAdd(&a.lora_rows[t], 1u);
  const int H = a.H, I = a.I, R = a.rank;
  const uint16_t* hr = a.h + (size_t)r * I;
  for (int i = threadIdx.x; i < I; i += LT) s_h[i] = bf16_to_f32(hr[i]);
  __syncthreads();
  const uint16_t* A2 = a.a2 + (size_t)e * R * I;
  const int wave = threadIdx.x >> 6;
  for (int j = wave; j < R; j += LT / 64) {
    const float d = wave_dot_bf16(A2 + (size_t)j * I, s_h, I);
    if ((threadIdx.x & 63) == 0) s_v[j] = d;
  }
  __syncthreads();
  const uint16_t* B2 = a.b2 + (size_t)e * H * R;
  uint16_t* y = a.y_perm + (size_t)r * H;
  for (int i = threadIdx.x; i < H; i += LT) {
    float dy = 0.f;
    for (int j = 0; j < R; ++j) dy += bf16_to_f32(B2[(size_t)i * R + j]) * s_v[j];
    if (tau) y[i] = (uint16_t)f32_to_bf16_rne(bf16_to_f32(y[i]) + a.scale * dy);
  }
}

}  // namespace

hipError_t launch_lora_pre(const LoraArgs& a, hipStream_t s) {
  const size_t lds = ((size_t)a.H + 2 * a.rank) * sizeof(float);
  lora_pre_kernel<<<a.T * a.k, LT, lds, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_lora_post(const LoraArgs& a, hipStream_t s) {
  const size_t lds = ((size_t)a.I + a.rank) * sizeof(float);
  lora_post_kernel<<<a.T * a.k, LT, lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace pmpe
