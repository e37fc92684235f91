// K1 - fused policy-masked router (Sec. 3.1 mask equation; App. B.1).
//
// One workgroup of 8 waves routes a tile of 32 tokens:
//  1. Decode each token's policy word: tau = (word == PMPE_POLICY_ALLOW); a NULL word
//     array, a malformed word or a missing private router all give deny.
//  2. Logits over the permitted pool only. For the public pass, rows of allow tokens are
//     fed as zeros and their results discarded; for the private pass the same holds for
//     deny tokens, so a deny token's x is never multiplied with a private router row,
//     and a pass with no token of its policy is skipped (its router rows are not read).
//     bf16 activations: the fp32 router row w is split exactly into three bf16 parts
//     w = hi + mid + lo (each truncation keeps the next 8 significant bits, so the sum
//     is exact for normal w); every product x * part is exact in fp32 and the MFMA
//     accumulates in fp32, so the logit carries fp32 accumulation error only.
//     fp32 activations use a plain fp32 dot product.
//  3. Top-k: one wave per token sorts 64-bit keys (descending-ordered fp32 logit, expert
//     id) with a bitonic network across the wave; the first k keys win, equal logits
//     going to the lower id (-0.0 == +0.0, NaN ranks as -inf).
//  4. Gates (RENORM over the k winners, or POOL_SOFTMAX over the whole pool) in fp32,
//     written in ascending expert-id order; kgap = z_(k) - z_(k+1).
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int RT_TOK = 32;
constexpr int RT_WAVES = 8;
constexpr int RT_THREADS = 64 * RT_WAVES;

// Descending sort key of an fp32 logit: smaller key = larger logit.
__device__ __forceinline__ uint32_t desc_key(float z) {
  uint32_t u = __float_as_uint(z);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) u = 0xFF800000u;  // NaN ranks as -inf
  if (u == 0x80000000u) u = 0u;                          // -0.0 == +0.0
  const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}

// Exact split of an fp32 value into three bf16 parts (bit patterns).
__device__ __forceinline__ void split3(float w, uint32_t& h, uint32_t& m, uint32_t& l) {
  const uint32_t uh = __float_as_uint(w) & 0xFFFF0000u;
  const float r1 = w - __uint_as_float(uh);
  const uint32_t um = __float_as_uint(r1) & 0xFFFF0000u;
  const float r2 = r1 - __uint_as_float(um);
  h = uh >> 16;
  m = um >> 16;
  l = __float_as_uint(r2) >> 16;
}

// Bitonic sort (ascending) of NPL*64 keys held NPL per lane; element i = r*64 + lane.
template <int NPL>
__device__ __forceinline__ void wave_bitonic_sort(uint64_t (&v)[NPL]) {
  const int lane = lane_id();
  constexpr int N = NPL * 64;
#pragma unroll
  for (int size = 2; size <= N; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= 64) {
        const int rs = stride >> 6;
#pragma unroll
        for (int r = 0; r < NPL; ++r) {
          const int q = r ^ rs;
          if (q > r) {
            const bool asc = (((r << 6) | lane) & size) == 0;
            const uint64_t a = v[r], b = v[q];
            const bool sw = asc ? (a > b) : (a < b);
            v[r] = sw ? b : a;
            v[q] = sw ? a : b;
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < NPL; ++r) {
          const uint64_t o = shfl_xor_u64(v[r], stride);
          const bool asc = (((r << 6) | lane) & size) == 0;
          const bool lower = (lane & stride) == 0;
          const uint64_t mn = v[r] < o ? v[r] : o;
          const uint64_t mx = v[r] < o ? o : v[r];
          v[r] = (lower == asc) ? mn : mx;
        }
      }
    }
  }
}

struct TopkCtx {
  int T, n_pub, n_priv, k, gate_mode;
  int32_t* topk_idx;
  float* topk_gate;
  uint8_t* allow;
  float* kgap;
};

template <int NPL>
__device__ void topk_one_token(const TopkCtx& c, int t, int tau, const float* z) {
  const int lane = lane_id();
  const int N = tau ? c.n_priv : c.n_pub;
  const int base = tau ? c.n_pub : 0;
  const int k = c.k;
  uint64_t key[NPL];
#pragma unroll
  for (int r = 0; r < NPL; ++r) {
    const int s = r * 64 + lane;
    key[r] = (s < N) ? (((uint64_t)desc_key(z[s]) << 32) | (uint32_t)s) : ~0ull;
  }
  wave_bitonic_sort<NPL>(key);
  // element i of the sorted order lives in lane i (r = 0) for i < 64 > k
  const uint32_t uslot = (uint32_t)key[0];  // padding keys carry 0xFFFFFFFF
  const int slot = (uslot < (uint32_t)N) ? (int)uslot : N;
  const float zl = (slot < N) ? z[slot] : -INFINITY;
  const float m = __shfl(zl, 0, 64);
  float den;
  const float ex = (lane < k) ? __expf(zl - m) : 0.0f;
  if (c.gate_mode == PMPE_GATE_POOL_SOFTMAX) {
    float part = 0.0f;
#pragma unroll
    for (int r = 0; r < NPL; ++r) {
      const int s = r * 64 + lane;
      if (s < N) part += __expf(z[s] - m);
    }
    den = wave_sum(part);
  } else {
    den = wave_sum(ex);
  }
  // ascending-id output position among the k winners
  int pos = 0;
  for (int q = 0; q < k; ++q) {
    const int sq = __shfl(slot, q, 64);
    pos += (sq < slot) ? 1 : 0;
  }
  if (lane < k) {
    c.topk_idx[(size_t)t * k + pos] = base + slot;
    c.topk_gate[(size_t)t * k + pos] = ex / den;
  }
  const float zk = __shfl(zl, k - 1, 64);
  const float zk1 = __shfl(zl, k < 64 ? k : 63, 64);
  if (lane == 0) {
    c.allow[t] = (uint8_t)tau;
    if (c.kgap) {
      float g = (N == k) ? INFINITY : (zk - zk1);
      if (g != g) g = 0.0f;  // both -inf (NaN-ranked): a tie
      c.kgap[t] = g;
    }
  }
}

template <bool ACT_BF16>
__global__ __launch_bounds__(RT_THREADS) void route_kernel(RouteArgs a) {
  __shared__ int s_tau[RT_TOK];
  __shared__ int s_need[2];
  __shared__ float s_z[RT_TOK][PMPE_MAX_POOL];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int t0 = blockIdx.x * RT_TOK;

  if (tid < 2) s_need[tid] = 0;
  __syncthreads();
  if (tid < RT_TOK) {
    const int t = t0 + tid;
    int tau = -1;
    if (t < a.T) {
      tau = (a.words != nullptr && a.words[t] == PMPE_POLICY_ALLOW) ? 1 : 0;
      if (tau == 1 && a.wr_priv == nullptr) {
        tau = 0;  // fail closed: no private router, the row is routed as deny
        if (a.dev_status) atomicOr(a.dev_status, PMPE_DEV_PRIV_ROUTER_MISSING);
      }
      s_need[tau] = 1;
    }
    s_tau[tid] = tau;
  }
  __syncthreads();

  for (int pass = 0; pass < 2; ++pass) {
    if (!s_need[pass]) continue;  // uniform: no token of this policy in the tile
    const float* wr = pass ? a.wr_priv : a.wr_pub;
    const int N = pass ? a.n_priv : a.n_pub;
    const int bias_base = pass ? a.n_pub : 0;
    const int H = a.H;
    if constexpr (ACT_BF16) {
      const uint16_t* x = (const uint16_t*)a.x;
      const int nblk = (N + 15) >> 4;
      for (int j = wave; j < nblk; j += RT_WAVES) {
        const int n = (j << 4) + (lane & 15);
        const bool nv = n < N;
        const int koff = (lane >> 4) * 8;
        const float* wrow = wr + (size_t)(nv ? n : 0) * H + koff;
        bool av[2];
        const uint16_t* xrow[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
          const int tt = mb * 16 + (lane & 15);
          av[mb] = s_tau[tt] == pass;
          xrow[mb] = x + (size_t)(av[mb] ? t0 + tt : 0) * H + koff;
        }
        f32x4 acc[2] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
#pragma unroll 4
        for (int kk = 0; kk < H; kk += 32) {
          float4 w0 = make_float4(0, 0, 0, 0), w1 = w0;
          if (nv) {
            w0 = *(const float4*)(wrow + kk);
            w1 = *(const float4*)(wrow + kk + 4);
          }
          u32x4 xa[2];
#pragma unroll
          for (int mb = 0; mb < 2; ++mb) {
            xa[mb] = av[mb] ? *(const u32x4*)(xrow[mb] + kk) : u32x4{0, 0, 0, 0};
          }
          const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
          uint32_t ph[8], pm[8], pl[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) split3(wv[i], ph[i], pm[i], pl[i]);
          const bf16x8 bh = as_bf16x8(u32x4{ph[0] | (ph[1] << 16), ph[2] | (ph[3] << 16),
                                            ph[4] | (ph[5] << 16), ph[6] | (ph[7] << 16)});
          const bf16x8 bm = as_bf16x8(u32x4{pm[0] | (pm[1] << 16), pm[2] | (pm[3] << 16),
                                            pm[4] | (pm[5] << 16), pm[6] | (pm[7] << 16)});
          const bf16x8 bl = as_bf16x8(u32x4{pl[0] | (pl[1] << 16), pl[2] | (pl[3] << 16),
                                            pl[4] | (pl[5] << 16), pl[6] | (pl[7] << 16)});
#pragma unroll
          for (int mb = 0; mb < 2; ++mb) {
            const bf16x8 av8 = as_bf16x8(xa[mb]);
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bh, acc[mb], 0, 0, 0);
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bm, acc[mb], 0, 0, 0);
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bl, acc[mb], 0, 0, 0);
          }
        }
        const float b = (nv && a.bias) ? a.bias[bias_base + n] : 0.0f;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int tt = mb * 16 + (lane >> 4) * 4 + i;
            if (nv && s_tau[tt] == pass) s_z[tt][n] = a.bias ? acc[mb][i] + b : acc[mb][i];
          }
        }
      }
    } else {
      const float* x = (const float*)a.x;
      for (int p = tid; p < RT_TOK * N; p += RT_THREADS) {
        const int tt = p / N, n = p - tt * N;
        if (s_tau[tt] != pass) continue;
        const float* xr = x + (size_t)(t0 + tt) * H;
        const float* wrow = wr + (size_t)n * H;
        float acc = 0.0f;
        for (int h0 = 0; h0 < H; h0 += 64) {  // blocked: partial sums of 64 terms
          float part = 0.0f;
          for (int h = h0; h < h0 + 64; ++h) part = fmaf(xr[h], wrow[h], part);
          acc += part;
        }
        s_z[tt][n] = a.bias ? acc + a.bias[bias_base + n] : acc;
      }
    }
  }
  __syncthreads();

  TopkCtx c{a.T, a.n_pub, a.n_priv, a.k, a.gate_mode, a.topk_idx, a.topk_gate, a.allow, a.kgap};
  for (int tt = wave; tt < RT_TOK; tt += RT_WAVES) {
    const int tau = s_tau[tt];
    if (tau < 0) continue;
    const int N = tau ? a.n_priv : a.n_pub;
    if (N <= 64)
      topk_one_token<1>(c, t0 + tt, tau, s_z[tt]);
    else if (N <= 128)
      topk_one_token<2>(c, t0 + tt, tau, s_z[tt]);
    else
      topk_one_token<4>(c, t0 + tt, tau, s_z[tt]);
  }
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  const dim3 grid((a.T + RT_TOK - 1) / RT_TOK), block(RT_THREADS);
  if (a.act_bf16)
    hipLaunchKernelGGL(route_kernel<true>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(route_kernel<false>, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace pmpe
