// K1 - fused policy-masked router (Sec. 3.1 mask equation; App. B.1).
//
// A logits kernel over (token tile, 16-expert group of one pool) blocks, then a top-k
// kernel with one wave per token:
//  1. Decode each token's policy word: tau = (word == PMPE_POLICY_ALLOW); a NULL word
//     array, a malformed word or a missing private router all give deny.
//  2. Logits over the permitted pool only. A block feeds only the tokens whose policy
//     selects its pool: other rows load a token of this pool's policy and their results
//     are discarded, so a deny token's x is never multiplied with a private router row,
//     and a block with no token of its policy returns before reading its router rows.
//     Up to 2048 tokens the operands are loaded straight into registers (16-token tiles,
//     H split across the four waves); larger batches stage them in LDS (64 tokens x 64
//     experts, H split across up to four blocks whose partial logits the top-k adds).
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
#include "lds_dma.h"
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int RT_WAVES = 4;
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

// The value of lane (lane ^ stride) for the strides of a wave bitonic network, without the
// LDS crossbar where a lane-permuting move does it: DPP quad permutations for strides 1 and 2,
// a rotation by 8 within each row of 16 lanes for stride 8 (a rotation by 8 of 16 lanes is
// the xor), ds_swizzle (xor mask within 32 lanes) for 4 and 16, a full shuffle for 32.
__device__ __forceinline__ uint32_t xor_lanes(uint32_t x, int stride) {
  const int v = (int)x;
  if (stride == 1) return (uint32_t)__builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);  // [1,0,3,2]
  if (stride == 2) return (uint32_t)__builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);  // [2,3,0,1]
  if (stride == 8) return (uint32_t)__builtin_amdgcn_mov_dpp(v, 0x128, 0xF, 0xF, false);  // row_ror:8
  if (stride == 4) return (uint32_t)__builtin_amdgcn_ds_swizzle(v, (4 << 10) | 0x1F);
  if (stride == 16) return (uint32_t)__builtin_amdgcn_ds_swizzle(v, (16 << 10) | 0x1F);
  return (uint32_t)__shfl_xor(v, stride, 64);
}
__device__ __forceinline__ uint64_t xor_lanes_u64(uint64_t v, int stride) {
  const uint32_t lo = xor_lanes((uint32_t)v, stride), hi = xor_lanes((uint32_t)(v >> 32), stride);
  return ((uint64_t)hi << 32) | lo;
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
          const uint64_t o = xor_lanes_u64(v[r], stride);
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

// tau of token t: only the exact allow word allows; with no private router the token
// fails closed to deny (and the status bit is raised).
__device__ __forceinline__ int token_tau(const RouteArgs& a, int t) {
  int tau = (a.words != nullptr && a.words[t] == PMPE_POLICY_ALLOW) ? 1 : 0;
  if (tau == 1 && a.wr_priv == nullptr) {
    tau = 0;
    if (a.dev_status) atomicOr(a.dev_status, PMPE_DEV_PRIV_ROUTER_MISSING);
  }
  return tau;
}

struct TopkCtx {
  int T, n_pub, n_priv, k, gate_mode;
  int32_t* topk_idx;
  float* topk_gate;
  uint8_t* allow;
  float* kgap;
};

// Top-k of token t over its pool: N logits z[0..N) of expert ids base + s.
template <int NPL>
__device__ void topk_one_token(const TopkCtx& c, int t, int tau, int N, int base, const float* z) {
  const int lane = lane_id();
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

// Token-tile x expert-group logits. Block (tile, g): TT tokens against 16 experts of
// one pool; the four waves split H in quarters (each wave starts its quarter at a
// block-dependent step so that concurrent blocks read different router columns) and
// their partial sums are added in fixed wave order, then the bias. Only tokens whose
// policy selects this pool are fed and written.
template <int TT>
__global__ __launch_bounds__(RT_THREADS) void route_logits_bf16_kernel(RouteArgs a, int ntiles, int ngroups) {
  constexpr int NMB = TT / 16;
  __shared__ int s_tau[TT];
  __shared__ int s_first;
  __shared__ float s_part[RT_WAVES][TT][16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // 1-D grid, (token tile, expert group) with the group fastest; XCD blockIdx % 8
  // takes a contiguous range of that order, so a token tile is fetched into one L2.
  const int total = ntiles * ngroups;
  const int b = blockIdx.x, xcd = b & 7, j = b >> 3;
  const int cnt_x = (total >> 3) + (xcd < (total & 7) ? 1 : 0);
  if (j >= cnt_x) return;  // past this XCD's range
  const int L = xcd * (total >> 3) + min(xcd, total & 7) + j;
  const int tile = L / ngroups, grp = L - tile * ngroups;
  const int t0 = tile * TT;
  const int gpub = (a.n_pub + 15) >> 4;
  const int pass = grp < gpub ? 0 : 1;
  const int n0 = (pass ? grp - gpub : grp) * 16;
  const int N = pass ? a.n_priv : a.n_pub;
  if (tid == 0) s_first = TT;
  __syncthreads();
  int mine = 0;
  if (tid < TT) {
    const int tau = (t0 + tid < a.T) ? token_tau(a, t0 + tid) : -1;
    s_tau[tid] = tau;
    mine = (a.soft ? tau >= 0 : tau == pass) ? 1 : 0;
    if (mine) atomicMin(&s_first, tid);
  }
  // no token of this pool's policy in the tile: its router rows are never read
  if (!__syncthreads_or(mine)) return;
  const float* wr = pass ? a.wr_priv : a.wr_pub;
  const int H = a.H;
  const uint16_t* x = (const uint16_t*)a.x;
  // Operand rows of this lane. A lane whose expert is past the pool, or whose token
  // has the other policy, reads a row that belongs to this pass (expert n0, the
  // tile's first token of this policy) and its results are discarded: a token's x
  // is only ever loaded for the pool its policy permits (in the soft control arm every
  // token takes part in both pools).
  const int n = n0 + (lane & 15);
  const int koff = (lane >> 4) * 8;
  const float* wrow = wr + (size_t)(n < N ? n : n0) * H + koff;
  const int first = s_first;
  const uint16_t* xrow[NMB];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) {
    const int tt = mb * 16 + (lane & 15);
    const bool part = a.soft ? s_tau[tt] >= 0 : s_tau[tt] == pass;
    xrow[mb] = x + (size_t)(t0 + (part ? tt : first)) * H + koff;
  }
  const int nsteps = H / (32 * RT_WAVES);  // K steps of this wave's quarter
  const int kbase = wave * nsteps;
  const int rot = (tile * 5 + grp * 3) % nsteps;
  f32x4 acc[NMB];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) acc[mb] = f32x4{0, 0, 0, 0};
  // A ring of D K steps of loads (D-1 in flight while one is multiplied). Loads are
  // unconditional (a step past the end reloads the last one and is not used), so the
  // loop is straight-line and the compiler's wait counts keep the ring full; each
  // refill stays right after the step that freed its slot.
  constexpr int D = 2;
  float4 w[D][2];
  u32x4 xa[D][NMB];
  auto load = [&](int d, int st) {
    st = min(st, nsteps - 1);
    const int kk = (kbase + (st + rot) % nsteps) * 32;
    w[d][0] = *(const float4*)(wrow + kk);
    w[d][1] = *(const float4*)(wrow + kk + 4);
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) xa[d][mb] = *(const u32x4*)(xrow[mb] + kk);
  };
  auto step = [&](int d) {
    const float wv[8] = {w[d][0].x, w[d][0].y, w[d][0].z, w[d][0].w,
                         w[d][1].x, w[d][1].y, w[d][1].z, w[d][1].w};
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
    for (int mb = 0; mb < NMB; ++mb) {
      const bf16x8 av8 = as_bf16x8(xa[d][mb]);
      acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bh, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bm, acc[mb], 0, 0, 0);
      acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bl, acc[mb], 0, 0, 0);
    }
  };
#pragma unroll
  for (int d = 0; d < D; ++d) load(d, d);
  const int nfull = nsteps - nsteps % D;
  for (int s0 = 0; s0 < nfull; s0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      step(d);
      load(d, s0 + d + D);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int d = 0; d < D; ++d)
    if (nfull + d < nsteps) step(d);
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) s_part[wave][mb * 16 + (lane >> 4) * 4 + i][lane & 15] = acc[mb][i];
  __syncthreads();
  for (int o = tid; o < TT * 16; o += RT_THREADS) {
    const int tt = o >> 4, c = o & 15;
    const int nn = n0 + c;
    if ((a.soft ? s_tau[tt] < 0 : s_tau[tt] != pass) || nn >= N) continue;
    float z = s_part[0][tt][c];
#pragma unroll
    for (int w2 = 1; w2 < RT_WAVES; ++w2) z += s_part[w2][tt][c];
    if (a.bias) z += a.bias[(pass ? a.n_pub : 0) + nn];
    a.z[(size_t)(t0 + tt) * a.zstride + (a.soft && pass ? a.n_pub : 0) + nn] = z;
  }
}

// Wait for the copies of the oldest step in flight: `younger` steps were issued after it
// (NDMA copies each, loads complete in order), at most Y of which may stay in flight.
template <int Y, int NDMA>
__device__ __forceinline__ void wait_steps(int younger) {
  if constexpr (Y == 0)
    wait_vmcnt<0>();
  else if (younger >= Y)
    wait_vmcnt<Y * NDMA>();
  else
    wait_steps<Y - 1, NDMA>(younger);
}

// Large batches, wide tile: 64 tokens x 64 experts of one pool per block. Wave w owns
// experts n0 + 16 w .. n0 + 16 w + 15 against all 64 tokens (four 16-token row blocks), so
// each fp32 router value is split into its three bf16 parts by one wave only (a tile of
// 16 experts whose four waves split H by tokens would split every router value four times)
// and a tile's x rows are copied once per 64 experts. K steps of BK: the step's x rows
// (64 x 2BK bytes) and router rows (64 x 4BK bytes) go through a ring of D stages of
// global->LDS copies, each wave copying the x rows and the router rows of its own 16-row
// blocks. The K range is split `ksplit` ways: split s writes its partial logits to
// z + s * T * zstride (split 0 adds the logit bias) and the top-k kernel adds the partials
// in split order, so the logits are bitwise reproducible. Token selection, the exact
// three-part split and the pool rule are those of the register kernel above; rows past the pool
// copy expert n0 and are discarded.
constexpr int RW_TT = 64, RW_NE = 64, RW_THREADS = 256;
template <int BK_, int D_>
struct RwCfg {
  static constexpr int BK = BK_, D = D_;
  static constexpr int XR = 2 * BK, WR = 4 * BK;          // bytes per x row, per router row
  static constexpr int XB = RW_TT * XR, WB = RW_NE * WR;  // bytes per stage
  static constexpr int STAGE = XB + WB;
  static constexpr int XC = 16 * XR / 1024, WC = 16 * WR / 1024;  // copies per wave per step
  static constexpr int XRPC = 1024 / XR, WRPC = 1024 / WR;        // rows per copy
  static constexpr int NDMA = XC + WC;
  static constexpr int SUB = BK / 32;                     // MFMA K sub-steps per step
  static_assert(BK == 32 || BK == 64, "wide router K step");
  static_assert(RW_TT == 16 * (RW_THREADS / 64) && RW_NE == 16 * (RW_THREADS / 64), "wide router tile");
};
using RwLarge = RwCfg<64, 3>;

// Physical 16-byte chunk of logical chunk c in row r, for rows of CPR chunks: XOR-swizzled
// by row so that the fragment reads of 16 consecutive rows at one logical chunk cover the 64
// LDS banks once (rows of 64 bytes: four rows per bank line; 128 bytes: two; 256: one).
template <int CPR>
__device__ __forceinline__ int rw_swz(int r, int c) {
  if constexpr (CPR == 4) return c ^ ((r >> 2) & 3);
  else if constexpr (CPR == 8) return c ^ ((r >> 1) & 7);
  else return c ^ (r & 15);
}

template <class R>
__global__ __launch_bounds__(RW_THREADS) void route_logits_wide_kernel(RouteArgs a, int ntiles, int ngroups,
                                                                      int ksplit) {
  constexpr int BK = R::BK, D = R::D, CX = R::XR / 16, CW = R::WR / 16;
  __shared__ __attribute__((aligned(16))) unsigned char smem[D * R::STAGE];
  __shared__ int s_tau[RW_TT];
  __shared__ int s_first;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // XCD x = b % 8 takes tiles x, x + 8, ...; on an XCD, block j is (local tile, group,
  // split) with the split fastest, so the blocks of one tile share its x rows in one L2
  const int b = blockIdx.x, xcd = b & 7, j = b >> 3;
  const int per_tile = ngroups * ksplit;
  const int lt = j / per_tile, rem = j - lt * per_tile;
  const int grp = rem / ksplit, split = rem - grp * ksplit;
  const int tile = lt * 8 + xcd;
  if (tile >= ntiles) return;
  const int t0 = tile * RW_TT;
  const int gpub = (a.n_pub + RW_NE - 1) / RW_NE;
  const int pass = grp < gpub ? 0 : 1;
  const int n0 = (pass ? grp - gpub : grp) * RW_NE;
  const int N = pass ? a.n_priv : a.n_pub;
  if (tid == 0) s_first = RW_TT;
  __syncthreads();
  int mine = 0;
  if (tid < RW_TT) {
    const int tau = (t0 + tid < a.T) ? token_tau(a, t0 + tid) : -1;
    s_tau[tid] = tau;
    mine = (a.soft ? tau >= 0 : tau == pass) ? 1 : 0;
    if (mine) atomicMin(&s_first, tid);
  }
  // no token of this pool's policy in the tile: its router rows are never read
  if (!__syncthreads_or(mine)) return;
  const int H = a.H;
  const int first = s_first;
  auto part = [&](int r) { return a.soft ? s_tau[r] >= 0 : s_tau[r] == pass; };
  // Copy sources as byte offsets from the step's base. x copy jj of wave w fills LDS rows
  // 16w + XRPC jj + l / CX, lane l's physical chunk l % CX holding logical chunk
  // rw_swz(row, l % CX); a row whose token has the other policy (or lies past T) copies the
  // tile's first token of this policy. Router copy jj of wave w fills rows
  // 16w + WRPC jj + l / CW in the same way.
  uint32_t offx[R::XC], offw[R::WC];
#pragma unroll
  for (int jj = 0; jj < R::XC; ++jj) {
    const int r = 16 * wave + R::XRPC * jj + lane / CX;
    const int c = rw_swz<CX>(r, lane % CX);
    const int tok = part(r) ? r : first;
    offx[jj] = ((uint32_t)tok * (uint32_t)H + c * 8) * 2;
  }
#pragma unroll
  for (int jj = 0; jj < R::WC; ++jj) {
    const int r = 16 * wave + R::WRPC * jj + lane / CW;
    const int c = rw_swz<CW>(r, lane % CW);
    const int n = n0 + r;
    offw[jj] = ((uint32_t)(n < N ? n : n0) * (uint32_t)H + c * 4) * 4;
  }
  const uint16_t* x = (const uint16_t*)a.x + (size_t)t0 * H;
  const float* wr = pass ? a.wr_priv : a.wr_pub;
  const int ns = H / BK / ksplit;  // K steps of this split
  const int k0 = split * ns;
  const int rot = (tile * 5 + grp * 3 + split) % ns;
  const uint32_t lds0 = lds_addr(smem);
  auto issue = [&](int st) {
    const int kk = (k0 + (st + rot) % ns) * BK;
    const uint32_t sx = __builtin_amdgcn_readfirstlane(lds0 + (st % D) * R::STAGE);
    const uint32_t wx = sx + wave * R::XC * 1024, ww = sx + R::XB + wave * R::WC * 1024;
    Unroll<0, R::XC>::run([&](auto jj) { dma16s<jj.value * 1024, false>(offx[jj.value], x + kk, wx); });
    Unroll<0, R::WC>::run([&](auto jj) { dma16s<jj.value * 1024, false>(offw[jj.value], wr + kk, ww); });
  };
  // Fragment addresses within a stage. A (row block mb, sub-step sub): row 16mb + (l&15),
  // 8 bf16 at logical chunk 4 sub + l/16. Router: row 16w + (l&15), the same 8 K values as
  // the fp32 chunks 8 sub + 2(l/16) and the next.
  const int g = lane >> 4, nr = 16 * wave + (lane & 15);
  uint32_t pa[R::SUB][4], pw[R::SUB][2];
#pragma unroll
  for (int sub = 0; sub < R::SUB; ++sub) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      const int ar = mb * 16 + (lane & 15);
      pa[sub][mb] = ar * R::XR + (rw_swz<CX>(ar, sub * 4 + g) << 4);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) pw[sub][h] = R::XB + nr * R::WR + (rw_swz<CW>(nr, sub * 8 + 2 * g + h) << 4);
  }
  f32x4 acc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) acc[mb] = f32x4{0, 0, 0, 0};
  int issued = 0;
  for (; issued < D - 1 && issued < ns; ++issued) issue(issued);
  for (int s = 0; s < ns; ++s) {
    // this wave's copies of step s landed (younger steps may stay in flight) ...
    wait_steps<D - 2, R::NDMA>(issued - 1 - s);
    // ... and every other wave's; every read of step s - 1 is finished
    barrier_raw();
    if (issued < ns) issue(issued++);  // into the slot of step s - 1
    const uint32_t st = (uint32_t)(s % D) * R::STAGE;
#pragma unroll
    for (int sub = 0; sub < R::SUB; ++sub) {
      const float4 w0 = *(const float4*)(smem + st + pw[sub][0]);
      const float4 w1 = *(const float4*)(smem + st + pw[sub][1]);
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
      for (int mb = 0; mb < 4; ++mb) {
        const bf16x8 av8 = as_bf16x8(*(const u32x4*)(smem + st + pa[sub][mb]));
        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bh, acc[mb], 0, 0, 0);
        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bm, acc[mb], 0, 0, 0);
        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bl, acc[mb], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's reads of the slot are done
  }
  // lane l holds tokens 16mb + 4(l/16) + i against expert n0 + 16w + (l&15)
  const int nn = n0 + nr;
  if (nn >= N) return;
  float* zp = a.z + (size_t)split * a.T * a.zstride;
  const float bias = (a.bias && split == 0) ? a.bias[(pass ? a.n_pub : 0) + nn] : 0.0f;
  const int zc = (a.soft && pass ? a.n_pub : 0) + nn;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tt = mb * 16 + g * 4 + i;
      if (!part(tt)) continue;
      float z = acc[mb][i];
      if (split == 0 && a.bias) z += bias;
      // non-temporal: the partial logits are read once, by the top-k kernel
      __builtin_nontemporal_store(z, &zp[(size_t)(t0 + tt) * a.zstride + zc]);
    }
}

// fp32 activations (small layers): one thread per (token, expert) pair, fp32 dot
// products in blocks of 64 terms.
__global__ __launch_bounds__(RT_THREADS) void route_logits_f32_kernel(RouteArgs a) {
  const int t = blockIdx.x;
  const int tau = token_tau(a, t);
  // masked: the permitted pool; soft (control arm): public then private rows
  const int N = a.soft ? a.n_pub + a.n_priv : (tau ? a.n_priv : a.n_pub);
  const int base = (a.soft || !tau) ? 0 : a.n_pub;
  const float* xr = (const float*)a.x + (size_t)t * a.H;
  for (int n = threadIdx.x; n < N; n += RT_THREADS) {
    const int e = base + n;  // global expert id
    const float* wrow = (e < a.n_pub) ? a.wr_pub + (size_t)e * a.H : a.wr_priv + (size_t)(e - a.n_pub) * a.H;
    float acc = 0.0f;
    for (int h0 = 0; h0 < a.H; h0 += 64) {
      float part = 0.0f;
      for (int h = h0; h < h0 + 64; ++h) part = fmaf(xr[h], wrow[h], part);
      acc += part;
    }
    if (a.bias) acc += a.bias[e];
    a.z[(size_t)t * a.zstride + n] = acc;
  }
}

// Top-k and gates: one wave per token over its pool's logits. With K-split logits the
// wave first adds the partial arrays in split order into LDS and ranks that row.
__global__ __launch_bounds__(RT_THREADS) void route_topk_kernel(RouteArgs a) {
  __shared__ float s_z[RT_WAVES][2 * PMPE_MAX_POOL];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * RT_WAVES + w;
  if (t >= a.T) return;  // wave-uniform; no block barrier follows
  const float* z = a.z + (size_t)t * a.zstride;
  if (a.zsplit > 1) {
    // the whole zstride-wide row of every split is loaded without waiting for the policy
    // word (entries past the pool are added but never ranked), then added in split order
    const size_t pstride = (size_t)a.T * a.zstride;
    if (a.zsplit == 4) {
      for (int s = lane; s < a.zstride; s += 64) {
        const float v0 = z[s], v1 = z[pstride + s], v2 = z[2 * pstride + s], v3 = z[3 * pstride + s];
        s_z[w][s] = ((v0 + v1) + v2) + v3;
      }
    } else {
      for (int s = lane; s < a.zstride; s += 64) {
        float v = z[s];
        for (int p = 1; p < a.zsplit; ++p) v += z[p * pstride + s];
        s_z[w][s] = v;
      }
    }
    // the wave's LDS writes complete before any lane reads another lane's entry
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    z = &s_z[w][0];
  }
  const int tau = token_tau(a, t);
  // masked: the permitted pool; soft (control arm): the concatenated pool
  const int N = a.soft ? a.n_pub + a.n_priv : (tau ? a.n_priv : a.n_pub);
  const int base = (a.soft || !tau) ? 0 : a.n_pub;
  TopkCtx c{a.T, a.n_pub, a.n_priv, a.k, a.gate_mode, a.topk_idx, a.topk_gate, a.allow, a.kgap};
  if (N <= 64)
    topk_one_token<1>(c, t, tau, N, base, z);
  else if (N <= 128)
    topk_one_token<2>(c, t, tau, N, base, z);
  else if (N <= 256)
    topk_one_token<4>(c, t, tau, N, base, z);
  else
    topk_one_token<8>(c, t, tau, N, base, z);
}

}  // namespace

int route_ksplit(int T, int H, int n_pub, int n_priv, int act_bf16) {
  if (!act_bf16 || T <= 2048) return 1;
  // enough blocks to fill the chip (two resident per CU) with the K range of a tile split
  // over up to four blocks
  const int64_t nt = (T + RW_TT - 1) / RW_TT;
  const int64_t groups = (n_pub + RW_NE - 1) / RW_NE + (n_priv + RW_NE - 1) / RW_NE;
  const int nsteps = H / RwLarge::BK;
  int S = 1;
  while (S < 4 && nt * groups * S < 1024 && nsteps % (2 * S) == 0) S *= 2;
  return S;
}

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  if (a.act_bf16) {
    if (a.T > 2048) {
      const int nt = (a.T + RW_TT - 1) / RW_TT;
      const int groups = (a.n_pub + RW_NE - 1) / RW_NE + (a.n_priv + RW_NE - 1) / RW_NE;
      // 8 XCDs x ceil(nt / 8) tiles each x the groups and K splits of a tile
      const int64_t grid = (int64_t)8 * ((nt + 7) / 8) * groups * a.zsplit;
      hipLaunchKernelGGL(route_logits_wide_kernel<RwLarge>, dim3((unsigned)grid), dim3(RW_THREADS), 0, s, a, nt,
                         groups, a.zsplit);
    } else {
      const int groups = (a.n_pub + 15) / 16 + (a.n_priv + 15) / 16;
      const int nt = (a.T + 15) / 16;
      hipLaunchKernelGGL(route_logits_bf16_kernel<16>, dim3((nt * groups + 7) / 8 * 8), dim3(RT_THREADS), 0, s, a, nt, groups);
    }
  } else {
    hipLaunchKernelGGL(route_logits_f32_kernel, dim3(a.T), dim3(RT_THREADS), 0, s, a);
  }
  hipLaunchKernelGGL(route_topk_kernel, dim3((a.T + RT_WAVES - 1) / RT_WAVES), dim3(RT_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace pmpe
