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
//     H split across the four waves); larger batches stage them in LDS (64-token tiles).
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

// Large batches: token-tile x expert-group logits with both operands staged in LDS.
// Block (tile, g): TT tokens against RL_NE experts of one pool; wave w owns the tile's
// 16-token row block w over the whole of H, so no partial sums are exchanged. K steps of
// 64: a step's x rows (TT x 128 bytes) and fp32 router rows (RL_NE x 256 bytes) are copied
// whole into a ring of D stages by global->LDS copies, so every request is a full
// 128-byte line (loads of 64-byte row pieces straight into the MFMA register layout
// bound the register kernel at this size). The 16-byte chunks of each LDS row are
// XOR-swizzled by row so that the fragment reads of 16 rows hit distinct banks. Token
// selection, the exact three-part split, the pool rule and the K rotation are those of
// the register kernel.
// 16 experts per block and 6 stages (72 KiB, two blocks per CU): the kernel is bound by the
// copies in flight per CU, so more concurrent blocks beat fewer re-reads (Qwen-shaped
// 4096-token batch: 32 experts per block 43 us, 16 experts with 4 stages 38 us, with 6
// stages 35 us, the register kernel 46 us, top-k included).
constexpr int RL_NE = 16, RL_BK = 64;
template <int TT_, int D_>
struct RlCfg {
  static constexpr int TT = TT_, D = D_;
  static constexpr int THREADS = 4 * TT;                 // one wave per 16-token row block
  static constexpr int WAVES = THREADS / 64;
  static constexpr int NB = RL_NE / 16;                  // 16-expert blocks per wave
  static constexpr int XB = TT * RL_BK * 2;              // x bytes per stage
  static constexpr int WB = RL_NE * RL_BK * 4;           // router bytes per stage
  static constexpr int STAGE = XB + WB;
  static constexpr int WDMA = WB / 1024 / WAVES;         // router copies (1 KiB, 4 rows) per wave per stage
  static constexpr int NDMA = 2 + WDMA;                  // copies per wave per stage: 2 of x, the router's
  static_assert(TT % 16 == 0 && RL_NE % 16 == 0 && WDMA >= 1 && WDMA * WAVES * 1024 == WB, "router tile");
};
using RlLarge = RlCfg<64, 6>;

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

// Block b runs on XCD b % 8. Token tiles are dealt round-robin to the XCDs (tile
// 8 i + x to XCD x) with the groups of one tile adjacent on its XCD, so the blocks
// that find tokens of their pool spread over all XCDs even when consecutive tiles share
// a policy (requests are contiguous token ranges), and a tile's x rows are shared in
// one L2.
template <class R>
__global__ __launch_bounds__(R::THREADS) void route_logits_lds_kernel(RouteArgs a, int ntiles, int ngroups) {
  constexpr int TT = R::TT, D = R::D, NB = R::NB, WDMA = R::WDMA;
  __shared__ __attribute__((aligned(16))) unsigned char smem[D * R::STAGE];
  __shared__ int s_tau[TT];
  __shared__ int s_first;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.x, xcd = b & 7, j = b >> 3;
  const int lt = j / ngroups, grp = j - lt * ngroups;
  const int tile = lt * 8 + xcd;
  if (tile >= ntiles) return;
  const int t0 = tile * TT;
  const int gpub = (a.n_pub + RL_NE - 1) / RL_NE;
  const int pass = grp < gpub ? 0 : 1;
  const int n0 = (pass ? grp - gpub : grp) * RL_NE;
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
  const int H = a.H;
  const int first = s_first;
  auto part = [&](int r) { return a.soft ? s_tau[r] >= 0 : s_tau[r] == pass; };
  // Copy sources, byte offsets from the step's base (x: the tile's first row, so every
  // offset is below TT rows of H bf16 whatever T). x: copy jj of wave w fills LDS rows
  // (2w + jj) * 8 + l / 8, lane l's physical chunk l % 8 holding logical chunk
  // (l % 8) ^ ((row >> 1) & 7); a row whose token has the other policy (or lies past T)
  // copies the tile's first token of this policy, so a token's x is only ever read for
  // the pool it is permitted. Router: copy jj of wave w fills rows (WDMA w + jj) * 4 +
  // l / 16, physical chunk l % 16 holding logical chunk (l % 16) ^ (row & 15); rows past
  // the pool copy expert n0 (their results are discarded).
  uint32_t offx[2];
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    const int r = (2 * wave + jj) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    const int tok = part(r) ? r : first;  // row within the tile
    offx[jj] = ((uint32_t)tok * (uint32_t)H + c * 8) * 2;
  }
  uint32_t offw[WDMA];
#pragma unroll
  for (int jj = 0; jj < WDMA; ++jj) {
    const int r = (WDMA * wave + jj) * 4 + (lane >> 4);
    const int c = (lane & 15) ^ (r & 15);
    const int n = n0 + r;
    offw[jj] = ((uint32_t)(n < N ? n : n0) * (uint32_t)H + c * 4) * 4;
  }
  const uint16_t* x = (const uint16_t*)a.x + (size_t)t0 * H;
  const float* wr = pass ? a.wr_priv : a.wr_pub;
  const int nsteps = H / RL_BK;
  const int rot = (tile * 5 + grp * 3) % nsteps;  // concurrent blocks read different columns
  const uint32_t lds0 = lds_addr(smem);
  auto issue = [&](int st) {
    const int kk = ((st + rot) % nsteps) * RL_BK;
    const uint32_t sx = __builtin_amdgcn_readfirstlane(lds0 + (st % D) * R::STAGE);
    dma16s<0, false>(offx[0], x + kk, sx + 2 * wave * 1024);
    dma16s<1024, false>(offx[1], x + kk, sx + 2 * wave * 1024);
    const uint32_t sw = sx + R::XB + WDMA * wave * 1024;
    Unroll<0, WDMA>::run([&](auto jj) { dma16s<jj.value * 1024, false>(offw[jj.value], wr + kk, sw); });
  };
  // Fragment addresses within a stage. A: row 16w + (l & 15), 8 bf16 of K sub-step sub at
  // logical chunk 4 sub + l / 16. Router block nb: row 16 nb + (l & 15), the same 8 K
  // values as two fp32 chunks 8 sub + 2 (l / 16) and the next.
  const int ar = wave * 16 + (lane & 15), nr = lane & 15, g = lane >> 4;
  uint32_t pa[2], pw[NB][2][2];
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    pa[sub] = ar * 128 + (((sub * 4 + g) ^ ((ar >> 1) & 7)) << 4);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int h = 0; h < 2; ++h)
        pw[nb][sub][h] = R::XB + (nb * 16 + nr) * 256 + (((sub * 8 + 2 * g + h) ^ nr) << 4);
  }
  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0, 0, 0, 0};
  int issued = 0;
  for (; issued < D - 1 && issued < nsteps; ++issued) issue(issued);
  for (int s = 0; s < nsteps; ++s) {
    // this wave's copies of step s landed (younger steps may stay in flight) ...
    wait_steps<D - 2, R::NDMA>(issued - 1 - s);
    // ... and every other wave's; every read of step s - 1 is finished
    barrier_raw();
    if (issued < nsteps) issue(issued++);  // into the slot of step s - 1
    const uint32_t st = (uint32_t)(s % D) * R::STAGE;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const bf16x8 av8 = as_bf16x8(*(const u32x4*)(smem + st + pa[sub]));
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const float4 w0 = *(const float4*)(smem + st + pw[nb][sub][0]);
        const float4 w1 = *(const float4*)(smem + st + pw[nb][sub][1]);
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
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bh, acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bm, acc[nb], 0, 0, 0);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av8, bl, acc[nb], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's reads of the slot are done
  }
  // lane l holds tokens 16w + 4 (l / 16) + i against experts n0 + 16 nb + (l & 15)
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tt = wave * 16 + g * 4 + i;
      const int nn = n0 + nb * 16 + nr;
      if (!part(tt) || nn >= N) continue;
      float z = acc[nb][i];
      if (a.bias) z += a.bias[(pass ? a.n_pub : 0) + nn];
      a.z[(size_t)(t0 + tt) * a.zstride + (a.soft && pass ? a.n_pub : 0) + nn] = z;
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

// Top-k and gates: one wave per token over its pool's logits.
__global__ __launch_bounds__(RT_THREADS) void route_topk_kernel(RouteArgs a) {
  const int t = blockIdx.x * RT_WAVES + (threadIdx.x >> 6);
  if (t >= a.T) return;
  const int tau = token_tau(a, t);
  // masked: the permitted pool; soft (control arm): the concatenated pool
  const int N = a.soft ? a.n_pub + a.n_priv : (tau ? a.n_priv : a.n_pub);
  const int base = (a.soft || !tau) ? 0 : a.n_pub;
  const float* z = a.z + (size_t)t * a.zstride;
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

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  if (a.act_bf16) {
    if (a.T > 2048) {
      using R = RlLarge;
      const int nt = (a.T + R::TT - 1) / R::TT;
      const int lgroups = (a.n_pub + RL_NE - 1) / RL_NE + (a.n_priv + RL_NE - 1) / RL_NE;
      // 8 XCDs x ceil(nt / 8) tiles each x the groups of a tile
      const int64_t grid = (int64_t)8 * ((nt + 7) / 8) * lgroups;
      hipLaunchKernelGGL(route_logits_lds_kernel<R>, dim3((unsigned)grid), dim3(R::THREADS), 0, s, a, nt, lgroups);
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
