// K3 - expert FFN: grouped SwiGLU GEMM over the experts that have rows (plus the
// always-on shared group), with the private-row execution audit written by the blocks
// that execute the rows.
//
// Groups: routed expert g < E owns permuted rows [offset[g], offset[g] + count[g]);
// the shared group (g = E, when present) owns all T tokens in token order. A tile is
// (group, M tile of BM rows, N tile). The tile list is built on the device from the
// expert counts (no host synchronisation): every block scans the per-group tile
// counts, so groups with zero rows get no tile and load nothing. Tiles are numbered
// group-major, then N tile, then M tile, so concurrent tiles share weight and row
// tiles; block ids are remapped so that each XCD (workgroups are dealt to the 8 XCDs
// round-robin) works on one contiguous range of the routed experts' tiles and its L2
// holds the shared operands; the shared group's tiles (longest K loop in GEMM2) are
// spread over the XCDs ahead of them.
//
//   GEMM1  [rows, H] x [H, 2I]: the N tile holds BN/2 gate columns and the matching
//          BN/2 up columns, so h = silu(g) * u is formed in registers and rounded once
//          to bf16 into the workspace h [T*k, I].
//   GEMM2  [rows, I] x [I, H] -> y_perm (bf16); the first N tile of each private M
//          tile adds its rows to the audit.
//
// bf16 path: v_mfma_f32_16x16x32_bf16 with fp32 accumulation; A and B tiles are
// copied straight from global memory into LDS (global_load_lds_dwordx4, no register
// staging) through a ring of STAGES buffers of BK-wide K steps, so STAGES-1 steps
// are in flight while one is multiplied (with few rows per expert every weight tile
// is read once, and the weight copies carry the non-temporal hint); the 16-byte chunks of each LDS row are
// XOR-swizzled by row so that MFMA operand reads do not conflict on banks. Rows past a tile's valid count are loaded from a valid
// row (their results are never stored), and MFMAs of 16-row blocks that hold no
// valid row are skipped. The output tile goes through LDS so that global stores are
// whole 16-byte vectors.
#include <type_traits>

#include "lds_dma.h"
#include "pmpe_internal.h"

namespace pmpe {
namespace {

// LDS operand tiles hold BK bf16 per row (RB = 2*BK bytes, CH = BK/8 chunks of 16
// bytes). Chunk c of row r is stored at chunk c ^ f(r): f(r) = r & 7 for 128-byte
// rows and (r >> 1) & 3 for 64-byte rows, so any 8 consecutive rows read at one
// logical chunk land in 8 distinct 16-byte bank groups of a 128-byte bank line.
template <int BK>
__device__ __forceinline__ int swz(int r, int c) {
  if constexpr (BK == 64)
    return r * 128 + ((c ^ (r & 7)) << 4);
  else
    return r * 64 + ((c ^ ((r >> 1) & 3)) << 4);
}

template <int BM_, int BN_, int WM_, int WN_, int STAGES_, int BK_, int FRAG_BUFS_ = 1, bool HALF_ = true,
          bool NT_B_ = false, bool W8_ = false>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, STAGES = STAGES_, BK = BK_;
  static constexpr int FRAG_BUFS = FRAG_BUFS_;  // 2: read the next K step's fragments early
  // a shorter K-loop variant for tiles whose valid rows fill at most half of each wave's
  // row blocks (needs the registers of a second accumulator set)
  static constexpr bool HALF = HALF_;
  // Weight copies carry the non-temporal hint: when every weight tile is read once
  // (few rows per expert) this keeps the streamed weights from evicting the reused
  // activation rows (decode-shaped batch: 245 -> 185 us on MI355X).
  static constexpr bool NT_B = NT_B_;
  // W8: expert weights are fp8 (e4m3) with a power-of-two scale per weight row; their
  // LDS rows hold BK bytes and are widened to bf16 when the MFMA fragments are read.
  static constexpr bool W8 = W8_;
  static constexpr int RB = 2 * BK, CH = BK / 8, RPD = 1024 / RB;  // rows per DMA instruction
  static constexpr int RB_B = W8 ? BK : RB, CH_B = RB_B / 16, RPD_B = 1024 / RB_B;
  static constexpr int WAVES = WM * WN, THREADS = 64 * WAVES;
  static constexpr int A_BYTES = BM * RB, B_BYTES = BN * RB_B, STAGE = A_BYTES + B_BYTES;
  static constexpr int A_DMA = BM / RPD / WAVES, B_DMA = BN / RPD_B / WAVES;  // per wave per stage
  // A wave owns MB 16-row blocks of the tile, interleaved with the other WM-1 row
  // waves (block j*WM + wm), so a partly filled tile loads every SIMD evenly.
  static constexpr int WROWS = BM / WM, MB = WROWS / 16;
  static constexpr int LDS = STAGES * STAGE;
  // resident blocks per CU: the ring plus up to 8 KiB of static tables per block
  static constexpr int PER_CU = (160 * 1024) / (LDS + 8 * 1024);
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(A_DMA * RPD * WAVES == BM && B_DMA * RPD_B * WAVES == BN, "DMA split");
  static_assert(!W8 || BK == 64, "fp8 weight rows are 64 bytes");
};
using CfgLarge = Cfg<256, 256, 4, 2, 2, 64>;  // prefill: 8 waves of 64 x 128, 2 x 64 KiB stages
// decode-shaped: 4 waves, 3 x 24 KiB stages, streamed weights
using CfgSmall = Cfg<64, 128, 1, 4, 3, 64, 2, true, true>;
// fp8 weights: the smaller weight tiles leave room for a third stage (3 x 48 KiB) in the
// prefill configuration. The decode one takes 256 weight rows per tile, so that a K step
// copies as many weight bytes (16 KiB) as the bf16 decode tile and two blocks per CU keep as
// much of the weight stream in flight; its copies carry no non-temporal hint, because a
// 64-byte fp8 row step reads half a line and the next step must find the other half in L2
// (with the hint: 1.35x the weight bytes fetched from HBM).
using CfgLarge8 = Cfg<256, 256, 4, 2, 3, 64, 1, true, false, true>;
using CfgSmall8 = Cfg<64, 256, 1, 4, 3, 64, 2, true, false, true>;

constexpr int MAXG = 2 * PMPE_MAX_POOL + 1;  // routed experts + the shared group

// DMA of 4 bytes per lane (int32 gather indices): lane l's word lands at lds_base + 4 * l.
__device__ __forceinline__ void dma4(const void* src, uint32_t lds_base_) {
  const uint32_t lds_base = __builtin_amdgcn_readfirstlane(lds_base_);
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %0, off" ::"v"(src),
      "s"(lds_base)
      : "memory", "m0");
}

// Rows of the output tile staged per epilogue pass: the largest multiple of 16 that
// divides BM and whose bf16 rows fit in one ring stage.
constexpr int epilogue_rows(int fit, int bm) {
  for (int d = (fit < bm ? fit : bm) / 16 * 16; d >= 16; d -= 16)
    if (bm % d == 0) return d;
  return 16;
}

struct TileInfo {
  int g;     // group: expert id, or E for the shared group
  int m0;    // first row of the tile within the group
  int n0;    // first output column (GEMM1: h column; GEMM2: y column)
  int rows;  // valid rows
  int base;  // first row of the tile in the group's row space (permuted row / token)
};

// Persistent bf16 grouped GEMM. GATED: GEMM1 (x -> h with SwiGLU); else GEMM2 (h -> y).
//
// Each block builds the group table once (tile counts, row counts and offsets in LDS),
// then walks its share of the tile list: XCD x = blockIdx % 8 owns a contiguous slice
// of the (group, N tile, M tile) order, dealt round-robin to the XCD's blocks. K steps
// of consecutive tiles form one stream: the copy ring keeps STAGES-1 steps in flight
// across tile boundaries, so the next tile's first operands load during the current
// tile's last MFMAs and its epilogue. Gather indices (row_token slices) are fetched by
// LDS-DMA as well, one tile ahead of their use, so no register-destined global load
// inside the stream forces the compiler to drain the ring.
// SAVE (GEMM1 only): also store the fp32 gate and up projections [a; b] of every routed
// row into ab_save [T*k, 2I], for a later backward pass. AUDIT (GEMM2 only): count the
// executed private rows; off when the kernel serves as a plain grouped GEMM (the
// backward's products with transposed weights).
// GATHER_A (GEMM2 form only): the A rows are gathered by token, row r of the product
// reading x[row_token[r]] (the backward's dh takes the upstream gradient rows so).
template <class C, bool GATED, bool SAVE = false, bool AUDIT = true, bool GATHER_A = false>
__global__ __launch_bounds__(C::THREADS) void gemm_bf16_kernel(FfnArgs a) {
  static_assert(!(GATED && GATHER_A), "GEMM1 gathers through x_perm == NULL");
  __shared__ __attribute__((aligned(16))) unsigned char smem[C::LDS];
  // Gather-index slices (row_token) of the tiles in flight. The producer runs up to
  // STAGES-1 K steps ahead of the consumer and fetches a tile's slice one tile before its
  // first step, so with one K step per tile (K = BK) the slices of tiles ci .. ci+STAGES
  // are live while tile ci is consumed: STAGES+1 slots.
  constexpr int NRT = C::STAGES + 1;
  __shared__ __attribute__((aligned(16))) int s_rt[NRT][C::BM];
  __shared__ int s_cum[MAXG + 1];
  __shared__ int s_cnt[MAXG];
  __shared__ int s_off[MAXG];
  // interleaved group order (prefill tiles only: the decode tiles' two blocks per CU have no
  // LDS to spare for the permutation)
  constexpr bool MIX = C::BM >= 256;
  __shared__ int s_perm[MIX ? MAXG : 1];
  constexpr int NCOLS = GATED ? C::BN / 2 : C::BN;  // output columns per tile
  constexpr int WCOLS = NCOLS / C::WN;               // output columns per wave
  constexpr int NBO = WCOLS / 16;                    // output 16-col blocks per wave
  constexpr int NB = GATED ? 2 * NBO : NBO;          // B operand blocks per wave
  constexpr int BK = C::BK, S = C::STAGES, NDMA = C::A_DMA + C::B_DMA;
  constexpr int ER = epilogue_rows(C::STAGE / (NCOLS * 2), C::BM);  // epilogue rows per pass
  static_assert(ER % 16 == 0 && C::BM % ER == 0, "an epilogue pass must hold whole 16-row blocks");
  static_assert(C::BM % 64 == 0, "row_token slices are copied 64 entries at a time");

  const int tid = threadIdx.x, lane = tid & 63;
  const int uwave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, scalar
  const int wm = uwave / C::WN, wn = uwave % C::WN;
  const int E = a.n_pub + a.n_priv;
  const int ngroups = E + (a.Is > 0 ? 1 : 0);
  const int H = a.H;
  const int TK = a.T * a.k;

  if (tid < 64) {
    // Tile order, prefill tiles (256 rows): the shared group first (all T tokens; in GEMM2
    // its K loop over 2 I_s is the longest, so its tiles must not be left for the end),
    // then the public and the private experts interleaved in proportion to the pool sizes
    // (public j before private p iff (2j+1) n_priv <= (2p+1) n_pub). Each XCD's slice of
    // the routed tiles then holds both kinds (the private experts' full tiles carry about
    // twice the MFMA work of the half-filled public ones), while the tiles of one expert
    // stay adjacent. Decode-shaped tiles keep the expert order (their two blocks per CU
    // have no LDS to spare for the permutation).
    const int sh = (ngroups > E) ? 1 : 0;
    for (int g = tid; MIX && g < ngroups; g += 64) {
      int pos;
      if (g < a.n_pub) {
        const int num = (2 * g + 1) * a.n_priv;  // private experts before public g
        pos = sh + g + min(a.n_priv, ((num + a.n_pub - 1) / a.n_pub) / 2);
      } else if (g < E) {
        const int p = g - a.n_pub;
        const int f = (2 * p + 1) * a.n_pub / a.n_priv;  // public experts before private p
        pos = sh + p + min(a.n_pub, (f + 1) / 2);
      } else {
        pos = 0;
      }
      s_perm[pos] = g;
    }
    // (this wave's LDS writes above precede its reads below)
    int running = 0;
    for (int o0 = 0; o0 < ngroups; o0 += 64) {
      const int o = o0 + tid;
      int nt = 0;
      if (o < ngroups) {
        const int g = MIX ? s_perm[o] : o;
        const int cnt = (g < E) ? a.count[g] : a.T;
        s_cnt[g] = cnt;
        s_off[g] = (g < E) ? a.offset[g] : 0;
        const int width = GATED ? ((g < E) ? a.I : a.Is) : H;
        nt = ((cnt + C::BM - 1) / C::BM) * ((width + NCOLS - 1) / NCOLS);
      }
      const int incl = wave_incl_scan(nt);
      if (o < ngroups) s_cum[o + 1] = running + incl;
      running += __shfl(incl, 63, 64);
    }
    if (tid == 0) s_cum[0] = 0;
  }
  __syncthreads();

  // Block ids are remapped so that XCD x (workgroups go to the 8 XCDs round-robin) takes
  // one contiguous slice of the routed tiles, dealt round-robin to its blocks: tiles that
  // share an expert's weights or rows then run on one XCD and meet in its L2. The shared
  // group's tiles (prefill) come before them in every XCD's list, dealt to the XCDs in
  // chunks of XCH consecutive tiles (M tiles of one weight tile), so that every XCD gets
  // its share of them.
  constexpr int XCH = 8;
  const int total = s_cum[ngroups];
  const int n_sh = (MIX && ngroups > E) ? s_cum[1] : 0;  // shared tiles, first in the order
  const int n_rt = total - n_sh;
  const int b = blockIdx.x, x = b & 7, q = b >> 3;
  const int nbx = ((int)gridDim.x - x + 7) >> 3;
  const int nch = (n_sh + XCH - 1) / XCH;               // chunks of shared tiles
  const int nch_x = (nch > x) ? (nch - x + 7) / 8 : 0;  // those of XCD x
  // the last chunk (nch - 1) is the only one that may be partial
  const int sh_x = nch_x * XCH - ((nch_x > 0 && (nch - 1) % 8 == x) ? (nch * XCH - n_sh) : 0);
  const int cnt_x = sh_x + (n_rt >> 3) + (x < (n_rt & 7) ? 1 : 0);
  const int start_x = n_sh + x * (n_rt >> 3) + min(x, n_rt & 7);
  const int ntl = (cnt_x > q && q < nbx) ? (cnt_x - q + nbx - 1) / nbx : 0;
  if (ntl == 0) return;

  auto tile_of = [&](int i) {
    const int j = q + i * nbx;  // index within the XCD's tiles
    const int L = (j < sh_x) ? (x + 8 * (j / XCH)) * XCH + (j % XCH) : start_x + (j - sh_x);
    int lo = 0, hi = ngroups - 1;  // last position o with s_cum[o] <= L (a group with tiles)
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_cum[mid] <= L) lo = mid; else hi = mid - 1;
    }
    TileInfo t;
    const int o = __builtin_amdgcn_readfirstlane(lo);
    t.g = MIX ? __builtin_amdgcn_readfirstlane(s_perm[o]) : o;
    const int cnt = __builtin_amdgcn_readfirstlane(s_cnt[t.g]);
    const int mt = (cnt + C::BM - 1) / C::BM;
    const int local = L - __builtin_amdgcn_readfirstlane(s_cum[o]);
    const int n = local / mt, m = local - n * mt;
    t.m0 = m * C::BM;
    t.n0 = n * NCOLS;
    t.rows = min(C::BM, cnt - t.m0);
    t.base = __builtin_amdgcn_readfirstlane(s_off[t.g]) + t.m0;
    return t;
  };
  // Does tile t read row_token? (gathered x rows in GEMM1; the audit in GEMM2)
  auto needs_rt = [&](const TileInfo& t) {
    if (t.g >= E) return false;
    return GATED ? (a.x_perm == nullptr) : (GATHER_A || (AUDIT && t.g >= a.n_pub));
  };
  const uint32_t lds0 = lds_addr(smem);
  const uint32_t rt0 = lds_addr(&s_rt[0][0]);
  // Copy row_token[base .. base + BM) of tile t into s_rt[slot] (wave 0; clamped reads).
  auto issue_rt = [&](const TileInfo& t, int slot) {
    if (uwave == 0 && needs_rt(t)) {
#pragma unroll
      for (int j = 0; j < (C::BM + 63) / 64; ++j) {
        const int idx = min(t.base + j * 64 + lane, TK - 1);
        dma4(a.row_token + idx, rt0 + (slot * C::BM + j * 64) * 4);
      }
    }
  };

  // Producer context: source pointers of the tile whose K steps are being issued.
  constexpr int CHK = C::CH;
  const int lrow = lane / CHK, lphys = lane % CHK;
  auto logical = [&](int r) { return (BK == 64) ? (lphys ^ (r & 7)) : (lphys ^ ((r >> 1) & 3)); };
  // weight rows of RB_B bytes (fp8: 64-byte rows, the 64-byte-row swizzle)
  const int lrow_b = lane / C::CH_B, lphys_b = lane % C::CH_B;
  auto logical_b = [&](int r) {
    if constexpr (C::W8) return lphys_b ^ ((r >> 1) & 3);
    else return logical(r);
  };
  constexpr int ESZ = C::W8 ? 1 : 2;  // bytes per weight element
  // Copy sources as 32-bit element offsets from tile-uniform bases (the host checks
  // that every offset fits).
  uint32_t offA[C::A_DMA], offB[C::B_DMA];
  const uint16_t* baseA = nullptr;
  const unsigned char* baseB = nullptr;  // weight bytes
  bool p_valid = true;  // producer tile has weights (private tiles may not)
  auto setup_ctx = [&](const TileInfo& t, int slot) {
    const bool shared = t.g >= E;
    const bool priv = !shared && t.g >= a.n_pub;
    const int I = shared ? a.Is : a.I;
    const int K = GATED ? H : I;
    const unsigned char* w;
    if (shared) {
      w = (const unsigned char*)(GATED ? a.w13_sh : a.w2_sh);
    } else if (!priv) {
      w = (const unsigned char*)(GATED ? a.w13_pub : a.w2_pub) + (size_t)t.g * (GATED ? 2 : 1) * I * H * ESZ;
    } else {
      w = (const unsigned char*)(GATED ? a.w13_priv : a.w2_priv);
      if (w) w += (size_t)(t.g - a.n_pub) * (GATED ? 2 : 1) * I * H * ESZ;
    }
    p_valid = (w != nullptr) && !(priv && (a.w13_priv == nullptr || a.w2_priv == nullptr));
    if (!p_valid) w = (const unsigned char*)(GATED ? a.w13_pub : a.w2_pub);  // read but never used
    if (GATED)
      baseA = (const uint16_t*)((!shared && a.x_perm) ? a.x_perm : a.x);
    else
      baseA = (const uint16_t*)(GATHER_A ? a.x : shared ? a.h_sh : a.h);
    baseB = w;
#pragma unroll
    for (int i = 0; i < C::A_DMA; ++i) {
      const int r = (uwave * C::A_DMA + i) * C::RPD + lrow;
      const int rr = min(r, t.rows - 1);  // rows past the valid count reload a valid row
      uint32_t row;
      if (GATED) {
        if (shared || a.x_perm)
          row = (uint32_t)(t.base + rr) * (uint32_t)H;
        else
          row = (uint32_t)s_rt[slot][rr] * (uint32_t)H;
      } else if (GATHER_A) {
        row = (uint32_t)s_rt[slot][rr] * (uint32_t)I;
      } else {
        row = (uint32_t)(t.base + rr) * (uint32_t)I;
      }
      offA[i] = (row + logical(r) * 8) * 2;  // bytes
    }
#pragma unroll
    for (int i = 0; i < C::B_DMA; ++i) {
      const int r = (uwave * C::B_DMA + i) * C::RPD_B + lrow_b;
      int wrow;
      if (GATED) {
        const int half = C::BN / 2;
        const int j = (r < half) ? r : r - half;
        const int col = min(t.n0 + j, I - 1);
        wrow = (r < half) ? col : I + col;
      } else {
        wrow = min(t.n0 + r, H - 1);
      }
      offB[i] = ((uint32_t)wrow * (uint32_t)K + logical_b(r) * (16 / ESZ)) * ESZ;  // bytes
    }
    return K / BK;
  };
  auto issue = [&](int slot, int k0) {
    // slot is wave-uniform; say so, so that the LDS base stays in an SGPR
    const uint32_t sa = __builtin_amdgcn_readfirstlane(lds0 + slot * C::STAGE);
    const uint32_t sb = sa + C::A_BYTES;
    const uint16_t* ba = baseA + k0;  // scalar bases advance by the K step
    const unsigned char* bb = baseB + k0 * ESZ;
    const uint32_t wa = sa + uwave * C::A_DMA * 1024, wb = sb + uwave * C::B_DMA * 1024;
    Unroll<0, C::A_DMA>::run([&](auto i) { dma16s<i.value * 1024, false>(offA[i.value], ba, wa); });
    Unroll<0, C::B_DMA>::run([&](auto i) { dma16s<i.value * 1024, C::NT_B>(offB[i.value], bb, wb); });
  };

  // Producer state: next step to issue is (pi, pk) of a tile with pnk steps; `issued`
  // counts the steps issued so far.
  int pi = 0, pk = 0, pnk = 0, issued = 0;
  TileInfo pt = tile_of(0);
  // prologue: gather indices of tiles 0 and 1, then the first S-1 steps
  issue_rt(pt, 0);
  wait_vmcnt<0>();
  __syncthreads();
  pnk = setup_ctx(pt, 0);
  if (ntl > 1) issue_rt(tile_of(1), 1);
  auto produce = [&](int slot) {  // issue the next step into `slot` (if any remain)
    if (pi >= ntl) return;
    if (pk == pnk) {  // advance to the next tile; its gather indices arrived earlier
      ++pi;
      pk = 0;
      if (pi >= ntl) return;
      pt = tile_of(pi);
      pnk = setup_ctx(pt, pi % NRT);
      if (pi + 1 < ntl) issue_rt(tile_of(pi + 1), (pi + 1) % NRT);
    }
    issue(slot, pk * BK);
    ++pk;
    ++issued;
  };
#pragma unroll
  for (int s = 0; s < S - 1; ++s) produce(s);

  // B operand row (within the tile) of block nb of this wave, minus the wave's offset
  auto bconst = [&](int nb) {
    if (GATED) return (nb < NBO) ? nb * 16 : C::BN / 2 + (nb - NBO) * 16;
    return nb * 16;
  };
  // row of 16-row block j of this wave within the tile
  auto arow = [&](int j) { return (j * C::WM + wm) * 16; };
  constexpr int SUB = BK / 32;
  constexpr int FB = C::FRAG_BUFS;
  bf16x8 fa[FB][C::MB], fb[FB][NB];
  // Every operand block starts at a multiple of 16 rows, so the swizzled position of a
  // lane's chunk depends on the lane alone: one per-lane offset per K sub-step, plus a
  // wave-uniform part, plus a compile-time part that fits the ds_read offset field.
  uint32_t lane_off[SUB], lane_off_b[SUB];
#pragma unroll
  for (int sub = 0; sub < SUB; ++sub) {
    lane_off[sub] = (uint32_t)swz<BK>(lane & 15, sub * 4 + (lane >> 4));
    // fp8 weights: 8 bytes (8 K values) per lane, half a 16-byte chunk of a 64-byte row
    lane_off_b[sub] = C::W8 ? (uint32_t)(swz<32>(lane & 15, sub * 2 + (lane >> 5)) + 8 * ((lane >> 4) & 1))
                            : lane_off[sub];
  }
  // Fragments of K sub-step `sub`: all NB operand blocks of B, and the first MBL
  // 16-row blocks of A (the blocks past MBL hold no valid row of the tile).
  auto read_frags = [&](auto mbl, int slot, int sub, int buf) {
    constexpr int MBL = decltype(mbl)::value;
    const uint32_t pa = lane_off[sub] + slot * C::STAGE + arow(0) * C::RB;
    const uint32_t pb = lane_off_b[sub] + slot * C::STAGE + C::A_BYTES + wn * WCOLS * C::RB_B;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if constexpr (C::W8) {
        // 8 fp8 values widened exactly to bf16 (scale 1; the row scale is applied to the
        // fp32 accumulators in the epilogue)
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        typedef __bf16 b16x2 __attribute__((ext_vector_type(2)));
        const u32x2 q = *(const u32x2*)(smem + pb + bconst(nb) * C::RB_B);
        const b16x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q.x, 1.0f, false);
        const b16x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q.x, 1.0f, true);
        const b16x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q.y, 1.0f, false);
        const b16x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(q.y, 1.0f, true);
        fb[buf][nb] = bf16x8{p0.x, p0.y, p1.x, p1.y, p2.x, p2.y, p3.x, p3.y};
      } else {
        fb[buf][nb] = as_bf16x8(*(const u32x4*)(smem + pb + bconst(nb) * C::RB));
      }
    }
#pragma unroll
    for (int mb = 0; mb < MBL; ++mb)
      fa[buf][mb] = as_bf16x8(*(const u32x4*)(smem + pa + mb * C::WM * 16 * C::RB));
  };
  // One K step on the first MBL row blocks of this wave.
  auto kstep = [&](auto mbl, int slot, f32x4 (&acc)[decltype(mbl)::value][NB]) {
    constexpr int MBL = decltype(mbl)::value;
    if (FB == 2) read_frags(mbl, slot, 0, 0);
#pragma unroll
    for (int sub = 0; sub < SUB; ++sub) {
      const int cur = (FB == 2) ? (sub & 1) : 0;
      if (FB == 2) {
        if (sub + 1 < SUB) read_frags(mbl, slot, sub + 1, (sub + 1) & 1);
      } else {
        read_frags(mbl, slot, sub, 0);
      }
#pragma unroll
      for (int mb = 0; mb < MBL; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[cur][mb], fb[cur][nb],
                                                               acc[mb][nb], 0, 0, 0);
      // single-buffered fragments: keep the next sub-step's reads below these MFMAs
      if (FB == 1) __builtin_amdgcn_sched_barrier(0);
    }
  };

  int gs = 0;  // global step index of the consumer (ring slot = gs % S)
  constexpr int VPR = NCOLS / 8;  // 16-byte vectors per output row
  // K loop and output of one tile for a wave whose valid row blocks all lie in its
  // first MBL blocks. The accumulators live only here, so the variants for fully and
  // partly filled tiles share no loop-carried registers. Every variant runs the same
  // sequence of barriers (one per K step, two per epilogue pass).
  auto tile_body = [&](auto mbl, const TileInfo& ct, int cnk, int mb_live, bool c_valid,
                       uint16_t* out, size_t ld, int width) {
    constexpr int MBL = decltype(mbl)::value;
    f32x4 acc[MBL][NB];
#pragma unroll
    for (int mb = 0; mb < MBL; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0, 0, 0, 0};
    for (int kc = 0; kc < cnk; ++kc, ++gs) {
      // this wave's copies of step gs are done (the S-2 younger steps, when they were
      // issued, may stay in flight) ...
      if (issued - 1 - gs >= S - 2)
        wait_vmcnt<(S - 2) * NDMA>();
      else
        wait_vmcnt<0>();
      // ... and every other wave's; every read of step gs-1 is finished
      barrier_raw();
      produce((gs + S - 1) % S);
      // straight-line MFMAs (rows past the valid count inside a live block are
      // computed but never stored; a wave with no valid row skips the step)
      if (mb_live > 0) kstep(mbl, gs % S, acc);
    }
    if (!c_valid) return;
    // Epilogue through the ring slot just consumed (younger slots hold the next
    // tile's operands in flight).
    uint16_t* so = (uint16_t*)(smem + ((gs - 1) % S) * C::STAGE);
    // fp8 weights: the per-row scales of this tile's expert (powers of two, so scaling
    // the fp32 accumulators equals multiplying by the dequantised weights)
    const float* sc = nullptr;
    if constexpr (C::W8) {
      const int rows_w = GATED ? 2 * width : width;
      sc = (ct.g < a.n_pub) ? (GATED ? a.w13_scale_pub : a.w2_scale_pub) + (size_t)ct.g * rows_w
                            : (GATED ? a.w13_scale_priv : a.w2_scale_priv) + (size_t)(ct.g - a.n_pub) * rows_w;
    }
    for (int pass = 0; pass < C::BM / ER; ++pass) {
      barrier_raw();  // the slot's previous contents are no longer read
#pragma unroll
      for (int mb = 0; mb < MBL; ++mb) {
        const int r0 = arow(mb);
        if (r0 / ER == pass && mb < mb_live) {
#pragma unroll
          for (int nb = 0; nb < NBO; ++nb) {
            float sg = 1.0f, su = 1.0f;
            if constexpr (C::W8) {
              const int col = min(ct.n0 + wn * WCOLS + nb * 16 + (lane & 15), width - 1);
              sg = sc[col];
              if (GATED) su = sc[width + col];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int r = r0 - pass * ER + (lane >> 4) * 4 + i;
              const int c = wn * WCOLS + nb * 16 + (lane & 15);
              const float v = GATED ? silu(acc[mb][nb][i] * sg) * (acc[mb][nb + NBO][i] * su)
                                    : acc[mb][nb][i] * sg;
              so[r * NCOLS + c] = (uint16_t)f32_to_bf16_rne(v);
              if constexpr (GATED && SAVE) {
                const int rt = r0 + (lane >> 4) * 4 + i;  // row within the tile
                const int col = ct.n0 + c;
                if (ct.g < E && rt < ct.rows && col < width) {
                  float* ab = a.ab_save + (size_t)(ct.base + rt) * (2 * width);
                  ab[col] = acc[mb][nb][i];
                  ab[width + col] = acc[mb][nb + NBO][i];
                }
              }
            }
          }
        }
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes landed
      barrier_raw();
      const int prow = min(ER, ct.rows - pass * ER);
      for (int i = tid; i < prow * VPR; i += C::THREADS) {
        const int r = i / VPR, v = i - r * VPR;
        const int c = ct.n0 + v * 8;
        if (c < width)
          *(u32x4*)(out + (size_t)(ct.base + pass * ER + r) * ld + c) = *(const u32x4*)(so + r * NCOLS + v * 8);
      }
    }
  };

  for (int ci = 0; ci < ntl; ++ci) {
    const TileInfo ct = tile_of(ci);
    const bool c_shared = ct.g >= E;
    const bool c_priv = !c_shared && ct.g >= a.n_pub;
    const int cI = c_shared ? a.Is : a.I;
    const int cnk = (GATED ? H : cI) / BK;
    const bool c_valid = !(c_priv && (a.w13_priv == nullptr || a.w2_priv == nullptr));
    // this wave's blocks j with a valid row (arow(j) < rows)
    const int nblk = (ct.rows + 15) / 16;
    const int mb_live = c_valid ? max(0, min(C::MB, (nblk - wm + C::WM - 1) / C::WM)) : 0;
    uint16_t* out;
    size_t ld;
    const int width = GATED ? cI : H;
    if (GATED) {
      out = (uint16_t*)(c_shared ? a.h_sh : a.h);
      ld = (size_t)cI;
    } else {
      out = (uint16_t*)(c_shared ? a.y_shared : a.y_perm);
      ld = (size_t)H;
    }
    // A partly filled tile (e.g. an expert with fewer rows than BM) runs the variant
    // that reads and multiplies only the first half of the wave's row blocks.
    if (C::HALF && C::MB >= 2 && mb_live <= C::MB / 2)
      tile_body(std::integral_constant<int, (C::MB >= 2 ? C::MB / 2 : C::MB)>{}, ct, cnk, mb_live,
                c_valid, out, ld, width);
    else
      tile_body(std::integral_constant<int, C::MB>{}, ct, cnk, mb_live, c_valid, out, ld, width);
    if (!c_valid && !GATED) {
      // private rows without private weights: not executed, not audited, y zeroed
      if (tid == 0 && a.dev_status) atomicOr(a.dev_status, PMPE_DEV_PRIV_WEIGHTS_MISSING);
      for (int i = tid; i < ct.rows * VPR; i += C::THREADS) {
        const int r = i / VPR, v = i - r * VPR;
        const int c = ct.n0 + v * 8;
        if (c < width) *(u32x4*)(out + (size_t)(ct.base + r) * ld + c) = u32x4{0, 0, 0, 0};
      }
    }
    // Execution audit: the first N tile of every executed private M tile counts its rows.
    if (!GATED && AUDIT && c_priv && c_valid && ct.n0 == 0) {
      for (int r = tid; r < ct.rows; r += C::THREADS) atomicAdd(&a.audit_rows[s_rt[ci % NRT][r]], 1u);
      if (ct.m0 == 0 && tid == 0 && a.audit_calls) atomicAdd(&a.audit_calls[ct.g - a.n_pub], 1u);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    barrier_raw();  // epilogue reads of the slot are done before it is refilled
  }
  wait_vmcnt<0>();  // no copy may still be writing LDS when the block exits
}

// ---------------------------------------------------------------------------
// Private-expert weight gradients: C[p] [M, N] = AT_p BT_p^T, K = private expert p's rows
// (padded to a multiple of 64 with zero rows), AT [M, P] and BT [N, P] K-contiguous. One
// block per (expert, N tile, M tile), consecutive indices on one XCD; the same 256 x 256 x 64
// tile, two-stage global->LDS copy ring, swizzle and MFMA fragments as the forward's
// prefill GEMM, fp32 results stored from the accumulators. An expert without rows gets
// zeros. The K order of every output element is fixed, so the result is deterministic.
// ---------------------------------------------------------------------------
template <class C>
__global__ __launch_bounds__(C::THREADS) void wgrad_kernel(WgradArgs a) {
  static_assert(C::STAGES == 2 && !C::W8 && C::BK == 64, "two stages of bf16 K steps of 64");
  __shared__ __attribute__((aligned(16))) unsigned char smem[C::LDS];
  __shared__ int s_k[2];
  constexpr int BK = C::BK, NB = C::BN / C::WN / 16, MB = C::MB, WCOLS = C::BN / C::WN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int uwave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = uwave / C::WN, wn = uwave % C::WN;
  const int mtiles = (a.M + C::BM - 1) / C::BM, ntiles = (a.N + C::BN - 1) / C::BN;
  const int total = a.n_priv * ntiles * mtiles;
  const int per = (int)gridDim.x >> 3;  // the grid is a multiple of 8
  const int L = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  if (L >= total) return;
  const int pe = L / (ntiles * mtiles), rem = L - pe * (ntiles * mtiles);
  const int nt = rem / mtiles, mt = rem - nt * mtiles;
  if (tid < 64) {  // padded offset and padded row count of expert pe
    int running = 0;
    for (int q0 = 0; q0 < pe; q0 += 64) {
      const int q = q0 + tid;
      running += wave_sum_int(q < pe ? (a.count[a.n_pub + q] + 63) / 64 * 64 : 0);
    }
    if (tid == 0) {
      s_k[0] = running;
      s_k[1] = (a.count[a.n_pub + pe] + 63) / 64 * 64;
    }
  }
  __syncthreads();
  const int po = s_k[0], nk = s_k[1] / BK;
  const int m0 = mt * C::BM, n0 = nt * C::BN;
  const int lrow = lane / C::CH, lphys = lane % C::CH;
  uint32_t offA[C::A_DMA], offB[C::B_DMA];
#pragma unroll
  for (int i = 0; i < C::A_DMA; ++i) {
    const int r = (uwave * C::A_DMA + i) * C::RPD + lrow;
    const int m = min(m0 + r, a.M - 1);  // rows past M reload row M-1 (never stored)
    offA[i] = ((uint32_t)m * (uint32_t)a.P + (uint32_t)po + (uint32_t)((lphys ^ (r & 7)) * 8)) * 2;
  }
#pragma unroll
  for (int i = 0; i < C::B_DMA; ++i) {
    const int r = (uwave * C::B_DMA + i) * C::RPD + lrow;
    const int n = min(n0 + r, a.N - 1);
    offB[i] = ((uint32_t)n * (uint32_t)a.P + (uint32_t)po + (uint32_t)((lphys ^ (r & 7)) * 8)) * 2;
  }
  const uint32_t lds0 = lds_addr(smem);
  auto issue = [&](int slot, int k0) {
    const uint32_t sa = __builtin_amdgcn_readfirstlane(lds0 + slot * C::STAGE);
    const uint32_t wa = sa + uwave * C::A_DMA * 1024, wb = sa + C::A_BYTES + uwave * C::B_DMA * 1024;
    const uint16_t* ba = a.AT + k0;
    const uint16_t* bb = a.BT + k0;
    Unroll<0, C::A_DMA>::run([&](auto i) { dma16s<i.value * 1024, false>(offA[i.value], ba, wa); });
    Unroll<0, C::B_DMA>::run([&](auto i) { dma16s<i.value * 1024, false>(offB[i.value], bb, wb); });
  };
  f32x4 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0, 0, 0, 0};
  uint32_t lane_off[BK / 32];
#pragma unroll
  for (int sub = 0; sub < BK / 32; ++sub) lane_off[sub] = (uint32_t)swz<BK>(lane & 15, sub * 4 + (lane >> 4));
  if (nk > 0) issue(0, 0);
  for (int kc = 0; kc < nk; ++kc) {
    wait_vmcnt<0>();  // this wave's copies of step kc landed ...
    barrier_raw();    // ... and every wave's; every read of step kc-1 is finished
    if (kc + 1 < nk) issue((kc + 1) & 1, (kc + 1) * BK);
    const int slot = kc & 1;
#pragma unroll
    for (int sub = 0; sub < BK / 32; ++sub) {
      bf16x8 fa[MB], fb[NB];
      const uint32_t pa = lane_off[sub] + slot * C::STAGE + wm * 16 * C::RB;
      const uint32_t pb = lane_off[sub] + slot * C::STAGE + C::A_BYTES + wn * WCOLS * C::RB;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) fb[nb] = as_bf16x8(*(const u32x4*)(smem + pb + nb * 16 * C::RB));
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) fa[mb] = as_bf16x8(*(const u32x4*)(smem + pa + mb * C::WM * 16 * C::RB));
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[mb], fb[nb], acc[mb][nb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // lane holds C[m = 4 (lane / 16) + i][n = lane % 16] of each 16 x 16 block
  float* cp = a.C + (size_t)pe * a.M * a.N;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + (mb * C::WM + wm) * 16 + (lane >> 4) * 4 + i;
      if (m >= a.M) continue;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int n = n0 + wn * WCOLS + nb * 16 + (lane & 15);
        if (n < a.N) cp[(size_t)m * a.N + n] = acc[mb][nb][i];
      }
    }
}

// ---------------------------------------------------------------------------
// fp32 path support: tile of F32_BM rows of one expert (same device-side lookup)
// ---------------------------------------------------------------------------
constexpr int F32_BM = 128;
constexpr int THREADS = 256;

struct Tile {
  int e;     // expert id, -1 for the shared group, -2 for no tile
  int m0;    // first row of the tile within the group
  int rows;  // valid rows (<= F32_BM)
  int base;  // first permuted row of the tile (shared group: first token)
};

__device__ Tile find_tile(const int32_t* count, const int32_t* offset, int E, int slot,
                          int* s_tile) {
  const int tid = threadIdx.x;
  if (tid < 64) {
    const int lane = tid;
    int running = 0;
    for (int e0 = 0; e0 < E; e0 += 64) {
      const int e = e0 + lane;
      const int c = (e < E) ? count[e] : 0;
      const int nt = (c + F32_BM - 1) / F32_BM;
      const int incl = wave_incl_scan(nt);
      const int excl = incl - nt;
      if (nt > 0 && slot >= running + excl && slot < running + incl) {
        s_tile[0] = e;
        s_tile[1] = (slot - running - excl) * F32_BM;
      }
      running += __shfl(incl, 63, 64);
      if (running > slot) break;
    }
    if (lane == 0 && running <= slot) s_tile[0] = -2;
  }
  __syncthreads();
  Tile t;
  t.e = s_tile[0];
  t.m0 = s_tile[1];
  if (t.e >= 0) {
    t.rows = min(F32_BM, count[t.e] - t.m0);
    t.base = offset[t.e] + t.m0;
  } else {
    t.rows = 0;
    t.base = 0;
  }
  return t;
}

// ---------------------------------------------------------------------------
// fp32 path (small layers): one thread per output element, fp32 dot products.
// ---------------------------------------------------------------------------
constexpr int F32_NT = 64;

__global__ __launch_bounds__(THREADS) void gemm1_f32_kernel(FfnArgs a, int shared_group) {
  __shared__ int s_tile[2];
  const int H = a.H;
  const int I = shared_group ? a.Is : a.I;
  const int n0 = blockIdx.x * F32_NT;
  Tile tile;
  const float* w13;
  if (shared_group) {
    tile.e = -1;
    tile.m0 = blockIdx.y * F32_BM;
    tile.rows = min(F32_BM, a.T - tile.m0);
    tile.base = tile.m0;
    w13 = (const float*)a.w13_sh;
  } else {
    tile = find_tile(a.count, a.offset, a.n_pub + a.n_priv, blockIdx.y, s_tile);
    if (tile.e < 0) return;
    if (tile.e < a.n_pub) {
      w13 = (const float*)a.w13_pub + (size_t)tile.e * 2 * I * H;
    } else {
      if (a.w13_priv == nullptr || a.w2_priv == nullptr) return;
      w13 = (const float*)a.w13_priv + (size_t)(tile.e - a.n_pub) * 2 * I * H;
    }
  }
  for (int idx = threadIdx.x; idx < tile.rows * F32_NT; idx += THREADS) {
    const int r = idx / F32_NT, c = n0 + idx % F32_NT;
    if (c >= I) continue;
    size_t xr;
    const float* xb;
    if (shared_group || !a.x_perm) {
      xb = (const float*)a.x;
      xr = shared_group ? (size_t)(tile.base + r) : (size_t)a.row_token[tile.base + r];
    } else {
      xb = (const float*)a.x_perm;
      xr = (size_t)(tile.base + r);
    }
    const float* xv = xb + xr * H;
    const float* wg = w13 + (size_t)c * H;
    const float* wu = w13 + (size_t)(I + c) * H;
    float g = 0.0f, u = 0.0f;
    for (int h = 0; h < H; ++h) {
      g = fmaf(xv[h], wg[h], g);
      u = fmaf(xv[h], wu[h], u);
    }
    float* hout = (float*)(shared_group ? a.h_sh : a.h);
    hout[(size_t)(tile.base + r) * I + c] = silu(g) * u;
  }
}

__global__ __launch_bounds__(THREADS) void gemm2_f32_kernel(FfnArgs a, int shared_group) {
  __shared__ int s_tile[2];
  const int H = a.H;
  const int I = shared_group ? a.Is : a.I;
  const int n0 = blockIdx.x * F32_NT;
  Tile tile;
  const float* w2;
  bool priv = false;
  if (shared_group) {
    tile.e = -1;
    tile.m0 = blockIdx.y * F32_BM;
    tile.rows = min(F32_BM, a.T - tile.m0);
    tile.base = tile.m0;
    w2 = (const float*)a.w2_sh;
  } else {
    tile = find_tile(a.count, a.offset, a.n_pub + a.n_priv, blockIdx.y, s_tile);
    if (tile.e < 0) return;
    if (tile.e < a.n_pub) {
      w2 = (const float*)a.w2_pub + (size_t)tile.e * H * I;
    } else {
      priv = true;
      if (a.w13_priv == nullptr || a.w2_priv == nullptr) {
        if (threadIdx.x == 0 && a.dev_status) atomicOr(a.dev_status, PMPE_DEV_PRIV_WEIGHTS_MISSING);
        float* y = (float*)a.y_perm;
        for (int idx = threadIdx.x; idx < tile.rows * F32_NT; idx += THREADS) {
          const int r = idx / F32_NT, c = n0 + idx % F32_NT;
          if (c < H) y[(size_t)(tile.base + r) * H + c] = 0.0f;
        }
        return;
      }
      w2 = (const float*)a.w2_priv + (size_t)(tile.e - a.n_pub) * H * I;
    }
  }
  const float* hin = (const float*)(shared_group ? a.h_sh : a.h);
  float* y = (float*)(shared_group ? a.y_shared : a.y_perm);
  for (int idx = threadIdx.x; idx < tile.rows * F32_NT; idx += THREADS) {
    const int r = idx / F32_NT, c = n0 + idx % F32_NT;
    if (c >= H) continue;
    const float* hv = hin + (size_t)(tile.base + r) * I;
    const float* wv = w2 + (size_t)c * I;
    float acc = 0.0f;
    for (int i = 0; i < I; ++i) acc = fmaf(hv[i], wv[i], acc);
    y[(size_t)(tile.base + r) * H + c] = acc;
  }
  if (priv && blockIdx.x == 0) {
    for (int r = threadIdx.x; r < tile.rows; r += THREADS) atomicAdd(&a.audit_rows[a.row_token[tile.base + r]], 1u);
    if (tile.m0 == 0 && threadIdx.x == 0 && a.audit_calls) atomicAdd(&a.audit_calls[tile.e - a.n_pub], 1u);
  }
}

}  // namespace

hipError_t launch_expert_ffn(const FfnArgs& a, hipStream_t s) { return launch_expert_ffn_parts(a, s, 3); }

// fp8 expert weights (routed experts only, no shared group): the same two GEMMs.
hipError_t launch_expert_ffn_fp8(const FfnArgs& a, hipStream_t s) {
  const int E = a.n_pub + a.n_priv;
  int dev = 0, ncu = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) ncu = v;
  }
  const bool large = (int64_t)a.T * a.k >= (int64_t)128 * E;
  auto run = [&](auto cfg) {
    using C = decltype(cfg);
    auto grid = [&](int ncols, bool gemm1) {
      const int64_t w = gemm1 ? a.I : a.H;
      int64_t tiles = ((int64_t)a.T * a.k / C::BM + E) * ((w + ncols - 1) / ncols);
      int64_t g = (int64_t)ncu * C::PER_CU;
      if (tiles < g) g = (tiles + 7) / 8 * 8;
      return dim3((unsigned)g);
    };
    hipLaunchKernelGGL((gemm_bf16_kernel<C, true>), grid(C::BN / 2, true), dim3(C::THREADS), 0, s, a);
    hipLaunchKernelGGL((gemm_bf16_kernel<C, false>), grid(C::BN, false), dim3(C::THREADS), 0, s, a);
  };
  if (large)
    run(CfgLarge8{});
  else
    run(CfgSmall8{});
  return hipGetLastError();
}

hipError_t launch_wgrad(const WgradArgs& a, hipStream_t s) {
  using C = Cfg<256, 256, 4, 2, 2, 64>;
  const int64_t total = (int64_t)a.n_priv * ((a.M + C::BM - 1) / C::BM) * ((a.N + C::BN - 1) / C::BN);
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(wgrad_kernel<C>, dim3((unsigned)((total + 7) / 8 * 8)), dim3(C::THREADS), 0, s, a);
  return hipGetLastError();
}

// The GEMM2 kernel as a plain grouped product without the audit: y[r] = h[r] W_g^T for the
// rows of every routed group g, W_g [H, I] (K = I contiguous), bf16 in and out. With
// a.gather_a, row r of the product reads x[row_token[r]] (x [T, I]) instead of h[r].
hipError_t launch_grouped_nt_gemm(const FfnArgs& a, hipStream_t s) {
  const int E = a.n_pub + a.n_priv;
  int dev = 0, ncu = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) ncu = v;
  }
  const bool large = (int64_t)a.T * a.k >= (int64_t)128 * E;
  auto run = [&](auto cfg) {
    using C = decltype(cfg);
    int64_t tiles = ((int64_t)a.T * a.k / C::BM + E) * ((a.H + C::BN - 1) / C::BN);
    int64_t g = (int64_t)ncu * C::PER_CU;
    if (tiles < g) g = (tiles + 7) / 8 * 8;
    if (a.gather_a)
      hipLaunchKernelGGL((gemm_bf16_kernel<C, false, false, false, true>), dim3((unsigned)g), dim3(C::THREADS), 0, s, a);
    else
      hipLaunchKernelGGL((gemm_bf16_kernel<C, false, false, false>), dim3((unsigned)g), dim3(C::THREADS), 0, s, a);
  };
  if (large)
    run(CfgLarge{});
  else
    run(CfgSmall{});
  return hipGetLastError();
}

// parts: bit 0 runs GEMM1 (x -> h), bit 1 runs GEMM2 (h -> y)
hipError_t launch_expert_ffn_parts(const FfnArgs& a, hipStream_t s, int parts) {
  const int E = a.n_pub + a.n_priv;
  if (a.act_bf16) {
    // Average rows per routed expert picks the tile shape.
    const bool large = (int64_t)a.T * a.k >= (int64_t)128 * E;
    int dev = 0, ncu = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
      int v = 0;
      if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) ncu = v;
    }
    // Persistent grid: blocks resident at once (a multiple of the 8 XCDs), never more
    // than the tiles there can be.
    auto grid = [&](int BMv, int ncols, bool gemm1, int per_cu) {
      const int64_t w = gemm1 ? a.I : a.H;
      int64_t tiles = ((int64_t)a.T * a.k / BMv + E) * ((w + ncols - 1) / ncols);
      if (a.Is > 0) {
        const int64_t ws = gemm1 ? a.Is : a.H;
        tiles += ((a.T + BMv - 1) / BMv) * ((ws + ncols - 1) / ncols);
      }
      int64_t g = (int64_t)ncu * per_cu;
      if (tiles < g) g = (tiles + 7) / 8 * 8;
      return dim3((unsigned)g);
    };
    if (large) {
      using C = CfgLarge;
      if ((parts & 1) && a.ab_save)
        hipLaunchKernelGGL((gemm_bf16_kernel<C, true, true>), grid(C::BM, C::BN / 2, true, C::PER_CU), dim3(C::THREADS), 0, s, a);
      else if (parts & 1)
        hipLaunchKernelGGL((gemm_bf16_kernel<C, true>), grid(C::BM, C::BN / 2, true, C::PER_CU), dim3(C::THREADS), 0, s, a);
      if (parts & 2)
        hipLaunchKernelGGL((gemm_bf16_kernel<C, false>), grid(C::BM, C::BN, false, C::PER_CU), dim3(C::THREADS), 0, s, a);
    } else {
      using C = CfgSmall;
      if ((parts & 1) && a.ab_save)
        hipLaunchKernelGGL((gemm_bf16_kernel<C, true, true>), grid(C::BM, C::BN / 2, true, C::PER_CU), dim3(C::THREADS), 0, s, a);
      else if (parts & 1)
        hipLaunchKernelGGL((gemm_bf16_kernel<C, true>), grid(C::BM, C::BN / 2, true, C::PER_CU), dim3(C::THREADS), 0, s, a);
      if (parts & 2)
        hipLaunchKernelGGL((gemm_bf16_kernel<C, false>), grid(C::BM, C::BN, false, C::PER_CU), dim3(C::THREADS), 0, s, a);
    }
  } else {
    const int m_slots = (a.T * a.k + F32_BM - 1) / F32_BM + E;
    const int sh_slots = (a.T + F32_BM - 1) / F32_BM;
    if (parts & 1) {
      hipLaunchKernelGGL(gemm1_f32_kernel, dim3((a.I + F32_NT - 1) / F32_NT, m_slots), dim3(THREADS), 0, s, a, 0);
      if (a.Is > 0)
        hipLaunchKernelGGL(gemm1_f32_kernel, dim3((a.Is + F32_NT - 1) / F32_NT, sh_slots), dim3(THREADS), 0, s, a, 1);
    }
    if (parts & 2) {
      hipLaunchKernelGGL(gemm2_f32_kernel, dim3((a.H + F32_NT - 1) / F32_NT, m_slots), dim3(THREADS), 0, s, a, 0);
      if (a.Is > 0)
        hipLaunchKernelGGL(gemm2_f32_kernel, dim3((a.H + F32_NT - 1) / F32_NT, sh_slots), dim3(THREADS), 0, s, a, 1);
    }
  }
  return hipGetLastError();
}

}  // namespace pmpe
