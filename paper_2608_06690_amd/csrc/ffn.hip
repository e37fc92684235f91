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
// round-robin) works on one contiguous range of that order and its L2 holds the
// shared operands.
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
// are in flight while one is multiplied; the 16-byte chunks of each LDS row are
// XOR-swizzled by row so that MFMA operand reads do not conflict on banks. Rows past a tile's valid count are loaded from a valid
// row (their results are never stored), and MFMAs of 16-row blocks that hold no
// valid row are skipped. The output tile goes through LDS so that global stores are
// whole 16-byte vectors.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

typedef __attribute__((address_space(3))) unsigned char lds_u8;

// 32-bit LDS address of a shared-memory pointer.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const lds_u8*)p;
}

// Global -> LDS copy of 16 bytes per lane: lane l's bytes land at lds_base + 16 * l
// (lds_base is wave-uniform, held in M0). Written as inline assembly so that the
// compiler does not treat the copy as a pending LDS write that every later LDS read
// must wait for; the kernel waits for its own copies explicitly (wait_vmcnt) before
// a barrier and only then reads the stage they filled.
__device__ __forceinline__ void dma16(const void* src, uint32_t lds_base) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off" ::"v"(src),
      "s"(lds_base)
      : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier without the full memory drain that __syncthreads() implies: the
// copies a stage depends on were already waited for (wait_vmcnt), and every LDS read
// of the previous stage was consumed by an MFMA before this point. Later stages'
// copies stay in flight across it.
__device__ __forceinline__ void barrier_raw() { asm volatile("s_barrier" ::: "memory"); }

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

template <int BM_, int BN_, int WM_, int WN_, int STAGES_, int BK_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, STAGES = STAGES_, BK = BK_;
  static constexpr int RB = 2 * BK, CH = BK / 8, RPD = 1024 / RB;  // rows per DMA instruction
  static constexpr int WAVES = WM * WN, THREADS = 64 * WAVES;
  static constexpr int A_BYTES = BM * RB, B_BYTES = BN * RB, STAGE = A_BYTES + B_BYTES;
  static constexpr int A_DMA = BM / RPD / WAVES, B_DMA = BN / RPD / WAVES;  // per wave per stage
  static constexpr int WROWS = BM / WM, MB = WROWS / 16;
  static constexpr int LDS = STAGES * STAGE;
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(A_DMA * RPD * WAVES == BM && B_DMA * RPD * WAVES == BN, "DMA split");
};
#ifndef PMPE_CFG_LARGE
#define PMPE_CFG_LARGE 256, 256, 4, 2, 2, 64
#endif
#ifndef PMPE_CFG_SMALL
#define PMPE_CFG_SMALL 64, 128, 1, 4, 3, 64
#endif
using CfgLarge = Cfg<PMPE_CFG_LARGE>;  // prefill: 8 waves, 2 x 64 KiB stages
using CfgSmall = Cfg<PMPE_CFG_SMALL>;  // decode-shaped: 4 waves, 3 x 24 KiB stages

struct GTile {
  int g;     // group: expert id, or E for the shared group; -1: no tile
  int m0;    // first row of the tile within the group
  int n0;    // first output column (GEMM1: h column; GEMM2: y column)
  int rows;  // valid rows
  int base;  // first row of the tile in the group's row space (permuted row / token)
};

// Block-uniform tile lookup. ncols = output columns per N tile.
__device__ GTile lookup_tile(const FfnArgs& a, bool gemm1, int BMv, int ncols, int* s_cum) {
  const int E = a.n_pub + a.n_priv;
  const int ngroups = E + (a.Is > 0 ? 1 : 0);
  const int tid = threadIdx.x;
  if (tid < 64) {
    int running = 0;
    for (int g0 = 0; g0 < ngroups; g0 += 64) {
      const int g = g0 + tid;
      int nt = 0;
      if (g < ngroups) {
        const int cnt = (g < E) ? a.count[g] : a.T;
        const int width = gemm1 ? ((g < E) ? a.I : a.Is) : a.H;
        nt = ((cnt + BMv - 1) / BMv) * ((width + ncols - 1) / ncols);
      }
      const int incl = wave_incl_scan(nt);
      if (g < ngroups) s_cum[g + 1] = running + incl;
      running += __shfl(incl, 63, 64);
    }
    if (tid == 0) s_cum[0] = 0;
  }
  __syncthreads();
  GTile t;
  t.g = -1;
  const int total = s_cum[ngroups];
  const int b = blockIdx.x;
  if (b >= total) return t;
  // XCD-aware order: XCD x = b % 8 takes a contiguous range of the tile order
  const int x = b & 7, j = b >> 3;
  const int L = x * (total >> 3) + min(x, total & 7) + j;
  int lo = 0, hi = ngroups - 1;  // last g with s_cum[g] <= L
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_cum[mid] <= L) lo = mid; else hi = mid - 1;
  }
  const int g = lo;
  const int cnt = (g < E) ? a.count[g] : a.T;
  const int mt = (cnt + BMv - 1) / BMv;
  const int local = L - s_cum[g];
  const int n = local / mt, m = local - n * mt;
  t.g = g;
  t.m0 = m * BMv;
  t.n0 = n * ncols;
  t.rows = min(BMv, cnt - t.m0);
  t.base = ((g < E) ? a.offset[g] : 0) + t.m0;
  return t;
}

// One bf16 GEMM tile. GATED: GEMM1 (x -> h with SwiGLU); else GEMM2 (h -> y).
template <class C, bool GATED>
__global__ __launch_bounds__(C::THREADS) void gemm_bf16_kernel(FfnArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[C::LDS];
  __shared__ int s_cum[2 * PMPE_MAX_POOL + 2];
  constexpr int NCOLS = GATED ? C::BN / 2 : C::BN;  // output columns per tile
  constexpr int WCOLS = NCOLS / C::WN;               // output columns per wave
  constexpr int NBO = WCOLS / 16;                    // output 16-col blocks per wave
  constexpr int NB = GATED ? 2 * NBO : NBO;          // B operand blocks per wave
  static_assert(C::BM * NCOLS * 2 <= C::LDS, "output tile must fit the LDS ring");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  const int E = a.n_pub + a.n_priv;

  const GTile t = lookup_tile(a, GATED, C::BM, NCOLS, s_cum);
  if (t.g < 0) return;
  const bool shared = t.g >= E;
  const bool priv = !shared && t.g >= a.n_pub;
  const int I = shared ? a.Is : a.I;
  const int H = a.H;
  const int K = GATED ? H : I;
  const int width = GATED ? I : H;  // valid output columns

  const uint16_t* w;
  if (shared) {
    w = (const uint16_t*)(GATED ? a.w13_sh : a.w2_sh);
  } else if (!priv) {
    w = (const uint16_t*)(GATED ? a.w13_pub : a.w2_pub) + (size_t)t.g * 2 * I * H / (GATED ? 1 : 2);
  } else {
    if (a.w13_priv == nullptr || a.w2_priv == nullptr) {
      if (!GATED) {
        // private rows without private weights: not executed, not audited, y zeroed
        if (tid == 0 && a.dev_status) atomicOr(a.dev_status, PMPE_DEV_PRIV_WEIGHTS_MISSING);
        uint16_t* y = (uint16_t*)a.y_perm;
        for (int i = tid; i < t.rows * NCOLS; i += C::THREADS) {
          const int r = i / NCOLS, c = t.n0 + i % NCOLS;
          if (c < width) y[(size_t)(t.base + r) * H + c] = 0;
        }
      }
      return;
    }
    w = (const uint16_t*)(GATED ? a.w13_priv : a.w2_priv) +
        (size_t)(t.g - a.n_pub) * 2 * I * H / (GATED ? 1 : 2);
  }

  // Per-lane source rows of this wave's DMA instructions. DMA instruction i of wave
  // `wave` fills the RPD operand rows r0 = (wave * n + i) * RPD ..; lane l writes LDS
  // chunk (row r0 + l / CH, physical chunk l % CH), which holds the logical chunk whose
  // swizzled position that is.
  constexpr int BK = C::BK;
  const int lrow = lane / C::CH, lphys = lane % C::CH;
  auto logical = [&](int r) { return (BK == 64) ? (lphys ^ (r & 7)) : (lphys ^ ((r >> 1) & 3)); };
  const uint16_t* srcA[C::A_DMA];
  const uint16_t* srcB[C::B_DMA];
#pragma unroll
  for (int i = 0; i < C::A_DMA; ++i) {
    const int r = (wave * C::A_DMA + i) * C::RPD + lrow;
    const int rr = min(r, t.rows - 1);  // rows past the valid count reload a valid row
    const int c = logical(r);
    const uint16_t* row;
    if (GATED) {
      if (shared)
        row = (const uint16_t*)a.x + (size_t)(t.base + rr) * H;
      else if (a.x_perm)
        row = (const uint16_t*)a.x_perm + (size_t)(t.base + rr) * H;
      else
        row = (const uint16_t*)a.x + (size_t)a.row_token[t.base + rr] * H;
    } else {
      row = (const uint16_t*)(shared ? a.h_sh : a.h) + (size_t)(t.base + rr) * I;
    }
    srcA[i] = row + c * 8;
  }
#pragma unroll
  for (int i = 0; i < C::B_DMA; ++i) {
    const int r = (wave * C::B_DMA + i) * C::RPD + lrow;
    const int c = logical(r);
    int wrow;
    if (GATED) {
      const int half = C::BN / 2;
      const int j = (r < half) ? r : r - half;
      const int col = min(t.n0 + j, I - 1);
      wrow = (r < half) ? col : I + col;
    } else {
      wrow = min(t.n0 + r, H - 1);
    }
    srcB[i] = w + (size_t)wrow * K + c * 8;
  }

  const uint32_t lds0 = lds_addr(smem);
  const int uwave = __builtin_amdgcn_readfirstlane(wave);  // wave index as a scalar
  auto issue = [&](int stage, int k0) {
    const uint32_t sa = lds0 + stage * C::STAGE;
    const uint32_t sb = sa + C::A_BYTES;
#pragma unroll
    for (int i = 0; i < C::A_DMA; ++i) dma16(srcA[i] + k0, sa + (uwave * C::A_DMA + i) * 1024);
#pragma unroll
    for (int i = 0; i < C::B_DMA; ++i) dma16(srcB[i] + k0, sb + (uwave * C::B_DMA + i) * 1024);
  };

  f32x4 acc[C::MB][NB];
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0, 0, 0, 0};

  // 16-row blocks of this wave that hold at least one valid row
  const int wrow0 = wm * C::WROWS;
  const int mb_live = max(0, min(C::MB, (t.rows - wrow0 + 15) / 16));

  // B operand row (within the tile) of this wave's block nb, for lane row l16
  auto brow = [&](int nb) {
    if (GATED) {
      const int half = C::BN / 2;
      return (nb < NBO) ? wn * WCOLS + nb * 16 : half + wn * WCOLS + (nb - NBO) * 16;
    }
    return wn * WCOLS + nb * 16;
  };

  const int nk = K / BK;
#pragma unroll
  for (int s = 0; s < C::STAGES - 1; ++s)
    if (s < nk) issue(s, s * BK);

  constexpr int SUB = BK / 32;  // MFMA K steps per stage
  bf16x8 fa[2][C::MB], fb[2][NB];
  auto read_frags = [&](const unsigned char* sa, const unsigned char* sb, int sub, int buf) {
    const int ch = sub * 4 + (lane >> 4);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      fb[buf][nb] = as_bf16x8(*(const u32x4*)(sb + swz<BK>(brow(nb) + (lane & 15), ch)));
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
      fa[buf][mb] = as_bf16x8(*(const u32x4*)(sa + swz<BK>(wrow0 + mb * 16 + (lane & 15), ch)));
  };

  for (int kc = 0; kc < nk; ++kc) {
    // this wave's copies of stage kc are done (later stages may stay in flight) ...
    if (kc + C::STAGES - 2 < nk) {
      wait_vmcnt<(C::STAGES - 2) * (C::A_DMA + C::B_DMA)>();
    } else {
      wait_vmcnt<0>();
    }
    // ... and so are every other wave's; all reads of stage kc-1 are finished
    barrier_raw();
    if (kc + C::STAGES - 1 < nk) issue((kc + C::STAGES - 1) % C::STAGES, (kc + C::STAGES - 1) * BK);
    if (mb_live > 0) {
      const unsigned char* sa = smem + (kc % C::STAGES) * C::STAGE;
      const unsigned char* sb = sa + C::A_BYTES;
      read_frags(sa, sb, 0, 0);
#pragma unroll
      for (int sub = 0; sub < SUB; ++sub) {
        if (sub + 1 < SUB) read_frags(sa, sb, sub + 1, (sub + 1) & 1);
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb) {
          if (mb < mb_live) {
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
              acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[sub & 1][mb], fb[sub & 1][nb],
                                                                   acc[mb][nb], 0, 0, 0);
          }
        }
      }
    }
  }
  __syncthreads();  // all MFMA reads of LDS done: reuse it for the output tile

  // Output tile [BM][NCOLS] bf16 in LDS, then 16-byte stores of the valid part.
  uint16_t* so = (uint16_t*)smem;
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBO; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wrow0 + mb * 16 + (lane >> 4) * 4 + i;
        const int c = wn * WCOLS + nb * 16 + (lane & 15);
        float v;
        if (GATED)
          v = silu(acc[mb][nb][i]) * acc[mb][nb + NBO][i];
        else
          v = acc[mb][nb][i];
        so[r * NCOLS + c] = (uint16_t)f32_to_bf16_rne(v);
      }
  __syncthreads();
  uint16_t* out;
  size_t ld;
  if (GATED) {
    out = (uint16_t*)(shared ? a.h_sh : a.h);
    ld = (size_t)I;
  } else {
    out = (uint16_t*)(shared ? a.y_shared : a.y_perm);
    ld = (size_t)H;
  }
  constexpr int VPR = NCOLS / 8;  // 16-byte vectors per output row
  for (int i = tid; i < t.rows * VPR; i += C::THREADS) {
    const int r = i / VPR, v = i - r * VPR;
    const int c = t.n0 + v * 8;
    if (c < width) *(u32x4*)(out + (size_t)(t.base + r) * ld + c) = *(const u32x4*)(so + r * NCOLS + v * 8);
  }

  // Execution audit: the first N tile of every private M tile counts its rows once.
  if (!GATED && priv && t.n0 == 0) {
    for (int r = tid; r < t.rows; r += C::THREADS) atomicAdd(&a.audit_rows[a.row_token[t.base + r]], 1u);
    if (t.m0 == 0 && tid == 0 && a.audit_calls) atomicAdd(&a.audit_calls[t.g - a.n_pub], 1u);
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

hipError_t launch_expert_ffn(const FfnArgs& a, hipStream_t s) {
  const int E = a.n_pub + a.n_priv;
  if (a.act_bf16) {
    // Average rows per routed expert picks the tile shape.
    const bool large = (int64_t)a.T * a.k >= (int64_t)128 * E;
    auto grid = [&](int BMv, int ncols, bool gemm1) {
      const int64_t w = gemm1 ? a.I : a.H;
      int64_t tiles = ((int64_t)a.T * a.k / BMv + E) * ((w + ncols - 1) / ncols);
      if (a.Is > 0) {
        const int64_t ws = gemm1 ? a.Is : a.H;
        tiles += ((a.T + BMv - 1) / BMv) * ((ws + ncols - 1) / ncols);
      }
      return dim3((unsigned)tiles);
    };
    if (large) {
      using C = CfgLarge;
      hipLaunchKernelGGL((gemm_bf16_kernel<C, true>), grid(C::BM, C::BN / 2, true), dim3(C::THREADS), 0, s, a);
      hipLaunchKernelGGL((gemm_bf16_kernel<C, false>), grid(C::BM, C::BN, false), dim3(C::THREADS), 0, s, a);
    } else {
      using C = CfgSmall;
      hipLaunchKernelGGL((gemm_bf16_kernel<C, true>), grid(C::BM, C::BN / 2, true), dim3(C::THREADS), 0, s, a);
      hipLaunchKernelGGL((gemm_bf16_kernel<C, false>), grid(C::BM, C::BN, false), dim3(C::THREADS), 0, s, a);
    }
  } else {
    const int m_slots = (a.T * a.k + F32_BM - 1) / F32_BM + E;
    const int sh_slots = (a.T + F32_BM - 1) / F32_BM;
    hipLaunchKernelGGL(gemm1_f32_kernel, dim3((a.I + F32_NT - 1) / F32_NT, m_slots), dim3(THREADS), 0, s, a, 0);
    if (a.Is > 0)
      hipLaunchKernelGGL(gemm1_f32_kernel, dim3((a.Is + F32_NT - 1) / F32_NT, sh_slots), dim3(THREADS), 0, s, a, 1);
    hipLaunchKernelGGL(gemm2_f32_kernel, dim3((a.H + F32_NT - 1) / F32_NT, m_slots), dim3(THREADS), 0, s, a, 0);
    if (a.Is > 0)
      hipLaunchKernelGGL(gemm2_f32_kernel, dim3((a.H + F32_NT - 1) / F32_NT, sh_slots), dim3(THREADS), 0, s, a, 1);
  }
  return hipGetLastError();
}

}  // namespace pmpe
