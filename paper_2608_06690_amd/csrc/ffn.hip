// K3 - expert FFN: grouped SwiGLU GEMM over the experts that have rows, with the
// private-row execution audit written by the blocks that execute the rows.
//
// Expert e owns permuted rows [offset[e], offset[e] + count[e]). A tile is (expert,
// 128-row M tile, N tile). Tile slots are numbered expert by expert, ceil(count/128)
// per expert, so a launch of ceil(T*k/128) + E slots covers every tile; each block
// finds its tile by a wave scan over the per-expert tile counts read on the device
// (no host synchronisation, experts with zero rows get no tile and load nothing).
//
//   GEMM1  [rows, H] x [H, 2I]: the N tile is 64 gate columns plus the matching 64 up
//          columns, so the SwiGLU h = silu(g) * u is formed in registers and stored as
//          act_dtype h [T*k, I] in the workspace.
//   GEMM2  [rows, I] x [I, H]: N tile of 128 output columns -> y_perm.
//
// bf16 tiles: 256 threads = 4 waves in a 2 x 2 layout, v_mfma_f32_16x16x32_bf16,
// K step 64, A and B tiles staged in LDS (double buffered; the next K step's global
// loads are issued before the current step's MFMAs), 16-byte chunks XOR-swizzled by
// row so that 16 lanes reading 16 rows hit distinct banks. fp32 is accumulated, h and
// y are rounded once to bf16 (round to nearest even).
//
// The shared experts (always on, independent of the policy) run through the same
// kernels as one more group whose rows are all T tokens.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int BM = 128;
constexpr int BK = 64;
constexpr int NT1 = 64;   // GEMM1: h columns per tile (64 gate + 64 up weight rows)
constexpr int NT2 = 128;  // GEMM2: output columns per tile
constexpr int THREADS = 256;

struct Tile {
  int e;     // expert id, -1 for the shared group, -2 for no tile
  int m0;    // first row of the tile within the group
  int rows;  // valid rows (<= BM)
  int base;  // first permuted row of the tile (shared group: first token)
};

// Block-uniform lookup of the tile of slot `slot` (wave 0 scans, result via LDS).
__device__ Tile find_tile(const int32_t* count, const int32_t* offset, int E, int slot,
                          int* s_tile) {
  const int tid = threadIdx.x;
  if (tid < 64) {
    const int lane = tid;
    int running = 0;
    for (int e0 = 0; e0 < E; e0 += 64) {
      const int e = e0 + lane;
      const int c = (e < E) ? count[e] : 0;
      const int nt = (c + BM - 1) / BM;
      const int incl = wave_incl_scan(nt);
      const int excl = incl - nt;
      if (nt > 0 && slot >= running + excl && slot < running + incl) {
        s_tile[0] = e;
        s_tile[1] = (slot - running - excl) * BM;
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
    t.rows = min(BM, count[t.e] - t.m0);
    t.base = offset[t.e] + t.m0;
  } else {
    t.rows = 0;
    t.base = 0;
  }
  return t;
}

// LDS tile of R rows x 64 bf16 (128 bytes per row, eight 16-byte chunks, swizzled).
template <int R>
struct LdsTile {
  u32x4 v[R * 8];
  __device__ __forceinline__ u32x4& at(int row, int chunk) { return v[row * 8 + (chunk ^ (row & 7))]; }
};

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) { return *(const u32x4*)p; }

// ---------------------------------------------------------------------------
// bf16 GEMM1 (+ SwiGLU)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(THREADS) void gemm1_bf16_kernel(FfnArgs a, int shared_group) {
  __shared__ LdsTile<BM> sA[2];
  __shared__ LdsTile<2 * NT1> sB[2];
  __shared__ int s_tile[2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int H = a.H;
  const int I = shared_group ? a.Is : a.I;
  const int n0 = blockIdx.x * NT1;

  Tile tile;
  const uint16_t* w13;
  if (shared_group) {
    tile.e = -1;
    tile.m0 = blockIdx.y * BM;
    tile.rows = min(BM, a.T - tile.m0);
    tile.base = tile.m0;
    w13 = (const uint16_t*)a.w13_sh;
  } else {
    tile = find_tile(a.count, a.offset, a.n_pub + a.n_priv, blockIdx.y, s_tile);
    if (tile.e < 0) return;
    if (tile.e < a.n_pub) {
      w13 = (const uint16_t*)a.w13_pub + (size_t)tile.e * 2 * I * H;
    } else {
      if (a.w13_priv == nullptr || a.w2_priv == nullptr) return;  // reported by GEMM2
      w13 = (const uint16_t*)a.w13_priv + (size_t)(tile.e - a.n_pub) * 2 * I * H;
    }
  }
  if (tile.rows <= 0) return;

  // Global source rows of this thread's four A chunks and four B chunks.
  const int lrow = tid >> 3;  // 0..31
  const int lch = tid & 7;
  const uint16_t* srcA[4];
  const uint16_t* srcB[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lrow + 32 * i;
    if (r < tile.rows) {
      size_t xr;
      if (shared_group)
        xr = (size_t)(tile.base + r);
      else if (a.x_perm)
        xr = (size_t)(tile.base + r);
      else
        xr = (size_t)a.row_token[tile.base + r];
      const uint16_t* xb = (const uint16_t*)((shared_group || !a.x_perm) ? a.x : a.x_perm);
      srcA[i] = xb + xr * H + lch * 8;
    } else {
      srcA[i] = nullptr;
    }
    const int br = lrow + 32 * i;  // 0..127: gate rows then up rows
    const int wrow = (br < NT1) ? (n0 + br) : (I + n0 + br - NT1);
    srcB[i] = w13 + (size_t)wrow * H + lch * 8;
  }

  u32x4 ra[4], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = srcA[i] ? ld16(srcA[i] + k0) : u32x4{0, 0, 0, 0};
      rb[i] = ld16(srcB[i] + k0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sA[buf].at(lrow + 32 * i, lch) = ra[i];
      sB[buf].at(lrow + 32 * i, lch) = rb[i];
    }
  };

  f32x4 accG[4][2], accU[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      accG[mb][nb] = f32x4{0, 0, 0, 0};
      accU[mb][nb] = f32x4{0, 0, 0, 0};
    }

  const int nk = H / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int buf = kc & 1;
    if (kc + 1 < nk) gload((kc + 1) * BK);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int ch = s * 4 + (lane >> 4);
      bf16x8 fa[4], fg[2], fu[2];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) fa[mb] = as_bf16x8(sA[buf].at(wm * 64 + mb * 16 + (lane & 15), ch));
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        fg[nb] = as_bf16x8(sB[buf].at(wn * 32 + nb * 16 + (lane & 15), ch));
        fu[nb] = as_bf16x8(sB[buf].at(NT1 + wn * 32 + nb * 16 + (lane & 15), ch));
      }
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          accG[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[mb], fg[nb], accG[mb][nb], 0, 0, 0);
          accU[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[mb], fu[nb], accU[mb][nb], 0, 0, 0);
        }
    }
    if (kc + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: h = silu(g) * u, rounded to bf16.
  uint16_t* hout = (uint16_t*)(shared_group ? a.h_sh : a.h);
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * 64 + mb * 16 + (lane >> 4) * 4 + i;
        const int col = n0 + wn * 32 + nb * 16 + (lane & 15);
        if (r < tile.rows) {
          const float hv = silu(accG[mb][nb][i]) * accU[mb][nb][i];
          hout[(size_t)(tile.base + r) * I + col] = (uint16_t)f32_to_bf16_rne(hv);
        }
      }
}

// ---------------------------------------------------------------------------
// bf16 GEMM2 (down projection) + audit
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(THREADS) void gemm2_bf16_kernel(FfnArgs a, int shared_group) {
  __shared__ LdsTile<BM> sA[2];
  __shared__ LdsTile<NT2> sB[2];
  __shared__ int s_tile[2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int H = a.H;
  const int I = shared_group ? a.Is : a.I;
  const int n0 = blockIdx.x * NT2;

  Tile tile;
  const uint16_t* w2;
  bool priv = false;
  if (shared_group) {
    tile.e = -1;
    tile.m0 = blockIdx.y * BM;
    tile.rows = min(BM, a.T - tile.m0);
    tile.base = tile.m0;
    w2 = (const uint16_t*)a.w2_sh;
  } else {
    tile = find_tile(a.count, a.offset, a.n_pub + a.n_priv, blockIdx.y, s_tile);
    if (tile.e < 0) return;
    if (tile.e < a.n_pub) {
      w2 = (const uint16_t*)a.w2_pub + (size_t)tile.e * H * I;
    } else {
      priv = true;
      if (a.w13_priv == nullptr || a.w2_priv == nullptr) {
        // Private rows without private weights: not executed, not audited, zeroed.
        if (tid == 0 && a.dev_status) atomicOr(a.dev_status, PMPE_DEV_PRIV_WEIGHTS_MISSING);
        uint16_t* y = (uint16_t*)a.y_perm;
        for (int idx = tid; idx < tile.rows * NT2; idx += THREADS) {
          const int r = idx / NT2, c = idx - r * NT2;
          y[(size_t)(tile.base + r) * H + n0 + c] = 0;
        }
        return;
      }
      w2 = (const uint16_t*)a.w2_priv + (size_t)(tile.e - a.n_pub) * H * I;
    }
  }
  if (tile.rows <= 0) return;

  const uint16_t* hin = (const uint16_t*)(shared_group ? a.h_sh : a.h);
  const int lrow = tid >> 3;
  const int lch = tid & 7;
  const uint16_t* srcA[4];
  const uint16_t* srcB[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lrow + 32 * i;
    srcA[i] = (r < tile.rows) ? hin + (size_t)(tile.base + r) * I + lch * 8 : nullptr;
    srcB[i] = w2 + (size_t)(n0 + r) * I + lch * 8;
  }
  u32x4 ra[4], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = srcA[i] ? ld16(srcA[i] + k0) : u32x4{0, 0, 0, 0};
      rb[i] = ld16(srcB[i] + k0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sA[buf].at(lrow + 32 * i, lch) = ra[i];
      sB[buf].at(lrow + 32 * i, lch) = rb[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x4{0, 0, 0, 0};

  const int nk = I / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int buf = kc & 1;
    if (kc + 1 < nk) gload((kc + 1) * BK);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int ch = s * 4 + (lane >> 4);
      bf16x8 fa[4], fb[4];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) fa[mb] = as_bf16x8(sA[buf].at(wm * 64 + mb * 16 + (lane & 15), ch));
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) fb[nb] = as_bf16x8(sB[buf].at(wn * 64 + nb * 16 + (lane & 15), ch));
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[mb], fb[nb], acc[mb][nb], 0, 0, 0);
    }
    if (kc + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  uint16_t* y = (uint16_t*)(shared_group ? a.y_shared : a.y_perm);
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * 64 + mb * 16 + (lane >> 4) * 4 + i;
        const int col = n0 + wn * 64 + nb * 16 + (lane & 15);
        if (r < tile.rows) y[(size_t)(tile.base + r) * H + col] = (uint16_t)f32_to_bf16_rne(acc[mb][nb][i]);
      }

  // Execution audit: the first N tile of each private tile counts its rows once.
  if (priv && blockIdx.x == 0) {
    for (int r = tid; r < tile.rows; r += THREADS) atomicAdd(&a.audit_rows[a.row_token[tile.base + r]], 1u);
    if (tile.m0 == 0 && tid == 0 && a.audit_calls) atomicAdd(&a.audit_calls[tile.e - a.n_pub], 1u);
  }
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
    tile.m0 = blockIdx.y * BM;
    tile.rows = min(BM, a.T - tile.m0);
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
    tile.m0 = blockIdx.y * BM;
    tile.rows = min(BM, a.T - tile.m0);
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
  const int m_slots = (a.T * a.k + BM - 1) / BM + E;
  const int sh_slots = (a.T + BM - 1) / BM;
  if (a.act_bf16) {
    hipLaunchKernelGGL(gemm1_bf16_kernel, dim3(a.I / NT1, m_slots), dim3(THREADS), 0, s, a, 0);
    if (a.Is > 0)
      hipLaunchKernelGGL(gemm1_bf16_kernel, dim3(a.Is / NT1, sh_slots), dim3(THREADS), 0, s, a, 1);
    hipLaunchKernelGGL(gemm2_bf16_kernel, dim3(a.H / NT2, m_slots), dim3(THREADS), 0, s, a, 0);
    if (a.Is > 0)
      hipLaunchKernelGGL(gemm2_bf16_kernel, dim3(a.H / NT2, sh_slots), dim3(THREADS), 0, s, a, 1);
  } else {
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
