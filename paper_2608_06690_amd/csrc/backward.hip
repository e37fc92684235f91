// Private-only backward of one policy-masked MoE layer.
//
// Only the private experts and the private router rows are trainable (G2 of Sec. 2.2:
// frozen public parameters are not optimised; Sec. 3.2: only the private gate and
// expert weights require gradients). The input gradient still flows through every
// executed expert (public ones too), through the router logits of the selected
// experts and the gates. The route is the forward's: the selection is piecewise
// constant, so gradients flow through the gate values only.
//
// For a row r = (token t, selected expert e, gate g) with upstream gradient G_t:
//   dg      = G_t . y_e(x_t)                      (forward expert output, y_perm)
//   u_r     = g G_t                               (bf16, the expert's upstream row)
//   [a; b]  = W13_e x_t                           (fp32, saved by the forward or recomputed)
//   dh      = W2_e^T u_r
//   da      = dh b s (1 + a (1 - s)),  db = dh a s,  s = sigmoid(a),  h = a s b
//   dx_t   += W13_e^T [da; db]
//   dW2_e  += u_r h^T,  dW13_e += [da; db] x_t^T   (private e only)
// and per token, with the k selected gates renormalised by a softmax (RENORM):
//   dz_j = g_j (dg_j - sum_i g_i dg_i),  dx_t += sum_j dz_j W_r[e_j],
//   dW_r[e] += dz x_t for private e.
//
// Kernels: a per-token row pass (dg, dz, u rows, gathered x rows); launches of one
// grouped bf16 MFMA GEMM template: the gate and up projections (only when the forward
// did not save them), dh with the SwiGLU backward in its epilogue, the row input
// gradients, and the weight gradients, which cover the private experts only, so no
// public gradient is ever formed; then per-token input-gradient and
// per-private-expert router-gradient reductions. Every output element is summed by
// one thread in a fixed order, so the results are bitwise reproducible.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int BT = 256;      // threads of every kernel here
constexpr int TM = 128;      // GEMM tile rows (M)
constexpr int TN = 128;      // GEMM tile columns (N)
constexpr int TK = 64;       // GEMM K step
constexpr int ROWB = 2 * TK; // bytes of one LDS operand row (64 bf16)
constexpr int OPB = TM * ROWB;  // bytes of one LDS operand tile (16 KiB)
constexpr int MAXG = 2 * PMPE_MAX_POOL;

// ---------------------------------------------------------------------------
// Per-token row pass
// ---------------------------------------------------------------------------
// Block t: dg_j = G_t . y_perm[r_j] (fixed-order block reduction), dz_j (RENORM),
// dY[r_j] = bf16(g_j G_t) and Xp[r_j] = x_t (when a later pass reads them), dz_row[r_j] = dz_j,
// g_row[r_j] = g_j.
__global__ __launch_bounds__(BT) void bwd_rows_kernel(BwdArgs a) {
  __shared__ float s_part[BT / 64][PMPE_MAX_TOPK];
  __shared__ float s_dz[PMPE_MAX_TOPK];
  __shared__ int s_row[PMPE_MAX_TOPK];
  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int H = a.H, k = a.k, nch = H / 8;
  const uint16_t* G = (const uint16_t*)a.dout + (size_t)t * H;
  const uint16_t* y = (const uint16_t*)a.y_perm;
  if (tid < k) s_row[tid] = a.token_row[t * k + tid];
  __syncthreads();
  float part[PMPE_MAX_TOPK];
#pragma unroll
  for (int j = 0; j < PMPE_MAX_TOPK; ++j) part[j] = 0.f;
  for (int c = tid; c < nch; c += BT) {
    const u32x4 gv = *(const u32x4*)(G + c * 8);
    float gf[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      gf[2 * q] = bf16_to_f32(gv[q] & 0xFFFFu);
      gf[2 * q + 1] = bf16_to_f32(gv[q] >> 16);
    }
    // eight rows' loads at a time, unconditional (slots past k reload slot k - 1, unused)
#pragma unroll
    for (int j0 = 0; j0 < PMPE_MAX_TOPK; j0 += 8) {
      if (j0 < k) {
        u32x4 yv[8];
#pragma unroll
        for (int jj = 0; jj < 8; ++jj)
          yv[jj] = __builtin_nontemporal_load((const u32x4*)(y + (size_t)s_row[min(j0 + jj, k - 1)] * H + c * 8));
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
          if (j0 + jj < k) {
            float s = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q)
              s += gf[2 * q] * bf16_to_f32(yv[jj][q] & 0xFFFFu) + gf[2 * q + 1] * bf16_to_f32(yv[jj][q] >> 16);
            part[j0 + jj] += s;
          }
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < PMPE_MAX_TOPK; ++j) {
    if (j < k) {
      const float v = wave_sum(part[j]);
      if (lane == 0) s_part[wave][j] = v;
    }
  }
  __syncthreads();
  if (tid == 0) {
    float dg[PMPE_MAX_TOPK], g[PMPE_MAX_TOPK], sum = 0.f;
    for (int j = 0; j < k; ++j) {
      float v = 0.f;
      for (int w = 0; w < BT / 64; ++w) v += s_part[w][j];
      dg[j] = v;
      g[j] = a.topk_gate[t * k + j];
      sum += g[j] * v;
    }
    // RENORM: the logit gradient lives on the k selected experts; POOL_SOFTMAX keeps
    // dg (per slot) for the pool pass, which needs every pool logit
    for (int j = 0; j < k; ++j) s_dz[j] = a.pool_gates ? dg[j] : g[j] * (dg[j] - sum);
  }
  __syncthreads();
  if (tid < k) {
    a.dz_row[s_row[tid]] = s_dz[tid];
    a.g_row[s_row[tid]] = a.topk_gate[t * k + tid];
  }
  const uint16_t* xt = (const uint16_t*)a.x + (size_t)t * H;
  // The gathered copy of x feeds the recomputed [a; b] and the transposing weight-gradient
  // GEMM; the K-contiguous private copies gather x by token themselves. The scaled rows dY
  // feed the transposing GEMMs only: on the NT path dh gathers dout by token (its rows are
  // scaled by g_row in the SwiGLU pass) and the K-contiguous private dY is made from dout.
  const bool need_xp = a.ab == nullptr || (a.n_priv > 0 && a.tr == nullptr);
  const bool need_dy = a.w2t_pub == nullptr || (a.n_priv > 0 && a.tr == nullptr);
  if (!need_xp && !need_dy) return;
  for (int c = tid; c < nch; c += BT) {
    const u32x4 gv = *(const u32x4*)(G + c * 8);
    const u32x4 xv = *(const u32x4*)(xt + c * 8);
    for (int j = 0; j < k; ++j) {
      const float g = a.topk_gate[t * k + j];
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        o[q] = pack_bf16x2(g * bf16_to_f32(gv[q] & 0xFFFFu), g * bf16_to_f32(gv[q] >> 16));
      const size_t r = (size_t)s_row[j];
      if (need_dy) *(u32x4*)(a.dY + r * H + c * 8) = o;
      if (need_xp) *(u32x4*)(a.Xp + r * H + c * 8) = xv;
    }
  }
}

// ---------------------------------------------------------------------------
// Grouped bf16 GEMM, C[M, N] = A[M, K] B[N, K]^T per group, fp32 accumulation
// ---------------------------------------------------------------------------
// Operand views: a non-transposed operand is stored with K contiguous (row m at
// P + row * ld); a transposed one is stored [K, M] with M contiguous (element (m, k) at
// P + k * ld + m). Both are staged through registers into the same K-contiguous LDS
// layout; a transposed operand is turned in registers from 4 K-rows x 8 columns into
// 8 rows x 4 K values per thread.
//
// ROWS mode: group g owns rows [offset[g], offset[g] + count[g]) of A and of C, K and N
// are fixed, B is the group's weight matrix. K-ROWS mode: the contraction runs over the
// group's rows (K = count[g]; rows past it are read as zeros), M and N are fixed, and
// C is the group's own [M, N] matrix.
// EPI_SWIGLU_BWD also writes h for the weight gradient; EPI_SWIGLU_BWD_NOH (frozen
// shared experts, no weight gradient) does not.
enum { EPI_F32 = 0, EPI_SWIGLU_BWD = 1, EPI_SWIGLU_BWD_NOH = 2 };

struct GemmArgs {
  const uint16_t* A;
  int lda;
  const uint16_t* B;       // K-ROWS: activation rows; ROWS: public weight base
  const uint16_t* B_priv;  // ROWS: private weight base
  size_t strideB;          // ROWS: elements per expert weight matrix
  int ldb;
  float* C;
  int ldc;
  size_t strideC;          // K-ROWS: elements per group output
  const int32_t* count;
  const int32_t* offset;
  int g_begin, g_end, n_pub;
  int M, N, K;
  int fixed_rows;          // ROWS: > 0 means one group of this many rows at row 0, weights B
  // EPI_SWIGLU_BWD: [a; b] rows (fp32, 2I per row) in, [da; db] and h (bf16, if Hh) out
  const float* AB;
  uint16_t* dA13;
  uint16_t* Hh;
  int I;
};

// LDS position of 16-byte chunk c of operand row r: XOR-swizzled by the row's low and
// next three bits, so that 16 consecutive rows read at one chunk and the transposed
// stores of 16 rows eight apart both spread over the bank groups.
__device__ __forceinline__ int lds_pos(int r, int c) {
  return r * ROWB + ((c ^ (r & 7) ^ ((r >> 3) & 7)) << 4);
}

template <bool TA, bool TB, bool KROWS, int EPI>
__global__ __launch_bounds__(BT) void bwd_gemm_kernel(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[2][2][OPB];
  __shared__ int s_cum[MAXG + 1];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves of 64 x 64
  const int ng = p.g_end - p.g_begin;
  const int ntn = p.N / TN;

  // tile index with consecutive indices on one XCD (blocks are dealt round-robin)
  const int per = (int)gridDim.x >> 3;
  const int L = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
  int g, m0, n0, Kg, base, rows;
  if (KROWS) {
    const int tpg = (p.M / TM) * ntn;
    if (L >= ng * tpg) return;
    const int gi = L / tpg, loc = L - gi * tpg;
    g = p.g_begin + gi;
    m0 = (loc / ntn) * TM;
    n0 = (loc % ntn) * TN;
    Kg = p.count[g];
    base = p.offset[g];
    rows = TM;
  } else if (p.fixed_rows > 0) {
    const int mt = (p.fixed_rows + TM - 1) / TM;
    if (L >= mt * ntn) return;
    g = 0;
    n0 = (L / mt) * TN;
    m0 = (L % mt) * TM;
    rows = min(TM, p.fixed_rows - m0);
    base = m0;
    Kg = p.K;
  } else {
    if (tid < 64) {
      int running = 0;
      for (int i0 = 0; i0 < ng; i0 += 64) {
        const int i = i0 + tid;
        const int nt = i < ng ? ((p.count[p.g_begin + i] + TM - 1) / TM) * ntn : 0;
        const int incl = wave_incl_scan(nt);
        if (i < ng) s_cum[i + 1] = running + incl;
        running += __shfl(incl, 63, 64);
      }
      if (tid == 0) s_cum[0] = 0;
    }
    __syncthreads();
    if (L >= s_cum[ng]) return;
    int lo = 0, hi = ng - 1;  // last group with s_cum[i] <= L
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_cum[mid] <= L) lo = mid; else hi = mid - 1;
    }
    g = p.g_begin + lo;
    const int cnt = p.count[g];
    const int mt = (cnt + TM - 1) / TM;
    const int loc = L - s_cum[lo];
    n0 = (loc / mt) * TN;
    m0 = (loc % mt) * TM;
    rows = min(TM, cnt - m0);
    base = p.offset[g] + m0;
    Kg = p.K;
  }
  const uint16_t* Bg = p.B;
  if (!KROWS && p.fixed_rows == 0) Bg = (g < p.n_pub) ? p.B + (size_t)g * p.strideB : p.B_priv + (size_t)(g - p.n_pub) * p.strideB;

  u32x4 ra[4], rb[4];
  // Registers of K step k0: direct operands 4 x 16 bytes of rows (t + 256 i) / 8,
  // transposed operands 4 consecutive K rows x 8 columns.
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (!TA) {
        const int q = tid + BT * i, r = q >> 3, c = q & 7;
        const int rr = min(r, rows - 1);
        ra[i] = *(const u32x4*)(p.A + (size_t)(base + rr) * p.lda + k0 + c * 8);
      } else {
        const int kk = k0 + (tid >> 4) * 4 + i, col = m0 + (tid & 15) * 8;
        const int kc = min(kk, Kg - 1);
        u32x4 v = *(const u32x4*)(p.A + (size_t)(base + kc) * p.lda + col);
        ra[i] = kk < Kg ? v : u32x4{0, 0, 0, 0};
      }
      if (!TB) {
        const int q = tid + BT * i, r = q >> 3, c = q & 7;
        rb[i] = *(const u32x4*)(Bg + (size_t)(n0 + r) * p.ldb + k0 + c * 8);
      } else {
        const int kk = k0 + (tid >> 4) * 4 + i, col = n0 + (tid & 15) * 8;
        if (KROWS) {
          const int kc = min(kk, Kg - 1);
          u32x4 v = *(const u32x4*)(Bg + (size_t)(base + kc) * p.ldb + col);
          rb[i] = kk < Kg ? v : u32x4{0, 0, 0, 0};
        } else {
          rb[i] = *(const u32x4*)(Bg + (size_t)kk * p.ldb + col);
        }
      }
    }
  };
  auto store_op = [&](unsigned char* dst, const u32x4 (&v)[4], bool transposed) {
    if (!transposed) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = tid + BT * i;
        *(u32x4*)(dst + lds_pos(q >> 3, q & 7)) = v[i];
      }
    } else {
      const int kg = tid >> 4, r0 = (tid & 15) * 8;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int w = j >> 1;
        uint32_t d0, d1;
        if (j & 1) {
          d0 = (v[0][w] >> 16) | (v[1][w] & 0xFFFF0000u);
          d1 = (v[2][w] >> 16) | (v[3][w] & 0xFFFF0000u);
        } else {
          d0 = (v[0][w] & 0xFFFFu) | (v[1][w] << 16);
          d1 = (v[2][w] & 0xFFFFu) | (v[3][w] << 16);
        }
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        *(u32x2*)(dst + lds_pos(r0 + j, kg >> 1) + (kg & 1) * 8) = u32x2{d0, d1};
      }
    }
  };
  auto lstore = [&](int buf) {
    store_op(smem[buf][0], ra, TA);
    store_op(smem[buf][1], rb, TB);
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0, 0, 0, 0};

  const int nk = (Kg + TK - 1) / TK;
  if (nk > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    gload(min(kt + 1, nk - 1) * TK);  // the last step reloads itself; its store is unused
#pragma unroll
    for (int sub = 0; sub < TK / 32; ++sub) {
      const int ch = sub * 4 + (lane >> 4);
      bf16x8 fa[4], fb[4];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        fa[mb] = as_bf16x8(*(const u32x4*)(smem[cur][0] + lds_pos(wm * 64 + mb * 16 + (lane & 15), ch)));
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        fb[nb] = as_bf16x8(*(const u32x4*)(smem[cur][1] + lds_pos(wn * 64 + nb * 16 + (lane & 15), ch)));
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[mb], fb[nb], acc[mb][nb], 0, 0, 0);
    }
    lstore(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: lane holds C[m = 4 (lane / 16) + i][n = lane % 16] of each 16 x 16 block.
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = wm * 64 + mb * 16 + (lane >> 4) * 4 + i;
      if (m >= rows) continue;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int n = n0 + wn * 64 + nb * 16 + (lane & 15);
        const float v = acc[mb][nb][i];
        if (EPI == EPI_F32) {
          if (KROWS)
            p.C[(size_t)(g - p.g_begin) * p.strideC + (size_t)(m0 + m) * p.ldc + n] = v;
          else
            p.C[(size_t)(base + m) * p.ldc + n] = v;
        } else {
          const size_t r = (size_t)(base + m);
          const float ga = p.AB[r * 2 * p.I + n], ub = p.AB[r * 2 * p.I + p.I + n];
          const float s = 1.0f / (1.0f + __expf(-ga));
          const float da = v * ub * s * (1.0f + ga * (1.0f - s));
          const float db = v * ga * s;
          p.dA13[r * 2 * p.I + n] = (uint16_t)f32_to_bf16_rne(da);
          p.dA13[r * 2 * p.I + p.I + n] = (uint16_t)f32_to_bf16_rne(db);
          if (EPI == EPI_SWIGLU_BWD) p.Hh[r * p.I + n] = (uint16_t)f32_to_bf16_rne(ga * s * ub);
        }
      }
    }
}

// ---------------------------------------------------------------------------
// Reductions
// ---------------------------------------------------------------------------
// SwiGLU backward on the rows of dh (NT path, where dH[r] = dout[t] W2^T and the row's
// upstream is g_row[r] dH[r]): da = dh b s (1 + a (1 - s)),
// db = dh a s, h = a s b, with [a; b] the saved fp32 gate and up projections; four
// columns per thread. With pub_only, block r stops at the first private row (the private
// rows' tile pass writes theirs together with their K-contiguous copies) and h is not
// written (only the private experts' weight gradients read it).
__global__ __launch_bounds__(BT) void bwd_swiglu_kernel(BwdArgs a, const float* AB, int pub_only) {
  const int r = blockIdx.x, I = a.I;
  if (pub_only && r >= a.offset[a.n_pub]) return;
  const uint16_t* dh = a.dH + (size_t)r * I;
  const float gr = a.g_row[r];  // dh here is dout W2^T; the row's upstream is g_row[r] times it
  const float* ab = AB + (size_t)r * 2 * I;
  uint16_t* da = a.dA13 + (size_t)r * 2 * I;
  uint16_t* hh = a.Hh + (size_t)r * I;
  for (int i = threadIdx.x * 4; i < I; i += BT * 4) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 dv = *(const u32x2*)(dh + i);
    const f32x4 g = *(const f32x4*)(ab + i), u = *(const f32x4*)(ab + I + i);
    float dga[4], dub[4], h[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      swiglu_bwd(gr * bf16_to_f32(j & 1 ? dv[j >> 1] >> 16 : dv[j >> 1] & 0xFFFFu), g[j], u[j], dga[j], dub[j], h[j]);
    *(u32x2*)(da + i) = u32x2{pack_bf16x2(dga[0], dga[1]), pack_bf16x2(dga[2], dga[3])};
    *(u32x2*)(da + I + i) = u32x2{pack_bf16x2(dub[0], dub[1]), pack_bf16x2(dub[2], dub[3])};
    if (!pub_only) *(u32x2*)(hh + i) = u32x2{pack_bf16x2(h[0], h[1]), pack_bf16x2(h[2], h[3])};
  }
}

// Softmax over the whole permitted pool (POOL_SOFTMAX), block t: the pool logits
// z_e = x_t . W_r[e] (+ b_e) are recomputed in fp32 (one wave per logit, fixed-order
// reduction), p = softmax(z), and dz_e = p_e ([e selected] dg_e - sum_sel p_i dg_i) for
// every pool member e, written to dz_pool[t, e - first id of the pool].
__global__ __launch_bounds__(BT) void bwd_pool_dz_kernel(BwdArgs a) {
  extern __shared__ float s_dyn[];
  float* s_x = s_dyn;               // [H]
  float* s_z = s_dyn + a.H;         // [pool]
  __shared__ float s_red[2];
  const int t = blockIdx.x, H = a.H, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // the pool of the token is the one its selection lies in (a masked route never mixes
  // pools; the soft control ranks the concatenated pool)
  const bool priv = a.topk_idx[t * a.k] >= a.n_pub;
  const int first = a.soft ? 0 : (priv ? a.n_pub : 0);
  const int pool = a.soft ? a.n_pub + a.n_priv : (priv ? a.n_priv : a.n_pub);
  const uint16_t* xt = (const uint16_t*)a.x + (size_t)t * H;
  for (int h = tid; h < H; h += BT) s_x[h] = bf16_to_f32(xt[h]);
  __syncthreads();
  for (int i = wave; i < pool; i += BT / 64) {
    const int e = first + i;
    const float* w = e < a.n_pub ? a.wr_pub + (size_t)e * H : a.wr_priv + (size_t)(e - a.n_pub) * H;
    float s = 0.f;
    for (int h = lane; h < H; h += 64) s += s_x[h] * w[h];
    s = wave_sum(s);
    if (lane == 0) s_z[i] = a.bias ? s + a.bias[e] : s;
  }
  __syncthreads();
  if (tid == 0) {
    float mx = -INFINITY;
    for (int i = 0; i < pool; ++i) mx = fmaxf(mx, s_z[i]);
    float den = 0.f;
    for (int i = 0; i < pool; ++i) den += __expf(s_z[i] - mx);
    // sum over the selection of p_i dg_i (dg per slot from the row pass)
    float sel = 0.f;
    for (int j = 0; j < a.k; ++j) {
      const int e = a.topk_idx[t * a.k + j];
      sel += __expf(s_z[e - first] - mx) / den * a.dz_row[a.token_row[t * a.k + j]];
    }
    s_red[0] = mx;
    s_red[1] = den;
    s_z[pool] = sel;  // scratch slot after the pool
  }
  __syncthreads();
  const float mx = s_red[0], den = s_red[1], sel = s_z[pool];
  float* dzp = a.dz_pool + (size_t)t * a.pool_stride;
  for (int i = tid; i < pool; i += BT) {
    const float pe = __expf(s_z[i] - mx) / den;
    float u = 0.f;
    for (int j = 0; j < a.k; ++j)
      if (a.topk_idx[t * a.k + j] == first + i) u = a.dz_row[a.token_row[t * a.k + j]];
    dzp[i] = pe * (u - sel);
  }
}

// dx_t = sum_j dXr[r_j] (slot order) + router term + shared-expert term, eight columns per
// thread (the k rows' loads are all issued before the ordered sum). Router term: RENORM
// sum_j dz_j W_r[e_j]; POOL_SOFTMAX sum over the pool of dz_e W_r[e] in id order.
template <bool NT>  // NT: bf16 row input gradients (the NT path), else fp32
__global__ __launch_bounds__(BT) void bwd_dx_kernel(BwdArgs a) {
  __shared__ int s_r[PMPE_MAX_TOPK];
  __shared__ int s_e[PMPE_MAX_TOPK];
  __shared__ float s_dz[PMPE_MAX_TOPK];
  const int t = blockIdx.x, H = a.H, k = a.k, tid = threadIdx.x;
  if (tid < k) {
    const int r = a.token_row[t * k + tid];
    s_r[tid] = r;
    s_e[tid] = a.topk_idx[t * k + tid];
    s_dz[tid] = a.pool_gates ? 0.f : a.dz_row[r];
  }
  __syncthreads();
  const bool priv = a.topk_idx[t * k] >= a.n_pub;
  const int first = a.soft ? 0 : (priv ? a.n_pub : 0);
  const int pool = a.soft ? a.n_pub + a.n_priv : (priv ? a.n_priv : a.n_pub);
  const float* dzp = a.pool_gates ? a.dz_pool + (size_t)t * a.pool_stride : nullptr;
  for (int h = tid * 8; h < H; h += BT * 8) {
    f32x4 s[2] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
    // up to eight rows in flight, summed in slot order. The slots' rows, experts and dz are
    // read from LDS before any global load (an LDS read waits for every older LDS-counted
    // operation), the router rows are addressed from the kernel's own global pointers, and
    // the loads are unconditional (slots past k reload slot k - 1 and are not added).
    for (int j0 = 0; j0 < k; j0 += 8) {
      int rj[8], ej[8];
      float dzj[8];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const int j = min(j0 + jj, k - 1);
        rj[jj] = s_r[j];
        ej[jj] = s_e[j];
        dzj[jj] = s_dz[j];
      }
      f32x4 d[8][2], w[8][2];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        if constexpr (NT) {
          // read once: keep the L2 for the router rows that every token re-reads
          const u32x4 v = __builtin_nontemporal_load((const u32x4*)((const uint16_t*)a.dXr + (size_t)rj[jj] * H + h));
#pragma unroll
          for (int q = 0; q < 2; ++q)
            d[jj][q] = f32x4{bf16_to_f32(v[2 * q] & 0xFFFFu), bf16_to_f32(v[2 * q] >> 16),
                             bf16_to_f32(v[2 * q + 1] & 0xFFFFu), bf16_to_f32(v[2 * q + 1] >> 16)};
        } else {
          d[jj][0] = *(const f32x4*)(a.dXr + (size_t)rj[jj] * H + h);
          d[jj][1] = *(const f32x4*)(a.dXr + (size_t)rj[jj] * H + h + 4);
        }
        const int e = ej[jj];
        const float* wr = e < a.n_pub ? a.wr_pub + (size_t)e * H : a.wr_priv + (size_t)(e - a.n_pub) * H;
        w[jj][0] = *(const f32x4*)(wr + h);
        w[jj][1] = *(const f32x4*)(wr + h + 4);
      }
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        if (j0 + jj < k) {
#pragma unroll
          for (int q = 0; q < 2; ++q) s[q] += d[jj][q] + dzj[jj] * w[jj][q];
        }
      }
    }
    for (int i = 0; dzp && i < pool; ++i) {
      const int e = first + i;
      const float* w = e < a.n_pub ? a.wr_pub + (size_t)e * H : a.wr_priv + (size_t)(e - a.n_pub) * H;
#pragma unroll
      for (int q = 0; q < 2; ++q) s[q] += dzp[i] * *(const f32x4*)(w + h + 4 * q);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      if (a.dXsh) s[q] += *(const f32x4*)(a.dXsh + (size_t)t * H + h + 4 * q);
      *(f32x4*)(a.dx + (size_t)t * H + h + 4 * q) = s[q];
    }
  }
}

// POOL_SOFTMAX router-row gradient of private expert p: every token whose pool holds p
// contributes dz x_t (the gradient is dense over the pool). Block (p, c) sums a fixed
// chunk of tokens in ascending order, eight columns per thread.
__global__ __launch_bounds__(BT) void bwd_dwr_pool_part_kernel(BwdArgs a) {
  const int pe = blockIdx.x, c = blockIdx.y, H = a.H, T = a.T;
  if (c == 0 && threadIdx.x == 0 && a.grad_rows) a.grad_rows[pe] = (uint32_t)a.count[a.n_pub + pe];
  const int per = (T + BWD_DWR_SPLIT - 1) / BWD_DWR_SPLIT;
  const int t0 = min(T, c * per), t1 = min(T, (c + 1) * per);
  float* part = a.dwr_part + ((size_t)pe * BWD_DWR_SPLIT + c) * H;
  const uint16_t* x = (const uint16_t*)a.x;
  for (int h = threadIdx.x * 8; h < H; h += BT * 8) {
    float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int t = t0; t < t1; ++t) {
      if (!a.soft && a.topk_idx[t * a.k] < a.n_pub) continue;  // a public-pool token
      const int idx = a.soft ? a.n_pub + pe : pe;
      const float dz = a.dz_pool[(size_t)t * a.pool_stride + idx];
      const u32x4 v = *(const u32x4*)(x + (size_t)t * H + h);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        s[2 * q] += dz * bf16_to_f32(v[q] & 0xFFFFu);
        s[2 * q + 1] += dz * bf16_to_f32(v[q] >> 16);
      }
    }
    *(f32x4*)(part + h) = f32x4{s[0], s[1], s[2], s[3]};
    *(f32x4*)(part + h + 4) = f32x4{s[4], s[5], s[6], s[7]};
  }
}

// Router-row gradient of private expert p, in two fixed-order stages: block (p, c) sums
// dz_r x[token of r] over the c-th of BWD_DWR_SPLIT equal chunks of p's rows (ascending), eight
// columns per thread; then dW_r[p] = sum over the chunks in order. grad_rows[p] = rows.
__global__ __launch_bounds__(BT) void bwd_dwr_part_kernel(BwdArgs a) {
  const int pe = blockIdx.x, c = blockIdx.y, e = a.n_pub + pe, H = a.H;
  const int cnt = a.count[e], off = a.offset[e];
  if (c == 0 && threadIdx.x == 0 && a.grad_rows) a.grad_rows[pe] = (uint32_t)cnt;
  const int per = (cnt + BWD_DWR_SPLIT - 1) / BWD_DWR_SPLIT;
  const int r0 = off + min(cnt, c * per), r1 = off + min(cnt, (c + 1) * per);
  float* part = a.dwr_part + ((size_t)pe * BWD_DWR_SPLIT + c) * H;
  const uint16_t* x = (const uint16_t*)a.x;
  for (int h = threadIdx.x * 8; h < H; h += BT * 8) {
    float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    // eight rows' loads in flight (rows past r1 reload row r1 - 1 and are not added)
    for (int rb = r0; rb < r1; rb += 8) {
      u32x4 v[8];
      float dz[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = min(rb + i, r1 - 1);
        dz[i] = a.dz_row[r];
        v[i] = *(const u32x4*)(x + (size_t)a.row_token[r] * H + h);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        if (rb + i < r1) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            s[2 * q] += dz[i] * bf16_to_f32(v[i][q] & 0xFFFFu);
            s[2 * q + 1] += dz[i] * bf16_to_f32(v[i][q] >> 16);
          }
        }
      }
    }
    *(f32x4*)(part + h) = f32x4{s[0], s[1], s[2], s[3]};
    *(f32x4*)(part + h + 4) = f32x4{s[4], s[5], s[6], s[7]};
  }
}

__global__ __launch_bounds__(BT) void bwd_dwr_sum_kernel(BwdArgs a) {
  const int pe = blockIdx.y, H = a.H;
  const int h = blockIdx.x * BT + threadIdx.x;
  if (h >= H) return;
  float s = 0.f;
  for (int c = 0; c < BWD_DWR_SPLIT; ++c) s += a.dwr_part[((size_t)pe * BWD_DWR_SPLIT + c) * H + h];
  a.dwr_priv[(size_t)pe * H + h] = s;
}

template <bool TA, bool TB, bool KROWS, int EPI>
hipError_t launch_gemm(const GemmArgs& g, int tiles, hipStream_t s) {
  if (tiles <= 0) return hipSuccess;
  const int grid = (tiles + 7) / 8 * 8;
  bwd_gemm_kernel<TA, TB, KROWS, EPI><<<grid, BT, 0, s>>>(g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_backward(const BwdArgs& a, hipStream_t s) {
  const int E = a.n_pub + a.n_priv, H = a.H, I = a.I, R = a.T * a.k;
  bwd_rows_kernel<<<a.T, BT, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.pool_gates) {
    const size_t lds = ((size_t)H + a.pool_stride + 1) * sizeof(float);
    bwd_pool_dz_kernel<<<a.T, BT, lds, s>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.Is > 0) {
    // shared experts: one group of all T tokens, gate 1, frozen weights (input gradient only)
    GemmArgs sh{};
    sh.fixed_rows = a.T;
    sh.A = (const uint16_t*)a.x; sh.lda = H;
    sh.B = (const uint16_t*)a.w13_sh; sh.ldb = H;
    sh.C = a.AB_sh; sh.ldc = 2 * a.Is; sh.N = 2 * a.Is; sh.K = H;
    const int mt = (a.T + TM - 1) / TM;
    e = launch_gemm<false, false, false, EPI_F32>(sh, mt * (sh.N / TN), s);
    if (e != hipSuccess) return e;
    sh.A = (const uint16_t*)a.dout; sh.lda = H;
    sh.B = (const uint16_t*)a.w2_sh; sh.ldb = a.Is;
    sh.C = nullptr; sh.N = a.Is; sh.K = H;
    sh.AB = a.AB_sh; sh.dA13 = a.dA13_sh; sh.Hh = nullptr; sh.I = a.Is;
    e = launch_gemm<false, true, false, EPI_SWIGLU_BWD_NOH>(sh, mt * (sh.N / TN), s);
    if (e != hipSuccess) return e;
    sh.A = a.dA13_sh; sh.lda = 2 * a.Is;
    sh.B = (const uint16_t*)a.w13_sh; sh.ldb = H;
    sh.C = a.dXsh; sh.ldc = H; sh.N = H; sh.K = 2 * a.Is;
    e = launch_gemm<false, true, false, EPI_F32>(sh, mt * (sh.N / TN), s);
    if (e != hipSuccess) return e;
  }
  // ROWS launches: at most R / TM + E row tiles over all groups
  const int mt_max = R / TM + E;
  GemmArgs g{};
  g.count = a.count;
  g.offset = a.offset;
  g.n_pub = a.n_pub;
  g.I = I;
  g.g_begin = 0;
  g.g_end = E;
  const float* AB = a.ab;
  if (!AB) {
    // [a; b] = Xp W13^T over every executed expert (not saved by the forward)
    g.A = a.Xp; g.lda = H;
    g.B = (const uint16_t*)a.w13_pub; g.B_priv = (const uint16_t*)a.w13_priv;
    g.strideB = (size_t)2 * I * H; g.ldb = H;
    g.C = a.AB; g.ldc = 2 * I;
    g.N = 2 * I; g.K = H;
    e = launch_gemm<false, false, false, EPI_F32>(g, mt_max * (g.N / TN), s);
    if (e != hipSuccess) return e;
    AB = a.AB;
  }
  if (a.w2t_pub) {  // host validation: all transposed weights or none
    // NT path: dh = dY (W2^T)^T and the row input gradients = [da; db] (W13^T)^T on the
    // forward's grouped GEMM (bf16 out), the SwiGLU backward as its own pass
    FfnArgs f{};
    f.T = a.T; f.k = a.k; f.n_pub = a.n_pub; f.n_priv = a.n_priv; f.act_bf16 = 1; f.Is = 0;
    f.count = a.count; f.offset = a.offset; f.row_token = a.row_token;
    f.H = I; f.I = H;  // N = I, K = H
    f.w13_pub = f.w2_pub = a.w2t_pub;
    f.w13_priv = f.w2_priv = a.w2t_priv;
    f.x = a.dout;  // row r reads dout[row_token[r]]; its gate is applied in the SwiGLU pass
    f.gather_a = 1;
    f.y_perm = a.dH;
    e = launch_grouped_nt_gemm(f, s);
    f.gather_a = 0;
    if (e != hipSuccess) return e;
    // with K-contiguous private copies, the private rows go through the tile pass that
    // also writes [da; db] and h transposed for the weight gradients
    const bool priv_t = a.n_priv > 0 && a.tr;
    bwd_swiglu_kernel<<<R, BT, 0, s>>>(a, AB, priv_t ? 1 : 0);
    e = hipGetLastError();
    if (e == hipSuccess && priv_t)
      e = launch_swiglu_priv_t(a.dH, a.g_row, AB, a.dA13, a.tr, a.tr + (size_t)2 * I * a.P, R, I, a.P,
                               a.count, a.offset, a.n_pub, a.n_priv, s);
    if (e != hipSuccess) return e;
    f.H = H; f.I = 2 * I;  // N = H, K = 2I
    f.w13_pub = f.w2_pub = a.w13t_pub;
    f.w13_priv = f.w2_priv = a.w13t_priv;
    f.h = a.dA13;
    f.y_perm = a.dXr;  // bf16 rows in the fp32 buffer
    e = launch_grouped_nt_gemm(f, s);
    if (e != hipSuccess) return e;
  } else {
  // dh = dY W2 (W2 stored [H, I]: K rows of N columns), SwiGLU backward in the epilogue
  g.A = a.dY; g.lda = H;
  g.B = (const uint16_t*)a.w2_pub; g.B_priv = (const uint16_t*)a.w2_priv;
  g.strideB = (size_t)H * I; g.ldb = I;
  g.C = nullptr; g.N = I; g.K = H;
  g.AB = AB; g.dA13 = a.dA13; g.Hh = a.Hh;
  e = launch_gemm<false, true, false, EPI_SWIGLU_BWD>(g, mt_max * (g.N / TN), s);
  if (e != hipSuccess) return e;
  // dXr = [da; db] W13 (W13 stored [2I, H])
  g.A = a.dA13; g.lda = 2 * I;
  g.B = (const uint16_t*)a.w13_pub; g.B_priv = (const uint16_t*)a.w13_priv;
  g.strideB = (size_t)2 * I * H; g.ldb = H;
  g.C = a.dXr; g.ldc = H; g.N = H; g.K = 2 * I;
  e = launch_gemm<false, true, false, EPI_F32>(g, mt_max * (g.N / TN), s);
  if (e != hipSuccess) return e;
  }
  if (a.n_priv > 0 && a.tr) {
    // K-contiguous copies of the private rows (zero-padded per expert to multiples of 64),
    // then the weight gradients on MFMA with 256 x 256 tiles. Regions of tr: [da; db]^T
    // [2I, P], h^T [I, P] (both written by the private SwiGLU tile pass on the NT path),
    // and one [H, P] region that holds x^T for dW13 and then dY^T for dW2.
    uint16_t* daT = a.tr;
    uint16_t* hT = a.tr + (size_t)2 * I * a.P;
    uint16_t* cT = a.tr + (size_t)3 * I * a.P;
    if (!a.w2t_pub) {
      e = launch_transpose_priv(a.dA13, nullptr, nullptr, daT, R, 2 * I, a.P, a.count, a.offset, a.n_pub,
                                a.n_priv, s);
      if (e == hipSuccess)
        e = launch_transpose_priv(a.Hh, nullptr, nullptr, hT, R, I, a.P, a.count, a.offset, a.n_pub, a.n_priv, s);
      if (e != hipSuccess) return e;
    }
    // dW13[p] = [da; db]^T X over private expert p's rows (x gathered by token): M = 2I, N = H
    e = launch_transpose_priv(a.x, a.row_token, nullptr, cT, R, H, a.P, a.count, a.offset, a.n_pub, a.n_priv, s);
    if (e == hipSuccess) e = launch_wgrad(WgradArgs{2 * I, H, a.P, a.n_pub, a.n_priv, daT, cT, a.count, a.dw13_priv}, s);
    // dW2[p] = dY^T h: M = H, N = I; dY rows are bf16(g_row[r] dout[t]), made here from dout
    // on the NT path (the transposing path stored them)
    if (e == hipSuccess) {
      if (a.w2t_pub)
        e = launch_transpose_priv(a.dout, a.row_token, a.g_row, cT, R, H, a.P, a.count, a.offset, a.n_pub,
                                  a.n_priv, s);
      else
        e = launch_transpose_priv(a.dY, nullptr, nullptr, cT, R, H, a.P, a.count, a.offset, a.n_pub, a.n_priv, s);
    }
    if (e == hipSuccess) e = launch_wgrad(WgradArgs{H, I, a.P, a.n_pub, a.n_priv, cT, hT, a.count, a.dw2_priv}, s);
    if (e != hipSuccess) return e;
  } else if (a.n_priv > 0) {
    // dW2[p] = dY^T Hh over private expert p's rows: M = H, N = I
    GemmArgs w{};
    w.count = a.count; w.offset = a.offset; w.n_pub = a.n_pub;
    w.g_begin = a.n_pub; w.g_end = E;
    w.A = a.dY; w.lda = H; w.B = a.Hh; w.ldb = I;
    w.C = a.dw2_priv; w.ldc = I; w.strideC = (size_t)H * I; w.M = H; w.N = I;
    e = launch_gemm<true, true, true, EPI_F32>(w, a.n_priv * (H / TM) * (I / TN), s);
    if (e != hipSuccess) return e;
    // dW13[p] = [da; db]^T Xp: M = 2I, N = H
    w.A = a.dA13; w.lda = 2 * I; w.B = a.Xp; w.ldb = H;
    w.C = a.dw13_priv; w.ldc = H; w.strideC = (size_t)2 * I * H; w.M = 2 * I; w.N = H;
    e = launch_gemm<true, true, true, EPI_F32>(w, a.n_priv * (2 * I / TM) * (H / TN), s);
    if (e != hipSuccess) return e;
  }
  if (a.n_priv > 0) {
    if (a.pool_gates)
      bwd_dwr_pool_part_kernel<<<dim3(a.n_priv, BWD_DWR_SPLIT), BT, 0, s>>>(a);
    else
      bwd_dwr_part_kernel<<<dim3(a.n_priv, BWD_DWR_SPLIT), BT, 0, s>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    bwd_dwr_sum_kernel<<<dim3((H + BT - 1) / BT, a.n_priv), BT, 0, s>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.w2t_pub)
    bwd_dx_kernel<true><<<a.T, BT, 0, s>>>(a);
  else
    bwd_dx_kernel<false><<<a.T, BT, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace pmpe
