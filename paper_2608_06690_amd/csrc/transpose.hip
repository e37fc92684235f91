// Per-expert transposes of bf16 weight matrices: dst[e] = src[e]^T for n matrices of
// [rows, cols]. The backward multiplies by W2 and W13 along their output dimension; with
// transposed copies (K contiguous) those products run on the same grouped NT GEMM as the
// forward. 64 x 64 tiles staged through LDS, 16-byte loads and stores along the
// contiguous dimension on both sides.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int TT = 64;

// LDS tile of 64 rows x 64 bf16 columns stored by row pairs: dword (c, m) holds rows 2m
// (low half) and 2m + 1 of column c, so a column reads back as 16-byte chunks of 8 rows.
// The pair index is XOR-swizzled by column bits 3-4: the 64 lanes of a wave that put the
// same element e of chunks q = 0..7 for 8 pairs touch 32 distinct banks twice (the
// minimum for 64 dword writes), and a column's chunks stay 16-byte aligned.
struct PairTile {
  uint32_t d[TT][TT / 2];
};
__device__ __forceinline__ int pt_idx(int c, int m) { return m ^ (((c >> 3) & 3) << 3); }
// Rows 2m (lo) and 2m + 1 (hi), columns 8q .. 8q + 7.
__device__ __forceinline__ void pt_put(PairTile& t, int m, int q, const u32x4& lo, const u32x4& hi) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int c = 8 * q + e, sh = 16 * (e & 1);
    t.d[c][pt_idx(c, m)] = ((lo[e >> 1] >> sh) & 0xFFFFu) | (((hi[e >> 1] >> sh) & 0xFFFFu) << 16);
  }
}
// Rows 8 ch .. 8 ch + 7 of column c.
__device__ __forceinline__ u32x4 pt_get(const PairTile& t, int c, int ch) {
  return *(const u32x4*)&t.d[c][pt_idx(c, 4 * ch)];
}

// NC 64 x 64 tiles side by side: rows r of the source (row_ptr(r) or nullptr for a zero
// row, 16-byte aligned; NC * 64 columns from there) to dst rows c, dst[c * ld_dst + r].
// Thread (m, q) loads 16 bytes of rows 2m and 2m + 1 per tile (8 lanes per 128-byte row
// segment), every load of the NC tiles issued before the first LDS write; the stores go
// out as 16-byte chunks, 8 lanes per 128-byte dst row segment.
// With a row scale (row_scale(r) != nullptr), element (r, c) becomes bf16(scale * value).
__device__ __forceinline__ u32x4 scale_bf16x8(const u32x4& v, float g) {
  u32x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(g * bf16_to_f32(v[e] & 0xFFFFu), g * bf16_to_f32(v[e] >> 16));
  return o;
}
template <int NC, class RowPtr, class RowScale>
__device__ __forceinline__ void tile_transpose(RowPtr row_ptr, RowScale row_scale, uint16_t* __restrict__ dst,
                                               size_t ld_dst) {
  __shared__ __attribute__((aligned(16))) PairTile tile[NC];
  const int tid = threadIdx.x, m = tid >> 3, q = tid & 7;
  u32x4 lo[NC], hi[NC];
  const uint16_t* s0 = row_ptr(2 * m);
  const uint16_t* s1 = row_ptr(2 * m + 1);
#pragma unroll
  for (int n = 0; n < NC; ++n) {
    lo[n] = s0 ? *(const u32x4*)(s0 + n * TT + q * 8) : u32x4{0, 0, 0, 0};
    hi[n] = s1 ? *(const u32x4*)(s1 + n * TT + q * 8) : u32x4{0, 0, 0, 0};
  }
  const float* g0 = row_scale(2 * m);
  const float* g1 = row_scale(2 * m + 1);
  if (g0) {
    const float f = *g0;
#pragma unroll
    for (int n = 0; n < NC; ++n) lo[n] = scale_bf16x8(lo[n], f);
  }
  if (g1) {
    const float f = *g1;
#pragma unroll
    for (int n = 0; n < NC; ++n) hi[n] = scale_bf16x8(hi[n], f);
  }
#pragma unroll
  for (int n = 0; n < NC; ++n) pt_put(tile[n], m, q, lo[n], hi[n]);
  __syncthreads();
#pragma unroll
  for (int n = 0; n < NC; ++n) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = (tid >> 3) + 32 * i;
      *(u32x4*)(dst + (size_t)(n * TT + c) * ld_dst + q * 8) = pt_get(tile[n], c, q);
    }
  }
}

__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ src,
                                                         uint16_t* __restrict__ dst, int rows,
                                                         int cols) {
  const size_t mat = (size_t)rows * cols;
  const uint16_t* s = src + (size_t)blockIdx.z * mat;
  uint16_t* d = dst + (size_t)blockIdx.z * mat;
  const int r0 = blockIdx.y * TT, c0 = blockIdx.x * TT;
  tile_transpose<1>([&](int r) { return s + (size_t)(r0 + r) * cols + c0; },
                    [](int) -> const float* { return nullptr; }, d + (size_t)c0 * rows + r0,
                 (size_t)rows);
}

// Padded private-row tiles. Private expert p owns the permuted rows [offset[n_pub + p],
// offset[n_pub + p + 1]); its K-contiguous copies hold them at columns po_p .. po_p +
// count_p - 1 of a [cols, P] matrix, zero up to the next multiple of 64, with po_p the
// sum of the earlier private experts' padded counts. Block x covers padded columns
// j0 = 64 x .. j0 + 63, which lie in one expert; past the last padded column it has no tile.
struct PrivTile {
  int j0;    // first padded column of the tile
  int jl;    // first row of the tile within its expert
  int cnt;   // rows of the expert
  int src0;  // permuted row of the tile's first row
};

// Called by every thread of the block; false (for all of them) when the block has no tile.
__device__ bool priv_tile(const int32_t* count, const int32_t* offset, int n_pub, int n_priv, PrivTile& pt) {
  __shared__ int s_po[PMPE_MAX_POOL + 1];
  const int tid = threadIdx.x;
  if (tid < 64) {
    int running = 0;
    for (int q0 = 0; q0 < n_priv; q0 += 64) {
      const int q = q0 + tid;
      const int v = (q < n_priv) ? (count[n_pub + q] + TT - 1) / TT * TT : 0;
      const int incl = wave_incl_scan(v);
      if (q < n_priv) s_po[q + 1] = running + incl;
      running += __shfl(incl, 63, 64);
    }
    if (tid == 0) s_po[0] = 0;
  }
  __syncthreads();
  pt.j0 = blockIdx.x * TT;
  if (pt.j0 >= s_po[n_priv]) return false;
  int lo = 0, hi = n_priv - 1;  // last expert with s_po[q] <= j0
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_po[mid] <= pt.j0) lo = mid; else hi = mid - 1;
  }
  pt.jl = pt.j0 - s_po[lo];
  pt.cnt = count[n_pub + lo];
  pt.src0 = offset[n_pub + lo] + pt.jl;
  return true;
}

// dst [cols, P] = the private rows of src [rows, cols], transposed and padded. With
// row_token, src is [T, cols] indexed by token: permuted row r reads src[row_token[r]]
// (the gathered rows are never stored row by row); with row_scale, element (r, c) is
// bf16(row_scale[r] * value). One block per 64 padded rows (x) x 64 NC columns (y).
template <int NC>
__global__ __launch_bounds__(256) void transpose_priv_kernel(const uint16_t* __restrict__ src,
                                                              const int32_t* __restrict__ row_token,
                                                              const float* __restrict__ row_scale,
                                                              uint16_t* __restrict__ dst, int cols,
                                                              int P, const int32_t* count,
                                                              const int32_t* offset, int n_pub,
                                                              int n_priv) {
  PrivTile pt;
  if (!priv_tile(count, offset, n_pub, n_priv, pt)) return;
  const int c0 = blockIdx.y * TT * NC;
  tile_transpose<NC>([&](int r) -> const uint16_t* {
    if (pt.jl + r >= pt.cnt) return nullptr;
    const int row = row_token ? row_token[pt.src0 + r] : pt.src0 + r;
    return src + (size_t)row * cols + c0;
  }, [&](int r) -> const float* {
    return (row_scale && pt.jl + r < pt.cnt) ? row_scale + pt.src0 + r : nullptr;
  }, dst + (size_t)c0 * P + pt.j0, (size_t)P);
}

// SwiGLU backward of the private rows (the rows of the NT backward's dh, I columns, whose
// upstream gradient is g_row[r] * dH[r]), with
// their outputs in both layouts: [da; db] row by row into dA13 [rows, 2I] (the row input
// gradients read them so), and K contiguous into daT [2I, P] (da in rows 0..I-1, db in
// rows I..2I-1) and h into hT [I, P] for the weight gradients. Block: 64 padded rows (x)
// x 64 columns (y); each thread computes 8 columns of two rows, and the three tiles go out
// transposed through LDS. Padding columns get zeros.
__global__ __launch_bounds__(256) void swiglu_priv_t_kernel(const uint16_t* __restrict__ dH,
                                                             const float* __restrict__ g_row,
                                                             const float* __restrict__ AB,
                                                             uint16_t* __restrict__ dA13,
                                                             uint16_t* __restrict__ daT,
                                                             uint16_t* __restrict__ hT, int I, int P,
                                                             const int32_t* count, const int32_t* offset,
                                                             int n_pub, int n_priv) {
  __shared__ __attribute__((aligned(16))) PairTile t_da, t_db, t_h;
  PrivTile pt;
  if (!priv_tile(count, offset, n_pub, n_priv, pt)) return;
  const int c0 = blockIdx.y * TT, tid = threadIdx.x;
  const int m = tid >> 3, q = tid & 7;  // rows 2m and 2m + 1 of the tile, columns 8q .. 8q + 7
  u32x4 oa[2], ob[2], oh[2];
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    oa[v] = ob[v] = oh[v] = u32x4{0, 0, 0, 0};
    const int r = 2 * m + v;
    if (pt.jl + r < pt.cnt) {
      const size_t row = (size_t)(pt.src0 + r);
      const u32x4 dv = *(const u32x4*)(dH + row * I + c0 + q * 8);
      const float gr = g_row[row];
      const float* g = AB + row * 2 * I + c0 + q * 8;
      const f32x4 g0 = *(const f32x4*)g, g1 = *(const f32x4*)(g + 4);
      const f32x4 u0 = *(const f32x4*)(g + I), u1 = *(const f32x4*)(g + I + 4);
      const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
      const float uu[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
      float da[8], db[8], h[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        swiglu_bwd(gr * bf16_to_f32(j & 1 ? dv[j >> 1] >> 16 : dv[j >> 1] & 0xFFFFu), gg[j], uu[j], da[j], db[j], h[j]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        oa[v][e] = pack_bf16x2(da[2 * e], da[2 * e + 1]);
        ob[v][e] = pack_bf16x2(db[2 * e], db[2 * e + 1]);
        oh[v][e] = pack_bf16x2(h[2 * e], h[2 * e + 1]);
      }
      uint16_t* d13 = dA13 + row * 2 * I + c0 + q * 8;
      *(u32x4*)d13 = oa[v];
      *(u32x4*)(d13 + I) = ob[v];
    }
  }
  pt_put(t_da, m, q, oa[0], oa[1]);
  pt_put(t_db, m, q, ob[0], ob[1]);
  pt_put(t_h, m, q, oh[0], oh[1]);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = (tid >> 3) + 32 * i;
    const size_t col = (size_t)pt.j0 + q * 8;
    *(u32x4*)(daT + (size_t)(c0 + c) * P + col) = pt_get(t_da, c, q);
    *(u32x4*)(daT + (size_t)(I + c0 + c) * P + col) = pt_get(t_db, c, q);
    *(u32x4*)(hT + (size_t)(c0 + c) * P + col) = pt_get(t_h, c, q);
  }
}

}  // namespace

// padded private rows never exceed rows_max rounded up to 64, plus 64 per private expert
static int priv_xtiles(int rows_max, int n_priv) { return (rows_max + TT - 1) / TT + n_priv; }

hipError_t launch_transpose_priv(const void* src, const int32_t* row_token, const float* row_scale,
                                 void* dst, int rows_max, int cols, int P, const int32_t* count,
                                 const int32_t* offset, int n_pub, int n_priv, hipStream_t s) {
  // four 64 x 64 tiles per block where the columns allow (more loads in flight per block)
  const int nc = cols % (4 * TT) == 0 ? 4 : cols % (2 * TT) == 0 ? 2 : 1;
  const dim3 grid(priv_xtiles(rows_max, n_priv), cols / (TT * nc));
  const uint16_t* in = (const uint16_t*)src;
  uint16_t* out = (uint16_t*)dst;
  if (nc == 4)
    transpose_priv_kernel<4><<<grid, 256, 0, s>>>(in, row_token, row_scale, out, cols, P, count, offset, n_pub, n_priv);
  else if (nc == 2)
    transpose_priv_kernel<2><<<grid, 256, 0, s>>>(in, row_token, row_scale, out, cols, P, count, offset, n_pub, n_priv);
  else
    transpose_priv_kernel<1><<<grid, 256, 0, s>>>(in, row_token, row_scale, out, cols, P, count, offset, n_pub, n_priv);
  return hipGetLastError();
}

hipError_t launch_swiglu_priv_t(const uint16_t* dH, const float* g_row, const float* AB, uint16_t* dA13,
                                uint16_t* daT, uint16_t* hT, int rows_max, int I, int P,
                                const int32_t* count, const int32_t* offset, int n_pub, int n_priv,
                                hipStream_t s) {
  swiglu_priv_t_kernel<<<dim3(priv_xtiles(rows_max, n_priv), I / TT), 256, 0, s>>>(
      dH, g_row, AB, dA13, daT, hT, I, P, count, offset, n_pub, n_priv);
  return hipGetLastError();
}

hipError_t launch_transpose(const void* src, void* dst, int n, int rows, int cols, hipStream_t s) {
  transpose_kernel<<<dim3(cols / TT, rows / TT, n), 256, 0, s>>>((const uint16_t*)src,
                                                                  (uint16_t*)dst, rows, cols);
  return hipGetLastError();
}

}  // namespace pmpe
