// K2 - dispatch: group the T*k (token, expert) pairs by expert, stably.
//
// Pairs are numbered token-major, p = t*k + j. A stable counting sort by expert id
// gives each expert's rows in ascending token order:
//  rank     one workgroup per chunk of 64 tokens: each pair's rank among the earlier
//           pairs of the chunk with the same expert (an in-order count, so the order is
//           deterministic) and the chunk's per-expert histogram (LDS atomics; integer
//           counts do not depend on the atomics' order).
//  scan     one workgroup: per expert, the running sum over chunks gives each chunk's
//           base; expert_count; exclusive scan over experts gives expert_offset.
//  scatter  row = offset[e] + chunk base + rank; token_row[p] = row; row_token[row] = t.
//  gather   (optional) one wave per permuted row copies x[row_token[row]] to x_perm[row]:
//           whole 16-byte-vector rows, so reads and writes are coalesced.
// Expert ids outside [0, E) are not counted and get token_row = -1.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int DP_TOK = 64;
constexpr int DP_THREADS = 256;
constexpr int DP_MAX_E = 2 * PMPE_MAX_POOL;

__global__ __launch_bounds__(DP_THREADS) void dispatch_rank_kernel(DispatchArgs a) {
  __shared__ int s_key[DP_TOK * PMPE_MAX_TOPK];
  __shared__ int s_hist[DP_MAX_E];
  const int tid = threadIdx.x;
  const int c = blockIdx.x;
  const int t0 = c * DP_TOK;
  const int ntok = min(DP_TOK, a.T - t0);
  const int np = ntok * a.k;
  const size_t p0 = (size_t)t0 * a.k;
  for (int e = tid; e < a.E; e += DP_THREADS) s_hist[e] = 0;
  for (int i = tid; i < np; i += DP_THREADS) {
    const int e = a.topk_idx[p0 + i];
    s_key[i] = (e >= 0 && e < a.E) ? e : -1;
  }
  __syncthreads();
  for (int i = tid; i < np; i += DP_THREADS) {
    const int key = s_key[i];
    int r = -1;
    if (key >= 0) {
      r = 0;
      for (int q = 0; q < i; ++q) r += (s_key[q] == key) ? 1 : 0;
      atomicAdd(&s_hist[key], 1);
    }
    a.rank[p0 + i] = r;
  }
  __syncthreads();
  for (int e = tid; e < a.E; e += DP_THREADS) a.chunk_base[(size_t)c * a.E + e] = s_hist[e];
}

constexpr int SC_THREADS = 1024;

__global__ __launch_bounds__(SC_THREADS) void dispatch_scan_kernel(DispatchArgs a, int nchunks) {
  __shared__ int s_tot[SC_THREADS];
  const int tid = threadIdx.x;
  const int E = a.E;
  // per expert: running sum over chunks (chunk counts -> chunk bases, in place)
  int tot = 0;
  if (tid < E) {
    for (int c = 0; c < nchunks; ++c) {
      const size_t i = (size_t)c * E + tid;
      const int v = a.chunk_base[i];
      a.chunk_base[i] = tot;
      tot += v;
    }
    a.count[tid] = tot;
  }
  s_tot[tid] = (tid < E) ? tot : 0;
  __syncthreads();
  // inclusive Hillis-Steele scan over experts
  for (int off = 1; off < SC_THREADS; off <<= 1) {
    const int v = (tid >= off) ? s_tot[tid - off] : 0;
    __syncthreads();
    s_tot[tid] += v;
    __syncthreads();
  }
  if (tid < E) {
    const int excl = s_tot[tid] - tot;
    a.offset[tid] = excl;
    for (int c = 0; c < nchunks; ++c) a.chunk_base[(size_t)c * E + tid] += excl;
  }
  if (tid == E - 1) a.offset[E] = s_tot[tid];
}

__global__ __launch_bounds__(DP_THREADS) void dispatch_scatter_kernel(DispatchArgs a) {
  const int tid = threadIdx.x;
  const int c = blockIdx.x;
  const int t0 = c * DP_TOK;
  const int np = min(DP_TOK, a.T - t0) * a.k;
  const size_t p0 = (size_t)t0 * a.k;
  for (int i = tid; i < np; i += DP_THREADS) {
    const size_t p = p0 + i;
    const int r = a.rank[p];
    int row = -1;
    if (r >= 0) {
      const int e = a.topk_idx[p];
      row = a.chunk_base[(size_t)c * a.E + e] + r;
      a.row_token[row] = (int32_t)(p / a.k);
    }
    a.token_row[p] = row;
  }
}

constexpr int GA_WAVES = 4;

__global__ __launch_bounds__(64 * GA_WAVES) void gather_rows_kernel(DispatchArgs a, int nrows) {
  const int row = blockIdx.x * GA_WAVES + (threadIdx.x >> 6);
  if (row >= nrows || row >= a.offset[a.E]) return;  // rows past the valid count are unset
  const int lane = threadIdx.x & 63;
  const int t = a.row_token[row];
  if (t < 0 || t >= a.T) return;
  const size_t row_bytes = (size_t)a.H * (a.act_bf16 ? 2 : 4);
  const u32x4* src = (const u32x4*)((const char*)a.x + (size_t)t * row_bytes);
  u32x4* dst = (u32x4*)((char*)a.x_perm + (size_t)row * row_bytes);
  const int nvec = (int)(row_bytes / 16);
  for (int v = lane; v < nvec; v += 64) dst[v] = src[v];
}

}  // namespace

int dispatch_chunks(int T) { return (T + DP_TOK - 1) / DP_TOK; }

hipError_t launch_dispatch(const DispatchArgs& a, hipStream_t s) {
  const int nchunks = dispatch_chunks(a.T);
  hipLaunchKernelGGL(dispatch_rank_kernel, dim3(nchunks), dim3(DP_THREADS), 0, s, a);
  hipLaunchKernelGGL(dispatch_scan_kernel, dim3(1), dim3(SC_THREADS), 0, s, a, nchunks);
  hipLaunchKernelGGL(dispatch_scatter_kernel, dim3(nchunks), dim3(DP_THREADS), 0, s, a);
  if (a.x_perm) {
    const int nrows = a.T * a.k;
    hipLaunchKernelGGL(gather_rows_kernel, dim3((nrows + GA_WAVES - 1) / GA_WAVES),
                       dim3(64 * GA_WAVES), 0, s, a, nrows);
  }
  return hipGetLastError();
}

}  // namespace pmpe
