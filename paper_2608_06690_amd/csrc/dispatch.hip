// K2 - dispatch: group the T*k (token, expert) pairs by expert, stably.
//
// Tokens are cut into chunks of 64. A stable counting sort by expert id gives every
// expert its rows in ascending token order:
//  hist     one workgroup per chunk builds, for every expert, the 64-bit mask of the
//           chunk's tokens that selected it (LDS 64-bit atomic OR: the result does not
//           depend on the order of the atomics). popcount(mask) is the chunk's
//           histogram, and the rank of token t among the chunk's rows of expert e is
//           popcount(mask_e & ((1 << t) - 1)).
//  count    one workgroup per expert: expert_count and a scan over the chunks' counts
//           (each chunk's first row within the expert).
//  scatter  one workgroup per chunk: expert_offset is the exclusive scan of the counts;
//           row = offset + chunk base + rank; token_row[t*k+j] = row; row_token[row] = t.
//           Up to 128 chunks every scatter block recounts the masks of all chunks itself
//           (dispatch_count_scatter_kernel), so count needs no launch of its own.
//  gather   (optional) one wave per permuted row copies x[row_token[row]] to
//           x_perm[row] in 16-byte vectors, so reads and writes are coalesced.
// Small batches (up to 8192 (token, slot) pairs, e.g. decode) whose masks and chunk
// bases fit in LDS run hist, count and scatter back to back in one workgroup
// (dispatch_fused_kernel): one launch instead of three, and the same outputs.
// No order-dependent atomics: the permutation is deterministic. Expert ids outside
// [0, E) are not counted and get token_row = -1. A token lists an expert at most once:
// if its row repeats an id, the first slot holding it gets the row and every later
// slot gets token_row = -1 (the router never repeats an id; a caller-built index may).
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int DP_TOK = 64;
constexpr int DP_THREADS = 256;
constexpr int DP_MAX_E = 2 * PMPE_MAX_POOL;

__device__ __forceinline__ int popc64(uint64_t v) { return __popcll(v); }

// Does slot j of a token's id row (ids[0..k)) repeat an id of an earlier slot?
__device__ __forceinline__ bool repeats_earlier(const int32_t* ids, int j, int e) {
  for (int i = 0; i < j; ++i)
    if (ids[i] == e) return true;
  return false;
}

__global__ __launch_bounds__(DP_THREADS) void dispatch_hist_kernel(DispatchArgs a) {
  __shared__ unsigned long long s_mask[DP_MAX_E];
  const int tid = threadIdx.x;
  const int c = blockIdx.x;
  const int t0 = c * DP_TOK;
  const int np = min(DP_TOK, a.T - t0) * a.k;
  const size_t p0 = (size_t)t0 * a.k;
  for (int e = tid; e < a.E; e += DP_THREADS) s_mask[e] = 0ull;
  __syncthreads();
  for (int i = tid; i < np; i += DP_THREADS) {
    const int e = a.topk_idx[p0 + i];
    if (e >= 0 && e < a.E) atomicOr(&s_mask[e], 1ull << (i / a.k));
  }
  __syncthreads();
  for (int e = tid; e < a.E; e += DP_THREADS) a.mask[(size_t)c * a.E + e] = s_mask[e];
}

// One workgroup per expert e: count[e] and the scan of its column of chunk counts
// (chunk_base relative to the expert's first row).
__global__ __launch_bounds__(DP_THREADS) void dispatch_count_kernel(DispatchArgs a, int nchunks) {
  __shared__ int s_wsum[DP_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int e = blockIdx.x;
  const int E = a.E;
  int running = 0;
  for (int c0 = 0; c0 < nchunks; c0 += DP_THREADS) {
    const int c = c0 + tid;
    const int v = (c < nchunks) ? popc64(a.mask[(size_t)c * E + e]) : 0;
    const int incl = wave_incl_scan(v);
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int before = running;
    for (int w = 0; w < wave; ++w) before += s_wsum[w];
    if (c < nchunks) a.chunk_base[(size_t)c * E + e] = before + incl - v;
    int tot = 0;
    for (int w = 0; w < DP_THREADS / 64; ++w) tot += s_wsum[w];
    running += tot;
    __syncthreads();
  }
  if (tid == 0) a.count[e] = running;
}

// Scatter, one workgroup per chunk: the expert offsets are an exclusive scan of
// count[] (recomputed in LDS by every block; block 0 writes expert_offset), then
// row = offset[e] + chunk base + popcount of the chunk's earlier tokens of e.
__global__ __launch_bounds__(DP_THREADS) void dispatch_scatter_kernel(DispatchArgs a) {
  __shared__ int s_off[DP_MAX_E + 1];
  __shared__ int s_wsum[DP_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = blockIdx.x;
  const int E = a.E;
  int running = 0;
  for (int e0 = 0; e0 < E; e0 += DP_THREADS) {
    const int e = e0 + tid;
    const int v = (e < E) ? a.count[e] : 0;
    const int incl = wave_incl_scan(v);
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int before = running;
    for (int w = 0; w < wave; ++w) before += s_wsum[w];
    if (e < E) s_off[e] = before + incl - v;
    int tot = 0;
    for (int w = 0; w < DP_THREADS / 64; ++w) tot += s_wsum[w];
    running += tot;
    __syncthreads();
  }
  if (tid == 0) s_off[E] = running;
  __syncthreads();
  if (c == 0)
    for (int e = tid; e <= E; e += DP_THREADS) a.offset[e] = s_off[e];
  const int t0 = c * DP_TOK;
  const int np = min(DP_TOK, a.T - t0) * a.k;
  const size_t p0 = (size_t)t0 * a.k;
  for (int i = tid; i < np; i += DP_THREADS) {
    const size_t p = p0 + i;
    const int e = a.topk_idx[p];
    int row = -1;
    const int tl = i / a.k, j = i - tl * a.k;
    if (e >= 0 && e < E && !repeats_earlier(a.topk_idx + (p - j), j, e)) {
      const uint64_t below = (tl == 0) ? 0ull : (a.mask[(size_t)c * E + e] & ((1ull << tl) - 1ull));
      row = s_off[e] + a.chunk_base[(size_t)c * E + e] + popc64(below);
      a.row_token[row] = t0 + tl;
    }
    a.token_row[p] = row;
  }
}

constexpr int DC_MAX_CHUNKS = 128;  // chunks up to which count runs inside the scatter blocks

// Count and scatter in one launch, one workgroup per chunk: every block re-reads the
// masks of all chunks (nchunks * E * 8 bytes, L2-resident after hist) for each expert's
// count and this chunk's base, scans the counts into offsets and scatters its chunk;
// block 0 writes expert_count and expert_offset. The same outputs as count + scatter.
__global__ __launch_bounds__(DP_THREADS) void dispatch_count_scatter_kernel(DispatchArgs a, int nchunks) {
  __shared__ int s_off[DP_MAX_E + 1];
  __shared__ int s_base[DP_MAX_E];
  __shared__ int s_wsum[DP_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = blockIdx.x;
  const int E = a.E;
  for (int e = tid; e < E; e += DP_THREADS) {
    int before = 0, total = 0;
#pragma unroll 8
    for (int cc = 0; cc < nchunks; ++cc) {
      const int v = popc64(a.mask[(size_t)cc * E + e]);
      before += (cc < c) ? v : 0;
      total += v;
    }
    s_base[e] = before;
    s_off[e] = total;
    if (c == 0) a.count[e] = total;
  }
  __syncthreads();
  // expert offsets: exclusive scan of the counts, in place
  int running = 0;
  for (int e0 = 0; e0 < E; e0 += DP_THREADS) {
    const int e = e0 + tid;
    const int v = (e < E) ? s_off[e] : 0;
    const int incl = wave_incl_scan(v);
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int before = running;
    for (int w = 0; w < wave; ++w) before += s_wsum[w];
    int tot = 0;
    for (int w = 0; w < DP_THREADS / 64; ++w) tot += s_wsum[w];
    __syncthreads();  // every count of this range is read before the offsets replace them
    if (e < E) s_off[e] = before + incl - v;
    running += tot;
  }
  if (tid == 0) s_off[E] = running;
  __syncthreads();
  if (c == 0)
    for (int e = tid; e <= E; e += DP_THREADS) a.offset[e] = s_off[e];
  const int t0 = c * DP_TOK;
  const int np = min(DP_TOK, a.T - t0) * a.k;
  const size_t p0 = (size_t)t0 * a.k;
  for (int i = tid; i < np; i += DP_THREADS) {
    const size_t p = p0 + i;
    const int e = a.topk_idx[p];
    int row = -1;
    const int tl = i / a.k, j = i - tl * a.k;
    if (e >= 0 && e < E && !repeats_earlier(a.topk_idx + (p - j), j, e)) {
      const uint64_t below = (tl == 0) ? 0ull : (a.mask[(size_t)c * E + e] & ((1ull << tl) - 1ull));
      row = s_off[e] + s_base[e] + popc64(below);
      a.row_token[row] = t0 + tl;
    }
    a.token_row[p] = row;
  }
}

constexpr int DF_THREADS = 1024;
constexpr size_t DF_MAX_LDS = 144 * 1024;  // masks (8 B) and chunk bases (4 B) of every (chunk, expert)
constexpr int64_t DF_MAX_PAIRS = 8192;      // (token, slot) pairs up to which one workgroup is used

// Single-workgroup dispatch: the same three steps as hist / count / scatter, with the
// chunk masks and chunk bases in LDS.
__global__ __launch_bounds__(DF_THREADS) void dispatch_fused_kernel(DispatchArgs a, int nchunks) {
  __shared__ __attribute__((aligned(16))) unsigned char df_smem[DF_MAX_LDS];
  __shared__ int s_off[DP_MAX_E + 1];
  __shared__ int s_wsum[DF_THREADS / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E = a.E, k = a.k;
  const int np = a.T * k;
  unsigned long long* s_mask = (unsigned long long*)df_smem;  // [nchunks][E]
  int* s_base = (int*)(df_smem + (size_t)nchunks * E * 8);    // [nchunks][E]
  for (int i = tid; i < nchunks * E; i += DF_THREADS) s_mask[i] = 0ull;
  __syncthreads();
  // hist: bit (token mod 64) of mask[chunk][expert] (64-bit atomic OR, order independent)
  for (int p = tid; p < np; p += DF_THREADS) {
    const int e = a.topk_idx[p];
    const int t = p / k;
    if (e >= 0 && e < E) atomicOr(&s_mask[(t / DP_TOK) * E + e], 1ull << (t % DP_TOK));
  }
  __syncthreads();
  // count: per expert, its chunks' popcounts in chunk order
  for (int e = tid; e < E; e += DF_THREADS) {
    int running = 0;
    for (int c = 0; c < nchunks; ++c) {
      s_base[c * E + e] = running;
      running += popc64(s_mask[c * E + e]);
    }
    a.count[e] = running;
    s_off[e] = running;
  }
  __syncthreads();
  // expert offsets: exclusive scan of the counts
  int running = 0;
  for (int e0 = 0; e0 < E; e0 += DF_THREADS) {
    const int e = e0 + tid;
    const int v = (e < E) ? s_off[e] : 0;
    const int incl = wave_incl_scan(v);
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int before = running;
    for (int w = 0; w < wave; ++w) before += s_wsum[w];
    int tot = 0;
    for (int w = 0; w < DF_THREADS / 64; ++w) tot += s_wsum[w];
    __syncthreads();  // every count of this range is read before the offsets replace them
    if (e < E) s_off[e] = before + incl - v;
    running += tot;
  }
  __syncthreads();
  if (tid == 0) s_off[E] = running;
  __syncthreads();
  for (int e = tid; e <= E; e += DF_THREADS) a.offset[e] = s_off[e];
  // scatter: row = offset + chunk base + rank of the token among its chunk's rows of e
  for (int p = tid; p < np; p += DF_THREADS) {
    const int e = a.topk_idx[p];
    int row = -1;
    const int t = p / k, j = p - t * k;
    if (e >= 0 && e < E && !repeats_earlier(a.topk_idx + (p - j), j, e)) {
      const int c = t / DP_TOK, tl = t % DP_TOK;
      const uint64_t below = (tl == 0) ? 0ull : (s_mask[c * E + e] & ((1ull << tl) - 1ull));
      row = s_off[e] + s_base[c * E + e] + popc64(below);
      a.row_token[row] = t;
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
  const size_t fused_lds = (size_t)nchunks * a.E * 12;
  // one workgroup is faster only while the pairs are few (measured: 256 x 8 pairs 12.6 -> 8 us;
  // 4096 x 8 pairs 13 -> 36 us)
  if (fused_lds <= DF_MAX_LDS && (int64_t)a.T * a.k <= DF_MAX_PAIRS) {
    hipLaunchKernelGGL(dispatch_fused_kernel, dim3(1), dim3(DF_THREADS), 0, s, a, nchunks);
  } else {
    hipLaunchKernelGGL(dispatch_hist_kernel, dim3(nchunks), dim3(DP_THREADS), 0, s, a);
    if (nchunks <= DC_MAX_CHUNKS) {
      hipLaunchKernelGGL(dispatch_count_scatter_kernel, dim3(nchunks), dim3(DP_THREADS), 0, s, a, nchunks);
    } else {
      hipLaunchKernelGGL(dispatch_count_kernel, dim3(a.E), dim3(DP_THREADS), 0, s, a, nchunks);
      hipLaunchKernelGGL(dispatch_scatter_kernel, dim3(nchunks), dim3(DP_THREADS), 0, s, a);
    }
  }
  if (a.x_perm) {
    const int nrows = a.T * a.k;
    hipLaunchKernelGGL(gather_rows_kernel, dim3((nrows + GA_WAVES - 1) / GA_WAVES),
                       dim3(64 * GA_WAVES), 0, s, a, nrows);
  }
  return hipGetLastError();
}

}  // namespace pmpe
