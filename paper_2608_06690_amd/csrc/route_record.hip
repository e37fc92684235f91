// Route records: one fixed-size record per token of a wrapped layer, holding what the
// fail-closed request procedure logs for the route audit - layer, request row, token,
// selected pool and policy decision (App. B.1, fifth step of the procedure) - so that
// the route log can be reconciled against the independent execution counters of the
// expert kernel (App. B.2 route counters indexed by row and layer; App. F.1).
//
// One thread per token: the request row is the last r with req_offset[r] <= t (binary
// search over the non-decreasing offsets), the private mask marks the slots whose
// selected expert id is private.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

__global__ __launch_bounds__(256) void route_record_kernel(RecordArgs a) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= a.T) return;
  int lo = 0, hi = a.R - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.req_offset[mid] <= t) lo = mid; else hi = mid - 1;
  }
  uint32_t mask = 0;
  for (int j = 0; j < a.k; ++j)
    if (a.topk_idx[t * a.k + j] >= a.n_pub) mask |= 1u << j;
  const uint32_t full = (1u << a.k) - 1u;  // k <= 16
  const uint32_t pool = mask == 0 ? PMPE_POOL_PUBLIC : (mask == full ? PMPE_POOL_PRIVATE : PMPE_POOL_MIXED);
  const uint32_t w0 = (uint32_t)(a.layer & 0xFFFF) | ((uint32_t)(a.allow[t] ? 1 : 0) << 16) | (pool << 24);
  const int row = lo;
  const int tok = t - a.req_offset[row];
  *(u32x4*)(a.rec + (size_t)t * 4) = u32x4{w0, (uint32_t)row, (uint32_t)tok, mask};
}

}  // namespace

hipError_t launch_route_record(const RecordArgs& a, hipStream_t s) {
  route_record_kernel<<<(a.T + 255) / 256, 256, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace pmpe
