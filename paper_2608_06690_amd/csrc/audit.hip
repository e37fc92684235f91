// K5 - audit reduce (App. B.2 row-indexed route counters; G1 zero private execution
// under deny). One workgroup of 16 waves. Long requests: wave w reduces requests w,
// w+16, ...; short requests (e.g. one token each): one lane per request. Each request
// gets the sum of its tokens' executed-private-row counts (64-bit integer sums, order
// independent) and its deny violations (tokens with allow == 0 and a nonzero count);
// a fixed-order reduction over the waves gives the total. All outputs are overwritten.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int AU_WAVES = 16;

__global__ __launch_bounds__(64 * AU_WAVES) void audit_kernel(AuditArgs a) {
  __shared__ unsigned long long s_tot[AU_WAVES];
  __shared__ unsigned int s_viol[AU_WAVES];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned long long wtot = 0;
  unsigned int wviol = 0;
  if (a.R >= 64 * AU_WAVES / 4 && a.T <= 16 * a.R) {
    // short requests: one lane per request
    for (int r = threadIdx.x; r < a.R; r += 64 * AU_WAVES) {
      const int lo = min(max(a.req_offset[r], 0), a.T);
      const int hi = min(max(a.req_offset[r + 1], lo), a.T);
      unsigned long long sum = 0;
      for (int t = lo; t < hi; ++t) {
        const uint32_t v = a.rows[t];
        sum += v;
        wviol += (a.allow[t] == 0 && v > 0) ? 1u : 0u;
      }
      a.req_rows[r] = sum;
      wtot += sum;
    }
    for (int off = 32; off > 0; off >>= 1) {
      wtot += __shfl_xor(wtot, off, 64);
      wviol += __shfl_xor(wviol, off, 64);
    }
  } else
  for (int r = wave; r < a.R; r += AU_WAVES) {
    const int lo = min(max(a.req_offset[r], 0), a.T);
    const int hi = min(max(a.req_offset[r + 1], lo), a.T);
    unsigned long long sum = 0;
    unsigned int viol = 0;
#pragma unroll 8
    for (int t = lo + lane; t < hi; t += 64) {  // unrolled: several loads in flight per lane
      const uint32_t v = a.rows[t];
      sum += v;
      viol += (a.allow[t] == 0 && v > 0) ? 1u : 0u;
    }
    for (int off = 32; off > 0; off >>= 1) {
      sum += __shfl_xor(sum, off, 64);
      viol += __shfl_xor(viol, off, 64);
    }
    if (lane == 0) a.req_rows[r] = sum;
    wtot += sum;
    wviol += viol;
  }
  if (lane == 0) {
    s_tot[wave] = wtot;
    s_viol[wave] = wviol;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long tot = 0;
    unsigned int viol = 0;
    for (int w = 0; w < AU_WAVES; ++w) {
      tot += s_tot[w];
      viol += s_viol[w];
    }
    *a.total = tot;
    *a.violations = viol;
  }
}

}  // namespace

hipError_t launch_audit(const AuditArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(audit_kernel, dim3(1), dim3(64 * AU_WAVES), 0, s, a);
  return hipGetLastError();
}

}  // namespace pmpe
