// K5 - audit reduce (App. B.2 row-indexed route counters; G1 zero private execution
// under deny). One workgroup: per-request sums of the executed-private-row counts
// (LDS 64-bit atomics; integer sums do not depend on order), their total, and the
// number of deny tokens with a nonzero count. All outputs are overwritten.
#include "pmpe_internal.h"

namespace pmpe {
namespace {

constexpr int AU_THREADS = 1024;
constexpr int AU_REQ = 1024;  // requests handled per round

__global__ __launch_bounds__(AU_THREADS) void audit_kernel(AuditArgs a) {
  __shared__ unsigned long long s_req[AU_REQ];
  __shared__ int s_off[AU_REQ + 1];
  __shared__ unsigned long long s_red[AU_THREADS / 64];
  __shared__ unsigned int s_vred[AU_THREADS / 64];
  const int tid = threadIdx.x;
  unsigned long long my_total = 0;
  unsigned int my_viol = 0;

  // deny violations over all tokens
  for (int t = tid; t < a.T; t += AU_THREADS) my_viol += (a.allow[t] == 0 && a.rows[t] > 0) ? 1u : 0u;

  for (int r0 = 0; r0 < a.R; r0 += AU_REQ) {
    const int nr = min(AU_REQ, a.R - r0);
    for (int i = tid; i < nr; i += AU_THREADS) s_req[i] = 0;
    for (int i = tid; i <= nr; i += AU_THREADS) s_off[i] = min(max(a.req_offset[r0 + i], 0), a.T);
    __syncthreads();
    const int lo = s_off[0], hi = s_off[nr];
    for (int t = lo + tid; t < hi; t += AU_THREADS) {
      // request of token t: last r with s_off[r] <= t
      int l = 0, h = nr - 1;
      while (l < h) {
        const int mid = (l + h + 1) >> 1;
        if (s_off[mid] <= t) l = mid; else h = mid - 1;
      }
      if (t < s_off[l + 1]) atomicAdd(&s_req[l], (unsigned long long)a.rows[t]);
    }
    __syncthreads();
    for (int i = tid; i < nr; i += AU_THREADS) {
      a.req_rows[r0 + i] = s_req[i];
      my_total += s_req[i];
    }
    __syncthreads();
  }

  // block reduction of the total and the violation count
  for (int off = 32; off > 0; off >>= 1) {
    my_total += __shfl_xor(my_total, off, 64);
    my_viol += __shfl_xor(my_viol, off, 64);
  }
  if ((tid & 63) == 0) {
    s_red[tid >> 6] = my_total;
    s_vred[tid >> 6] = my_viol;
  }
  __syncthreads();
  if (tid == 0) {
    unsigned long long tot = 0;
    unsigned int viol = 0;
    for (int w = 0; w < AU_THREADS / 64; ++w) {
      tot += s_red[w];
      viol += s_vred[w];
    }
    *a.total = tot;
    *a.violations = viol;
  }
}

}  // namespace

hipError_t launch_audit(const AuditArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(audit_kernel, dim3(1), dim3(AU_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace pmpe
