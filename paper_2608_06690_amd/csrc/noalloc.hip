// Allocation-free dispatch (pmpe_dispatch_noalloc): the dispatch kernels with their
// per-chunk expert masks and chunk bases in a file-scope device array instead of a
// caller-provided workspace, for callers that cannot allocate device memory.
//
// Each GPU holds its own copy of `scratch` at its own address. Host code never passes the
// array's name to a kernel or a copy (on the host it is only a stand-in for the symbol):
// the first call on a device looks up that device's address with hipGetSymbolAddress,
// with the device current, and every launch takes that address.
#include <mutex>

#include "pmpe_internal.h"

using namespace pmpe;

namespace {

__device__ __attribute__((aligned(256))) unsigned char scratch[PMPE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void* g_addr[kMaxDevices];
hipError_t g_err[kMaxDevices];
std::once_flag g_once[kMaxDevices];

// Device address of the current device's copy of `scratch` (looked up once per device).
hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  try {
    std::call_once(g_once[dev], [dev] {
      void* p = nullptr;
      const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      g_err[dev] = r;
      g_addr[dev] = (r == hipSuccess) ? p : nullptr;
    });
  } catch (...) {
    return hipErrorUnknown;
  }
  *out = g_addr[dev];
  return (g_err[dev] == hipSuccess && g_addr[dev] != nullptr) ? hipSuccess : hipErrorInvalidSymbol;
}

}  // namespace

extern "C" {

pmpe_status pmpe_dispatch_noalloc(const pmpe_layer_desc* d, int32_t T, const int32_t* topk_idx,
                                  const void* x, int32_t* expert_count, int32_t* expert_offset,
                                  int32_t* row_token, int32_t* token_row, void* x_perm,
                                  pmpe_stream_t stream) {
  // the size limit is checked before the device is touched; everything else is checked by
  // pmpe_dispatch with the scratch array as its workspace
  pmpe_status st = pmpe_check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (dispatch_workspace_bytes(d, T) > PMPE_NOALLOC_SCRATCH_BYTES) return PMPE_ERR_SCRATCH;
  if (!topk_idx || !expert_count || !expert_offset || !row_token || !token_row) return PMPE_ERR_NULL;
  if (T == 0) return PMPE_OK;
  void* ws = nullptr;
  if (scratch_address(&ws) != hipSuccess) return PMPE_ERR_LAUNCH;
  return pmpe_dispatch(d, T, topk_idx, x, expert_count, expert_offset, row_token, token_row,
                       x_perm, ws, PMPE_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
