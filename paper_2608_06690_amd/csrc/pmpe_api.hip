// C ABI of libpmpe: argument validation (host only, before any launch) and dispatch to
// the kernel launchers. No exception crosses this boundary; nothing is allocated.
#include <cmath>
#include <new>

#include "pmpe_internal.h"

using namespace pmpe;

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

size_t elem_bytes(const pmpe_layer_desc* d) { return d->act_dtype == PMPE_BF16 ? 2 : 4; }

pmpe_status check_desc(const pmpe_layer_desc* d, int32_t T) {
  if (d == nullptr) return PMPE_ERR_NULL;
  if (T < 0 || T > PMPE_MAX_TOKENS) return PMPE_ERR_SHAPE;
  if (d->act_dtype != PMPE_F32 && d->act_dtype != PMPE_BF16) return PMPE_ERR_DTYPE;
  if (d->w_dtype != d->act_dtype) return PMPE_ERR_DTYPE;
  if (d->hidden < 128 || d->hidden > 16384 || d->hidden % 128 != 0) return PMPE_ERR_SHAPE;
  if (d->inter < 64 || d->inter > 65536 || d->inter % 64 != 0) return PMPE_ERR_SHAPE;
  if (d->top_k < 1 || d->top_k > PMPE_MAX_TOPK) return PMPE_ERR_SHAPE;
  if (d->n_pub < 1 || d->n_pub > PMPE_MAX_POOL || d->n_priv < 0 || d->n_priv > PMPE_MAX_POOL)
    return PMPE_ERR_SHAPE;
  if (d->top_k > d->n_pub || d->top_k > d->n_priv) return PMPE_ERR_K_EXCEEDS_POOL;
  if (d->n_shared < 0 || d->n_shared > 64) return PMPE_ERR_SHAPE;
  if (d->n_shared > 0) {
    if (d->shared_inter < 64 || d->shared_inter % 64 != 0) return PMPE_ERR_SHAPE;
    if ((int64_t)d->n_shared * d->shared_inter > 65536) return PMPE_ERR_SHAPE;
  }
  if (d->gate_mode != PMPE_GATE_RENORM_TOPK && d->gate_mode != PMPE_GATE_POOL_SOFTMAX)
    return PMPE_ERR_SHAPE;
  if (d->route_mode != PMPE_ROUTE_MASKED && d->route_mode != PMPE_ROUTE_SOFT) return PMPE_ERR_SHAPE;
  if (d->route_mode == PMPE_ROUTE_SOFT && d->n_pub + d->n_priv > 2 * PMPE_MAX_POOL) return PMPE_ERR_SHAPE;
  if ((int64_t)T * d->top_k > (int64_t)INT32_MAX / 2) return PMPE_ERR_SHAPE;
  // the expert kernels address rows of x, x_perm, h and of one expert's weights with
  // 32-bit byte offsets (bf16 elements, so fewer than 2^31 elements)
  const int64_t lim = (int64_t)1 << 31;
  const int64_t wmax = d->hidden > d->inter ? d->hidden : d->inter;
  const int64_t ish = (int64_t)d->n_shared * d->shared_inter;
  if ((int64_t)T * d->top_k * wmax >= lim) return PMPE_ERR_SHAPE;
  if ((int64_t)T * ish >= lim) return PMPE_ERR_SHAPE;
  if ((int64_t)T * d->hidden >= lim) return PMPE_ERR_SHAPE;
  if (2 * (int64_t)d->inter * d->hidden >= lim || 2 * ish * d->hidden >= lim) return PMPE_ERR_SHAPE;
  return PMPE_OK;
}

// logits row: the permitted pool (masked), or the concatenated pool (soft control)
int route_zstride(const pmpe_layer_desc* d) {
  if (d->route_mode == PMPE_ROUTE_SOFT) return d->n_pub + d->n_priv;
  return d->n_pub > d->n_priv ? d->n_pub : d->n_priv;
}

size_t route_ws(const pmpe_layer_desc* d, int32_t T) {
  const int S = route_ksplit(T, d->hidden, d->n_pub, d->n_priv, d->act_dtype == PMPE_BF16);
  return round_up((size_t)S * T * route_zstride(d) * 4);
}

size_t dispatch_ws(const pmpe_layer_desc* d, int32_t T) {
  const size_t E = (size_t)d->n_pub + d->n_priv;
  return round_up((size_t)dispatch_chunks(T) * E * 8) + round_up((size_t)dispatch_chunks(T) * E * 4);
}

size_t ffn_ws(const pmpe_layer_desc* d, int32_t T) {
  const size_t el = elem_bytes(d);
  const size_t Is = (size_t)d->n_shared * d->shared_inter;
  return round_up((size_t)T * d->top_k * d->inter * el) + round_up((size_t)T * Is * el);
}

pmpe_status launched(hipError_t e) { return e == hipSuccess ? PMPE_OK : PMPE_ERR_LAUNCH; }

// backward workspace: Xp, dY, [a; b], h, [da; db], row input gradients, row dz and gates
struct BwdLayout {
  size_t xp, dy, ab, hh, da, dxr, dz, grow, part, dzp, absh, dash, dxsh, dh, tr, total;
  int P;  // row stride of the transposed private rows (0: weight gradients on the transposing GEMM)
};
int bwd_pool_stride(const pmpe_layer_desc* d) {
  if (d->route_mode == PMPE_ROUTE_SOFT) return d->n_pub + d->n_priv;
  return d->n_pub > d->n_priv ? d->n_pub : d->n_priv;
}
BwdLayout bwd_layout(const pmpe_layer_desc* d, int32_t T) {
  const size_t R = (size_t)T * d->top_k, H = d->hidden, I = d->inter;
  BwdLayout L;
  size_t o = 0;
  L.xp = o; o += round_up(R * H * 2);
  L.dy = o; o += round_up(R * H * 2);
  L.ab = o; o += round_up(R * 2 * I * 4);
  L.hh = o; o += round_up(R * I * 2);
  L.da = o; o += round_up(R * 2 * I * 2);
  L.dxr = o; o += round_up(R * H * 4);
  L.dz = o; o += round_up(R * 4);
  L.grow = o; o += round_up(R * 4);
  L.part = o; o += round_up((size_t)d->n_priv * BWD_DWR_SPLIT * H * 4);
  const size_t Tt = (size_t)T, Is = (size_t)d->n_shared * d->shared_inter;
  L.dzp = o; o += d->gate_mode == PMPE_GATE_POOL_SOFTMAX ? round_up(Tt * bwd_pool_stride(d) * 4) : 0;
  L.absh = o; o += round_up(Tt * 2 * Is * 4);
  L.dash = o; o += round_up(Tt * 2 * Is * 2);
  L.dxsh = o; o += Is > 0 ? round_up(Tt * H * 4) : 0;
  L.dh = o; o += round_up(R * I * 2);
  // private rows transposed and padded per expert: [3I + H, P] bf16 ([da; db], h, and one
  // region for x and then dY), used when every byte offset of the weight-gradient copies
  // fits in 31 bits
  const size_t P = (R + 63) / 64 * 64 + 64 * (size_t)d->n_priv;
  const size_t wmax = 2 * I > H ? 2 * I : H;
  L.P = 0;
  L.tr = o;
  if (d->n_priv > 0 && wmax * P * 2 < ((size_t)1 << 31)) {
    L.P = (int)P;
    o += round_up((3 * I + H) * P * 2);
  }
  L.total = o;
  return L;
}

pmpe_status check_backward_desc(const pmpe_layer_desc* d, int32_t T) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (d->act_dtype != PMPE_BF16) return PMPE_ERR_DTYPE;
  if (d->inter % 128 != 0) return PMPE_ERR_SHAPE;
  // the grouped GEMMs address [T*k, 2I] rows with 32-bit element offsets
  if ((int64_t)T * d->top_k * 2 * d->inter >= ((int64_t)1 << 31)) return PMPE_ERR_SHAPE;
  if (d->n_shared > 0 && ((int64_t)d->n_shared * d->shared_inter) % 128 != 0) return PMPE_ERR_SHAPE;
  // the pool-softmax pass stages one x row in fp32 LDS
  if (d->gate_mode == PMPE_GATE_POOL_SOFTMAX && d->hidden > 8192) return PMPE_ERR_SHAPE;
  return PMPE_OK;
}

// two ping-pong digest arrays: every level fits in the one it does not read
size_t fingerprint_ws_parts(uint64_t nbytes, size_t* part0) {
  const uint64_t n = fingerprint_leaves(nbytes);
  if (n <= 1) {
    *part0 = 0;
    return 0;
  }
  *part0 = round_up((size_t)n * 32);
  return *part0 + round_up((size_t)((n + kFpFanout - 1) / kFpFanout) * 32);
}

pmpe_status expert_ffn_impl(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                            const void* x, const int32_t* expert_count,
                            const int32_t* expert_offset, const int32_t* row_token,
                            const void* w13_pub, const void* w2_pub, const void* w13_priv,
                            const void* w2_priv, const void* w13_sh, const void* w2_sh,
                            void* y_shared, void* y_perm, uint32_t* audit_token_rows,
                            uint32_t* audit_priv_calls, uint32_t* dev_status, void* ws,
                            size_t ws_bytes, pmpe_stream_t stream, float* ab_save) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (!expert_count || !expert_offset || !row_token || !w13_pub || !w2_pub || !y_perm ||
      !audit_token_rows)
    return PMPE_ERR_NULL;
  if (!x_perm && !x) return PMPE_ERR_NULL;
  if (d->n_shared > 0 && (!x || !w13_sh || !w2_sh || !y_shared)) return PMPE_ERR_NULL;
  const void* al[] = {x_perm, x, w13_pub, w2_pub, w13_priv, w2_priv, w13_sh, w2_sh, y_shared, y_perm};
  for (const void* p : al)
    if (p && !aligned16(p)) return PMPE_ERR_ALIGN;
  if (ab_save && d->act_dtype != PMPE_BF16) return PMPE_ERR_DTYPE;
  if (ab_save && !aligned16(ab_save)) return PMPE_ERR_ALIGN;
  if (T == 0) return PMPE_OK;
  if (!ws || ws_bytes < ffn_ws(d, T)) return PMPE_ERR_WORKSPACE;
  if (!aligned16(ws)) return PMPE_ERR_ALIGN;
  const size_t el = elem_bytes(d);
  const int Is = d->n_shared * d->shared_inter;
  void* h = ws;
  void* h_sh = (char*)ws + round_up((size_t)T * d->top_k * d->inter * el);
  FfnArgs a{T, d->hidden, d->inter, d->n_pub, d->n_priv, d->top_k, d->act_dtype == PMPE_BF16,
            d->n_shared > 0 ? Is : 0, x_perm, x, expert_count, expert_offset, row_token,
            w13_pub, w2_pub, w13_priv, w2_priv, w13_sh, w2_sh, y_shared, y_perm,
            audit_token_rows, audit_priv_calls, dev_status, h, h_sh, ab_save};
  return launched(launch_expert_ffn(a, (hipStream_t)stream));
}

}  // namespace

namespace pmpe {
size_t dispatch_workspace_bytes(const pmpe_layer_desc* d, int32_t T) { return dispatch_ws(d, T); }
}  // namespace pmpe

extern "C" {

int32_t pmpe_version(void) { return 10000; }

const char* pmpe_status_string(int32_t status) {
  switch (status) {
    case PMPE_OK: return "ok";
    case PMPE_ERR_NULL: return "a required pointer is NULL";
    case PMPE_ERR_SHAPE: return "a size is out of the supported range";
    case PMPE_ERR_K_EXCEEDS_POOL: return "top_k exceeds the public or the private pool";
    case PMPE_ERR_DTYPE: return "unsupported dtype combination";
    case PMPE_ERR_ALIGN: return "a pointer is not 16-byte aligned";
    case PMPE_ERR_WORKSPACE: return "workspace missing or too small";
    case PMPE_ERR_LAUNCH: return "the HIP runtime refused a kernel launch";
    case PMPE_ERR_TAG_MISMATCH: return "cache tag does not match the request; reuse refused";
    case PMPE_ERR_SCRATCH:
      return "the batch needs more scratch than the allocation-free entry point holds";
    default: return "unknown status";
  }
}

pmpe_status pmpe_check_desc(const pmpe_layer_desc* d, int32_t T) { return check_desc(d, T); }

size_t pmpe_workspace_bytes(const pmpe_layer_desc* d, int32_t T) {
  if (check_desc(d, T) != PMPE_OK) return 0;
  size_t m = route_ws(d, T);
  if (dispatch_ws(d, T) > m) m = dispatch_ws(d, T);
  if (ffn_ws(d, T) > m) m = ffn_ws(d, T);
  return m;
}

pmpe_status pmpe_route(const pmpe_layer_desc* d, int32_t T, const void* x, const float* wr_pub,
                       const float* wr_priv, const float* logit_bias, const uint32_t* policy_word,
                       int32_t* topk_idx, float* topk_gate, uint8_t* allow, float* kgap,
                       uint32_t* dev_status, void* ws, size_t ws_bytes, pmpe_stream_t stream) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (!x || !wr_pub || !topk_idx || !topk_gate || !allow) return PMPE_ERR_NULL;
  if (!aligned16(x) || !aligned16(wr_pub) || (wr_priv && !aligned16(wr_priv))) return PMPE_ERR_ALIGN;
  if (T == 0) return PMPE_OK;
  if (!ws || ws_bytes < route_ws(d, T)) return PMPE_ERR_WORKSPACE;
  if (!aligned16(ws)) return PMPE_ERR_ALIGN;
  if (d->route_mode == PMPE_ROUTE_SOFT && !wr_priv) return PMPE_ERR_NULL;
  RouteArgs a{T, d->hidden, d->n_pub, d->n_priv, d->top_k, d->gate_mode,
              d->act_dtype == PMPE_BF16, x, wr_pub, wr_priv, logit_bias, policy_word,
              topk_idx, topk_gate, allow, kgap, dev_status, (float*)ws, route_zstride(d),
              d->route_mode == PMPE_ROUTE_SOFT ? 1 : 0,
              route_ksplit(T, d->hidden, d->n_pub, d->n_priv, d->act_dtype == PMPE_BF16)};
  return launched(launch_route(a, (hipStream_t)stream));
}

pmpe_status pmpe_dispatch(const pmpe_layer_desc* d, int32_t T, const int32_t* topk_idx,
                          const void* x, int32_t* expert_count, int32_t* expert_offset,
                          int32_t* row_token, int32_t* token_row, void* x_perm, void* ws,
                          size_t ws_bytes, pmpe_stream_t stream) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (!topk_idx || !expert_count || !expert_offset || !row_token || !token_row) return PMPE_ERR_NULL;
  if (x_perm && !x) return PMPE_ERR_NULL;
  if (x_perm && (!aligned16(x) || !aligned16(x_perm))) return PMPE_ERR_ALIGN;
  if (T == 0) return PMPE_OK;
  if (!ws || ws_bytes < dispatch_ws(d, T)) return PMPE_ERR_WORKSPACE;
  if (!aligned16(ws)) return PMPE_ERR_ALIGN;
  const int E = d->n_pub + d->n_priv;
  uint64_t* mask = (uint64_t*)ws;
  int32_t* chunk_base = (int32_t*)((char*)ws + round_up((size_t)dispatch_chunks(T) * E * 8));
  DispatchArgs a{T, d->top_k, E, d->hidden, d->act_dtype == PMPE_BF16, topk_idx, x,
                 expert_count, expert_offset, row_token, token_row, x_perm, mask, chunk_base};
  return launched(launch_dispatch(a, (hipStream_t)stream));
}

pmpe_status pmpe_expert_ffn(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                            const void* x, const int32_t* expert_count,
                            const int32_t* expert_offset, const int32_t* row_token,
                            const void* w13_pub, const void* w2_pub, const void* w13_priv,
                            const void* w2_priv, const void* w13_sh, const void* w2_sh,
                            void* y_shared, void* y_perm, uint32_t* audit_token_rows,
                            uint32_t* audit_priv_calls, uint32_t* dev_status, void* ws,
                            size_t ws_bytes, pmpe_stream_t stream) {
  return expert_ffn_impl(d, T, x_perm, x, expert_count, expert_offset, row_token, w13_pub, w2_pub,
                         w13_priv, w2_priv, w13_sh, w2_sh, y_shared, y_perm, audit_token_rows,
                         audit_priv_calls, dev_status, ws, ws_bytes, stream, nullptr);
}

pmpe_status pmpe_expert_ffn_train(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                                  const void* x, const int32_t* expert_count,
                                  const int32_t* expert_offset, const int32_t* row_token,
                                  const void* w13_pub, const void* w2_pub, const void* w13_priv,
                                  const void* w2_priv, const void* w13_sh, const void* w2_sh,
                                  void* y_shared, void* y_perm, uint32_t* audit_token_rows,
                                  uint32_t* audit_priv_calls, uint32_t* dev_status, float* ab,
                                  void* ws, size_t ws_bytes, pmpe_stream_t stream) {
  if (!ab) return PMPE_ERR_NULL;
  return expert_ffn_impl(d, T, x_perm, x, expert_count, expert_offset, row_token, w13_pub, w2_pub,
                         w13_priv, w2_priv, w13_sh, w2_sh, y_shared, y_perm, audit_token_rows,
                         audit_priv_calls, dev_status, ws, ws_bytes, stream, ab);
}

pmpe_status pmpe_combine(const pmpe_layer_desc* d, int32_t T, const void* y_perm,
                         const int32_t* token_row, const float* topk_gate,
                         const void* y_shared, void* out, pmpe_stream_t stream) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (!y_perm || !token_row || !topk_gate || !out) return PMPE_ERR_NULL;
  if (d->n_shared > 0 && !y_shared) return PMPE_ERR_NULL;
  if (!aligned16(y_perm) || !aligned16(out) || (y_shared && !aligned16(y_shared))) return PMPE_ERR_ALIGN;
  if (T == 0) return PMPE_OK;
  CombineArgs a{T, d->hidden, d->top_k, d->act_dtype == PMPE_BF16, y_perm, token_row,
                topk_gate, d->n_shared > 0 ? y_shared : nullptr, out};
  return launched(launch_combine(a, (hipStream_t)stream));
}

pmpe_status pmpe_audit(const pmpe_layer_desc* d, int32_t T, const uint32_t* audit_token_rows,
                       const uint8_t* allow, const int32_t* req_offset, int32_t R,
                       uint64_t* req_private_rows, uint64_t* total_private_rows,
                       uint32_t* deny_violations, pmpe_stream_t stream) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (R < 0 || R > PMPE_MAX_TOKENS) return PMPE_ERR_SHAPE;
  if (!total_private_rows || !deny_violations) return PMPE_ERR_NULL;
  if (T > 0 && (!audit_token_rows || !allow)) return PMPE_ERR_NULL;
  if (R > 0 && (!req_offset || !req_private_rows)) return PMPE_ERR_NULL;
  AuditArgs a{T, R, audit_token_rows, allow, req_offset, req_private_rows, total_private_rows,
              deny_violations};
  return launched(launch_audit(a, (hipStream_t)stream));
}

pmpe_status pmpe_expert_ffn_fp8(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                                const void* x, const int32_t* expert_count,
                                const int32_t* expert_offset, const int32_t* row_token,
                                const void* w13_pub, const void* w2_pub, const void* w13_priv,
                                const void* w2_priv, const float* w13s_pub, const float* w2s_pub,
                                const float* w13s_priv, const float* w2s_priv, void* y_perm,
                                uint32_t* audit_token_rows, uint32_t* audit_priv_calls,
                                uint32_t* dev_status, void* ws, size_t ws_bytes,
                                pmpe_stream_t stream) {
  if (!d) return PMPE_ERR_NULL;
  if (d->act_dtype != PMPE_BF16 || d->w_dtype != PMPE_FP8_E4M3) return PMPE_ERR_DTYPE;
  // the descriptor checks of the bf16 path, with the weight dtype read as bf16
  pmpe_layer_desc db = *d;
  db.w_dtype = PMPE_BF16;
  pmpe_status st = check_desc(&db, T);
  if (st != PMPE_OK) return st;
  if (d->n_shared != 0) return PMPE_ERR_SHAPE;
  if (!expert_count || !expert_offset || !row_token || !w13_pub || !w2_pub || !y_perm ||
      !audit_token_rows || !w13s_pub || !w2s_pub)
    return PMPE_ERR_NULL;
  if (!x_perm && !x) return PMPE_ERR_NULL;
  if ((w13_priv != nullptr) != (w13s_priv != nullptr) || (w2_priv != nullptr) != (w2s_priv != nullptr))
    return PMPE_ERR_NULL;
  const void* al[] = {x_perm, x, w13_pub, w2_pub, w13_priv, w2_priv, y_perm};
  for (const void* p : al)
    if (p && !aligned16(p)) return PMPE_ERR_ALIGN;
  if (T == 0) return PMPE_OK;
  if (!ws || ws_bytes < ffn_ws(&db, T)) return PMPE_ERR_WORKSPACE;
  if (!aligned16(ws)) return PMPE_ERR_ALIGN;
  FfnArgs a{T, d->hidden, d->inter, d->n_pub, d->n_priv, d->top_k, 1, 0, x_perm, x, expert_count,
            expert_offset, row_token, w13_pub, w2_pub, w13_priv, w2_priv, nullptr, nullptr, nullptr,
            y_perm, audit_token_rows, audit_priv_calls, dev_status, ws, nullptr, nullptr,
            w13s_pub, w2s_pub, w13s_priv, w2s_priv};
  return launched(launch_expert_ffn_fp8(a, (hipStream_t)stream));
}

size_t pmpe_expert_ffn_lora_workspace_bytes(const pmpe_layer_desc* d, int32_t T) {
  if (check_desc(d, T) != PMPE_OK) return 0;
  return ffn_ws(d, T) + round_up((size_t)T * d->top_k * 2 * d->inter * 4);
}

pmpe_status pmpe_expert_ffn_lora(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                                 const void* x, const int32_t* expert_count,
                                 const int32_t* expert_offset, const int32_t* row_token,
                                 const uint32_t* policy_word, const void* w13_pub,
                                 const void* w2_pub, const void* a13, const void* b1,
                                 const void* b3, const void* a2, const void* b2, int32_t rank,
                                 float scale, int32_t gate, void* y_perm, uint32_t* lora_rows,
                                 uint32_t* dev_status, void* ws, size_t ws_bytes,
                                 pmpe_stream_t stream) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (d->act_dtype != PMPE_BF16) return PMPE_ERR_DTYPE;
  if (rank < 1 || rank > 128 || gate < PMPE_LORA_GATE_ROW || gate > PMPE_LORA_GATE_POSTHOC ||
      d->hidden > 8192 || d->inter > 8192 || d->n_shared != 0)
    return PMPE_ERR_SHAPE;
  if (!expert_count || !expert_offset || !row_token || !w13_pub || !w2_pub || !y_perm ||
      !a13 || !b1 || !b3 || !a2 || !b2 || !lora_rows)
    return PMPE_ERR_NULL;
  if (!x_perm && !x) return PMPE_ERR_NULL;
  const void* al[] = {x_perm, x, w13_pub, w2_pub, a13, b1, b3, a2, b2, y_perm};
  for (const void* p : al)
    if (p && !aligned16(p)) return PMPE_ERR_ALIGN;
  if (T == 0) return PMPE_OK;
  const size_t fws = ffn_ws(d, T);
  if (!ws || ws_bytes < fws + round_up((size_t)T * d->top_k * 2 * d->inter * 4)) return PMPE_ERR_WORKSPACE;
  if (!aligned16(ws)) return PMPE_ERR_ALIGN;
  float* ab = (float*)((char*)ws + fws);
  // the adapters sit on the public experts; private rows (if any) run without weights
  FfnArgs f{T, d->hidden, d->inter, d->n_pub, d->n_priv, d->top_k, 1, 0, x_perm, x, expert_count,
            expert_offset, row_token, w13_pub, w2_pub, nullptr, nullptr, nullptr, nullptr, nullptr,
            y_perm, lora_rows, nullptr, dev_status, ws, nullptr, ab};
  // GEMM1 never touches the audit; GEMM2 only audits private rows, which run without
  // weights here and are therefore neither executed nor counted
  LoraArgs l{T, d->hidden, d->inter, d->top_k, d->n_pub, d->n_priv, rank, gate, scale,
             expert_count, expert_offset, row_token, policy_word, x, x_perm,
             (const uint16_t*)a13, (const uint16_t*)b1, (const uint16_t*)b3, (const uint16_t*)a2,
             (const uint16_t*)b2, ab, (uint16_t*)ws, (uint16_t*)y_perm, lora_rows};
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = launch_expert_ffn_parts(f, s, 1);
  if (e == hipSuccess) e = launch_lora_pre(l, s);
  if (e == hipSuccess) e = launch_expert_ffn_parts(f, s, 2);
  if (e == hipSuccess) e = launch_lora_post(l, s);
  return launched(e);
}

static_assert(sizeof(pmpe_route_rec) == 16, "one record is one 16-byte store");
static_assert(sizeof(pmpe_cache_tag) == 68, "cache tag layout");

pmpe_status pmpe_route_record(const pmpe_layer_desc* d, int32_t T, int32_t layer,
                              const int32_t* topk_idx, const uint8_t* allow,
                              const int32_t* req_offset, int32_t R, pmpe_route_rec* rec,
                              pmpe_stream_t stream) {
  pmpe_status st = check_desc(d, T);
  if (st != PMPE_OK) return st;
  if (layer < 0 || layer > 0xFFFF || R < 0 || R > PMPE_MAX_TOKENS) return PMPE_ERR_SHAPE;
  if (T == 0) return PMPE_OK;
  if (R < 1) return PMPE_ERR_SHAPE;
  if (!topk_idx || !allow || !req_offset || !rec) return PMPE_ERR_NULL;
  if (!aligned16(rec)) return PMPE_ERR_ALIGN;
  RecordArgs a{T, R, d->top_k, d->n_pub, layer, topk_idx, allow, req_offset, (uint32_t*)rec};
  return launched(launch_route_record(a, (hipStream_t)stream));
}

pmpe_status pmpe_cache_tag_check(const pmpe_cache_tag* cache, const pmpe_cache_tag* request) {
  if (!cache || !request) return PMPE_ERR_TAG_MISMATCH;
  if (cache->decision > 1u || request->decision > 1u) return PMPE_ERR_TAG_MISMATCH;
  unsigned diff = cache->decision ^ request->decision;
  for (int i = 0; i < 32; ++i) {
    diff |= (unsigned)(cache->model_revision[i] ^ request->model_revision[i]);
    diff |= (unsigned)(cache->checkpoint_fingerprint[i] ^ request->checkpoint_fingerprint[i]);
  }
  return diff == 0 ? PMPE_OK : PMPE_ERR_TAG_MISMATCH;
}

size_t pmpe_backward_workspace_bytes(const pmpe_layer_desc* d, int32_t T) {
  if (check_backward_desc(d, T) != PMPE_OK) return 0;
  return bwd_layout(d, T).total;
}

pmpe_status pmpe_backward(const pmpe_layer_desc* d, int32_t T, const void* x, const void* dout,
                          const int32_t* topk_idx, const float* topk_gate,
                          const int32_t* expert_count, const int32_t* expert_offset,
                          const int32_t* row_token, const int32_t* token_row, const void* y_perm,
                          const float* wr_pub, const float* wr_priv, const void* w13_pub,
                          const void* w2_pub, const void* w13_priv, const void* w2_priv,
                          const float* logit_bias, const void* w13_sh, const void* w2_sh,
                          const void* w2t_pub, const void* w13t_pub, const void* w2t_priv,
                          const void* w13t_priv, const float* ab, float* dx, float* dw13_priv,
                          float* dw2_priv, float* dwr_priv, uint32_t* grad_rows, void* ws,
                          size_t ws_bytes, pmpe_stream_t stream) {
  pmpe_status st = check_backward_desc(d, T);
  if (st != PMPE_OK) return st;
  if (!x || !dout || !topk_idx || !topk_gate || !expert_count || !expert_offset || !row_token ||
      !token_row || !y_perm || !wr_pub || !w13_pub || !w2_pub || !dx)
    return PMPE_ERR_NULL;
  if (d->n_priv > 0 && (!wr_priv || !w13_priv || !w2_priv || !dw13_priv || !dw2_priv || !dwr_priv))
    return PMPE_ERR_NULL;
  if (d->n_shared > 0 && (!w13_sh || !w2_sh)) return PMPE_ERR_NULL;
  // transposed weights: all of them (private ones when there is a private pool) or none
  const bool any_t = w2t_pub || w13t_pub || w2t_priv || w13t_priv;
  if (any_t && (!w2t_pub || !w13t_pub || (d->n_priv > 0 && (!w2t_priv || !w13t_priv))))
    return PMPE_ERR_NULL;
  const void* al[] = {x, dout, y_perm, w13_pub, w2_pub, w13_priv, w2_priv, ab, w13_sh, w2_sh,
                      w2t_pub, w13t_pub, w2t_priv, w13t_priv, dx, dw13_priv, dw2_priv, dwr_priv};
  for (const void* p : al)
    if (p && !aligned16(p)) return PMPE_ERR_ALIGN;
  if (T == 0) return PMPE_OK;
  const BwdLayout L = bwd_layout(d, T);
  if (!ws || ws_bytes < L.total) return PMPE_ERR_WORKSPACE;
  if (!aligned16(ws)) return PMPE_ERR_ALIGN;
  char* w = (char*)ws;
  BwdArgs a{T, d->hidden, d->inter, d->top_k, d->n_pub, d->n_priv, x, dout, topk_idx, topk_gate,
            expert_count, expert_offset, row_token, token_row, y_perm, wr_pub, wr_priv, w13_pub,
            w2_pub, w13_priv, w2_priv, ab, dx, dw13_priv, dw2_priv, dwr_priv, grad_rows,
            (uint16_t*)(w + L.xp), (uint16_t*)(w + L.dy), (float*)(w + L.ab), (uint16_t*)(w + L.hh),
            (uint16_t*)(w + L.da), (float*)(w + L.dxr), (float*)(w + L.dz), (float*)(w + L.part),
            d->gate_mode == PMPE_GATE_POOL_SOFTMAX ? 1 : 0, d->route_mode == PMPE_ROUTE_SOFT ? 1 : 0,
            bwd_pool_stride(d), logit_bias, (float*)(w + L.dzp),
            d->n_shared > 0 ? d->n_shared * d->shared_inter : 0, w13_sh, w2_sh,
            (float*)(w + L.absh), (uint16_t*)(w + L.dash),
            d->n_shared > 0 ? (float*)(w + L.dxsh) : nullptr,
            any_t ? w2t_pub : nullptr, w13t_pub, w2t_priv, w13t_priv, (uint16_t*)(w + L.dh),
            L.P > 0 ? (uint16_t*)(w + L.tr) : nullptr, L.P, (float*)(w + L.grow)};
  return launched(launch_backward(a, (hipStream_t)stream));
}

pmpe_status pmpe_adamw(void* param, int32_t param_dtype, float* master, const float* grad,
                       float* m, float* v, uint64_t n, int32_t step, float lr, float beta1,
                       float beta2, float eps, float weight_decay, pmpe_stream_t stream) {
  if (param_dtype != PMPE_F32 && param_dtype != PMPE_BF16) return PMPE_ERR_DTYPE;
  if ((param_dtype == PMPE_BF16) != (master != nullptr)) return PMPE_ERR_DTYPE;
  if (step < 1 || !std::isfinite(lr) || !std::isfinite(eps) || !std::isfinite(weight_decay) ||
      !(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f))
    return PMPE_ERR_SHAPE;
  if (n == 0) return PMPE_OK;
  if (!param || !grad || !m || !v) return PMPE_ERR_NULL;
  const void* al[] = {param, master, grad, m, v};
  for (const void* p : al)
    if (p && !aligned16(p)) return PMPE_ERR_ALIGN;
  const float c1 = (float)(1.0 - std::pow((double)beta1, (double)step));
  const float c2 = (float)(1.0 - std::pow((double)beta2, (double)step));
  AdamwArgs a{param, master, grad, m, v, n, lr, beta1, beta2, eps, 1.0f - lr * weight_decay, c1, c2};
  return launched(launch_adamw(a, (hipStream_t)stream));
}

pmpe_status pmpe_transpose_experts(const void* src, void* dst, int32_t n, int32_t rows,
                                   int32_t cols, pmpe_stream_t stream) {
  if (n < 0 || n > 65535 || rows < 0 || cols < 0 || rows % 64 != 0 || cols % 64 != 0)
    return PMPE_ERR_SHAPE;
  if ((int64_t)rows * cols >= ((int64_t)1 << 31)) return PMPE_ERR_SHAPE;
  if (n == 0 || rows == 0 || cols == 0) return PMPE_OK;
  if (!src || !dst) return PMPE_ERR_NULL;
  if (!aligned16(src) || !aligned16(dst)) return PMPE_ERR_ALIGN;
  if (src == dst) return PMPE_ERR_SHAPE;
  return launched(launch_transpose(src, dst, n, rows, cols, (hipStream_t)stream));
}

size_t pmpe_fingerprint_workspace_bytes(uint64_t nbytes) {
  if (nbytes > PMPE_FP_MAX_BYTES) return 0;
  size_t p0;
  return fingerprint_ws_parts(nbytes, &p0);
}

pmpe_status pmpe_fingerprint(const void* data, uint64_t nbytes, uint8_t* digest, void* ws,
                             size_t ws_bytes, pmpe_stream_t stream) {
  if (nbytes > PMPE_FP_MAX_BYTES) return PMPE_ERR_SHAPE;
  if (!digest || (nbytes > 0 && !data)) return PMPE_ERR_NULL;
  if (!aligned16(digest)) return PMPE_ERR_ALIGN;
  size_t p0;
  const size_t need = fingerprint_ws_parts(nbytes, &p0);
  if (need > 0) {
    if (!ws) return PMPE_ERR_NULL;
    if (ws_bytes < need) return PMPE_ERR_WORKSPACE;
    if (!aligned16(ws)) return PMPE_ERR_ALIGN;
  }
  FingerprintArgs a{data, nbytes, digest, (uint8_t*)ws, need > 0 ? (uint8_t*)ws + p0 : nullptr};
  return launched(launch_fingerprint(a, (hipStream_t)stream));
}

}  // extern "C"
