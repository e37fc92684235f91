// Internal declarations of libpmpe: device helpers and the launchers that the C ABI
// (pmpe_api.hip) calls after validating its arguments. gfx950 (CDNA4) only.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "pmpe.h"

namespace pmpe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// bf16 helpers (raw uint16 storage; conversions exact or round-to-nearest-even)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;  // quiet NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}
// Two floats -> packed bf16 pair (low half = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return f32_to_bf16_rne(a) | (f32_to_bf16_rne(b) << 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// SwiGLU backward of one element: upstream d = dL/dh, gate projection g, up projection u;
// h = silu(g) u, da = d u s (1 + g (1 - s)), db = d g s with s = sigmoid(g).
__device__ __forceinline__ void swiglu_bwd(float d, float g, float u, float& da, float& db, float& h) {
  const float s = 1.0f / (1.0f + __expf(-g));
  da = d * u * s * (1.0f + g * (1.0f - s));
  db = d * g * s;
  h = g * s * u;
}

// Wave-level helpers (wave64).
__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ float wave_sum(float v) {
  // butterfly: every lane ends with the bitwise-identical total
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = __shfl_xor(lo, mask, 64);
  hi = __shfl_xor(hi, mask, 64);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = __shfl(lo, src, 64);
  hi = __shfl(hi, src, 64);
  return ((uint64_t)hi << 32) | lo;
}

// ---------------------------------------------------------------------------
// Launchers (arguments already validated; T > 0)
// ---------------------------------------------------------------------------
struct RouteArgs {
  int T, H, n_pub, n_priv, k, gate_mode, act_bf16;
  const void* x;
  const float* wr_pub;
  const float* wr_priv;
  const float* bias;
  const uint32_t* words;
  int32_t* topk_idx;
  float* topk_gate;
  uint8_t* allow;
  float* kgap;
  uint32_t* dev_status;
  float* z;     // workspace [zsplit, T, zstride]: fp32 logits of each token's permitted pool
  int zstride;
  int soft;     // control arm: every token ranks the concatenated pool (z holds all E logits)
  int zsplit;   // partial logit arrays (K split of the logits); the top-k adds them in order
};
// K splits of the router logits for a batch (1 unless the wide large-batch kernel runs);
// the route workspace holds this many [T, zstride] fp32 arrays.
int route_ksplit(int T, int H, int n_pub, int n_priv, int act_bf16);
hipError_t launch_route(const RouteArgs& a, hipStream_t s);

struct DispatchArgs {
  int T, k, E, H, act_bf16;
  const int32_t* topk_idx;
  const void* x;
  int32_t* count;
  int32_t* offset;
  int32_t* row_token;
  int32_t* token_row;
  void* x_perm;
  uint64_t* mask;       // workspace [nchunks, E]: tokens of a chunk that selected an expert
  int32_t* chunk_base;  // workspace [nchunks, E]: first row of a chunk's tokens per expert
};
int dispatch_chunks(int T);
hipError_t launch_dispatch(const DispatchArgs& a, hipStream_t s);
// workspace pmpe_dispatch needs for a valid descriptor (its masks and chunk bases)
size_t dispatch_workspace_bytes(const pmpe_layer_desc* d, int32_t T);

struct FfnArgs {
  int T, H, I, n_pub, n_priv, k, act_bf16;
  int Is;  // shared intermediate (0 = no shared group)
  const void* x_perm;
  const void* x;
  const int32_t* count;
  const int32_t* offset;
  const int32_t* row_token;
  const void* w13_pub;
  const void* w2_pub;
  const void* w13_priv;
  const void* w2_priv;
  const void* w13_sh;
  const void* w2_sh;
  void* y_shared;
  void* y_perm;
  uint32_t* audit_rows;
  uint32_t* audit_calls;
  uint32_t* dev_status;
  void* h;     // workspace [T*k, I]
  void* h_sh;  // workspace [T, Is]
  float* ab_save = nullptr;  // optional [T*k, 2I]: fp32 gate and up projections (bf16 path)
  // fp8 (e4m3) expert weights: fp32 power-of-two scale per weight row, [n, 2I] and [n, H]
  const float* w13_scale_pub = nullptr;
  const float* w2_scale_pub = nullptr;
  const float* w13_scale_priv = nullptr;
  const float* w2_scale_priv = nullptr;
  int gather_a = 0;  // plain grouped product (launch_grouped_nt_gemm): A row r is x[row_token[r]]
};
hipError_t launch_expert_ffn(const FfnArgs& a, hipStream_t s);
hipError_t launch_expert_ffn_parts(const FfnArgs& a, hipStream_t s, int parts);
hipError_t launch_grouped_nt_gemm(const FfnArgs& a, hipStream_t s);
hipError_t launch_expert_ffn_fp8(const FfnArgs& a, hipStream_t s);

struct LoraArgs {
  int T, H, I, k, n_pub, n_priv, rank, gate;
  float scale;
  const int32_t* count;
  const int32_t* offset;
  const int32_t* row_token;
  const uint32_t* words;
  const void* x;
  const void* x_perm;
  const uint16_t* a13;
  const uint16_t* b1;
  const uint16_t* b3;
  const uint16_t* a2;
  const uint16_t* b2;
  const float* ab;     // [T*k, 2I] gate and up projections of the frozen expert
  uint16_t* h;         // [T*k, I]
  uint16_t* y_perm;    // [T*k, H]
  uint32_t* lora_rows; // [T] adapter executions per token
};
hipError_t launch_lora_pre(const LoraArgs& a, hipStream_t s);
hipError_t launch_lora_post(const LoraArgs& a, hipStream_t s);

struct CombineArgs {
  int T, H, k, act_bf16;
  const void* y_perm;
  const int32_t* token_row;
  const float* gate;
  const void* y_shared;
  void* out;
};
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

struct AuditArgs {
  int T, R;
  const uint32_t* rows;
  const uint8_t* allow;
  const int32_t* req_offset;
  uint64_t* req_rows;
  uint64_t* total;
  uint32_t* violations;
};
hipError_t launch_audit(const AuditArgs& a, hipStream_t s);

struct AdamwArgs {
  void* param;          // fp32, or bf16 when master is given
  float* master;        // fp32 master copy of a bf16 parameter, or NULL
  const float* grad;
  float* m;
  float* v;
  uint64_t n;
  float lr, beta1, beta2, eps, decay, c1, c2;  // decay = 1 - lr wd; c = bias corrections
};
hipError_t launch_adamw(const AdamwArgs& a, hipStream_t s);

struct RecordArgs {
  int T, R, k, n_pub, layer;
  const int32_t* topk_idx;
  const uint8_t* allow;
  const int32_t* req_offset;
  uint32_t* rec;  // [T, 4] words
};
hipError_t launch_route_record(const RecordArgs& a, hipStream_t s);

struct BwdArgs {
  int T, H, I, k, n_pub, n_priv;
  const void* x;          // [T, H] bf16
  const void* dout;       // [T, H] bf16
  const int32_t* topk_idx;
  const float* topk_gate;
  const int32_t* count;
  const int32_t* offset;
  const int32_t* row_token;
  const int32_t* token_row;
  const void* y_perm;     // [T*k, H] bf16
  const float* wr_pub;
  const float* wr_priv;
  const void* w13_pub;
  const void* w2_pub;
  const void* w13_priv;
  const void* w2_priv;
  const float* ab;        // [T*k, 2I] saved by the forward, or NULL: recomputed into AB
  float* dx;
  float* dw13_priv;
  float* dw2_priv;
  float* dwr_priv;
  uint32_t* grad_rows;
  // workspace
  uint16_t* Xp;    // [T*k, H]
  uint16_t* dY;    // [T*k, H] (written only where a later pass reads it)
  float* AB;       // [T*k, 2I]
  uint16_t* Hh;    // [T*k, I]
  uint16_t* dA13;  // [T*k, 2I]
  float* dXr;      // [T*k, H]
  float* dz_row;   // [T*k]: RENORM logit gradient per row; POOL_SOFTMAX gate gradient
  float* dwr_part; // [n_priv, BWD_DWR_SPLIT, H]
  // softmax over the whole pool and the soft-routing control
  int pool_gates, soft, pool_stride;
  const float* bias;      // [E] or NULL
  float* dz_pool;         // [T, pool_stride]
  // shared experts (frozen; input gradient only)
  int Is;
  const void* w13_sh;     // [2 Is, H]
  const void* w2_sh;      // [H, Is]
  float* AB_sh;           // [T, 2 Is]
  uint16_t* dA13_sh;      // [T, 2 Is]
  float* dXsh;            // [T, H] or NULL
  // transposed expert weights (K contiguous): W2^T [n, I, H], W13^T [n, H, 2I]; when all
  // are present the dh and row-input-gradient products run on the grouped NT GEMM
  const void* w2t_pub;
  const void* w13t_pub;
  const void* w2t_priv;
  const void* w13t_priv;
  uint16_t* dH;           // [T*k, I] bf16 (NT path)
  // private rows transposed and padded per expert ([3I + H, P] bf16), or NULL:
  // the weight gradients then run on the transposing GEMM
  uint16_t* tr;
  int P;
  float* g_row;           // [T*k]: the gate of each row (its upstream rows are g_row[r] dout[t])
};
constexpr int BWD_DWR_SPLIT = 16;  // row chunks per private expert in the router-row gradient

hipError_t launch_backward(const BwdArgs& a, hipStream_t s);
hipError_t launch_transpose(const void* src, void* dst, int n, int rows, int cols, hipStream_t s);
// dst [cols, P]: the private rows of src transposed and zero-padded per expert (src [rows,
// cols] in permuted row order, or [T, cols] read through row_token when that is not NULL);
// with row_scale, element (r, c) is bf16(row_scale[r] * src value).
hipError_t launch_transpose_priv(const void* src, const int32_t* row_token, const float* row_scale,
                                 void* dst, int rows_max, int cols, int P, const int32_t* count,
                                 const int32_t* offset, int n_pub, int n_priv, hipStream_t s);
// SwiGLU backward of the private rows of dH [rows, I] (row r's upstream gradient is
// g_row[r] * dH[r]) with [a; b] from AB [rows, 2I]: [da; db] into dA13 [rows, 2I] and,
// transposed and padded like launch_transpose_priv, into daT [2I, P]; h into hT [I, P].
hipError_t launch_swiglu_priv_t(const uint16_t* dH, const float* g_row, const float* AB, uint16_t* dA13,
                                uint16_t* daT, uint16_t* hT, int rows_max, int I, int P,
                                const int32_t* count, const int32_t* offset, int n_pub, int n_priv,
                                hipStream_t s);

// Weight gradients of the private experts on MFMA from K-contiguous operands:
// C[p] [M, N] fp32 = sum over the padded rows j of private expert p of AT[m][po_p + j] *
// BT[n][po_p + j], with AT [M, P] and BT [N, P] from launch_transpose_priv.
struct WgradArgs {
  int M, N, P, n_pub, n_priv;
  const uint16_t* AT;
  const uint16_t* BT;
  const int32_t* count;
  float* C;
};
hipError_t launch_wgrad(const WgradArgs& a, hipStream_t s);

// Fingerprint tree: 1 KiB leaves, 16 digests per inner node.
constexpr uint32_t kFpLeafBytes = 1024;
constexpr uint32_t kFpFanout = 16;

struct FingerprintArgs {
  const void* data;
  uint64_t nbytes;
  uint8_t* digest;  // 32 bytes out
  uint8_t* ws;      // >= 32 * leaves bytes (unused when there is one leaf)
  uint8_t* ws2;     // >= 32 * ceil(leaves / 16) bytes
};

uint64_t fingerprint_leaves(uint64_t nbytes);
hipError_t launch_fingerprint(const FingerprintArgs& a, hipStream_t s);

}  // namespace pmpe
