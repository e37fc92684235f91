/*
 * pmpe.h - C ABI of libpmpe, the forward pass of one policy-masked MoE layer on an
 * AMD Instinct MI355X (gfx950).
 *
 * Method: Policy-Masked Private Experts (arXiv 2608.06690). Trusted per-request
 * authorization tau selects either the original public expert pool or a disjoint,
 * added private pool; the hard mask m(tau) is applied to the router logits BEFORE
 * top-k (Sec. 3.1, mask equation), so an ineligible expert never enters the
 * candidate set (App. B.1). Missing or malformed authorization resolves to deny
 * (Sec. 3.1 resolver paragraph; App. B.1). A separate execution audit counts the
 * private rows that were physically executed (App. F.1, independent hooks; App. B.2,
 * row-indexed route counters).
 *
 * One layer forward is five calls, all asynchronous on one HIP stream:
 *
 *   pmpe_route       policy decode, masked fp32 router logits, top-k, gates
 *   pmpe_dispatch    per-expert counts, offsets, stable permutation, row gather
 *   pmpe_expert_ffn  SwiGLU experts (grouped GEMM) + private-row execution audit
 *   pmpe_combine     out[t] = sum_j gate[t,j] * y[t, expert j] (+ shared experts)
 *   pmpe_audit       per-request private rows, total, deny violations
 *
 * Conventions for every call
 * - All pointers except `d` are DEVICE pointers unless stated otherwise; `d` (the
 *   layer descriptor) is a host pointer read during the call only.
 * - The caller owns and allocates every buffer, including the workspace. The library
 *   allocates nothing and keeps no pointer after a call returns.
 * - Host-side validation runs before any launch; on failure the call returns a
 *   negative pmpe_status, launches nothing and writes nothing. Errors inside kernels
 *   surface at the caller's next synchronisation; conditions only the device can
 *   see (e.g. private rows reaching a NULL private weight pointer) set bits in the
 *   optional `dev_status` word.
 * - Calls are stream-ordered; a workspace may be shared by calls on one stream.
 * - T = 0 is valid: nothing is launched and PMPE_OK is returned (pmpe_audit still
 *   writes its outputs).
 * - Row-major layouts throughout. Expert ids: public [0, n_pub), private
 *   [n_pub, n_pub + n_priv).
 * - No C++ exception crosses this ABI.
 */
#ifndef PMPE_H
#define PMPE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque HIP stream handle (identical to hipStream_t); NULL = the default stream. */
typedef struct ihipStream_t* pmpe_stream_t;

typedef enum {
  PMPE_OK = 0,
  PMPE_ERR_NULL = -1,            /* a required pointer is NULL */
  PMPE_ERR_SHAPE = -2,           /* a size is out of the supported range */
  PMPE_ERR_K_EXCEEDS_POOL = -3,  /* top_k > n_pub or top_k > n_priv */
  PMPE_ERR_DTYPE = -4,           /* unsupported dtype combination */
  PMPE_ERR_ALIGN = -5,           /* a pointer is not 16-byte aligned */
  PMPE_ERR_WORKSPACE = -6,       /* workspace missing or smaller than pmpe_workspace_bytes */
  PMPE_ERR_LAUNCH = -7,          /* the HIP runtime refused a launch */
  PMPE_ERR_TAG_MISMATCH = -8,    /* a cache tag does not match the request (reuse refused) */
  PMPE_ERR_SCRATCH = -9          /* needs more scratch than the allocation-free entry holds */
} pmpe_status;

typedef enum { PMPE_F32 = 0, PMPE_BF16 = 1, PMPE_FP8_E4M3 = 2 } pmpe_dtype;

/* Gate normalisation (the paper does not fix it):
 * RENORM        softmax over the k selected logits (= pool softmax renormalised over
 *               the top-k);
 * POOL_SOFTMAX  softmax over the whole permitted pool, gates not renormalised. */
typedef enum { PMPE_GATE_RENORM_TOPK = 0, PMPE_GATE_POOL_SOFTMAX = 1 } pmpe_gate_mode;

/* Routing mode. MASKED is the method: the policy mask is applied before top-k. SOFT is
 * the paper's soft-routing control (Sec. 4.2, third row of the control matrix; App. E):
 * one router over the concatenated public and private pool, no mask, for every token
 * whatever its policy word. It exists to show what the mask prevents (deny tokens then
 * reach private experts and the execution audit counts them as violations); it is not
 * a safe configuration. */
typedef enum { PMPE_ROUTE_MASKED = 0, PMPE_ROUTE_SOFT = 1 } pmpe_route_mode;

/* Policy words. Exactly one 32-bit value allows; every other value - including
 * corrupted words - is malformed and resolves to deny (fail closed). */
#define PMPE_POLICY_ALLOW 0xA11C0DE5u
#define PMPE_POLICY_DENY 0x00000000u

/* Bits of the optional device status word. */
#define PMPE_DEV_PRIV_ROUTER_MISSING 0x1u  /* allow rows met wr_priv == NULL: routed as deny */
#define PMPE_DEV_PRIV_WEIGHTS_MISSING 0x2u /* private rows met NULL private expert weights:
                                              those rows were NOT executed, outputs zeroed */

/* Supported ranges (checked by host validation). */
#define PMPE_MAX_POOL 256  /* n_pub and n_priv each in [top_k, 256] */
#define PMPE_MAX_TOPK 16
#define PMPE_MAX_TOKENS (1 << 24)

typedef struct {
  int32_t hidden;       /* H, multiple of 128, 128..16384 */
  int32_t inter;        /* I of one routed expert, multiple of 64 */
  int32_t n_pub;        /* public (original, frozen) experts */
  int32_t n_priv;       /* private (added) experts */
  int32_t top_k;        /* k, 1..16, k <= min(n_pub, n_priv) */
  int32_t n_shared;     /* always-on shared experts (0 = none) */
  int32_t shared_inter; /* I of one shared expert (multiple of 64 when n_shared > 0) */
  int32_t act_dtype;    /* pmpe_dtype of x, x_perm, y_perm, y_shared, out */
  int32_t w_dtype;      /* pmpe_dtype of expert weights; must equal act_dtype */
  int32_t gate_mode;    /* pmpe_gate_mode */
  int32_t route_mode;   /* pmpe_route_mode; 0 (zero-initialised) = MASKED */
} pmpe_layer_desc;
/* The expert kernels use 32-bit byte offsets, so validation also requires fewer than
 * 2^31 elements in: T*top_k*max(hidden, inter), T*hidden, T*n_shared*shared_inter,
 * 2*inter*hidden (one expert's w13) and 2*n_shared*shared_inter*hidden. */

/* Bytes of workspace that any call below may need for T tokens (the maximum over
 * the calls, so one buffer serves all of them). 0 if the descriptor is invalid. */
size_t pmpe_workspace_bytes(const pmpe_layer_desc* d, int32_t T);

/* Static, NUL-terminated description of a pmpe_status value. */
const char* pmpe_status_string(int32_t status);

/* Library version, major * 10000 + minor * 100 + patch. */
int32_t pmpe_version(void);

/* Validation only: PMPE_OK if the descriptor and T are supported, else the status every
 * call would return for them. Launches nothing, so it also runs on a host without a GPU. */
pmpe_status pmpe_check_desc(const pmpe_layer_desc* d, int32_t T);

/*
 * pmpe_route - policy decode, masked router logits, top-k and gates.
 * (Sec. 3.1 mask equation and the sentence after it; App. B.1 masked routing and
 * steps 2 and 4 of the fail-closed request procedure.)
 *
 * For token t: tau_t = (policy_word[t] == PMPE_POLICY_ALLOW). The permitted pool is
 * the private ids if tau_t, else the public ids. Logits z_e = fp32(x_t . W_r[e]) (+
 * logit_bias[e], one fp32 add) are computed for the permitted pool ONLY: the other
 * pool's logits are never formed, and a deny token's x is never multiplied with
 * private router rows. The k largest logits win, equal fp32 values going to the
 * lower expert id (-0.0 == +0.0). With route_mode SOFT (control arm only) every token
 * ranks all n_pub + n_priv logits, wr_priv must not be NULL (else PMPE_ERR_NULL), and the
 * allow output still reports the resolved policy decision.
 *
 *   x            [T, H] act_dtype
 *   wr_pub       [n_pub, H] fp32, frozen router rows
 *   wr_priv      [n_priv, H] fp32, private gate rows; never read unless some token
 *                allows; may be NULL (allow tokens then route as deny and
 *                PMPE_DEV_PRIV_ROUTER_MISSING is set)
 *   logit_bias   [n_pub + n_priv] fp32 or NULL
 *   policy_word  [T] uint32 or NULL (NULL: every token denies)
 *   topk_idx     [T, k] int32 out: global expert ids, ascending within a token
 *   topk_gate    [T, k] fp32 out, aligned with topk_idx
 *   allow        [T] uint8 out: resolved tau (the route log's policy decision)
 *   kgap         [T] fp32 out or NULL: k-th minus (k+1)-th largest masked logit,
 *                +inf when the pool has exactly k experts
 *   dev_status   [1] uint32 in/out or NULL: status bits are OR-ed in
 *   ws, ws_bytes workspace (holds the fp32 pool logits; for bf16 batches of more than
 *                2048 tokens up to four partial arrays of a split over H, added in a
 *                fixed order), at least pmpe_workspace_bytes(d, T)
 */
pmpe_status pmpe_route(const pmpe_layer_desc* d, int32_t T, const void* x, const float* wr_pub,
                       const float* wr_priv, const float* logit_bias, const uint32_t* policy_word,
                       int32_t* topk_idx, float* topk_gate, uint8_t* allow, float* kgap,
                       uint32_t* dev_status, void* ws, size_t ws_bytes, pmpe_stream_t stream);

/*
 * pmpe_dispatch - group the T*k (token, expert) pairs by expert.
 * (Token permutation of the MoE forward; no passage of the paper describes it.)
 *
 * Rows of expert e are the tokens that selected e, in ascending token order; experts
 * are laid out in ascending id order. Deterministic (no order-dependent atomics).
 * Ids outside [0, E) get no row (token_row = -1) and are not counted. A token that
 * lists the same expert in several slots gets one row for it, in the first such slot;
 * the later slots get token_row = -1 (pmpe_route never repeats an id).
 *
 *   topk_idx       [T, k] int32 from pmpe_route (or any caller-built index)
 *   x              [T, H] act_dtype (read only if x_perm != NULL)
 *   expert_count   [E] int32 out, E = n_pub + n_priv
 *   expert_offset  [E + 1] int32 out: exclusive prefix sum of expert_count
 *   row_token      [T*k] int32 out: permuted row -> token
 *   token_row      [T*k] int32 out: (t, j) -> permuted row of token t's j-th expert
 *   x_perm         [T*k, H] act_dtype out or NULL: x gathered in permuted order; with
 *                  NULL, pmpe_expert_ffn gathers rows from x itself
 *   ws, ws_bytes   workspace, at least pmpe_workspace_bytes(d, T)
 */
pmpe_status pmpe_dispatch(const pmpe_layer_desc* d, int32_t T, const int32_t* topk_idx,
                          const void* x, int32_t* expert_count, int32_t* expert_offset,
                          int32_t* row_token, int32_t* token_row, void* x_perm, void* ws,
                          size_t ws_bytes, pmpe_stream_t stream);

/*
 * pmpe_dispatch_noalloc - pmpe_dispatch without a workspace argument.
 * For callers that cannot allocate device memory: code under HIP graph capture, serving
 * loops and harnesses that forbid hipMalloc.
 *
 * Same outputs, arguments (minus ws / ws_bytes), validation and errors as pmpe_dispatch.
 * Its per-chunk expert masks and chunk bases live in a file-scope device array of
 * PMPE_NOALLOC_SCRATCH_BYTES on each GPU the library runs on, held until the process
 * ends; a batch needing more (about T / 64 * (n_pub + n_priv) * 12 bytes) returns
 * PMPE_ERR_SCRATCH before anything is launched. Calls no hipMalloc, hipFree or other
 * allocating routine; the first call on a device (the current device, which must be the
 * stream's) looks up that device's copy of the array once. Every call on one GPU uses
 * that GPU's single array: calls that overlap on one GPU (two streams, two threads)
 * race. Nothing in the array has to start at zero: every call writes what it reads.
 */
#define PMPE_NOALLOC_SCRATCH_BYTES ((size_t)2 << 20)
pmpe_status pmpe_dispatch_noalloc(const pmpe_layer_desc* d, int32_t T, const int32_t* topk_idx,
                                  const void* x, int32_t* expert_count, int32_t* expert_offset,
                                  int32_t* row_token, int32_t* token_row, void* x_perm,
                                  pmpe_stream_t stream);

/*
 * pmpe_expert_ffn - run every expert with at least one row, and the shared group.
 * (Disjoint private pool copying the expert architecture, Sec. 3.1; bias-free SwiGLU
 * with gate, up and down projections, Sec. 4.2; execution audit, App. F.1.)
 *
 * For expert e with n_e = expert_count[e] > 0 rows X (rows offset_e .. offset_e+n_e-1
 * of x_perm, or x[row_token[r]] when x_perm is NULL):
 *   h = silu(X Wg^T) * (X Wu^T)   (fp32 accumulate, h rounded to act_dtype)
 *   y_perm[rows] = h Wd^T         (fp32 accumulate, rounded to act_dtype)
 * Experts with zero rows load no weights and write nothing. Private weights are read
 * only for private experts that have rows, so an all-deny batch works with every
 * private pointer NULL.
 *
 * Audit (written here, by the code that executes the rows, not from the route log):
 *   audit_token_rows[row_token[r]] += 1 for every executed private row r;
 *   audit_priv_calls[e - n_pub]     += 1 for every private expert run with >= 1 row.
 * Both accumulate across calls; the caller zeroes them between decisions.
 *
 *   w13_pub   [n_pub, 2I, H]: rows [0, I) gate projection, rows [I, 2I) up projection
 *   w2_pub    [n_pub, H, I]: down projection
 *   w13_priv  [n_priv, 2I, H], w2_priv [n_priv, H, I]; may be NULL when no private row
 *             exists (otherwise PMPE_DEV_PRIV_WEIGHTS_MISSING is set, the rows are not
 *             executed, not audited, and their y_perm rows are zero)
 *   x         [T, H] act_dtype: needed if x_perm == NULL or n_shared > 0
 *   w13_sh    [2 Is, H], w2_sh [H, Is], Is = n_shared * shared_inter: the shared
 *             experts as one SwiGLU whose intermediate is their concatenation
 *             (gate rows of all shared experts, then their up rows); NULL if
 *             n_shared == 0
 *   y_shared  [T, H] act_dtype out (shared-group output), NULL if n_shared == 0
 *   y_perm    [T*k, H] act_dtype out
 *   audit_token_rows [T] uint32 in/out;  audit_priv_calls [n_priv] uint32 in/out or NULL
 *   dev_status [1] uint32 in/out or NULL
 */
pmpe_status pmpe_expert_ffn(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                            const void* x, const int32_t* expert_count,
                            const int32_t* expert_offset, const int32_t* row_token,
                            const void* w13_pub, const void* w2_pub, const void* w13_priv,
                            const void* w2_priv, const void* w13_sh, const void* w2_sh,
                            void* y_shared, void* y_perm, uint32_t* audit_token_rows,
                            uint32_t* audit_priv_calls, uint32_t* dev_status, void* ws,
                            size_t ws_bytes, pmpe_stream_t stream);

/*
 * pmpe_expert_ffn_train - pmpe_expert_ffn that also stores, for every routed row r, the
 * fp32 gate and up projections ab[r] = [W1 x; W3 x] (2I values) that pmpe_backward needs
 * (Sec. 3.2: the private pool is trained through the same forward). Same arguments and
 * errors as pmpe_expert_ffn plus ab (device, [T*k, 2I] fp32, 16-byte aligned, not NULL);
 * bf16 only (PMPE_ERR_DTYPE otherwise). The shared group's projections are not stored.
 * Rows of private experts whose weights are NULL are not executed and their ab rows are
 * left unwritten.
 */
pmpe_status pmpe_expert_ffn_train(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                                  const void* x, const int32_t* expert_count,
                                  const int32_t* expert_offset, const int32_t* row_token,
                                  const void* w13_pub, const void* w2_pub, const void* w13_priv,
                                  const void* w2_priv, const void* w13_sh, const void* w2_sh,
                                  void* y_shared, void* y_perm, uint32_t* audit_token_rows,
                                  uint32_t* audit_priv_calls, uint32_t* dev_status, float* ab,
                                  void* ws, size_t ws_bytes, pmpe_stream_t stream);

/*
 * pmpe_combine - merge the selected experts' outputs into the layer output.
 * (Merge into the frozen upper transformer, Fig. 1 and Sec. 3.1.)
 *
 *   out[t] = sum_{j<k} topk_gate[t,j] * y_perm[token_row[t,j]]  (+ y_shared[t])
 * accumulated in fp32 in slot order j = 0..k-1 and rounded once to act_dtype, so
 * the result is bitwise deterministic.
 *
 *   y_perm [T*k, H], token_row [T*k], topk_gate [T*k] fp32, y_shared [T, H] or NULL,
 *   out [T, H] act_dtype
 */
pmpe_status pmpe_combine(const pmpe_layer_desc* d, int32_t T, const void* y_perm,
                         const int32_t* token_row, const float* topk_gate,
                         const void* y_shared, void* out, pmpe_stream_t stream);

/*
 * pmpe_audit - reduce the execution audit per request.
 * (Route counters indexed by row, App. B.2; zero private execution under deny, G1.)
 *
 *   audit_token_rows   [T] uint32 from pmpe_expert_ffn
 *   allow              [T] uint8 from pmpe_route
 *   req_offset         [R + 1] int32: request r owns tokens [req_offset[r],
 *                      req_offset[r+1]); non-decreasing, req_offset[0] = 0,
 *                      req_offset[R] = T (a device array)
 *   req_private_rows   [R] uint64 out
 *   total_private_rows [1] uint64 out
 *   deny_violations    [1] uint32 out: tokens inside the requests with allow == 0 and
 *                      a nonzero count
 */
pmpe_status pmpe_audit(const pmpe_layer_desc* d, int32_t T, const uint32_t* audit_token_rows,
                       const uint8_t* allow, const int32_t* req_offset, int32_t R,
                       uint64_t* req_private_rows, uint64_t* total_private_rows,
                       uint32_t* deny_violations, pmpe_stream_t stream);

/*
 * pmpe_expert_ffn_fp8 - pmpe_expert_ffn with expert weights stored as fp8 (OCP e4m3) and
 * one fp32 scale per weight row that is a power of two: the weight is q * scale. A
 * precision variant (the paper's models ran in bf16); activations, accumulation and
 * outputs stay as in the bf16 path. Because the scales are powers of two and every e4m3
 * value is exactly a bf16 value, the products equal those of the bf16 kernel on the
 * dequantised weights; the weight bytes read from HBM halve.
 *
 *   d->act_dtype PMPE_BF16, d->w_dtype PMPE_FP8_E4M3, d->n_shared == 0
 *   w13_* [n, 2I, H] and w2_* [n, H, I] fp8 bytes; w13s_* [n, 2I] and w2s_* [n, H] fp32
 *   scales (NULL exactly when the matching private weights are NULL)
 * Other arguments, the audit and the errors as pmpe_expert_ffn; PMPE_ERR_DTYPE for other
 * dtypes, PMPE_ERR_SHAPE with shared experts. The scales are not checked on the device.
 */
pmpe_status pmpe_expert_ffn_fp8(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                                const void* x, const int32_t* expert_count,
                                const int32_t* expert_offset, const int32_t* row_token,
                                const void* w13_pub, const void* w2_pub, const void* w13_priv,
                                const void* w2_priv, const float* w13s_pub, const float* w2s_pub,
                                const float* w13s_priv, const float* w2s_priv, void* y_perm,
                                uint32_t* audit_token_rows, uint32_t* audit_priv_calls,
                                uint32_t* dev_status, void* ws, size_t ws_bytes,
                                pmpe_stream_t stream);

/*
 * pmpe_expert_ffn_lora - the request-gated LoRA control arm (Sec. 4.2 matched expert-LoRA
 * baseline; Sec. 5.2 and App. F.2: a request gate on an adapter is a logical switch,
 * and the paper's gated adapter still executed 1,225 times under deny). It exists to show
 * that failure class next to the disjoint private pool; it is not a safe configuration.
 *
 * The frozen public experts run as in pmpe_expert_ffn, with rank-r adapters on each
 * expert's gate, up and down projections scaled by s and by the row's decision tau
 * (policy_word of its token == PMPE_POLICY_ALLOW):
 *   g = Wg x + tau s Bg (Ag x),  u = Wu x + tau s Bu (Au x),  h = silu(g) u,
 *   y = Wd h + tau s Bd (Ad h).
 * gate selects where the decision is applied (PMPE_LORA_GATE_*): before any adapter work
 * per row, per tile of PMPE_LORA_TILE_ROWS consecutive rows of one expert (a tile with
 * an allowed row runs its adapters for all its rows), or only on the result. y_perm is
 * the same under every gate; lora_rows[t] (uint32 [T], accumulated, not cleared) gains 2
 * for every row of token t whose adapters physically ran (one for the gate/up adapters,
 * one for the down adapter), so pmpe_audit over it reports denied tokens that executed
 * adapters. Rows of private experts (none when the route used deny words only) get no
 * adapter.
 *
 *   a13 [n_pub, 2r, H], b1 and b3 [n_pub, I, r], a2 [n_pub, r, I], b2 [n_pub, H, r] bf16
 *   rank 1..128, scale the adapter scale s (alpha / r)
 * Other arguments as pmpe_expert_ffn; ws: pmpe_expert_ffn_lora_workspace_bytes(d, T).
 * Errors: as pmpe_expert_ffn, PMPE_ERR_DTYPE unless bf16, PMPE_ERR_SHAPE for a rank or gate
 * out of range or hidden / inter above 8192.
 */
typedef enum {
  PMPE_LORA_GATE_ROW = 0,     /* a denied row is skipped before any adapter work */
  PMPE_LORA_GATE_TILE = 1,    /* the decision is taken per tile of rows */
  PMPE_LORA_GATE_POSTHOC = 2  /* every row runs the adapters; the decision selects the result */
} pmpe_lora_gate;
#define PMPE_LORA_TILE_ROWS 64

size_t pmpe_expert_ffn_lora_workspace_bytes(const pmpe_layer_desc* d, int32_t T);

pmpe_status pmpe_expert_ffn_lora(const pmpe_layer_desc* d, int32_t T, const void* x_perm,
                                 const void* x, const int32_t* expert_count,
                                 const int32_t* expert_offset, const int32_t* row_token,
                                 const uint32_t* policy_word, const void* w13_pub,
                                 const void* w2_pub, const void* a13, const void* b1,
                                 const void* b3, const void* a2, const void* b2, int32_t rank,
                                 float scale, int32_t gate, void* y_perm, uint32_t* lora_rows,
                                 uint32_t* dev_status, void* ws, size_t ws_bytes,
                                 pmpe_stream_t stream);

/*
 * pmpe_route_record - export the route audit of one layer call: one record per token
 * with the layer, the request row, the token's position in the request, the selected
 * pool and the policy decision (App. B.1, fifth step of the fail-closed request
 * procedure; App. B.2: route counters are indexed by row and layer, so a batch total
 * cannot hide cross-row leakage). The records come from the route log (topk_idx,
 * allow), not from the expert kernels, so they can be reconciled against the
 * independent execution counters of pmpe_expert_ffn / pmpe_audit.
 *
 *   layer        layer index written into every record (0..65535)
 *   topk_idx     [T*k], allow [T]        from pmpe_route
 *   req_offset   [R + 1] device, as in pmpe_audit (R >= 1 when T > 0)
 *   rec          [T] pmpe_route_rec out, 16-byte aligned
 */
#define PMPE_POOL_PUBLIC 0u  /* every selected expert is public */
#define PMPE_POOL_PRIVATE 1u /* every selected expert is private */
#define PMPE_POOL_MIXED 2u   /* both (only the soft-routing control can do this) */
typedef struct {
  uint32_t layer_decision_pool; /* bits 0-15 layer, bit 16 decision (1 allow), bits 24-31 pool */
  int32_t row;                  /* request (batch row) index */
  int32_t token;                /* position of the token in its request */
  uint32_t private_mask;        /* bit j: the expert in slot j (ascending ids) is private */
} pmpe_route_rec;

pmpe_status pmpe_route_record(const pmpe_layer_desc* d, int32_t T, int32_t layer,
                              const int32_t* topk_idx, const uint8_t* allow,
                              const int32_t* req_offset, int32_t R, pmpe_route_rec* rec,
                              pmpe_stream_t stream);

/*
 * pmpe_cache_tag_check - host-side guard for cached attention state (App. B.1, third
 * step of the fail-closed request procedure; App. B.2: caches are tagged with the
 * policy decision, the model revision and the checkpoint fingerprint, and reuse across
 * tags is refused before a model call).
 *
 * Returns PMPE_OK only when both tags are present, both decisions are well formed (0
 * deny or 1 allow) and every field is equal; PMPE_ERR_TAG_MISMATCH otherwise (a missing
 * or malformed tag is refused, never treated as a match). Host pointers; no GPU work.
 */
typedef struct {
  uint32_t decision;                 /* resolved policy of the request: 1 allow, 0 deny */
  uint8_t model_revision[32];        /* e.g. SHA-256 of the model revision string */
  uint8_t checkpoint_fingerprint[32]; /* pmpe_fingerprint of the loaded weights */
} pmpe_cache_tag;

pmpe_status pmpe_cache_tag_check(const pmpe_cache_tag* cache, const pmpe_cache_tag* request);

/*
 * pmpe_backward - private-only backward of one layer for an upstream gradient dout.
 * (G2 of Sec. 2.2: frozen public parameters are not optimised and stay unchanged;
 * Sec. 3.2: only the private gate and the private expert weights require gradients.)
 *
 * Gradients are formed for the private expert weights and the private router rows
 * only; the public experts, the public router rows and the logit bias are frozen and
 * no gradient of theirs is ever formed or written. The input gradient flows through
 * every expert the forward executed (public ones included) and through the router:
 *
 *   dg_tj   = dout_t . y_{e_tj}(x_t)                     (y_perm of the forward)
 *   dz_tj   = g_tj (dg_tj - sum_i g_ti dg_ti)            (RENORM gates)
 *   dz_te   = p_te ([e selected] dg_te - sum_i p_ti dg_ti) (POOL_SOFTMAX, every pool
 *             member e, p = softmax of the recomputed fp32 pool logits)
 *   dx_t    = sum_j W13_e^T (da; db)_tj + sum_e dz_te W_r[e] (+ the shared experts'
 *             input gradient for upstream dout_t)
 *   dW2_p   = sum over rows of private expert p of (g dout_t) h^T
 *   dW13_p  = sum over rows of p of (da; db) x_t^T
 *   dW_r[p] = sum over rows of p of dz x_t
 * with a = W1 x, b = W3 x, s = sigmoid(a), h = a s b, dh = W2^T (g dout_t),
 * da = dh b s (1 + a (1 - s)), db = dh a s. The route (selection and gates) is the
 * forward's. Every output element is summed by one thread in a fixed order: two calls
 * on the same inputs give bitwise equal results.
 *
 * Supported: bf16, both gate modes (POOL_SOFTMAX with hidden <= 8192), shared experts
 * (frozen), inter and n_shared * shared_inter multiples of 128; either route mode (under PMPE_ROUTE_SOFT,
 * deny rows that reached private experts also feed private gradients - the control
 * shows what the mask prevents).
 *
 *   x [T, H], dout [T, H]                       bf16
 *   topk_idx, topk_gate [T*k], expert_count, expert_offset [E], row_token, token_row
 *   [T*k], y_perm [T*k, H]                      the forward's route, dispatch and
 *                                               expert outputs
 *   wr_pub, wr_priv, w13_*, w2_*                the forward's weights
 *   logit_bias [E] fp32 or NULL                 the route's logit bias (POOL_SOFTMAX
 *                                               recomputes the pool logits; a token's
 *                                               pool is the one its selection lies in)
 *   w13_sh, w2_sh                               shared experts (n_shared > 0)
 *   w2t_pub [n_pub, I, H], w13t_pub [n_pub, H, 2I], w2t_priv, w13t_priv
 *                                               transposed expert weights
 *                                               (pmpe_transpose_experts), all or none
 *                                               (the private ones only when n_priv > 0):
 *                                               with them the products with W2 and W13
 *                                               run on the forward's grouped GEMM
 *   ab [T*k, 2I] fp32 or NULL                   the gate and up projections saved by
 *                                               pmpe_expert_ffn_train; NULL recomputes
 *                                               them (one more grouped GEMM)
 *   dx [T, H] fp32                              out
 *   dw13_priv [n_priv, 2I, H], dw2_priv [n_priv, H, I], dwr_priv [n_priv, H]
 *                                               fp32 out, overwritten (an expert with
 *                                               no rows gets zeros)
 *   grad_rows [n_priv] uint32 out or NULL       rows that entered each private
 *                                               expert's gradient
 *   ws                                          pmpe_backward_workspace_bytes(d, T)
 *                                               bytes
 * x, dout, y_perm, every weight array, ab, ws, dx and the three gradient outputs are
 * 16-byte aligned (dx is written in 16-byte vectors).
 *
 * Errors: PMPE_ERR_DTYPE (not bf16), PMPE_ERR_SHAPE (inter or the shared width not a
 * multiple of 128), PMPE_ERR_NULL, PMPE_ERR_ALIGN, PMPE_ERR_WORKSPACE.
 */
size_t pmpe_backward_workspace_bytes(const pmpe_layer_desc* d, int32_t T);

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
                          size_t ws_bytes, pmpe_stream_t stream);

/*
 * pmpe_adamw - one AdamW step over one private parameter tensor (G2 of Sec. 2.2: the
 * optimizer is given the private parameters only, so a frozen public tensor is never
 * an argument of this call; Sec. 3.2 and App. C.1: fused AdamW). Decoupled weight decay:
 *   p <- p (1 - lr wd); m <- b1 m + (1 - b1) g; v <- b2 v + (1 - b2) g^2;
 *   p <- p - lr (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps)
 * in fp32. A bf16 parameter (param_dtype PMPE_BF16) needs an fp32 master copy that takes
 * the update; the bf16 weight is then its round-to-nearest-even value.
 *
 *   param     device, n elements of param_dtype (updated)
 *   master    device fp32 [n] (updated) for PMPE_BF16, must be NULL for PMPE_F32
 *   grad      device fp32 [n]; m, v device fp32 [n] (updated; zero before step 1)
 *   step      1-based step count
 * All pointers 16-byte aligned. Errors: PMPE_ERR_NULL, PMPE_ERR_ALIGN, PMPE_ERR_DTYPE,
 * PMPE_ERR_SHAPE (step < 1, or a hyper-parameter that is not finite, or betas outside [0,1)).
 */
pmpe_status pmpe_adamw(void* param, int32_t param_dtype, float* master, const float* grad,
                       float* m, float* v, uint64_t n, int32_t step, float lr, float beta1,
                       float beta2, float eps, float weight_decay, pmpe_stream_t stream);

/*
 * pmpe_transpose_experts - dst[e] = src[e]^T for n bf16 matrices of [rows, cols] (rows and
 * cols multiples of 64, fewer than 2^31 elements each, n <= 65535, src and dst distinct
 * and 16-byte aligned). Makes the transposed expert weights pmpe_backward can use; frozen
 * public weights need it once, trained private weights after every optimizer step.
 */
pmpe_status pmpe_transpose_experts(const void* src, void* dst, int32_t n, int32_t rows,
                                   int32_t cols, pmpe_stream_t stream);

/*
 * pmpe_fingerprint - SHA-256 tree digest of a device buffer, to show that the frozen
 * public weights are unchanged (hashed before and after training and after a reload,
 * Sec. 3.2 training and checkpointing, Sec. 5.1, App. C.1).
 *
 * Definition: level 0 is the SHA-256 digest (FIPS 180-4) of every PMPE_FP_LEAF_BYTES
 * chunk of the buffer, in order (the last chunk may be short; an empty buffer is one
 * empty chunk). Level j+1 is the SHA-256 digest of the concatenation of each run of up
 * to PMPE_FP_FANOUT consecutive level-j digests. The fingerprint is the single digest
 * of the first level that has one; a buffer of at most PMPE_FP_LEAF_BYTES bytes thus
 * has SHA-256(buffer) as its fingerprint. A set of tensors is fingerprinted by
 * fingerprinting the concatenation of their fingerprints.
 *
 *   data     device, nbytes bytes, any alignment (16-byte aligned data loads whole
 *            64-byte blocks as vectors; other data is read byte by byte, more slowly);
 *            may be NULL only when nbytes == 0
 *   nbytes   0 .. PMPE_FP_MAX_BYTES
 *   digest   device, 32 bytes out, 16-byte aligned: the digest bytes in standard order
 *   ws       device workspace of pmpe_fingerprint_workspace_bytes(nbytes) bytes,
 *            16-byte aligned; may be NULL when that size is 0
 *
 * Errors: PMPE_ERR_NULL (data with nbytes > 0, or digest, or a needed ws is NULL),
 * PMPE_ERR_SHAPE (nbytes too large), PMPE_ERR_ALIGN (digest or ws), PMPE_ERR_WORKSPACE.
 * The call is asynchronous on `stream`; data must not change until it has completed.
 */
#define PMPE_FP_LEAF_BYTES 1024
#define PMPE_FP_FANOUT 16
#define PMPE_FP_MAX_BYTES ((uint64_t)1 << 46)

size_t pmpe_fingerprint_workspace_bytes(uint64_t nbytes);

pmpe_status pmpe_fingerprint(const void* data, uint64_t nbytes, uint8_t* digest, void* ws,
                             size_t ws_bytes, pmpe_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PMPE_H */
