"""MI355X-native policy-masked MoE layer (Policy-Masked Private Experts, arXiv 2608.06690).

The computation lives in libpmpe.so (HIP kernels for gfx950 behind the C ABI of
include/pmpe.h); this package is its binding."""
from ._native import (PMPE_BF16, PMPE_F32, PMPE_GATE_POOL_SOFTMAX, PMPE_GATE_RENORM_TOPK,  # noqa: F401
                      PMPE_POLICY_ALLOW, PMPE_POLICY_DENY, PMPE_ROUTE_MASKED, PMPE_ROUTE_SOFT,
                      PMPE_FP_FANOUT, PMPE_FP_LEAF_BYTES, LayerDesc, PmpeError,
                      fingerprint_tensors, make_desc, pmpe_fingerprint,
                      pmpe_fingerprint_workspace_bytes, pmpe_backward,
                      pmpe_backward_workspace_bytes, pmpe_expert_ffn_train,
                      PMPE_POOL_MIXED, PMPE_POOL_PRIVATE, PMPE_POOL_PUBLIC, CacheTag,
                      make_cache_tag, pmpe_cache_tag_check, pmpe_route_record,
                      PMPE_LORA_GATE_POSTHOC, PMPE_LORA_GATE_ROW, PMPE_LORA_GATE_TILE,
                      PMPE_LORA_TILE_ROWS, pmpe_expert_ffn_lora, pmpe_expert_ffn_lora_workspace_bytes,
                      pmpe_adamw, pmpe_transpose_experts, PMPE_FP8_E4M3, pmpe_expert_ffn_fp8,
                      pmpe_audit, pmpe_check_desc, pmpe_combine, pmpe_dispatch, pmpe_expert_ffn,
                      pmpe_dispatch_noalloc, PMPE_ERR_SCRATCH, PMPE_NOALLOC_SCRATCH_BYTES,
                      pmpe_route, pmpe_version, pmpe_workspace_bytes)
from .layer import (AuditBuffers, GradBuffers, LayerBuffers, PolicyMaskedMoE,  # noqa: F401
                    PrivateAdamW)
from .policy import policy_word, request_offsets, resolve_policy, token_policy_words  # noqa: F401
