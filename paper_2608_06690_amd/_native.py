"""ctypes binding of libpmpe (include/pmpe.h): argument marshalling only.

Every function has the name of the C entry point and takes torch tensors (or None)
where the C call takes device pointers; the HIP stream defaults to torch's current
stream. A negative status raises PmpeError. Every step of the layer runs in the HIP
kernels of libpmpe; if the library is missing, importing this module fails.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# Only the library built in the package directory is loaded: it is the code that
# enforces the policy mask and writes the execution audit.
LIB_PATH = os.path.join(_PKG, "libpmpe.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is not built; run `python -m paper_2608_06690_amd.build` "
        "(or __graft_entry__.build()) first")

_lib = ctypes.CDLL(LIB_PATH)

PMPE_OK = 0
PMPE_F32 = 0
PMPE_BF16 = 1
PMPE_FP8_E4M3 = 2
PMPE_GATE_RENORM_TOPK = 0
PMPE_GATE_POOL_SOFTMAX = 1
PMPE_ROUTE_MASKED = 0
PMPE_ROUTE_SOFT = 1
PMPE_POLICY_ALLOW = 0xA11C0DE5
PMPE_POLICY_DENY = 0x00000000
PMPE_DEV_PRIV_ROUTER_MISSING = 0x1
PMPE_DEV_PRIV_WEIGHTS_MISSING = 0x2

STATUS_NAMES = {
    0: "PMPE_OK", -1: "PMPE_ERR_NULL", -2: "PMPE_ERR_SHAPE", -3: "PMPE_ERR_K_EXCEEDS_POOL",
    -4: "PMPE_ERR_DTYPE", -5: "PMPE_ERR_ALIGN", -6: "PMPE_ERR_WORKSPACE", -7: "PMPE_ERR_LAUNCH",
    -8: "PMPE_ERR_TAG_MISMATCH", -9: "PMPE_ERR_SCRATCH",
}
PMPE_ERR_TAG_MISMATCH = -8
PMPE_ERR_SCRATCH = -9
PMPE_NOALLOC_SCRATCH_BYTES = 2 << 20
PMPE_LORA_GATE_ROW = 0
PMPE_LORA_GATE_TILE = 1
PMPE_LORA_GATE_POSTHOC = 2
PMPE_LORA_TILE_ROWS = 64
PMPE_POOL_PUBLIC = 0
PMPE_POOL_PRIVATE = 1
PMPE_POOL_MIXED = 2


class PmpeError(RuntimeError):
    def __init__(self, status: int, call: str):
        self.status = status
        msg = _lib.pmpe_status_string(status).decode()
        super().__init__(f"{call}: {STATUS_NAMES.get(status, status)} ({msg})")


class LayerDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "hidden", "inter", "n_pub", "n_priv", "top_k", "n_shared", "shared_inter",
        "act_dtype", "w_dtype", "gate_mode", "route_mode")]


class CacheTag(ctypes.Structure):
    """pmpe_cache_tag: resolved decision (1 allow, 0 deny), model revision digest and
    checkpoint fingerprint (32 bytes each)."""
    _fields_ = [("decision", ctypes.c_uint32), ("model_revision", ctypes.c_uint8 * 32),
                ("checkpoint_fingerprint", ctypes.c_uint8 * 32)]


def make_cache_tag(decision: int, model_revision: bytes, checkpoint_fingerprint: bytes) -> CacheTag:
    if len(model_revision) != 32 or len(checkpoint_fingerprint) != 32:
        raise ValueError("model_revision and checkpoint_fingerprint are 32-byte digests")
    t = CacheTag()
    t.decision = decision
    t.model_revision[:] = list(model_revision)
    t.checkpoint_fingerprint[:] = list(checkpoint_fingerprint)
    return t


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t
_DESC = ctypes.POINTER(LayerDesc)

_lib.pmpe_version.restype = _I32
_lib.pmpe_version.argtypes = []
_lib.pmpe_status_string.restype = ctypes.c_char_p
_lib.pmpe_status_string.argtypes = [_I32]
_lib.pmpe_workspace_bytes.restype = _SZ
_lib.pmpe_workspace_bytes.argtypes = [_DESC, _I32]
_lib.pmpe_check_desc.restype = _I32
_lib.pmpe_check_desc.argtypes = [_DESC, _I32]
_lib.pmpe_route.restype = _I32
_lib.pmpe_route.argtypes = [_DESC, _I32] + [_P] * 10 + [_P, _SZ, _P]
_lib.pmpe_dispatch.restype = _I32
_lib.pmpe_dispatch.argtypes = [_DESC, _I32] + [_P] * 7 + [_P, _SZ, _P]
_lib.pmpe_dispatch_noalloc.restype = _I32
_lib.pmpe_dispatch_noalloc.argtypes = [_DESC, _I32] + [_P] * 7 + [_P]
_lib.pmpe_expert_ffn.restype = _I32
_lib.pmpe_expert_ffn.argtypes = [_DESC, _I32] + [_P] * 16 + [_P, _SZ, _P]
_lib.pmpe_combine.restype = _I32
_lib.pmpe_combine.argtypes = [_DESC, _I32] + [_P] * 5 + [_P]
_lib.pmpe_audit.restype = _I32
_lib.pmpe_audit.argtypes = [_DESC, _I32, _P, _P, _P, _I32, _P, _P, _P, _P]

_lib.pmpe_backward_workspace_bytes.restype = _SZ
_lib.pmpe_backward_workspace_bytes.argtypes = [_DESC, _I32]
_lib.pmpe_backward.restype = _I32
_lib.pmpe_backward.argtypes = [_DESC, _I32] + [_P] * 28 + [_P, _SZ, _P]
_lib.pmpe_transpose_experts.restype = _I32
_lib.pmpe_transpose_experts.argtypes = [_P, _P, _I32, _I32, _I32, _P]
_lib.pmpe_expert_ffn_train.restype = _I32
_lib.pmpe_expert_ffn_train.argtypes = [_DESC, _I32] + [_P] * 17 + [_P, _SZ, _P]
_lib.pmpe_expert_ffn_fp8.restype = _I32
_lib.pmpe_expert_ffn_fp8.argtypes = [_DESC, _I32] + [_P] * 17 + [_P, _SZ, _P]
_lib.pmpe_expert_ffn_lora_workspace_bytes.restype = _SZ
_lib.pmpe_expert_ffn_lora_workspace_bytes.argtypes = [_DESC, _I32]
_lib.pmpe_expert_ffn_lora.restype = _I32
_lib.pmpe_expert_ffn_lora.argtypes = ([_DESC, _I32] + [_P] * 13 + [_I32, ctypes.c_float, _I32]
                                      + [_P] * 3 + [_P, _SZ, _P])
_lib.pmpe_adamw.restype = _I32
_lib.pmpe_adamw.argtypes = [_P, _I32, _P, _P, _P, _P, ctypes.c_uint64, _I32] + [ctypes.c_float] * 5 + [_P]
_lib.pmpe_route_record.restype = _I32
_lib.pmpe_route_record.argtypes = [_DESC, _I32, _I32, _P, _P, _P, _I32, _P, _P]
_lib.pmpe_cache_tag_check.restype = _I32
_lib.pmpe_cache_tag_check.argtypes = [ctypes.POINTER(CacheTag), ctypes.POINTER(CacheTag)]
_lib.pmpe_fingerprint_workspace_bytes.restype = _SZ
_lib.pmpe_fingerprint_workspace_bytes.argtypes = [ctypes.c_uint64]
_lib.pmpe_fingerprint.restype = _I32
_lib.pmpe_fingerprint.argtypes = [_P, ctypes.c_uint64, _P, _P, _SZ, _P]

EXPORTED = ["pmpe_version", "pmpe_status_string", "pmpe_workspace_bytes", "pmpe_check_desc",
            "pmpe_route", "pmpe_dispatch", "pmpe_expert_ffn", "pmpe_combine", "pmpe_audit",
            "pmpe_fingerprint_workspace_bytes", "pmpe_fingerprint", "pmpe_backward_workspace_bytes",
            "pmpe_backward", "pmpe_expert_ffn_train", "pmpe_route_record", "pmpe_cache_tag_check",
            "pmpe_expert_ffn_lora_workspace_bytes", "pmpe_expert_ffn_lora", "pmpe_adamw",
            "pmpe_transpose_experts", "pmpe_expert_ffn_fp8"]

PMPE_FP_LEAF_BYTES = 1024
PMPE_FP_FANOUT = 16


def lib() -> ctypes.CDLL:
    return _lib


def make_desc(hidden: int, inter: int, n_pub: int, n_priv: int, top_k: int, n_shared: int = 0,
              shared_inter: int = 0, bf16: bool = True, gate_mode: int = PMPE_GATE_RENORM_TOPK,
              route_mode: int = 0) -> LayerDesc:
    dt = PMPE_BF16 if bf16 else PMPE_F32
    return LayerDesc(hidden, inter, n_pub, n_priv, top_k, n_shared, shared_inter, dt, dt, gate_mode,
                     route_mode)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libpmpe must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check(status: int, call: str) -> None:
    if status != PMPE_OK:
        raise PmpeError(status, call)


def pmpe_version() -> int:
    return int(_lib.pmpe_version())


def pmpe_workspace_bytes(desc: LayerDesc, T: int) -> int:
    return int(_lib.pmpe_workspace_bytes(ctypes.byref(desc), T))


def pmpe_check_desc(desc: LayerDesc, T: int) -> int:
    return int(_lib.pmpe_check_desc(ctypes.byref(desc), T))


def pmpe_route(desc, T, x, wr_pub, wr_priv, logit_bias, policy_word, topk_idx, topk_gate, allow,
               kgap, dev_status, ws, stream=None) -> None:
    _check(_lib.pmpe_route(ctypes.byref(desc), T, _ptr(x), _ptr(wr_pub), _ptr(wr_priv),
                           _ptr(logit_bias), _ptr(policy_word), _ptr(topk_idx), _ptr(topk_gate),
                           _ptr(allow), _ptr(kgap), _ptr(dev_status), _ptr(ws),
                           0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)),
           "pmpe_route")


def pmpe_dispatch(desc, T, topk_idx, x, expert_count, expert_offset, row_token, token_row, x_perm,
                  ws, stream=None) -> None:
    _check(_lib.pmpe_dispatch(ctypes.byref(desc), T, _ptr(topk_idx), _ptr(x), _ptr(expert_count),
                              _ptr(expert_offset), _ptr(row_token), _ptr(token_row), _ptr(x_perm),
                              _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                              _stream(stream)), "pmpe_dispatch")


def pmpe_dispatch_noalloc(desc, T, topk_idx, x, expert_count, expert_offset, row_token, token_row,
                          x_perm, stream=None) -> None:
    """pmpe_dispatch with the library's own per-device scratch array (no workspace)."""
    _check(_lib.pmpe_dispatch_noalloc(ctypes.byref(desc), T, _ptr(topk_idx), _ptr(x),
                                      _ptr(expert_count), _ptr(expert_offset), _ptr(row_token),
                                      _ptr(token_row), _ptr(x_perm), _stream(stream)),
           "pmpe_dispatch_noalloc")


def pmpe_expert_ffn(desc, T, x_perm, x, expert_count, expert_offset, row_token, w13_pub, w2_pub,
                    w13_priv, w2_priv, w13_sh, w2_sh, y_shared, y_perm, audit_token_rows,
                    audit_priv_calls, dev_status, ws, stream=None) -> None:
    _check(_lib.pmpe_expert_ffn(
        ctypes.byref(desc), T, _ptr(x_perm), _ptr(x), _ptr(expert_count), _ptr(expert_offset),
        _ptr(row_token), _ptr(w13_pub), _ptr(w2_pub), _ptr(w13_priv), _ptr(w2_priv), _ptr(w13_sh),
        _ptr(w2_sh), _ptr(y_shared), _ptr(y_perm), _ptr(audit_token_rows), _ptr(audit_priv_calls),
        _ptr(dev_status), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
        _stream(stream)), "pmpe_expert_ffn")


def pmpe_combine(desc, T, y_perm, token_row, topk_gate, y_shared, out, stream=None) -> None:
    _check(_lib.pmpe_combine(ctypes.byref(desc), T, _ptr(y_perm), _ptr(token_row), _ptr(topk_gate),
                             _ptr(y_shared), _ptr(out), _stream(stream)), "pmpe_combine")


def pmpe_audit(desc, T, audit_token_rows, allow, req_offset, R, req_private_rows,
               total_private_rows, deny_violations, stream=None) -> None:
    _check(_lib.pmpe_audit(ctypes.byref(desc), T, _ptr(audit_token_rows), _ptr(allow),
                           _ptr(req_offset), R, _ptr(req_private_rows), _ptr(total_private_rows),
                           _ptr(deny_violations), _stream(stream)), "pmpe_audit")


def pmpe_backward_workspace_bytes(desc: LayerDesc, T: int) -> int:
    return int(_lib.pmpe_backward_workspace_bytes(ctypes.byref(desc), T))


def pmpe_expert_ffn_train(desc, T, x_perm, x, expert_count, expert_offset, row_token, w13_pub,
                          w2_pub, w13_priv, w2_priv, w13_sh, w2_sh, y_shared, y_perm,
                          audit_token_rows, audit_priv_calls, dev_status, ab, ws,
                          stream=None) -> None:
    _check(_lib.pmpe_expert_ffn_train(
        ctypes.byref(desc), T, _ptr(x_perm), _ptr(x), _ptr(expert_count), _ptr(expert_offset),
        _ptr(row_token), _ptr(w13_pub), _ptr(w2_pub), _ptr(w13_priv), _ptr(w2_priv), _ptr(w13_sh),
        _ptr(w2_sh), _ptr(y_shared), _ptr(y_perm), _ptr(audit_token_rows), _ptr(audit_priv_calls),
        _ptr(dev_status), _ptr(ab), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
        _stream(stream)), "pmpe_expert_ffn_train")


def pmpe_backward(desc, T, x, dout, topk_idx, topk_gate, expert_count, expert_offset, row_token,
                  token_row, y_perm, wr_pub, wr_priv, w13_pub, w2_pub, w13_priv, w2_priv,
                  logit_bias, w13_sh, w2_sh, w2t_pub, w13t_pub, w2t_priv, w13t_priv, ab, dx,
                  dw13_priv, dw2_priv, dwr_priv,
                  grad_rows, ws, stream=None) -> None:
    _check(_lib.pmpe_backward(
        ctypes.byref(desc), T, _ptr(x), _ptr(dout), _ptr(topk_idx), _ptr(topk_gate),
        _ptr(expert_count), _ptr(expert_offset), _ptr(row_token), _ptr(token_row), _ptr(y_perm),
        _ptr(wr_pub), _ptr(wr_priv), _ptr(w13_pub), _ptr(w2_pub), _ptr(w13_priv), _ptr(w2_priv),
        _ptr(logit_bias), _ptr(w13_sh), _ptr(w2_sh), _ptr(w2t_pub), _ptr(w13t_pub),
        _ptr(w2t_priv), _ptr(w13t_priv), _ptr(ab), _ptr(dx), _ptr(dw13_priv), _ptr(dw2_priv), _ptr(dwr_priv), _ptr(grad_rows), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)), "pmpe_backward")


def pmpe_fingerprint_workspace_bytes(nbytes: int) -> int:
    return int(_lib.pmpe_fingerprint_workspace_bytes(nbytes))


def pmpe_fingerprint(data: Optional[torch.Tensor], digest: torch.Tensor, ws: Optional[torch.Tensor],
                     nbytes: Optional[int] = None, stream=None) -> None:
    """Fingerprint the bytes of `data` (all of them unless `nbytes` is given) into the
    32-byte device tensor `digest`."""
    if nbytes is None:
        nbytes = 0 if data is None else data.numel() * data.element_size()
    _check(_lib.pmpe_fingerprint(_ptr(data), nbytes, _ptr(digest), _ptr(ws),
                                 0 if ws is None else ws.numel() * ws.element_size(),
                                 _stream(stream)), "pmpe_fingerprint")


def fingerprint_tensors(*tensors: torch.Tensor, stream=None) -> torch.Tensor:
    """One fingerprint of several device tensors: the fingerprint of the concatenation of
    their fingerprints, in argument order. Returns a 32-byte uint8 device tensor."""
    if not tensors:
        raise ValueError("fingerprint_tensors needs at least one tensor")
    dev = tensors[0].device
    digests = torch.empty((len(tensors), 32), dtype=torch.uint8, device=dev)
    ws_bytes = max(pmpe_fingerprint_workspace_bytes(t.numel() * t.element_size()) for t in tensors)
    ws_bytes = max(ws_bytes, pmpe_fingerprint_workspace_bytes(32 * len(tensors)))
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    for i, t in enumerate(tensors):
        pmpe_fingerprint(t, digests[i], ws, stream=stream)
    root = torch.empty(32, dtype=torch.uint8, device=dev)
    pmpe_fingerprint(digests, root, ws, stream=stream)
    return root


def pmpe_route_record(desc, T, layer, topk_idx, allow, req_offset, R, rec, stream=None) -> None:
    """rec: [T, 4] int32 device tensor (pmpe_route_rec per token)."""
    _check(_lib.pmpe_route_record(ctypes.byref(desc), T, layer, _ptr(topk_idx), _ptr(allow),
                                  _ptr(req_offset), R, _ptr(rec), _stream(stream)),
           "pmpe_route_record")


def pmpe_cache_tag_check(cache: Optional[CacheTag], request: Optional[CacheTag]) -> bool:
    """True when the cached state may serve the request (every tag field equal)."""
    st = _lib.pmpe_cache_tag_check(None if cache is None else ctypes.byref(cache),
                                   None if request is None else ctypes.byref(request))
    if st not in (PMPE_OK, PMPE_ERR_TAG_MISMATCH):
        raise PmpeError(st, "pmpe_cache_tag_check")
    return st == PMPE_OK


def pmpe_expert_ffn_lora_workspace_bytes(desc: LayerDesc, T: int) -> int:
    return int(_lib.pmpe_expert_ffn_lora_workspace_bytes(ctypes.byref(desc), T))


def pmpe_expert_ffn_lora(desc, T, x_perm, x, expert_count, expert_offset, row_token, policy_word,
                         w13_pub, w2_pub, a13, b1, b3, a2, b2, rank, scale, gate, y_perm,
                         lora_rows, dev_status, ws, stream=None) -> None:
    _check(_lib.pmpe_expert_ffn_lora(
        ctypes.byref(desc), T, _ptr(x_perm), _ptr(x), _ptr(expert_count), _ptr(expert_offset),
        _ptr(row_token), _ptr(policy_word), _ptr(w13_pub), _ptr(w2_pub), _ptr(a13), _ptr(b1),
        _ptr(b3), _ptr(a2), _ptr(b2), rank, scale, gate, _ptr(y_perm), _ptr(lora_rows),
        _ptr(dev_status), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
        _stream(stream)), "pmpe_expert_ffn_lora")


def pmpe_adamw(param: torch.Tensor, master: Optional[torch.Tensor], grad: torch.Tensor,
               m: torch.Tensor, v: torch.Tensor, step: int, lr: float, beta1: float, beta2: float,
               eps: float, weight_decay: float, stream=None) -> None:
    """One AdamW step of one parameter tensor (fp32, or bf16 with an fp32 master copy)."""
    dt = PMPE_BF16 if param.dtype == torch.bfloat16 else PMPE_F32
    _check(_lib.pmpe_adamw(_ptr(param), dt, _ptr(master), _ptr(grad), _ptr(m), _ptr(v),
                           param.numel(), step, lr, beta1, beta2, eps, weight_decay,
                           _stream(stream)), "pmpe_adamw")


def pmpe_transpose_experts(src: torch.Tensor, dst: torch.Tensor, stream=None) -> None:
    """dst[e] = src[e]^T for a bf16 stack src [n, rows, cols] into dst [n, cols, rows]."""
    n, rows, cols = src.shape
    if tuple(dst.shape) != (n, cols, rows):
        raise ValueError("dst must be [n, cols, rows]")
    _check(_lib.pmpe_transpose_experts(_ptr(src), _ptr(dst), n, rows, cols, _stream(stream)),
           "pmpe_transpose_experts")


def pmpe_expert_ffn_fp8(desc, T, x_perm, x, expert_count, expert_offset, row_token, w13_pub,
                        w2_pub, w13_priv, w2_priv, w13s_pub, w2s_pub, w13s_priv, w2s_priv, y_perm,
                        audit_token_rows, audit_priv_calls, dev_status, ws, stream=None) -> None:
    """Expert FFN with fp8 (e4m3, uint8 storage) weights and fp32 power-of-two row scales."""
    _check(_lib.pmpe_expert_ffn_fp8(
        ctypes.byref(desc), T, _ptr(x_perm), _ptr(x), _ptr(expert_count), _ptr(expert_offset),
        _ptr(row_token), _ptr(w13_pub), _ptr(w2_pub), _ptr(w13_priv), _ptr(w2_priv),
        _ptr(w13s_pub), _ptr(w2s_pub), _ptr(w13s_priv), _ptr(w2s_priv), _ptr(y_perm),
        _ptr(audit_token_rows), _ptr(audit_priv_calls), _ptr(dev_status), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)), "pmpe_expert_ffn_fp8")
