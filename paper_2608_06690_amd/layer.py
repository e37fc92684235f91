"""PolicyMaskedMoE: owns one layer's device buffers and runs the five C-ABI calls in
order on one stream (route -> dispatch -> expert_ffn -> combine -> audit). It only
allocates torch tensors and passes pointers; all computation happens in libpmpe."""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

from . import _native as N


@dataclasses.dataclass
class LayerBuffers:
    topk_idx: torch.Tensor
    topk_gate: torch.Tensor
    allow: torch.Tensor
    kgap: torch.Tensor
    expert_count: torch.Tensor
    expert_offset: torch.Tensor
    row_token: torch.Tensor
    token_row: torch.Tensor
    x_perm: Optional[torch.Tensor]
    y_perm: torch.Tensor
    y_shared: Optional[torch.Tensor]
    out: torch.Tensor
    ws: torch.Tensor
    dev_status: torch.Tensor
    ab: Optional[torch.Tensor] = None   # [T*k, 2I] fp32, filled by a training forward


@dataclasses.dataclass
class GradBuffers:
    dx: torch.Tensor                    # [T, H] fp32
    dw13_priv: Optional[torch.Tensor]   # [n_priv, 2I, H] fp32
    dw2_priv: Optional[torch.Tensor]    # [n_priv, H, I] fp32
    dwr_priv: Optional[torch.Tensor]    # [n_priv, H] fp32
    grad_rows: torch.Tensor             # [n_priv] uint32 (int32 storage)
    ws: torch.Tensor


@dataclasses.dataclass
class AuditBuffers:
    token_rows: torch.Tensor    # [T] uint32 (int32 storage), accumulates across calls
    priv_calls: torch.Tensor    # [n_priv]
    req_rows: torch.Tensor      # [R] uint64 (int64 storage)
    total: torch.Tensor         # [1]
    violations: torch.Tensor    # [1]

    def zero_(self) -> "AuditBuffers":
        # fill kernels (torch's zero_), not memset nodes
        self.token_rows.zero_()
        self.priv_calls.zero_()
        return self


class PolicyMaskedMoE:
    """One policy-masked MoE layer with weights already on the device.

    Weights: wr_pub [n_pub, H] fp32, wr_priv [n_priv, H] fp32 (or None), bias [E] fp32 or
    None, w13_* [n, 2I, H], w2_* [n, H, I] in the activation dtype, shared group
    w13_sh [2 Is, H], w2_sh [H, Is] or None.
    """

    def __init__(self, desc: N.LayerDesc, wr_pub, wr_priv, bias, w13_pub, w2_pub, w13_priv,
                 w2_priv, w13_sh=None, w2_sh=None, gather_in_dispatch: bool = False):
        self.desc = desc
        self.wr_pub, self.wr_priv, self.bias = wr_pub, wr_priv, bias
        self.w13_pub, self.w2_pub = w13_pub, w2_pub
        self.w13_priv, self.w2_priv = w13_priv, w2_priv
        self.w13_sh, self.w2_sh = w13_sh, w2_sh
        self.gather_in_dispatch = gather_in_dispatch
        self._bufs = {}

    @property
    def device(self):
        return self.w13_pub.device

    @property
    def act_dtype(self):
        return torch.bfloat16 if self.desc.act_dtype == N.PMPE_BF16 else torch.float32

    def buffers(self, T: int) -> LayerBuffers:
        if T not in self._bufs:
            d, dev, k, H = self.desc, self.device, self.desc.top_k, self.desc.hidden
            E = d.n_pub + d.n_priv
            i32 = dict(dtype=torch.int32, device=dev)
            ws_bytes = max(N.pmpe_workspace_bytes(d, T), 256)
            self._bufs[T] = LayerBuffers(
                topk_idx=torch.empty(T * k, **i32), topk_gate=torch.empty(T * k, dtype=torch.float32, device=dev),
                allow=torch.empty(T, dtype=torch.uint8, device=dev),
                kgap=torch.empty(T, dtype=torch.float32, device=dev),
                expert_count=torch.empty(E, **i32), expert_offset=torch.empty(E + 1, **i32),
                row_token=torch.empty(T * k, **i32), token_row=torch.empty(T * k, **i32),
                x_perm=(torch.empty(T * k, H, dtype=self.act_dtype, device=dev)
                        if self.gather_in_dispatch else None),
                y_perm=torch.empty(T * k, H, dtype=self.act_dtype, device=dev),
                y_shared=(torch.empty(T, H, dtype=self.act_dtype, device=dev) if d.n_shared else None),
                out=torch.empty(T, H, dtype=self.act_dtype, device=dev),
                ws=torch.empty(ws_bytes, dtype=torch.uint8, device=dev),
                dev_status=torch.zeros(1, **i32))
        return self._bufs[T]

    def audit_buffers(self, T: int, R: int) -> AuditBuffers:
        dev = self.device
        return AuditBuffers(torch.zeros(T, dtype=torch.int32, device=dev),
                            torch.zeros(self.desc.n_priv, dtype=torch.int32, device=dev),
                            torch.zeros(R, dtype=torch.int64, device=dev),
                            torch.zeros(1, dtype=torch.int64, device=dev),
                            torch.zeros(1, dtype=torch.int32, device=dev))

    def route(self, x, words, b: LayerBuffers, stream=None):
        T = x.shape[0]
        N.pmpe_route(self.desc, T, x, self.wr_pub, self.wr_priv, self.bias, words, b.topk_idx,
                     b.topk_gate, b.allow, b.kgap, b.dev_status, b.ws, stream)

    def dispatch(self, x, b: LayerBuffers, stream=None):
        T = x.shape[0]
        N.pmpe_dispatch(self.desc, T, b.topk_idx, x, b.expert_count, b.expert_offset, b.row_token,
                        b.token_row, b.x_perm, b.ws, stream)

    def expert_ffn(self, x, b: LayerBuffers, audit: AuditBuffers, stream=None, train=False):
        T = x.shape[0]
        if train:
            if b.ab is None:
                b.ab = torch.empty(T * self.desc.top_k, 2 * self.desc.inter, dtype=torch.float32,
                                   device=self.device)
            N.pmpe_expert_ffn_train(
                self.desc, T, b.x_perm, x, b.expert_count, b.expert_offset, b.row_token,
                self.w13_pub, self.w2_pub, self.w13_priv, self.w2_priv, self.w13_sh, self.w2_sh,
                b.y_shared, b.y_perm, audit.token_rows, audit.priv_calls, b.dev_status, b.ab, b.ws,
                stream)
            return
        N.pmpe_expert_ffn(self.desc, T, b.x_perm, x, b.expert_count, b.expert_offset, b.row_token,
                          self.w13_pub, self.w2_pub, self.w13_priv, self.w2_priv, self.w13_sh,
                          self.w2_sh, b.y_shared, b.y_perm, audit.token_rows, audit.priv_calls,
                          b.dev_status, b.ws, stream)

    def combine(self, x, b: LayerBuffers, stream=None):
        T = x.shape[0]
        N.pmpe_combine(self.desc, T, b.y_perm, b.token_row, b.topk_gate, b.y_shared, b.out, stream)

    def forward_lora(self, x, words, lora, rank: int, scale: float, gate: int, audit: AuditBuffers,
                     lora_rows: torch.Tensor, req_offset=None, stream=None) -> LayerBuffers:
        """The request-gated LoRA control arm: every token routes in the public pool (deny
        words), the adapters `lora` = (a13, b1, b3, a2, b2) on the public experts are
        gated by the real `words`; lora_rows [T] int32 accumulates physical adapter rows."""
        T = x.shape[0]
        b = self.buffers(T)
        deny = torch.zeros_like(words)
        self.route(x, deny, b, stream)
        self.dispatch(x, b, stream)
        ws_bytes = N.pmpe_expert_ffn_lora_workspace_bytes(self.desc, T)
        if b.ws.numel() < ws_bytes:
            b.ws = torch.empty(ws_bytes, dtype=torch.uint8, device=self.device)
        N.pmpe_expert_ffn_lora(self.desc, T, b.x_perm, x, b.expert_count, b.expert_offset,
                               b.row_token, words, self.w13_pub, self.w2_pub, *lora, rank, scale,
                               gate, b.y_perm, lora_rows, b.dev_status, b.ws, stream)
        self.combine(x, b, stream)
        if req_offset is not None:
            self.audit(T, b, audit, req_offset, stream)
        return b

    def forward_fp8(self, x, words, fp8, audit: AuditBuffers, req_offset=None,
                    stream=None) -> LayerBuffers:
        """The layer with fp8 expert weights: fp8 = (w13_pub, w2_pub, w13_priv, w2_priv,
        w13s_pub, w2s_pub, w13s_priv, w2s_priv) (uint8 weights, fp32 row scales); routing,
        dispatch, combine and audit as in forward()."""
        T = x.shape[0]
        b = self.buffers(T)
        self.route(x, words, b, stream)
        self.dispatch(x, b, stream)
        d8 = N.LayerDesc(*[getattr(self.desc, f) for f, _ in N.LayerDesc._fields_])
        d8.w_dtype = N.PMPE_FP8_E4M3
        N.pmpe_expert_ffn_fp8(d8, T, b.x_perm, x, b.expert_count, b.expert_offset, b.row_token,
                              *fp8, b.y_perm, audit.token_rows, audit.priv_calls, b.dev_status,
                              b.ws, stream)
        self.combine(x, b, stream)
        if req_offset is not None:
            self.audit(T, b, audit, req_offset, stream)
        return b

    def route_record(self, T: int, b: LayerBuffers, req_offset, layer: int = 0,
                     rec: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Route records of the last forward of this T: [T, 4] int32 (pmpe_route_rec)."""
        rec = rec if rec is not None else torch.empty(T, 4, dtype=torch.int32, device=self.device)
        N.pmpe_route_record(self.desc, T, layer, b.topk_idx, b.allow, req_offset,
                            req_offset.numel() - 1, rec, stream)
        return rec

    def audit(self, T: int, b: LayerBuffers, audit: AuditBuffers, req_offset, stream=None):
        R = req_offset.numel() - 1
        N.pmpe_audit(self.desc, T, audit.token_rows, b.allow, req_offset, R, audit.req_rows,
                     audit.total, audit.violations, stream)

    def grad_buffers(self, T: int) -> GradBuffers:
        d, dev, H, I, P = self.desc, self.device, self.desc.hidden, self.desc.inter, self.desc.n_priv
        f32 = dict(dtype=torch.float32, device=dev)
        return GradBuffers(torch.empty(T, H, **f32),
                           torch.empty(P, 2 * I, H, **f32) if P else None,
                           torch.empty(P, H, I, **f32) if P else None,
                           torch.empty(P, H, **f32) if P else None,
                           torch.zeros(max(P, 1), dtype=torch.int32, device=dev),
                           torch.empty(max(N.pmpe_backward_workspace_bytes(d, T), 256),
                                       dtype=torch.uint8, device=dev))

    def _priv_key(self):
        # identity and torch version counter of the private expert weights: an in-place
        # torch update or a new tensor changes it (the optimizer's kernel writes through a
        # raw pointer and refreshes the copies itself)
        return tuple((w.data_ptr(), w._version) for w in (self.w2_priv, self.w13_priv))

    def refresh_private_transposes(self, stream=None) -> None:
        """Remake the transposed copies of the private expert weights (after they changed)."""
        if self.w13_priv is None or self.desc.n_priv == 0:
            return
        if getattr(self, "_wt_priv", None) is None:
            self._wt_priv = (
                torch.empty(self.w2_priv.shape[0], self.w2_priv.shape[2], self.w2_priv.shape[1],
                            dtype=self.w2_priv.dtype, device=self.device),
                torch.empty(self.w13_priv.shape[0], self.w13_priv.shape[2], self.w13_priv.shape[1],
                            dtype=self.w13_priv.dtype, device=self.device))
        N.pmpe_transpose_experts(self.w2_priv, self._wt_priv[0], stream)
        N.pmpe_transpose_experts(self.w13_priv, self._wt_priv[1], stream)
        self._wt_priv_key = self._priv_key()

    def transposed_weights(self, stream=None):
        """Transposed expert weights for the backward: the frozen public ones are made once
        and kept; the private ones are made once and remade only when the private weights
        change (an optimizer step, an in-place torch update or new tensors), not on every
        backward call."""
        if getattr(self, "_wt_pub", None) is None:
            w2t = torch.empty(self.w2_pub.shape[0], self.w2_pub.shape[2], self.w2_pub.shape[1],
                              dtype=self.w2_pub.dtype, device=self.device)
            w13t = torch.empty(self.w13_pub.shape[0], self.w13_pub.shape[2], self.w13_pub.shape[1],
                               dtype=self.w13_pub.dtype, device=self.device)
            N.pmpe_transpose_experts(self.w2_pub, w2t, stream)
            N.pmpe_transpose_experts(self.w13_pub, w13t, stream)
            self._wt_pub = (w2t, w13t)
        if self.w13_priv is None or self.desc.n_priv == 0:
            return self._wt_pub + (None, None)
        if getattr(self, "_wt_priv", None) is None or getattr(self, "_wt_priv_key", None) != self._priv_key():
            self.refresh_private_transposes(stream)
        return self._wt_pub + self._wt_priv

    def backward(self, x, dout, b: LayerBuffers, g: Optional[GradBuffers] = None,
                 stream=None, use_saved: bool = True, transposed: bool = True) -> GradBuffers:
        """Private-only backward of the forward that filled `b` (same x): input gradient
        and the gradients of the private experts and private router rows. The gate and
        up projections saved by a training forward are used when present (and
        `use_saved`), else recomputed; with `transposed` the products with W2 and W13 use
        transposed weight copies on the forward's grouped GEMM."""
        T = x.shape[0]
        g = g or self.grad_buffers(T)
        wt = self.transposed_weights(stream) if transposed else (None, None, None, None)
        N.pmpe_backward(self.desc, T, x, dout, b.topk_idx, b.topk_gate, b.expert_count,
                        b.expert_offset, b.row_token, b.token_row, b.y_perm, self.wr_pub,
                        self.wr_priv, self.w13_pub, self.w2_pub, self.w13_priv, self.w2_priv,
                        self.bias, self.w13_sh, self.w2_sh, *wt,
                        b.ab if use_saved else None, g.dx, g.dw13_priv, g.dw2_priv, g.dwr_priv, g.grad_rows, g.ws, stream)
        return g

    def forward(self, x, words, audit: AuditBuffers, req_offset=None, stream=None,
                train: bool = False) -> LayerBuffers:
        """Runs the layer; returns the buffers (out, route log, dispatch) of this T. A
        training forward also keeps what the backward needs (b.ab)."""
        b = self.buffers(x.shape[0])
        self.route(x, words, b, stream)
        self.dispatch(x, b, stream)
        self.expert_ffn(x, b, audit, stream, train)
        self.combine(x, b, stream)
        if req_offset is not None:
            self.audit(x.shape[0], b, audit, req_offset, stream)
        return b


class PrivateAdamW:
    """AdamW over a layer's private parameters only: the private router rows (fp32) and
    the private expert weights (bf16 with fp32 master copies). Public tensors are never
    handed to the optimizer (they are not arguments of any call here)."""

    def __init__(self, layer: PolicyMaskedMoE, lr: float = 1e-4, betas=(0.9, 0.999),
                 eps: float = 1e-8, weight_decay: float = 0.0):
        self.layer = layer
        self.lr, self.betas, self.eps, self.wd = lr, betas, eps, weight_decay
        self.params = [layer.wr_priv, layer.w13_priv, layer.w2_priv]
        self.master = [None if p.dtype == torch.float32 else p.float() for p in self.params]
        self.m = [torch.zeros(p.shape, dtype=torch.float32, device=p.device) for p in self.params]
        self.v = [torch.zeros(p.shape, dtype=torch.float32, device=p.device) for p in self.params]
        self.t = 0

    def step(self, g: GradBuffers, stream=None) -> None:
        self.t += 1
        grads = [g.dwr_priv, g.dw13_priv, g.dw2_priv]
        for p, mp, gr, m, v in zip(self.params, self.master, grads, self.m, self.v):
            N.pmpe_adamw(p, mp, gr, m, v, self.t, self.lr, self.betas[0], self.betas[1], self.eps,
                         self.wd, stream)
        # the backward's transposed copies of the private experts follow the update (once
        # per step, on the same stream), if the layer keeps them
        if getattr(self.layer, "_wt_priv", None) is not None:
            self.layer.refresh_private_transposes(stream)
