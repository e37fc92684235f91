"""Helpers for GPU parity tests: build a layer case from the seeded workloads, run it
through the C ABI on the device, and run the CPU oracle on the same inputs.

The oracle always receives inputs generated on the host; the device receives the
same tensors generated on the device (the generator is bit-identical on both)."""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

import workloads as W
from oracle import pmpe_oracle as O

RTOL_BF16 = 1e-2
RTOL_F32 = 1e-5
RTOL_GATE = 1e-5
# Per-row bars next to the aggregate ones: every (token, expert) row of y_perm and every
# token of the layer output on its own. bf16 experts round h, y and out once each to
# bf16 (unit roundoff u = 2^-8); each rounding adds a relative RMS error of u/sqrt(3) per
# element, and h's errors reach y through the down projection with the same relative RMS,
# so a y row carries about u*sqrt(2/3) = 3.2e-3 and an output row about u = 3.9e-3,
# averaged over H elements (spread of a few percent at H = 2048). 1e-2 is 2.5 u: above
# every correct row, far below a row computed from the wrong token, expert or columns
# (relative error of order 1).
RTOL_ROW_BF16 = 1e-2
RTOL_ROW_F32 = 1e-5


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


class _ExpertCache:
    """Host copies (fp64) of one layer's expert weights, generated on first use; the
    w13 and w2 banks of a layer share one cache, so each expert is generated once."""

    def __init__(self, cfg: W.LayerConfig, layer: int):
        self.cfg, self.layer = cfg, layer
        self.cache: Dict[int, tuple] = {}

    def get(self, e: int) -> tuple:
        if e not in self.cache:
            w13, w2 = W.make_expert(self.cfg, self.layer, e, "cpu")
            self.cache[e] = (np64(w13), np64(w2))
        return self.cache[e]


class ExpertBank:
    """Lazily generated host copies of one layer's expert weights, indexed by the
    expert's index within its pool (what the oracle's containers expect)."""

    def __init__(self, cfg: W.LayerConfig, layer: int, private: bool, which: str,
                 cache: Optional[_ExpertCache] = None):
        self.cfg, self.layer, self.private, self.which = cfg, layer, private, which
        self.store = cache or _ExpertCache(cfg, layer)

    def __getitem__(self, i: int) -> np.ndarray:
        e = i + (self.cfg.n_pub if self.private else 0)
        w13, w2 = self.store.get(e)
        return w13 if self.which == "w13" else w2


@dataclasses.dataclass
class OracleInputs:
    x: np.ndarray
    wr_pub: np.ndarray
    wr_priv: np.ndarray
    bias: Optional[np.ndarray]
    w13_pub: ExpertBank
    w2_pub: ExpertBank
    w13_priv: ExpertBank
    w2_priv: ExpertBank
    w13_sh: Optional[np.ndarray]
    w2_sh: Optional[np.ndarray]


def oracle_inputs(cfg: W.LayerConfig, layer: int = 0, x: Optional[torch.Tensor] = None) -> OracleInputs:
    wr_pub, wr_priv, bias = W.make_router(cfg, layer, "cpu")
    w13_sh, w2_sh = W.make_shared(cfg, layer, "cpu")
    xx = W.make_x(cfg, "cpu") if x is None else x.cpu()
    ec = _ExpertCache(cfg, layer)
    return OracleInputs(np64(xx), np64(wr_pub), np64(wr_priv), None if bias is None else np64(bias),
                        ExpertBank(cfg, layer, False, "w13", ec), ExpertBank(cfg, layer, False, "w2", ec),
                        ExpertBank(cfg, layer, True, "w13", ec), ExpertBank(cfg, layer, True, "w2", ec),
                        None if w13_sh is None else np64(w13_sh), None if w2_sh is None else np64(w2_sh))


def oracle_layer(cfg: W.LayerConfig, oi: OracleInputs, words: Sequence[int],
                 tokens: Optional[Sequence[int]] = None, soft: bool = False) -> O.LayerResult:
    return O.layer_forward(oi.x, oi.wr_pub, oi.wr_priv, oi.bias, oi.w13_pub, oi.w2_pub,
                           oi.w13_priv, oi.w2_priv, words, cfg.top_k, cfg.gate_mode,
                           oi.w13_sh, oi.w2_sh, tokens, soft=soft)


def make_desc(cfg: W.LayerConfig, soft: bool = False):
    import paper_2608_06690_amd as P
    gm = P.PMPE_GATE_POOL_SOFTMAX if cfg.gate_mode == "pool_softmax" else P.PMPE_GATE_RENORM_TOPK
    return P.make_desc(cfg.hidden, cfg.inter, cfg.n_pub, cfg.n_priv, cfg.top_k, cfg.n_shared,
                       cfg.shared_inter, cfg.dtype == "bf16", gm,
                       P.PMPE_ROUTE_SOFT if soft else P.PMPE_ROUTE_MASKED)


def device_layer(cfg: W.LayerConfig, layer: int = 0, device="cuda", gather_in_dispatch=False,
                 drop_private: bool = False, soft: bool = False):
    import paper_2608_06690_amd as P
    Lw = W.make_layer(cfg, layer, device)
    priv = (lambda t: None) if drop_private else (lambda t: t)
    return P.PolicyMaskedMoE(make_desc(cfg, soft), Lw.wr_pub, priv(Lw.wr_priv), Lw.bias, Lw.w13_pub,
                             Lw.w2_pub, priv(Lw.w13_priv), priv(Lw.w2_priv), Lw.w13_sh, Lw.w2_sh,
                             gather_in_dispatch=gather_in_dispatch), Lw


def words_tensor(words: Sequence[int], device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.asarray(words, np.uint32).view(np.int32).copy()).to(device)


@dataclasses.dataclass
class DeviceResult:
    idx: np.ndarray
    gate: np.ndarray
    allow: np.ndarray
    kgap: np.ndarray
    count: np.ndarray
    offset: np.ndarray
    row_token: np.ndarray
    token_row: np.ndarray
    out: torch.Tensor          # on host, act dtype
    y_perm: torch.Tensor       # [T*k, H] on host, act dtype: expert output rows
    audit_rows: np.ndarray
    audit_calls: np.ndarray
    req_rows: np.ndarray
    total: int
    violations: int
    dev_status: int


def run_device(layer, x: torch.Tensor, words: Optional[torch.Tensor], req_offset: torch.Tensor,
               audit=None) -> DeviceResult:
    T = x.shape[0]
    R = req_offset.numel() - 1
    k = layer.desc.top_k
    audit = audit or layer.audit_buffers(T, R)
    b = layer.forward(x, words, audit, req_offset)
    torch.cuda.synchronize()
    u32 = lambda t: t.cpu().numpy().view(np.uint32).astype(np.int64)  # noqa: E731
    return DeviceResult(
        idx=b.topk_idx.view(T, k).cpu().numpy().astype(np.int64),
        gate=b.topk_gate.view(T, k).cpu().numpy(), allow=b.allow.cpu().numpy(),
        kgap=b.kgap.cpu().numpy(), count=b.expert_count.cpu().numpy().astype(np.int64),
        offset=b.expert_offset.cpu().numpy().astype(np.int64),
        row_token=b.row_token.cpu().numpy().astype(np.int64),
        token_row=b.token_row.view(T, k).cpu().numpy().astype(np.int64),
        out=b.out.cpu().clone(), y_perm=b.y_perm.view(T * k, -1).cpu().clone(),
        audit_rows=u32(audit.token_rows), audit_calls=u32(audit.priv_calls),
        req_rows=audit.req_rows.cpu().numpy(), total=int(audit.total.item()),
        violations=int(audit.violations.item()), dev_status=int(b.dev_status.item()))


def rel_l2(a: np.ndarray, b: np.ndarray) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


def check_dispatch_consistent(d: DeviceResult, E: int) -> None:
    """Dispatch outputs are pure functions of the device's own topk_idx."""
    ref = O.dispatch(d.idx, E)
    assert np.array_equal(d.count, ref.count)
    assert np.array_equal(d.offset, ref.offset)
    assert np.array_equal(d.row_token, ref.row_token)
    assert np.array_equal(d.token_row, ref.token_row)


def compare_routes(cfg, d: DeviceResult, rt: O.Route, tokens=None) -> Dict[str, int]:
    """Routing parity: allow bit-exact everywhere; idx bit-exact off near-ties; gates
    within RTOL_GATE on tokens whose idx agree. Returns near-tie statistics."""
    toks = np.arange(d.idx.shape[0]) if tokens is None else np.asarray(tokens)
    assert np.array_equal(d.allow[toks], rt.allow[toks])
    nt = rt.near_tie[toks]
    same = np.all(d.idx[toks] == rt.idx[toks], axis=1)
    bad = toks[~same & ~nt]
    assert bad.size == 0, f"routing differs on non-near-tie tokens {bad[:10]}"
    ok = toks[same]
    assert rel_l2(d.gate[ok], rt.gate[ok]) <= RTOL_GATE
    return {"near_tie": int(nt.sum()), "near_tie_differ": int((~same & nt).sum()), "agree": int(same.sum())}


def row_rel_errors(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Relative L2 error of every row of a against the same row of b."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.linalg.norm(b, axis=1)
    num = np.linalg.norm(a - b, axis=1)
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), num)


def check_rows(cfg, d: DeviceResult, ref: O.LayerResult, toks: np.ndarray, tag: str = "") -> Dict[str, float]:
    """Per-row parity on tokens whose routes agree: every expert output row y_perm[token_row[t, j]]
    against the oracle's row for (t, idx[t, j]), and every token's layer output, each within
    the per-row bar; also the aggregate rel-L2 of the outputs. `ref.out` rows follow
    `ref.tokens`. Returns the largest errors."""
    bf16 = cfg.dtype == "bf16"
    rtol, rtol_row = (RTOL_BF16, RTOL_ROW_BF16) if bf16 else (RTOL_F32, RTOL_ROW_F32)
    toks = np.asarray(toks, np.int64)
    k = d.idx.shape[1]
    pos = {int(t): i for i, t in enumerate(np.asarray(ref.tokens))}
    out_ref = ref.out[[pos[int(t)] for t in toks]]
    out_dev = d.out.to(torch.float64).numpy()[toks]
    agg = rel_l2(out_dev, out_ref)
    tok_err = row_rel_errors(out_dev, out_ref)
    rows = d.token_row[toks].reshape(-1)
    assert np.all(rows >= 0)
    y_dev = d.y_perm[torch.from_numpy(rows)].to(torch.float64).numpy()
    y_ref = np.stack([ref.y[(int(t), int(d.idx[t, j]))] for t in toks for j in range(k)])
    row_err = row_rel_errors(y_dev, y_ref)
    worst_row = int(np.argmax(row_err))
    stats = {"agg": agg, "token_max": float(tok_err.max()), "row_max": float(row_err.max()),
             "row_mean": float(row_err.mean())}
    print(f"{tag} rows: aggregate {agg:.3e}, per-token max {stats['token_max']:.3e}, per-row max "
          f"{stats['row_max']:.3e} (mean {stats['row_mean']:.3e}) over {toks.size} tokens", flush=True)
    assert agg <= rtol
    assert tok_err.max() <= rtol_row, f"token {int(toks[int(np.argmax(tok_err))])}: {tok_err.max():.3e}"
    assert row_err.max() <= rtol_row, (
        f"row of token {int(toks[worst_row // k])} slot {worst_row % k}: {row_err.max():.3e}")
    return stats
