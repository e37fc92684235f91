"""CPU oracle of the policy-masked MoE layer: forward, private-only backward, and the
weight fingerprint.

TEST INFRASTRUCTURE ONLY. Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module. It shares no code with the
HIP path and must never be used to produce the library's results.

It is a plain, slow, fp64 definition of what one policy-masked MoE layer
computes, following Policy-Masked Private Experts (arXiv 2608.06690):

* resolve    trusted metadata -> tau in {0, 1}, failing closed
             (Sec. 3.1, resolver paragraph; App. B.1 "Policy resolution and masked routing")
* words      tau per request compiled to one 32-bit policy word and expanded per
             token row (App. B.1, second paragraph; App. B.2); on the device side a
             word allows only if it equals ALLOW_WORD exactly
* route      router logits z = x . W_r[e] (+ b_e) over the permitted pool, the hard
             mask m(tau) of Sec. 3.1 (mask equation) applied BEFORE top-k, top-k with
             the lowest expert id winning fp32 ties, gates
* dispatch   stable grouping of the selected (token, expert) pairs by expert
* experts    bias-free SwiGLU experts (gate, up, down projections as named in
             Sec. 4.2 "Matched adaptation and controls"); private experts are run by a
             separate function that counts the rows it executes, like the
             independent forward hooks of App. F.1
* combine    out_t = sum_j g_tj * y_{e_tj}(x_t) (+ shared experts)
* soft       the soft-routing control of Sec. 4.2 (third row of the control matrix)
             and App. E: one router over the concatenated public and private pool, no
             mask; kept only to show what the mask prevents
* audit      per-request private rows, deny violations (App. B.2 "route counters
             indexed by row and layer"; App. F.1)
* backward   gradients of the layer for an upstream gradient with only the private
             experts and private router rows trainable (G2 of Sec. 2.2; Sec. 3.2:
             only the private gate and experts require gradients); the input gradient
             flows through frozen public and shared experts and the router
* fingerprint  SHA-256 tree over the bytes of frozen weights (Sec. 3.2; App. C.1)

Readings where the paper is silent (the paper gives only the mask and top-k):

* Gates: RENORM (softmax over the k selected logits, i.e. pool softmax followed by
  top-k renormalisation) or POOL_SOFTMAX (softmax over the whole permitted pool,
  no renormalisation).
* Logits are fp32: the fp64 dot product of the exact inputs rounded once to fp32;
  a bias is then added in fp32.
* Ties: equal fp32 logits are broken by the lower expert id; -0.0 equals +0.0;
  a NaN logit ranks as -inf.
* The selected ids of a token are reported in ascending id order, with their
  gates aligned.
* Shared experts are always executed, independent of tau, added unweighted and
  never counted by the audit.
* Expert math is exact fp64 on the (fp32 or bf16) input values with no
  intermediate rounding.

Backward readings: the selection is the forward's (piecewise constant), gradients flow
through the gate values; the softmax derivative uses the fp64 softmax of the fp32
logits. It is pinned to torch autograd of a separately written fp64 forward, to central
finite differences and to exact special cases (all deny: no private gradient; k = 1
RENORM: no router gradient).

Parity of the floating-point expert outputs is pinned only by special cases (a
one-expert pool reduces to a dense SwiGLU MLP; all-deny equals a plain public-only
top-k MoE); the paper prints no numeric worked example of the layer.
"""
from __future__ import annotations

from collections.abc import Mapping
from dataclasses import dataclass, field
from typing import Any, Dict, List, Optional, Sequence

import numpy as np

ALLOW_WORD = 0xA11C0DE5   # the only policy word that allows
DENY_WORD = 0x00000000

GATE_RENORM = "renorm"
GATE_POOL_SOFTMAX = "pool_softmax"

NEAR_TIE = 1e-5


# ----------------------------------------------------------------------------
# Policy resolution (Sec. 3.1 resolver paragraph; App. B.1)
# ----------------------------------------------------------------------------

def resolve(meta: Any) -> int:
    """tau = 1 only for a trusted mapping whose 'allow_private' value has Boolean type
    and is true. Missing metadata, wrong keys, strings, numbers, lists, nested values,
    nulls and serialized JSON text all resolve to 0 (fail closed)."""
    if not isinstance(meta, Mapping):
        return 0
    if "allow_private" not in meta:
        return 0
    v = meta["allow_private"]
    if type(v) is bool and v is True:
        return 1
    return 0


def compile_words(metas: Sequence[Any], lengths: Sequence[int]) -> np.ndarray:
    """Per-token policy words: each request's resolved decision, repeated over its rows
    (App. B.1: the resolved vector is expanded per batch row before top-k)."""
    words: List[int] = []
    for meta, n in zip(metas, lengths):
        w = ALLOW_WORD if resolve(meta) == 1 else DENY_WORD
        words.extend([w] * int(n))
    return np.asarray(words, dtype=np.uint32)


def decode_word(word: int) -> int:
    """Device-side decode: exactly one value allows; anything else (malformed) denies."""
    return 1 if int(word) == ALLOW_WORD else 0


def pool(tau: int, n_pub: int, n_priv: int) -> np.ndarray:
    """Permitted expert ids: the mask m(tau) of Sec. 3.1 is 0 on this set and -inf
    elsewhere. tau=1 -> private ids [n_pub, n_pub+n_priv); tau=0 -> public [0, n_pub)."""
    if tau == 1:
        return np.arange(n_pub, n_pub + n_priv)
    return np.arange(0, n_pub)


# ----------------------------------------------------------------------------
# Routing (Sec. 3.1 mask equation and the sentence after it; App. B.1)
# ----------------------------------------------------------------------------

def logits(x_rows: np.ndarray, wr_rows: np.ndarray, bias: Optional[np.ndarray]) -> np.ndarray:
    """fp32 router logits of the given rows against the given router rows only.

    The dot products are taken in fp64 over the exact input values and rounded once
    to fp32; a bias is then added with one fp32 addition."""
    z = (np.asarray(x_rows, np.float64) @ np.asarray(wr_rows, np.float64).T).astype(np.float32)
    if bias is not None:
        z = (z + np.asarray(bias, np.float32)[None, :]).astype(np.float32)
    return z


def topk(z: np.ndarray, ids: np.ndarray, k: int):
    """Top-k of one token's permitted pool.

    Order the pool by (value descending, id ascending) with -0.0 == +0.0 and NaN as
    -inf; the first k form the selection. Returns (selected ids ascending, gap) where
    gap = z_(k) - z_(k+1) in fp64, +inf when the pool has exactly k experts."""
    zz = np.asarray(z, np.float64)
    zz = np.where(np.isnan(zz), -np.inf, zz) + 0.0
    order = sorted(range(len(ids)), key=lambda i: (-zz[i], int(ids[i])))
    sel = [int(ids[i]) for i in order[:k]]
    if len(ids) == k:
        gap = np.inf
    else:
        a, b = zz[order[k - 1]], zz[order[k]]
        gap = 0.0 if a == b else float(a - b)
    return np.asarray(sorted(sel), dtype=np.int64), gap


def gates(z_sel: np.ndarray, z_pool: np.ndarray, mode: str) -> np.ndarray:
    """Gate values in fp64, rounded to fp32. m is the largest selected logit, which is
    also the pool maximum."""
    zs = np.asarray(z_sel, np.float64)
    m = zs.max()
    num = np.exp(zs - m)
    if mode == GATE_RENORM:
        den = num.sum()
    elif mode == GATE_POOL_SOFTMAX:
        den = np.exp(np.asarray(z_pool, np.float64) - m).sum()
    else:
        raise ValueError(mode)
    return (num / den).astype(np.float32)


@dataclass
class Route:
    idx: np.ndarray        # [T, k] int64, ascending per token (global expert ids)
    gate: np.ndarray       # [T, k] fp32, aligned with idx
    allow: np.ndarray      # [T] uint8, resolved tau per token
    gap: np.ndarray        # [T] fp64, k-th minus (k+1)-th masked logit
    z: List[np.ndarray] = field(default_factory=list)  # per token: fp32 logits of its pool

    @property
    def near_tie(self) -> np.ndarray:
        return self.gap < NEAR_TIE


def route(x: np.ndarray, wr_pub: np.ndarray, wr_priv: np.ndarray, bias: Optional[np.ndarray],
          words: Sequence[int], k: int, gate_mode: str = GATE_RENORM, soft: bool = False) -> Route:
    """Masked top-k routing of every token. Private router rows are only ever read for
    tokens whose word allows; an ineligible expert never enters the candidate set.

    soft=True is the control arm of Sec. 4.2 / App. E: every token ranks the logits of
    the concatenated pool (public ids then private ids) with no mask; `allow` still
    records the resolved policy decision."""
    x = np.asarray(x)
    T = x.shape[0]
    n_pub, n_priv = wr_pub.shape[0], wr_priv.shape[0] if wr_priv is not None else 0
    idx = np.zeros((T, k), np.int64)
    gate = np.zeros((T, k), np.float32)
    allow = np.zeros(T, np.uint8)
    gap = np.zeros(T, np.float64)
    zs: List[np.ndarray] = [None] * T  # type: ignore
    taus = np.array([decode_word(w) for w in words], dtype=np.int64)
    if soft:
        ids = np.arange(n_pub + n_priv)
        wr = np.concatenate([np.asarray(wr_pub), np.asarray(wr_priv)], axis=0)
        b = None if bias is None else np.asarray(bias, np.float32)
        z = logits(x, wr, b)
        for t in range(T):
            sel, g = topk(z[t], ids, k)
            idx[t] = sel
            gate[t] = gates(z[t][sel], z[t], gate_mode)
            allow[t] = taus[t]
            gap[t] = g
            zs[t] = z[t]
        return Route(idx, gate, allow, gap, zs)
    for tau in (0, 1):
        toks = np.nonzero(taus == tau)[0]
        if len(toks) == 0:
            continue
        ids = pool(tau, n_pub, n_priv)
        wr = wr_priv if tau == 1 else wr_pub
        b = None if bias is None else np.asarray(bias, np.float32)[ids]
        z = logits(x[toks], wr, b)
        for row, t in enumerate(toks):
            sel, g = topk(z[row], ids, k)
            idx[t] = sel
            gate[t] = gates(z[row][sel - ids[0]], z[row], gate_mode)
            allow[t] = tau
            gap[t] = g
            zs[t] = z[row]
    return Route(idx, gate, allow, gap, zs)


# ----------------------------------------------------------------------------
# Dispatch: stable grouping of (token, expert) pairs by expert
# ----------------------------------------------------------------------------

@dataclass
class Dispatch:
    count: np.ndarray      # [E] int64
    offset: np.ndarray     # [E+1] int64, exclusive prefix sum of count
    row_token: np.ndarray  # [T*k] int64: permuted row -> token
    token_row: np.ndarray  # [T, k] int64: (token, slot) -> permuted row


def dispatch(idx: np.ndarray, n_experts: int) -> Dispatch:
    """Rows of expert e are the tokens that selected e, in ascending token order;
    experts follow each other in ascending id order."""
    T, k = idx.shape
    count = np.zeros(n_experts, np.int64)
    offset = np.zeros(n_experts + 1, np.int64)
    row_token = np.zeros(T * k, np.int64)
    token_row = np.full((T, k), -1, np.int64)
    r = 0
    for e in range(n_experts):
        offset[e] = r
        hit = idx == e
        tokens = np.nonzero(hit.any(axis=1))[0]
        for t in tokens:
            j = int(np.nonzero(hit[t])[0][0])
            row_token[r] = t
            token_row[t, j] = r
            r += 1
        count[e] = len(tokens)
    offset[n_experts] = r
    return Dispatch(count, offset, row_token, token_row)


# ----------------------------------------------------------------------------
# Experts
# ----------------------------------------------------------------------------

def swiglu(X: np.ndarray, w13: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """One bias-free SwiGLU expert: G = X Wg^T, U = X Wu^T, Y = (silu(G) * U) Wd^T, with
    w13 = [Wg; Wu] of shape [2I, H] and w2 = Wd of shape [H, I]."""
    X = np.asarray(X, np.float64)
    w13 = np.asarray(w13, np.float64)
    I = w13.shape[0] // 2
    G = X @ w13[:I].T
    U = X @ w13[I:].T
    A = G / (1.0 + np.exp(-G)) * U
    return A @ np.asarray(w2, np.float64).T


class ExecutionHook:
    """Counts what the private experts physically execute: rows per token and one call
    per private expert invoked with at least one row (App. F.1 independent hooks)."""

    def __init__(self, n_tokens: int, n_priv: int):
        self.rows = np.zeros(n_tokens, np.int64)
        self.calls = np.zeros(n_priv, np.int64)


def run_public_expert(X: np.ndarray, w13: np.ndarray, w2: np.ndarray) -> np.ndarray:
    return swiglu(X, w13, w2)


def run_private_expert(p: int, X: np.ndarray, tokens: np.ndarray, w13: np.ndarray,
                       w2: np.ndarray, hook: ExecutionHook) -> np.ndarray:
    """Private expert p (0-based within the private pool); the hook records every row."""
    Y = swiglu(X, w13, w2)
    for t in tokens:
        hook.rows[int(t)] += 1
    if len(tokens) > 0:
        hook.calls[p] += 1
    return Y


@dataclass
class LayerResult:
    route: Route
    disp: Dispatch
    out: np.ndarray               # [len(tokens), H] fp64 (rows of the evaluated tokens)
    tokens: np.ndarray            # evaluated token ids
    hook: ExecutionHook
    expert_count: np.ndarray      # [E]
    # (token, expert) -> that expert's output row for the token, before the gate
    y: Dict[tuple, np.ndarray] = field(default_factory=dict)


def layer_forward(x: np.ndarray, wr_pub, wr_priv, bias, w13_pub, w2_pub, w13_priv, w2_priv,
                  words: Sequence[int], k: int, gate_mode: str = GATE_RENORM,
                  w13_sh=None, w2_sh=None, tokens: Optional[Sequence[int]] = None,
                  soft: bool = False) -> LayerResult:
    """One policy-masked MoE layer. Routing and dispatch cover every token; expert
    outputs are evaluated for `tokens` (all by default). Weight containers are
    indexed by expert (e.g. w13_pub[e] -> [2I, H])."""
    x = np.asarray(x)
    T = x.shape[0]
    n_pub = wr_pub.shape[0]
    n_priv = wr_priv.shape[0] if wr_priv is not None else 0
    E = n_pub + n_priv
    rt = route(x, wr_pub, wr_priv, bias, words, k, gate_mode, soft=soft)
    dp = dispatch(rt.idx, E)
    toks = np.arange(T) if tokens is None else np.asarray(tokens, np.int64)
    hook = ExecutionHook(T, n_priv)
    y: Dict[tuple, np.ndarray] = {}
    for e in range(E):
        rows = toks[(rt.idx[toks] == e).any(axis=1)]   # the evaluated tokens that selected e
        if len(rows) == 0:
            continue
        X = x[rows]
        if e < n_pub:
            Y = run_public_expert(X, w13_pub[e], w2_pub[e])
        else:
            Y = run_private_expert(e - n_pub, X, rows, w13_priv[e - n_pub], w2_priv[e - n_pub], hook)
        for i, t in enumerate(rows):
            y[(int(t), e)] = Y[i]
    H = x.shape[1]
    out = np.zeros((len(toks), H), np.float64)
    ysh = swiglu(x[toks], w13_sh, w2_sh) if w13_sh is not None else None
    for i, t in enumerate(toks):
        acc = np.zeros(H, np.float64)
        for j in range(k):
            acc += np.float64(rt.gate[t, j]) * y[(int(t), int(rt.idx[t, j]))]
        if ysh is not None:
            acc += ysh[i]
        out[i] = acc
    return LayerResult(rt, dp, out, toks, hook, dp.count, y)


# ----------------------------------------------------------------------------
# Private-only backward (G2 of Sec. 2.2; Sec. 3.2 training and checkpointing)
# ----------------------------------------------------------------------------

def swiglu_backward(X: np.ndarray, w13: np.ndarray, w2: np.ndarray, dY: np.ndarray):
    """Gradients of one SwiGLU expert Y = (silu(X Wg^T) * (X Wu^T)) Wd^T for the upstream
    gradient dY: returns (dX, dW13, dW2) with dW13 = [dWg; dWu] of shape [2I, H] and
    dW2 = dWd of shape [H, I]. silu'(g) = s (1 + g (1 - s)) with s = sigmoid(g)."""
    X = np.asarray(X, np.float64)
    w13 = np.asarray(w13, np.float64)
    w2 = np.asarray(w2, np.float64)
    dY = np.asarray(dY, np.float64)
    I = w13.shape[0] // 2
    Wg, Wu = w13[:I], w13[I:]
    G = X @ Wg.T
    U = X @ Wu.T
    S = 1.0 / (1.0 + np.exp(-G))
    A = G * S * U                       # h = silu(G) * U
    dA = dY @ w2                        # [n, I]
    dW2 = dY.T @ A                      # [H, I]
    dG = dA * U * S * (1.0 + G * (1.0 - S))
    dU = dA * G * S
    dX = dG @ Wg + dU @ Wu
    dW13 = np.concatenate([dG.T @ X, dU.T @ X], axis=0)
    return dX, dW13, dW2


def gate_backward(z_sel: np.ndarray, z_pool: np.ndarray, sel_pos: np.ndarray, dg: np.ndarray,
                  mode: str) -> np.ndarray:
    """Logit gradient over the token's pool from the gate gradient dg of its k selected
    experts (positions sel_pos in the pool). Exact fp64 softmax derivative:
    RENORM   g = softmax(z_sel):  dz_j = g_j (dg_j - sum_i g_i dg_i) on the selection;
    POOL     p = softmax(z_pool), g_j = p_j:  dz_e = p_e ([e selected] dg_e - sum_i p_i dg_i)."""
    dz = np.zeros(len(z_pool), np.float64)
    dg = np.asarray(dg, np.float64)
    if mode == GATE_RENORM:
        zs = np.asarray(z_sel, np.float64)
        g = np.exp(zs - zs.max())
        g /= g.sum()
        dz[sel_pos] = g * (dg - (g * dg).sum())
    elif mode == GATE_POOL_SOFTMAX:
        zp = np.asarray(z_pool, np.float64)
        p = np.exp(zp - zp.max())
        p /= p.sum()
        up = np.zeros(len(zp), np.float64)
        up[sel_pos] = dg
        dz = p * (up - (p[sel_pos] * dg).sum())
    else:
        raise ValueError(mode)
    return dz


@dataclass
class LayerGrads:
    route: Route
    dx: np.ndarray          # [T, H] input gradient (through every expert, router, shared)
    dw13_priv: np.ndarray   # [n_priv, 2I, H]
    dw2_priv: np.ndarray    # [n_priv, H, I]
    dwr_priv: np.ndarray    # [n_priv, H] private router rows (the private gate)
    grad_rows: np.ndarray   # [n_priv] rows that entered each private expert's gradient


def layer_backward(x: np.ndarray, wr_pub, wr_priv, bias, w13_pub, w2_pub, w13_priv, w2_priv,
                   words: Sequence[int], k: int, dout: np.ndarray, gate_mode: str = GATE_RENORM,
                   w13_sh=None, w2_sh=None, soft: bool = False) -> LayerGrads:
    """Backward of layer_forward for the upstream gradient dout [T, H], with only the
    private experts and the private router rows trainable: public experts, public
    router rows, the logit bias and shared experts are frozen, so no gradient of theirs
    is formed, but the input gradient flows through all of them. The route (a
    piecewise-constant selection) is the forward's; gradients flow through the gate
    values of the selected experts."""
    x = np.asarray(x)
    T, H = x.shape
    n_pub = wr_pub.shape[0]
    n_priv = wr_priv.shape[0] if wr_priv is not None else 0
    E = n_pub + n_priv
    dout = np.asarray(dout, np.float64)
    rt = route(x, wr_pub, wr_priv, bias, words, k, gate_mode, soft=soft)
    x64 = np.asarray(x, np.float64)
    dx = np.zeros((T, H), np.float64)
    I = (np.asarray(w13_priv[0]).shape[0] // 2) if n_priv else np.asarray(w13_pub[0]).shape[0] // 2
    dw13 = np.zeros((n_priv, 2 * I, H), np.float64)
    dw2 = np.zeros((n_priv, H, I), np.float64)
    dwr = np.zeros((n_priv, H), np.float64)
    grad_rows = np.zeros(n_priv, np.int64)
    dg = np.zeros((T, k), np.float64)
    for e in range(E):
        hit = rt.idx == e
        rows = np.nonzero(hit.any(axis=1))[0]
        if len(rows) == 0:
            continue
        slot = np.argmax(hit[rows], axis=1)
        w13 = w13_pub[e] if e < n_pub else w13_priv[e - n_pub]
        w2 = w2_pub[e] if e < n_pub else w2_priv[e - n_pub]
        X = x64[rows]
        Y = swiglu(X, w13, w2)
        g = rt.gate[rows, slot].astype(np.float64)
        dg[rows, slot] = (dout[rows] * Y).sum(axis=1)
        dX, dW13, dW2 = swiglu_backward(X, w13, w2, g[:, None] * dout[rows])
        dx[rows] += dX
        if e >= n_pub:
            dw13[e - n_pub] = dW13
            dw2[e - n_pub] = dW2
            grad_rows[e - n_pub] = len(rows)
    taus = rt.allow.astype(np.int64)
    wr_all = np.concatenate([np.asarray(wr_pub, np.float64)]
                            + ([np.asarray(wr_priv, np.float64)] if n_priv else []), axis=0)
    for t in range(T):
        ids = np.arange(E) if soft else pool(int(taus[t]), n_pub, n_priv)
        sel_pos = np.searchsorted(ids, rt.idx[t])
        z_pool = rt.z[t]
        dz = gate_backward(z_pool[sel_pos], z_pool, sel_pos, dg[t], gate_mode)
        dx[t] += dz @ wr_all[ids]
        priv = ids >= n_pub
        if priv.any():
            dwr[ids[priv] - n_pub] += dz[priv][:, None] * x64[t][None, :]
    if w13_sh is not None:
        dxs, _, _ = swiglu_backward(x64, w13_sh, w2_sh, dout)
        dx += dxs
    return LayerGrads(rt, dx, dw13, dw2, dwr, grad_rows)


# ----------------------------------------------------------------------------
# Audit (App. B.2 row-indexed route counters; App. F.1)
# ----------------------------------------------------------------------------

def route_private_rows(idx: np.ndarray, n_pub: int) -> np.ndarray:
    """Route-log count per token: how many of its selected experts are private."""
    return (np.asarray(idx) >= n_pub).sum(axis=1).astype(np.int64)


@dataclass
class Audit:
    req_private_rows: np.ndarray   # [R] int64
    total_private_rows: int
    deny_violations: int           # tokens with allow == 0 and a nonzero private-row count


def audit(token_rows: np.ndarray, allow: np.ndarray, req_offset: Sequence[int]) -> Audit:
    token_rows = np.asarray(token_rows, np.int64)
    R = len(req_offset) - 1
    req = np.zeros(R, np.int64)
    for r in range(R):
        req[r] = int(token_rows[req_offset[r]:req_offset[r + 1]].sum())
    viol = int(((np.asarray(allow) == 0) & (token_rows > 0)).sum())
    return Audit(req, int(req.sum()), viol)


# ----------------------------------------------------------------------------
# Public-weight fingerprint: the frozen public weights are hashed before and after
# training and must be unchanged (Sec. 3.2 training and checkpointing; Sec. 5.1; App. C.1)
# ----------------------------------------------------------------------------

FP_LEAF = 1024     # bytes per leaf chunk
FP_FANOUT = 16     # child digests hashed together per inner node


def fingerprint(data: bytes) -> bytes:
    """16-ary SHA-256 tree over a byte string.

    Level 0: the SHA-256 digest of every 1024-byte chunk (the last chunk may be short;
    an empty input is one empty chunk). Level j+1: the SHA-256 digest of the
    concatenation of up to 16 consecutive level-j digests. The root, when one digest
    remains, is the fingerprint (an input of at most 1024 bytes has root SHA-256(data)).
    SHA-256 itself is FIPS 180-4, taken from hashlib."""
    import hashlib
    data = bytes(data)
    n = max(1, -(-len(data) // FP_LEAF))
    level = [hashlib.sha256(data[i * FP_LEAF:(i + 1) * FP_LEAF]).digest() for i in range(n)]
    while len(level) > 1:
        level = [hashlib.sha256(b"".join(level[i:i + FP_FANOUT])).digest()
                 for i in range(0, len(level), FP_FANOUT)]
    return level[0]


def fingerprint_set(parts: Sequence[bytes]) -> bytes:
    """Fingerprint of several buffers: the fingerprint of the concatenation of their
    fingerprints, in order."""
    return fingerprint(b"".join(fingerprint(p) for p in parts))


# ----------------------------------------------------------------------------
# Route records and cache tags (App. B.1 fail-closed request procedure, steps 3 and 5;
# App. B.2 state isolation and cache discipline)
# ----------------------------------------------------------------------------

POOL_PUBLIC, POOL_PRIVATE, POOL_MIXED = 0, 1, 2


def route_records(idx: np.ndarray, allow: np.ndarray, req_offset: Sequence[int], n_pub: int,
                  layer: int) -> np.ndarray:
    """One record per token: (layer | decision << 16 | pool << 24, request row, position in
    the request, mask of the slots whose selected expert is private), as uint32 [T, 4]."""
    T, k = idx.shape
    rec = np.zeros((T, 4), np.uint32)
    offs = list(req_offset)
    for t in range(T):
        row = max(r for r in range(len(offs) - 1) if offs[r] <= t)
        mask = sum(1 << j for j in range(k) if idx[t, j] >= n_pub)
        pool = POOL_PUBLIC if mask == 0 else (POOL_PRIVATE if mask == (1 << k) - 1 else POOL_MIXED)
        rec[t] = (layer | (int(allow[t]) << 16) | (pool << 24), row, t - offs[row], mask)
    return rec


def cache_tag_ok(cache: Optional[tuple], request: Optional[tuple]) -> bool:
    """Cached state may serve a request only when both tags exist, both decisions are
    well formed (0 or 1) and (decision, model revision, checkpoint fingerprint) are equal."""
    if cache is None or request is None:
        return False
    if cache[0] not in (0, 1) or request[0] not in (0, 1):
        return False
    return tuple(cache) == tuple(request)


# ----------------------------------------------------------------------------
# Request-gated LoRA control (Sec. 4.2 matched expert-LoRA baseline; Sec. 5.2 and
# App. F.2: a request gate on an adapter is a logical switch, so the adapter can still
# be physically executed for denied requests)
# ----------------------------------------------------------------------------

LORA_GATE_ROW, LORA_GATE_TILE, LORA_GATE_POSTHOC = 0, 1, 2
LORA_TILE_ROWS = 64


def lora_expert(X: np.ndarray, taus: np.ndarray, w13, w2, a13, b1, b3, a2, b2, scale: float):
    """One public expert with rank-r adapters on its gate, up and down projections, the
    adapter terms multiplied by the row's decision tau (1 allow, 0 deny):
        g = X Wg^T + tau s (X Ag^T) Bg^T,  u = X Wu^T + tau s (X Au^T) Bu^T,
        h = silu(g) u,  y = h Wd^T + tau s (h Ad^T) Bd^T
    with a13 = [Ag; Au] ([2r, H]), b1 = Bg [I, r], b3 = Bu [I, r], a2 = Ad [r, I],
    b2 = Bd [H, r]."""
    X = np.asarray(X, np.float64)
    t = np.asarray(taus, np.float64)[:, None]
    w13 = np.asarray(w13, np.float64)
    I = w13.shape[0] // 2
    r = np.asarray(a13).shape[0] // 2
    a13 = np.asarray(a13, np.float64)
    G = X @ w13[:I].T + t * scale * ((X @ a13[:r].T) @ np.asarray(b1, np.float64).T)
    U = X @ w13[I:].T + t * scale * ((X @ a13[r:].T) @ np.asarray(b3, np.float64).T)
    Hh = G / (1.0 + np.exp(-G)) * U
    return Hh @ np.asarray(w2, np.float64).T + t * scale * ((Hh @ np.asarray(a2, np.float64).T)
                                                           @ np.asarray(b2, np.float64).T)


def lora_physical_rows(idx: np.ndarray, taus: np.ndarray, n_experts: int, mode: int) -> np.ndarray:
    """Adapter rows physically executed per token under each gate granularity. Rows are
    the dispatch order (experts ascending, tokens ascending within an expert).
    ROW      the gate is applied per row before any adapter work: allow rows only;
    TILE     the gate is applied per tile of LORA_TILE_ROWS consecutive rows of one expert:
             a tile runs its adapter when any of its rows allows, so denied rows that
             share a tile with an allowed row are executed (and their result discarded);
    POSTHOC  every row runs the adapter; the decision only scales the result."""
    dp = dispatch(idx, n_experts)
    T = idx.shape[0]
    rows = np.zeros(T, np.int64)
    for e in range(n_experts):
        toks = dp.row_token[dp.offset[e]:dp.offset[e] + dp.count[e]]
        for s in range(0, len(toks), LORA_TILE_ROWS):
            tile = toks[s:s + LORA_TILE_ROWS]
            for t in tile:
                if mode == LORA_GATE_ROW:
                    run = taus[t] == 1
                elif mode == LORA_GATE_TILE:
                    run = any(taus[u] == 1 for u in tile)
                elif mode == LORA_GATE_POSTHOC:
                    run = True
                else:
                    raise ValueError(mode)
                rows[t] += int(run)
    return rows


# ----------------------------------------------------------------------------
# Optimizer step over the private parameters (G2 of Sec. 2.2: only private parameters
# are passed to the optimizer; Sec. 3.2 and App. C.1: fused AdamW)
# ----------------------------------------------------------------------------

def adamw_step(p: np.ndarray, g: np.ndarray, m: np.ndarray, v: np.ndarray, step: int, lr: float,
               beta1: float, beta2: float, eps: float, weight_decay: float):
    """AdamW (Loshchilov and Hutter, decoupled weight decay) in fp64: the parameter first
    decays by lr * wd * p, then moves by lr * m_hat / (sqrt(v_hat) + eps) with the
    bias-corrected moments of step `step` (1-based). Returns (p, m, v)."""
    p = np.asarray(p, np.float64) * (1.0 - lr * weight_decay)
    g = np.asarray(g, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    mh = m / (1.0 - beta1 ** step)
    vh = v / (1.0 - beta2 ** step)
    return p - lr * mh / (np.sqrt(vh) + eps), m, v
