"""Seeded synthetic inputs for the policy-masked MoE layer.

This module generates inputs only: random tensors, request lengths and request
metadata. It computes no step of the layer (no policy resolution, no routing, no
expert math), so the CPU oracle and the GPU path can both draw their inputs from
it without sharing any of the method's arithmetic.

Random tensors come from a counter-based generator so that the same values can be
produced on the host (for the oracle) or directly on the device (for large GPU
cases), bit for bit, and so that any single expert's weights can be regenerated
on its own:

* SplitMix64 (Steele, Lea and Flood, OOPSLA 2014; the published `splitmix64`
  finaliser) is evaluated on a per-tensor 64-bit key plus the word counter
  times the golden-ratio increment;
* each 64-bit output word yields four 16-bit uniforms u;
* u is mapped to an approximate standard normal deviate through a fixed fp32
  table of the inverse normal CDF at (u + 1/2) / 65536 (tails reach +-4.3);
* the deviate is scaled by the tensor's standard deviation with one fp32
  multiply and, for bf16 tensors, rounded to nearest even.

All integer steps are exact, the fp32 multiply and the bf16 rounding are
correctly rounded on both devices, and the table is built once on the host, so
host- and device-generated tensors are identical.

Workload recipes (the five layer configurations of the benchmark):

* ``tiny``     64 tokens in 4 requests of 16, H 128, I 256, 8 public + 4 private
               experts, top-2, fp32; every tensor N(0, 0.02); three passes
               (drawn policies, all deny, drawn policies again).
* ``qwen``     Qwen3-30B-A3B-shaped layer: 4096 tokens in 8 requests of 512,
               H 2048, I 768, 128 public + 32 private, top-8, bf16 experts,
               fp32 router; x ~ N(0, 1), router and experts N(0, 0.02);
               4 allow and 4 deny requests in a seeded order.
* ``deepseek`` DeepSeek-V2-Lite-shaped layer: 8192 tokens in 16 requests of 512,
               H 2048, I 1408, 2 shared + 64 public + 16 private, top-6 with
               pool-softmax gates, per-expert logit bias N(0, 1); policy
               Bernoulli(1/2) per request.
* ``decode``   256 requests of 1 token, Qwen shape, Zipf(1.1) logit bias
               b_e = -1.1 ln(rank_e) with ranks a seeded permutation within each
               pool; 64 allow, 26 malformed and 166 deny requests.
* ``stack``    48 independent Qwen-shaped layers, 16384 tokens in 32 requests of
               512; passes all allow, all deny, all allow.
"""
from __future__ import annotations

import dataclasses
from statistics import NormalDist
from typing import Any, Dict, List, Optional, Sequence

import numpy as np
import torch

BASE_SEED = 20260730

# ----------------------------------------------------------------------------
# Configurations
# ----------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    index: int            # position in the list of workloads; the seed is BASE_SEED + index
    tokens: int
    requests: int
    hidden: int
    inter: int
    n_pub: int
    n_priv: int
    top_k: int
    n_shared: int = 0
    shared_inter: int = 0
    dtype: str = "bf16"   # "f32" or "bf16": activations and expert weights
    gate_mode: str = "renorm"   # "renorm" or "pool_softmax"
    x_std: float = 1.0
    w_std: float = 0.02
    wr_std: float = 0.02
    bias: Optional[str] = None  # None, "normal" or "zipf"
    layers: int = 1
    passes: int = 1

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index

    @property
    def n_experts(self) -> int:
        return self.n_pub + self.n_priv

    @property
    def req_len(self) -> int:
        return self.tokens // self.requests


CONFIGS: Dict[str, LayerConfig] = {
    "tiny": LayerConfig("tiny", 0, 64, 4, 128, 256, 8, 4, 2, dtype="f32",
                        x_std=0.02, w_std=0.02, wr_std=0.02, passes=3),
    "qwen": LayerConfig("qwen", 1, 4096, 8, 2048, 768, 128, 32, 8),
    "deepseek": LayerConfig("deepseek", 2, 8192, 16, 2048, 1408, 64, 16, 6,
                            n_shared=2, shared_inter=1408, gate_mode="pool_softmax",
                            bias="normal"),
    "decode": LayerConfig("decode", 3, 256, 256, 2048, 768, 128, 32, 8, bias="zipf"),
    "stack": LayerConfig("stack", 4, 16384, 32, 2048, 768, 128, 32, 8, layers=48, passes=3),
}
ALIASES = {"c1": "tiny", "c2": "qwen", "c3": "deepseek", "c4": "decode", "c5": "stack"}


def get_config(name: str) -> LayerConfig:
    return CONFIGS[ALIASES.get(name, name)]


def scaled_config(cfg: LayerConfig, **changes) -> LayerConfig:
    """A copy of `cfg` with some fields replaced (smaller parity cases)."""
    return dataclasses.replace(cfg, **changes)


# ----------------------------------------------------------------------------
# Counter-based generator
# ----------------------------------------------------------------------------

_M64 = 1 << 64
_GOLDEN = 0x9E3779B97F4A7C15
_MIX1 = 0xBF58476D1CE4E5B9
_MIX2 = 0x94D049BB133111EB


def _signed(v: int) -> int:
    v &= _M64 - 1
    return v - _M64 if v >= (1 << 63) else v


def splitmix64_int(z: int) -> int:
    """SplitMix64 finaliser on a Python int (used to derive tensor keys)."""
    z &= _M64 - 1
    z = ((z ^ (z >> 30)) * _MIX1) & (_M64 - 1)
    z = ((z ^ (z >> 27)) * _MIX2) & (_M64 - 1)
    return z ^ (z >> 31)


def tensor_key(*parts: int) -> int:
    """64-bit key for one tensor slice, derived from integers (seed, layer, tensor id, ...)."""
    k = 0
    for p in parts:
        k = splitmix64_int((k + _GOLDEN + (int(p) & (_M64 - 1))) & (_M64 - 1))
    return k


def _lsr(z: torch.Tensor, s: int) -> torch.Tensor:
    # logical right shift of int64 lanes holding uint64 bit patterns
    return (z >> s) & ((1 << (64 - s)) - 1)


def splitmix64_words(key: int, n_words: int, device) -> torch.Tensor:
    """n_words outputs of SplitMix64 for counters 1..n_words under `key` (int64 bit patterns)."""
    ctr = torch.arange(1, n_words + 1, dtype=torch.int64, device=device)
    z = ctr * _signed(_GOLDEN) + _signed(key)
    z = (z ^ _lsr(z, 30)) * _signed(_MIX1)
    z = (z ^ _lsr(z, 27)) * _signed(_MIX2)
    return z ^ _lsr(z, 31)


_TABLE_CACHE: Dict[str, torch.Tensor] = {}


def normal_table(device="cpu") -> torch.Tensor:
    """fp32 table t[u] = inverse normal CDF at (u + 1/2) / 65536, u in [0, 65536)."""
    dev = str(torch.device(device))
    if dev not in _TABLE_CACHE:
        if "cpu" not in _TABLE_CACHE:
            nd = NormalDist()
            vals = [nd.inv_cdf((u + 0.5) / 65536.0) for u in range(65536)]
            _TABLE_CACHE["cpu"] = torch.tensor(vals, dtype=torch.float64).to(torch.float32)
        _TABLE_CACHE[dev] = _TABLE_CACHE["cpu"].to(device)
    return _TABLE_CACHE[dev]


_CHUNK_WORDS = 1 << 22


def normal(key: int, shape: Sequence[int], std: float, dtype: torch.dtype = torch.float32,
           device="cpu") -> torch.Tensor:
    """Tensor of approximately N(0, std^2) values from the counter-based generator."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = torch.empty(n, dtype=dtype, device=device)
    table = normal_table(device)
    scale = torch.tensor(std, dtype=torch.float32, device=device)
    n_words = (n + 3) // 4
    w0 = 0
    while w0 < n_words:
        nw = min(_CHUNK_WORDS, n_words - w0)
        ctr = torch.arange(w0 + 1, w0 + nw + 1, dtype=torch.int64, device=device)
        z = ctr * _signed(_GOLDEN) + _signed(key)
        z = (z ^ _lsr(z, 30)) * _signed(_MIX1)
        z = (z ^ _lsr(z, 27)) * _signed(_MIX2)
        z = z ^ _lsr(z, 31)
        # the four 16-bit fields of each word, lowest first (little-endian lanes)
        u = z.view(torch.int16).to(torch.int32) & 0xFFFF
        e0 = 4 * w0
        e1 = min(n, 4 * (w0 + nw))
        v = table[u[: e1 - e0]] * scale
        out[e0:e1] = v.to(dtype)
        w0 += nw
    return out.reshape(tuple(shape))


# tensor ids inside a layer's key space
T_X, T_WR_PUB, T_WR_PRIV, T_BIAS, T_W13_PUB, T_W2_PUB, T_W13_PRIV, T_W2_PRIV, T_W13_SH, T_W2_SH, T_DOUT = range(11)
T_LORA_A13, T_LORA_B1, T_LORA_B3, T_LORA_A2, T_LORA_B2 = range(11, 16)


def torch_dtype(cfg: LayerConfig) -> torch.dtype:
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


# ----------------------------------------------------------------------------
# Layer tensors
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class LayerWeights:
    """One layer's parameters. Expert weights: w13 [E, 2I, H] (gate rows, then up rows),
    w2 [E, H, I]; router rows fp32 [n, H]; shared group as one SwiGLU of intermediate
    n_shared * shared_inter: w13_sh [2 * Is, H], w2_sh [H, Is]."""
    wr_pub: torch.Tensor
    wr_priv: torch.Tensor
    bias: Optional[torch.Tensor]
    w13_pub: torch.Tensor
    w2_pub: torch.Tensor
    w13_priv: torch.Tensor
    w2_priv: torch.Tensor
    w13_sh: Optional[torch.Tensor] = None
    w2_sh: Optional[torch.Tensor] = None


def make_x(cfg: LayerConfig, device="cpu", tokens: Optional[Sequence[int]] = None) -> torch.Tensor:
    """Layer input x [T, H] (the first layer's input for the stack)."""
    x = normal(tensor_key(cfg.seed, 0, T_X, 0), (cfg.tokens, cfg.hidden), cfg.x_std,
               torch_dtype(cfg), device)
    return x if tokens is None else x[torch.as_tensor(tokens, device=x.device)]


def make_dout(cfg: LayerConfig, layer: int = 0, device="cpu", std: float = 1.0) -> torch.Tensor:
    """Upstream gradient of the layer output, [T, H] in the activation dtype."""
    return normal(tensor_key(cfg.seed, layer, T_DOUT, 0), (cfg.tokens, cfg.hidden), std,
                  torch_dtype(cfg), device)


def make_lora(cfg: LayerConfig, rank: int, layer: int = 0, device="cpu", std: float = 0.02):
    """Rank-`rank` adapters on every public expert's gate, up and down projections (the
    matched expert-LoRA control): a13 [n_pub, 2r, H] (gate rows then up rows), b1 and b3
    [n_pub, I, r], a2 [n_pub, r, I], b2 [n_pub, H, r], in the activation dtype. Both
    factors are drawn (not the zero-B initialisation), so the adapter is not a no-op."""
    s, dt, n, H, I = cfg.seed, torch_dtype(cfg), cfg.n_pub, cfg.hidden, cfg.inter
    k = lambda tid: tensor_key(s, layer, tid, rank)  # noqa: E731
    return (normal(k(T_LORA_A13), (n, 2 * rank, H), std, dt, device),
            normal(k(T_LORA_B1), (n, I, rank), std, dt, device),
            normal(k(T_LORA_B3), (n, I, rank), std, dt, device),
            normal(k(T_LORA_A2), (n, rank, I), std, dt, device),
            normal(k(T_LORA_B2), (n, H, rank), std, dt, device))


def quantize_fp8_rows(w: torch.Tensor):
    """Per-row power-of-two scaling of a weight stack [..., rows, cols] into OCP fp8 e4m3:
    scale = 2^ceil(log2(max|row| / 448)) (1 for an all-zero row), q = round-to-nearest-even
    of w / scale. Returns (q as uint8 bytes, fp32 scales [..., rows], the dequantised
    weights q * scale as fp32); q * scale is exact, and so is its bf16 value."""
    wf = w.float()
    amax = wf.abs().amax(dim=-1)
    e = torch.ceil(torch.log2(torch.clamp(amax, min=1e-30) / 448.0))
    scale = torch.where(amax > 0, torch.exp2(e), torch.ones_like(amax))
    q = (wf / scale.unsqueeze(-1)).to(torch.float8_e4m3fn)
    deq = q.float() * scale.unsqueeze(-1)
    return q.view(torch.uint8), scale.contiguous(), deq


def make_router(cfg: LayerConfig, layer: int = 0, device="cpu"):
    s = cfg.seed
    wr_pub = normal(tensor_key(s, layer, T_WR_PUB, 0), (cfg.n_pub, cfg.hidden), cfg.wr_std,
                    torch.float32, device)
    wr_priv = normal(tensor_key(s, layer, T_WR_PRIV, 0), (cfg.n_priv, cfg.hidden), cfg.wr_std,
                     torch.float32, device)
    bias = None
    if cfg.bias == "normal":
        bias = normal(tensor_key(s, layer, T_BIAS, 0), (cfg.n_experts,), 1.0, torch.float32, device)
    elif cfg.bias == "zipf":
        rng = np.random.default_rng([s, layer, T_BIAS])
        ranks = np.concatenate([rng.permutation(cfg.n_pub) + 1, rng.permutation(cfg.n_priv) + 1])
        bias = torch.from_numpy((-1.1 * np.log(ranks.astype(np.float64))).astype(np.float32)).to(device)
    return wr_pub, wr_priv, bias


def make_expert(cfg: LayerConfig, layer: int, expert: int, device="cpu"):
    """(w13 [2I, H], w2 [H, I]) of global expert id `expert` (public ids first)."""
    s, dt = cfg.seed, torch_dtype(cfg)
    if expert < cfg.n_pub:
        k13, k2, e = T_W13_PUB, T_W2_PUB, expert
    else:
        k13, k2, e = T_W13_PRIV, T_W2_PRIV, expert - cfg.n_pub
    w13 = normal(tensor_key(s, layer, k13, e), (2 * cfg.inter, cfg.hidden), cfg.w_std, dt, device)
    w2 = normal(tensor_key(s, layer, k2, e), (cfg.hidden, cfg.inter), cfg.w_std, dt, device)
    return w13, w2


def make_shared(cfg: LayerConfig, layer: int = 0, device="cpu"):
    if cfg.n_shared == 0:
        return None, None
    s, dt = cfg.seed, torch_dtype(cfg)
    i_sh = cfg.n_shared * cfg.shared_inter
    w13 = normal(tensor_key(s, layer, T_W13_SH, 0), (2 * i_sh, cfg.hidden), cfg.w_std, dt, device)
    w2 = normal(tensor_key(s, layer, T_W2_SH, 0), (cfg.hidden, i_sh), cfg.w_std, dt, device)
    return w13, w2


def make_layer(cfg: LayerConfig, layer: int = 0, device="cpu") -> LayerWeights:
    wr_pub, wr_priv, bias = make_router(cfg, layer, device)
    dt = torch_dtype(cfg)
    E, H, I = cfg.n_experts, cfg.hidden, cfg.inter
    w13 = torch.empty((E, 2 * I, H), dtype=dt, device=device)
    w2 = torch.empty((E, H, I), dtype=dt, device=device)
    for e in range(E):
        a, b = make_expert(cfg, layer, e, device)
        w13[e].copy_(a)
        w2[e].copy_(b)
    w13_sh, w2_sh = make_shared(cfg, layer, device)
    n = cfg.n_pub
    return LayerWeights(wr_pub, wr_priv, bias, w13[:n], w2[:n], w13[n:], w2[n:], w13_sh, w2_sh)


# ----------------------------------------------------------------------------
# Requests and trusted metadata
# ----------------------------------------------------------------------------

ALLOW_META = {"allow_private": True}
DENY_META = {"allow_private": False}

# Metadata forms that must all fail closed: missing metadata, wrong keys, strings,
# numbers, lists, nested values, nulls and serialized JSON text.
MALFORMED_META: List[Any] = [
    None,
    {},
    {"allow": True},
    {"Allow_Private": True},
    {"allow_private": "true"},
    {"allow_private": "True"},
    {"allow_private": 1},
    {"allow_private": 1.0},
    {"allow_private": [True]},
    {"allow_private": (True,)},
    {"allow_private": {"value": True}},
    {"allow_private": None},
    '{"allow_private": true}',
    b'{"allow_private": true}',
    [("allow_private", True)],
    {"user": {"allow_private": True}},
    {"allow_private": "1"},
    {"allow_private": "yes"},
]


@dataclasses.dataclass
class Requests:
    lengths: List[int]
    metas: List[Any]
    kinds: List[str]   # "allow", "deny" or "malformed": how the metadata was drawn

    @property
    def offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.lengths)]).astype(np.int32)


def _meta(kind: str, i: int) -> Any:
    if kind == "allow":
        return dict(ALLOW_META)
    if kind == "deny":
        return dict(DENY_META)
    return MALFORMED_META[i % len(MALFORMED_META)]


def make_requests(cfg: LayerConfig, pass_idx: int = 0) -> Requests:
    """Requests of one pass. Kinds per workload:

    tiny: one seeded request malformed, the rest Bernoulli(1/2) (redrawn until both
    decisions appear); pass 1 is all deny. qwen: seeded order of 4 allow + 4 deny.
    deepseek: Bernoulli(1/2), redrawn until both appear. decode: seeded order of 64
    allow, 26 malformed, 166 deny. stack: all allow, all deny, all allow.
    """
    R = cfg.requests
    rng = np.random.default_rng([cfg.seed, 7777])
    if cfg.name == "tiny":
        while True:
            bad = int(rng.integers(R))
            kinds = ["allow" if b else "deny" for b in rng.integers(0, 2, R)]
            kinds[bad] = "malformed"
            good = [k for i, k in enumerate(kinds) if i != bad]
            if "allow" in good and "deny" in good:
                break
        if pass_idx == 1:
            kinds = ["deny"] * R
    elif cfg.name == "qwen":
        kinds = list(rng.permutation(["allow"] * (R // 2) + ["deny"] * (R - R // 2)))
    elif cfg.name == "deepseek":
        while True:
            kinds = ["allow" if b else "deny" for b in rng.integers(0, 2, R)]
            if "allow" in kinds and "deny" in kinds:
                break
    elif cfg.name == "decode":
        n_allow, n_bad = round(0.25 * R), round(0.10 * R)
        kinds = list(rng.permutation(["allow"] * n_allow + ["malformed"] * n_bad
                                     + ["deny"] * (R - n_allow - n_bad)))
    elif cfg.name == "stack":
        kinds = ["deny" if pass_idx == 1 else "allow"] * R
    else:  # scaled-down copies of a workload keep its name; anything else alternates
        kinds = ["allow" if i % 2 == 0 else "deny" for i in range(R)]
    kinds = [str(k) for k in kinds]
    metas = [_meta(k, i) for i, k in enumerate(kinds)]
    lengths = [cfg.tokens // R] * R
    lengths[-1] += cfg.tokens - sum(lengths)
    return Requests(lengths, metas, kinds)


def alternating_requests(n_rows: int, row_len: int) -> Requests:
    """Mixed-policy batch: rows alternate allow and deny (the mixed-batch attack family)."""
    kinds = ["allow" if i % 2 == 0 else "deny" for i in range(n_rows)]
    return Requests([row_len] * n_rows, [_meta(k, i) for i, k in enumerate(kinds)], kinds)
