"""GPU parity of the policy-masked MoE layer against the CPU oracle (through the C ABI).

Acceptance: allow bit-exact; topk_idx bit-exact on every token the oracle does not
flag as a near tie (k-th/(k+1)-th fp32 logit gap < 1e-5); dispatch outputs exact
functions of the GPU's own topk_idx and equal to the oracle's where routes agree;
the private-row audit bit-exact always; gates rel-L2 <= 1e-5; layer output rel-L2
<= 1e-2 (bf16 experts) or 1e-5 (fp32 experts) over tokens whose routes agree.
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C
import paper_2608_06690_amd as P

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def words_for(cfg, pass_idx=0):
    req = W.make_requests(cfg, pass_idx)
    return req, O.compile_words(req.metas, req.lengths)


def full_check(cfg, layer, x_dev, words, req, oi=None, rtol=None):
    """Run the device layer and the full oracle; assert every acceptance rule, including
    the per-row bars on every expert output row and every token of every agreeing token."""
    d = C.run_device(layer, x_dev, C.words_tensor(words), torch.tensor(req.offsets, device="cuda"))
    oi = oi or C.oracle_inputs(cfg)
    ref = C.oracle_layer(cfg, oi, words)
    stats = C.compare_routes(cfg, d, ref.route)
    C.check_dispatch_consistent(d, cfg.n_experts)
    same = np.all(d.idx == ref.route.idx, axis=1)
    if same.all():
        assert np.array_equal(d.count, ref.disp.count)
        assert np.array_equal(d.row_token, ref.disp.row_token)
    # audit: bit-exact with the oracle's hooks (tie-independent: pools are disjoint)
    assert np.array_equal(d.audit_rows, ref.hook.rows)
    a = O.audit(ref.hook.rows, ref.route.allow, req.offsets)
    assert np.array_equal(d.req_rows, a.req_private_rows)
    assert d.total == a.total_private_rows == cfg.top_k * int(ref.route.allow.sum())
    assert d.violations == 0 and d.dev_status == 0
    # expert output rows and layer outputs, per row and in aggregate, on agreeing tokens
    rs = C.check_rows(cfg, d, ref, np.nonzero(same)[0], tag=f"{cfg.name}: T={cfg.tokens}")
    log(f"{cfg.name}: T={cfg.tokens} rel_l2={rs['agg']:.3e} {stats}")
    if rtol is not None:
        assert rs["agg"] <= rtol
    return d, ref


# ----------------------------------------------------------------------------
# Tiny fp32 layer: allow - deny - allow
# ----------------------------------------------------------------------------

def test_tiny_fp32_allow_deny_allow():
    cfg = W.get_config("tiny")
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    oi = C.oracle_inputs(cfg)
    res = []
    for p in range(3):
        req, words = words_for(cfg, p)
        log(f"tiny pass {p}: kinds={req.kinds}")
        res.append(full_check(cfg, layer, x, words, req, oi))
    d0, d1, d2 = (r[0] for r in res)
    assert d1.total == 0 and d1.audit_rows.sum() == 0 and np.all(d1.idx < cfg.n_pub)
    assert torch.equal(d0.out, d2.out)           # recovery reproduces allow bitwise
    assert np.array_equal(d0.idx, d2.idx) and np.array_equal(d0.gate, d2.gate)
    assert np.array_equal(d0.audit_rows, d2.audit_rows)


# ----------------------------------------------------------------------------
# Small bf16 layers with ragged sizes (several tiles, ragged tails)
# ----------------------------------------------------------------------------

SMALL = [
    dict(tokens=300, requests=6, hidden=256, inter=192, n_pub=24, n_priv=12, top_k=4),
    dict(tokens=77, requests=7, hidden=384, inter=128, n_pub=16, n_priv=8, top_k=8),
    dict(tokens=1, requests=1, hidden=128, inter=64, n_pub=8, n_priv=8, top_k=8),  # k = pool
    dict(tokens=520, requests=4, hidden=256, inter=256, n_pub=200, n_priv=40, top_k=6),
]


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: f"T{s['tokens']}_H{s['hidden']}_E{s['n_pub']}+{s['n_priv']}_k{s['top_k']}")
@pytest.mark.parametrize("gather", [False, True], ids=["fused_gather", "dispatch_gather"])
def test_small_bf16_layer(shape, gather):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    layer, _ = C.device_layer(cfg, gather_in_dispatch=gather)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    req.lengths[-1] += cfg.tokens - sum(req.lengths)
    words = O.compile_words(req.metas, req.lengths)
    full_check(cfg, layer, x, words, req)


# Batches above 2048 tokens take the router whose operands are staged in LDS (64-token
# tiles; 2048 tokens is the register kernel's largest batch): a ragged last tile, tiles that mix allow and deny tokens (request boundaries off
# the 64-token grid), pools that are not multiples of 16, and H = 384 (6 K steps, so the
# per-block K rotation wraps at an odd count).
LARGE_ROUTE = [
    dict(tokens=2048, requests=7, hidden=256, inter=128, n_pub=40, n_priv=12, top_k=4),  # last register-path size
    dict(tokens=2049, requests=7, hidden=256, inter=128, n_pub=40, n_priv=12, top_k=4),  # one-token last tile
    dict(tokens=2113, requests=9, hidden=256, inter=128, n_pub=40, n_priv=12, top_k=4),
    dict(tokens=4100, requests=5, hidden=384, inter=128, n_pub=128, n_priv=32, top_k=8),
    # both pools over several partly filled 64-expert groups, H split four ways
    dict(tokens=2500, requests=5, hidden=512, inter=128, n_pub=100, n_priv=70, top_k=6),
]


@pytest.mark.parametrize("shape", LARGE_ROUTE, ids=lambda s: f"T{s['tokens']}_H{s['hidden']}_E{s['n_pub']}+{s['n_priv']}")
def test_large_batch_router(shape):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    req.lengths[-1] += cfg.tokens - sum(req.lengths)
    words = O.compile_words(req.metas, req.lengths)
    full_check(cfg, layer, x, words, req)


# The large-batch top-k adds every split's whole partial-logit row of a token (the row is as
# wide as the larger pool) before the token's policy word has told it which pool it ranks, so
# entries past the pool hold whatever the workspace held. The routing must not depend on it:
# the same batch routed over a workspace of zeros, NaNs and huge values gives the same bits.
@pytest.mark.parametrize("soft", [False, True], ids=["masked", "soft"])
def test_large_batch_router_ignores_workspace_contents(soft):
    shape = dict(tokens=4100, requests=5, hidden=384, inter=128, n_pub=128, n_priv=32, top_k=8)
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    layer, _ = C.device_layer(cfg, soft=soft)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    req.lengths[-1] += cfg.tokens - sum(req.lengths)
    words = C.words_tensor(O.compile_words(req.metas, req.lengths))
    b = layer.buffers(cfg.tokens)
    log(f"router workspace fills: T={cfg.tokens} soft={soft}")
    outs = []
    for fill in (0.0, float("nan"), 3.0e38, -3.0e38):
        b.ws.view(torch.float32).fill_(fill)
        layer.route(x, words, b)
        torch.cuda.synchronize()
        outs.append([t.clone() for t in (b.topk_idx, b.topk_gate, b.allow, b.kgap)])
    for o in outs[1:]:
        for got, ref in zip(o, outs[0]):
            assert torch.equal(got, ref)
    assert int(b.dev_status.item()) == 0


# Expert intermediate 64: the down projection has a single K step per tile, so in a
# persistent block the copy producer runs up to STAGES-1 tiles ahead of the tile being
# multiplied, and the gather-index (row_token) slices of STAGES+1 tiles are live at once;
# the execution audit reads the slice of the tile it counts. Several private tiles per
# block (2048 alternating tokens) and a skewed decode batch (Zipf bias, malformed words),
# audit and per-request rows bit-exact.
INTER64 = [
    ("alternating_2048", dict(tokens=2048, requests=8, hidden=512, inter=64)),
    ("decode_zipf", dict(inter=64)),
]


@pytest.mark.parametrize("name,shape", INTER64, ids=[n for n, _ in INTER64])
def test_inter64_audit_several_tiles_per_block(name, shape):
    base = W.get_config("decode" if name.startswith("decode") else "qwen")
    cfg = W.scaled_config(base, **shape)
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    if name.startswith("decode"):
        req, words = words_for(cfg)
    else:
        req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
        words = O.compile_words(req.metas, req.lengths)
    d, ref = full_check(cfg, layer, x, words, req)
    assert d.total > 0
    if name.startswith("alternating"):  # private experts span several 64-row tiles
        assert ref.disp.count[cfg.n_pub:].min() > 64


def test_small_deepseek_like_shared_and_pool_softmax():
    cfg = W.scaled_config(W.get_config("deepseek"), tokens=400, requests=4, hidden=256, inter=128,
                          n_pub=32, n_priv=8, top_k=6, shared_inter=192)
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req, words = words_for(cfg)
    full_check(cfg, layer, x, words, req)


# ----------------------------------------------------------------------------
# Full-size workloads: every token through the oracle
# ----------------------------------------------------------------------------

@pytest.mark.timeout(600)
def test_qwen_layer_full_size():
    cfg = W.get_config("qwen")
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req, words = words_for(cfg)
    log(f"{cfg.name}: device run and oracle of all {cfg.tokens} tokens")
    d, ref = full_check(cfg, layer, x, words, req)
    assert int(d.allow.sum()) == 2048 and d.total == 2048 * cfg.top_k


@pytest.mark.timeout(600)
def test_deepseek_layer_full_size():
    cfg = W.get_config("deepseek")
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req, words = words_for(cfg)
    log(f"{cfg.name}: device run and oracle of all {cfg.tokens} tokens")
    d, ref = full_check(cfg, layer, x, words, req)
    # the skewed bias leaves routed experts without rows: they load nothing, and the
    # device's empty experts are exactly the oracle's once routes agree
    n_empty = int((ref.disp.count == 0).sum())
    assert n_empty > 0
    if np.all(d.idx == ref.route.idx):
        assert int((d.count == 0).sum()) == n_empty
        assert np.array_equal(d.count == 0, ref.disp.count == 0)


def test_decode_layer_full_oracle():
    cfg = W.get_config("decode")
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req, words = words_for(cfg)
    assert req.kinds.count("malformed") == 26 and req.kinds.count("allow") == 64
    d, ref = full_check(cfg, layer, x, words, req)
    assert int(d.allow.sum()) == 64


# ----------------------------------------------------------------------------
# Prefill batches on the 256 x 256 persistent expert kernel (T*k at least 128 rows per
# expert on average): several tiles per persistent block, ragged M tiles (private
# experts of ~2,460 rows, public ones of ~820), rows past a tile's valid count, both
# gather paths, the shared group, and the fail-closed paths (NULL or NaN private
# weights) at this size
# ----------------------------------------------------------------------------

PREFILL_MULTI = dict(tokens=4100, requests=5, hidden=1024, inter=512, n_pub=16, n_priv=8, top_k=8)


@pytest.mark.parametrize("gather", [False, True], ids=["fused_gather", "dispatch_gather"])
def test_prefill_multi_tile(gather):
    cfg = W.scaled_config(W.get_config("qwen"), **PREFILL_MULTI)
    layer, _ = C.device_layer(cfg, gather_in_dispatch=gather)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    words = O.compile_words(req.metas, req.lengths)
    d, ref = full_check(cfg, layer, x, words, req)
    cnt = ref.disp.count
    assert cnt[cfg.n_pub:].min() > 2 * 256 and cnt[:cfg.n_pub].min() > 256   # ragged multi-tile experts


# The shared group's tiles lead every XCD's tile list in chunks of 8: 2048 tokens give 16
# shared tiles per GEMM (whole chunks); 1300 tokens with 2 I_s = 384 give 18 (GEMM1) and 12
# (GEMM2), each ending in a partial chunk.
@pytest.mark.parametrize("tokens,shared_inter", [(2048, 128), (1300, 192)], ids=["whole_chunks", "partial_chunk"])
def test_prefill_shared_group_pool_softmax(tokens, shared_inter):
    cfg = W.scaled_config(W.get_config("deepseek"), tokens=tokens, requests=4, hidden=512, inter=256,
                          n_pub=32, n_priv=8, top_k=6, shared_inter=shared_inter)
    assert cfg.tokens * cfg.top_k >= 128 * (cfg.n_pub + cfg.n_priv)  # the 256 x 256 prefill tiles
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req, words = words_for(cfg)
    full_check(cfg, layer, x, words, req)


def test_prefill_fail_closed_private_weights():
    cfg = W.scaled_config(W.get_config("qwen"), **PREFILL_MULTI)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    words = O.compile_words(req.metas, req.lengths)
    offs = torch.tensor(req.offsets, device="cuda")
    ref_layer, Lw = C.device_layer(cfg)
    ref = C.run_device(ref_layer, x, C.words_tensor(words), offs)
    # allow rows with the private weights missing: not executed, not audited, zeroed
    nul = P.PolicyMaskedMoE(C.make_desc(cfg), Lw.wr_pub, Lw.wr_priv, None, Lw.w13_pub, Lw.w2_pub,
                            None, None)
    d = C.run_device(nul, x, C.words_tensor(words), offs)
    taus = np.array([O.decode_word(w) for w in words])
    assert d.dev_status & 0x2 and d.total == 0 and d.audit_rows.sum() == 0
    assert torch.all(d.out[torch.from_numpy(taus == 1)] == 0)
    deny = torch.from_numpy(taus == 0)
    assert torch.equal(d.out[deny], ref.out[deny])
    # all deny: NULL and NaN private tensors give the full layer's output bit for bit
    dreq = W.Requests([820] * 5, [W.DENY_META] * 5, ["deny"] * 5)
    dwords = C.words_tensor(O.compile_words(dreq.metas, dreq.lengths))
    base = C.run_device(ref_layer, x, dwords, offs)
    nulld = C.run_device(C.device_layer(cfg, drop_private=True)[0], x, dwords, offs)
    nan = P.PolicyMaskedMoE(C.make_desc(cfg), Lw.wr_pub, torch.full_like(Lw.wr_priv, float("nan")), None,
                            Lw.w13_pub, Lw.w2_pub, torch.full_like(Lw.w13_priv, float("nan")),
                            torch.full_like(Lw.w2_priv, float("nan")))
    dnan = C.run_device(nan, x, dwords, offs)
    for dd in (nulld, dnan):
        assert torch.equal(dd.out, base.out) and dd.total == 0 and dd.dev_status == 0
    log(f"prefill fail-closed: allow rows zeroed {int((taus == 1).sum())}, deny rows equal")
