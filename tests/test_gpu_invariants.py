"""GPU invariants and edge cases of the policy-masked MoE layer (through the C ABI).

* determinism: two runs give identical bits;
* deny isolation: an all-deny batch gives bitwise the same output with the private
  pointers NULL, present, or poisoned with NaN; private router rows scaled by 1e6 and
  inputs aligned with them still route deny tokens to public experts only;
* fail closed on the device: malformed words deny; allow words without a private
  router route as deny (status bit); private rows without private weights are not
  executed or audited (status bit);
* grouped-GEMM edge cases checked against the oracle on a given routing: an expert
  with exactly 152 rows, every token on one expert, empty experts, and shapes where
  each persistent block processes several tiles.
"""
import numpy as np
import pytest
import torch

import paper_2608_06690_amd as P
import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C

pytestmark = pytest.mark.gpu

SMALL = dict(tokens=320, requests=4, hidden=256, inter=128, n_pub=24, n_priv=8, top_k=4)


def small_cfg(**kw):
    d = dict(SMALL)
    d.update(kw)
    return W.scaled_config(W.get_config("qwen"), **d)


def run(layer, x, words, req):
    return C.run_device(layer, x, None if words is None else C.words_tensor(words),
                        torch.tensor(req.offsets, device="cuda"))


def test_determinism_bitwise():
    cfg = small_cfg()
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(4, 80)
    words = O.compile_words(req.metas, req.lengths)
    a = run(layer, x, words, req)
    b = run(layer, x, words, req)
    assert torch.equal(a.out, b.out)
    assert np.array_equal(a.idx, b.idx) and np.array_equal(a.gate, b.gate)
    assert np.array_equal(a.row_token, b.row_token) and np.array_equal(a.audit_rows, b.audit_rows)


def test_all_deny_equal_with_null_and_nan_private():
    cfg = small_cfg()
    x = W.make_x(cfg, "cuda")
    req = W.Requests([80] * 4, [W.DENY_META] * 4, ["deny"] * 4)
    words = O.compile_words(req.metas, req.lengths)
    layer, Lw = C.device_layer(cfg)
    ref = run(layer, x, words, req)
    null_layer, _ = C.device_layer(cfg, drop_private=True)
    d_null = run(null_layer, x, words, req)
    poisoned = P.PolicyMaskedMoE(layer.desc, Lw.wr_pub, torch.full_like(Lw.wr_priv, float("nan")),
                                 None, Lw.w13_pub, Lw.w2_pub, torch.full_like(Lw.w13_priv, float("nan")),
                                 torch.full_like(Lw.w2_priv, float("nan")))
    d_nan = run(poisoned, x, words, req)
    for d in (d_null, d_nan):
        assert torch.equal(d.out, ref.out)
        assert not torch.isnan(d.out.float()).any()
        assert d.total == 0 and d.audit_rows.sum() == 0 and d.dev_status == 0
        assert np.all(d.idx < cfg.n_pub)
    # public-only layer: a plain MoE over the public pool equals the deny output
    oi = C.oracle_inputs(cfg)
    res = C.oracle_layer(cfg, oi, words)
    assert np.array_equal(ref.audit_rows, res.hook.rows)


def test_adversarial_private_router_override_under_deny():
    cfg = small_cfg()
    layer, Lw = C.device_layer(cfg)
    wr_priv = (Lw.wr_priv * 1e6).contiguous()
    # every token's hidden state aligned with a private router row
    x = Lw.wr_priv[torch.arange(cfg.tokens, device="cuda") % cfg.n_priv].to(torch.bfloat16).contiguous()
    adv = P.PolicyMaskedMoE(layer.desc, Lw.wr_pub, wr_priv, None, Lw.w13_pub, Lw.w2_pub,
                            Lw.w13_priv, Lw.w2_priv)
    req = W.alternating_requests(4, 80)
    words = O.compile_words(req.metas, req.lengths)
    d = run(adv, x, words, req)
    taus = np.array([O.decode_word(w) for w in words])
    assert np.all(d.idx[taus == 0] < cfg.n_pub)
    assert np.all(d.idx[taus == 1] >= cfg.n_pub)
    assert np.all(d.audit_rows[taus == 0] == 0) and d.violations == 0


def test_malformed_words_deny_on_device():
    cfg = small_cfg(tokens=64, requests=1)
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    A = O.ALLOW_WORD
    bad = [A ^ (1 << b) for b in range(32)] + [0, 1, 0xFFFFFFFF, A + 1, A - 1,
                                               int.from_bytes(A.to_bytes(4, "little"), "big")]
    words = np.array(bad + [A] * (64 - len(bad)), np.uint32)
    req = W.Requests([64], [None], ["malformed"])
    d = run(layer, x, words, req)
    assert np.all(d.allow[:len(bad)] == 0) and np.all(d.allow[len(bad):] == 1)
    assert np.all(d.idx[:len(bad)] < cfg.n_pub) and np.all(d.idx[len(bad):] >= cfg.n_pub)
    # NULL word array: every token denies
    d0 = run(layer, x, None, req)
    assert np.all(d0.allow == 0) and d0.total == 0


def test_allow_without_private_router_fails_closed():
    cfg = small_cfg()
    _, Lw = C.device_layer(cfg)
    layer = P.PolicyMaskedMoE(C.make_desc(cfg), Lw.wr_pub, None, None, Lw.w13_pub, Lw.w2_pub,
                              Lw.w13_priv, Lw.w2_priv)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(4, 80)
    words = O.compile_words(req.metas, req.lengths)
    d = run(layer, x, words, req)
    assert d.dev_status & 0x1
    assert np.all(d.allow == 0) and np.all(d.idx < cfg.n_pub) and d.total == 0


def test_private_rows_without_private_weights_not_executed():
    cfg = small_cfg()
    _, Lw = C.device_layer(cfg)
    layer = P.PolicyMaskedMoE(C.make_desc(cfg), Lw.wr_pub, Lw.wr_priv, None, Lw.w13_pub, Lw.w2_pub,
                              None, None)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(4, 80)
    words = O.compile_words(req.metas, req.lengths)
    d = run(layer, x, words, req)
    assert d.dev_status & 0x2
    assert d.total == 0 and d.audit_rows.sum() == 0
    taus = np.array([O.decode_word(w) for w in words])
    assert torch.all(d.out[torch.from_numpy(taus == 1)] == 0)   # zeroed private rows
    ref, _ = C.device_layer(cfg)
    d_ref = run(ref, x, words, req)
    deny = torch.from_numpy(taus == 0)
    assert torch.equal(d.out[deny], d_ref.out[deny])               # deny rows unaffected


# ----------------------------------------------------------------------------
# Grouped-GEMM edge cases on a given routing (dispatch -> expert_ffn -> combine)
# ----------------------------------------------------------------------------

def ffn_on_routing(cfg, idx, gates):
    """Run dispatch, expert FFN and combine on a given routing; returns out and counts."""
    layer, Lw = C.device_layer(cfg)
    T, k = idx.shape
    x = W.make_x(cfg, "cuda")
    b = layer.buffers(T)
    b.topk_idx.copy_(torch.from_numpy(idx.astype(np.int32).ravel()))
    b.topk_gate.copy_(torch.from_numpy(gates.astype(np.float32).ravel()))
    audit = layer.audit_buffers(T, 1)
    layer.dispatch(x, b)
    layer.expert_ffn(x, b, audit)
    layer.combine(x, b)
    torch.cuda.synchronize()
    return b.out.cpu(), b.expert_count.cpu().numpy(), audit.token_rows.cpu().numpy().view(np.uint32)


def oracle_on_routing(cfg, idx, gates, tokens):
    oi = C.oracle_inputs(cfg)
    n_pub = cfg.n_pub
    out = np.zeros((len(tokens), cfg.hidden))
    for i, t in enumerate(tokens):
        for j in range(idx.shape[1]):
            e = int(idx[t, j])
            w13 = oi.w13_pub[e] if e < n_pub else oi.w13_priv[e - n_pub]
            w2 = oi.w2_pub[e] if e < n_pub else oi.w2_priv[e - n_pub]
            out[i] += np.float64(gates[t, j]) * O.swiglu(oi.x[t:t + 1], w13, w2)[0]
    return out


def edge_case(cfg, idx, n_check=40, seed=0):
    gates = np.random.default_rng(seed).random(idx.shape).astype(np.float32)
    out, count, audit = ffn_on_routing(cfg, idx, gates)
    assert np.array_equal(count, np.bincount(idx.ravel(), minlength=cfg.n_experts))
    assert np.array_equal(audit.astype(np.int64), O.route_private_rows(idx, cfg.n_pub))
    rng = np.random.default_rng(seed + 1)
    toks = np.sort(rng.choice(idx.shape[0], size=min(n_check, idx.shape[0]), replace=False))
    ref = oracle_on_routing(cfg, idx, gates, toks)
    err = C.rel_l2(out.double().numpy()[toks], ref)
    print(f"edge case {cfg.tokens}x{cfg.hidden}: rel_l2={err:.3e}", flush=True)
    assert err <= C.RTOL_BF16
    return count


def test_expert_with_exactly_152_rows_and_empty_experts():
    cfg = small_cfg(tokens=400, n_pub=16, n_priv=8, top_k=2)
    rng = np.random.default_rng(7)
    idx = np.zeros((400, 2), np.int64)
    for t in range(400):
        if t < 152:
            idx[t] = [3, 20]                       # expert 3: exactly 152 rows
        else:
            idx[t] = np.sort(rng.choice([0, 1, 2, 5, 6, 17, 18], 2, replace=False))
    count = edge_case(cfg, idx)
    assert count[3] == 152 and (count == 0).sum() >= 8


def test_all_tokens_on_one_expert():
    cfg = small_cfg(tokens=1000, n_pub=8, n_priv=8, top_k=1)
    idx = np.full((1000, 1), 5, np.int64)
    count = edge_case(cfg, idx)
    assert count[5] == 1000


@pytest.mark.parametrize("shape", [
    dict(tokens=4096, hidden=256, inter=1024, n_pub=16, n_priv=8, top_k=4),   # 256x256 tiles, ~3 per block
    dict(tokens=2048, hidden=256, inter=512, n_pub=64, n_priv=32, top_k=2),   # 64x128 tiles, ~2.5 per block
], ids=["large_tiles", "small_tiles"])
def test_persistent_blocks_run_several_tiles(shape):
    cfg = small_cfg(requests=8, **shape)
    rng = np.random.default_rng(3)
    idx = np.stack([np.sort(rng.choice(cfg.n_experts, cfg.top_k, replace=False)) for _ in range(cfg.tokens)])
    edge_case(cfg, idx, n_check=32)
