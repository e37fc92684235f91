"""GPU parity of the private-only backward (G2 of Sec. 2.2; Sec. 3.2) against the CPU
oracle: input gradient, private expert weight gradients and private router-row
gradients, element by element at small sizes and on sampled private experts at the
Qwen-shaped layer's full size. Also: bitwise determinism, public weights untouched,
the soft-routing control feeding private gradients from deny rows."""
import sys

import numpy as np
import pytest
import torch

import paper_2608_06690_amd as P
import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C

pytestmark = pytest.mark.gpu

RTOL = C.RTOL_BF16


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def forward_backward(cfg, soft=False, dout=None, saved=True, transposed=True):
    """Training forward (keeps the gate and up projections) then the backward, which
    uses them (saved=True) or recomputes them, with transposed weight copies on the
    grouped NT GEMM (transposed=True) or the transposing GEMM."""
    layer, Lw = C.device_layer(cfg, soft=soft)
    req = W.make_requests(cfg)
    words = O.compile_words(req.metas, req.lengths)
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda")
    audit = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
    b = layer.forward(x, C.words_tensor(words), audit, offs, train=True)
    g = layer.backward(x, dout.to("cuda"), b, use_saved=saved, transposed=transposed)
    torch.cuda.synchronize()
    return layer, Lw, b, g, words, x


def oracle_route_and_dout(cfg, oi, words, soft=False):
    """Oracle route and the upstream gradient with near-tie tokens zeroed (their
    selection may legitimately differ between fp32 implementations)."""
    rt = O.route(oi.x, oi.wr_pub, oi.wr_priv, oi.bias, words, cfg.top_k, cfg.gate_mode, soft=soft)
    dout = W.make_dout(cfg)
    dout[torch.from_numpy(rt.near_tie)] = 0
    return rt, dout


def stacked(bank, n):
    return np.stack([bank[i] for i in range(n)]) if n else None


SMALL = [
    dict(tokens=512, requests=4, hidden=512, inter=256, n_pub=32, n_priv=8, top_k=4),
    dict(tokens=300, requests=3, hidden=256, inter=128, n_pub=16, n_priv=8, top_k=8),
    dict(tokens=1024, requests=8, hidden=256, inter=384, n_pub=8, n_priv=4, top_k=2),
]


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: f"T{s['tokens']}_H{s['hidden']}_I{s['inter']}_k{s['top_k']}")
@pytest.mark.parametrize("soft,saved,transposed", [(False, True, True), (False, False, True),
                                                   (False, True, False), (True, True, True)],
                         ids=["masked", "masked-recompute", "masked-transposing", "soft"])
def test_backward_matches_oracle(shape, soft, saved, transposed):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    log(f"backward {shape} soft={soft} saved={saved} transposed={transposed}")
    oi = C.oracle_inputs(cfg)
    req = W.make_requests(cfg)
    words = O.compile_words(req.metas, req.lengths)
    rt, dout = oracle_route_and_dout(cfg, oi, words, soft)
    layer, Lw, b, g, _, _ = forward_backward(cfg, soft, dout, saved, transposed)
    idx = b.topk_idx.view(cfg.tokens, cfg.top_k).cpu().numpy()
    keep = ~rt.near_tie
    assert np.array_equal(idx[keep], rt.idx[keep])
    ref = O.layer_backward(oi.x, oi.wr_pub, oi.wr_priv, oi.bias, stacked(oi.w13_pub, cfg.n_pub),
                           stacked(oi.w2_pub, cfg.n_pub), stacked(oi.w13_priv, cfg.n_priv),
                           stacked(oi.w2_priv, cfg.n_priv), words, cfg.top_k, C.np64(dout),
                           cfg.gate_mode, soft=soft)
    errs = {
        "dx": C.rel_l2(g.dx.cpu().numpy(), ref.dx),
        "dw13": C.rel_l2(g.dw13_priv.cpu().numpy(), ref.dw13_priv),
        "dw2": C.rel_l2(g.dw2_priv.cpu().numpy(), ref.dw2_priv),
        "dwr": C.rel_l2(g.dwr_priv.cpu().numpy(), ref.dwr_priv),
    }
    log(f"  rel_l2 {errs}  grad_rows {g.grad_rows.cpu().numpy().tolist()}")
    for k_, v in errs.items():
        assert v <= RTOL, (k_, v)
    rows = g.grad_rows.cpu().numpy().astype(np.int64)
    assert np.array_equal(rows, b.expert_count[cfg.n_pub:].cpu().numpy())
    if np.array_equal(idx, rt.idx):
        assert np.array_equal(rows, ref.grad_rows)
    # private experts without rows get exactly zero gradient
    empty = rows == 0
    assert not g.dw13_priv[torch.from_numpy(empty).cuda()].any()


def test_training_forward_output_equals_inference_forward():
    """The forward that keeps the projections for the backward computes the same layer
    output and audit, bit for bit."""
    cfg = W.scaled_config(W.get_config("qwen"), **SMALL[0])
    layer, Lw = C.device_layer(cfg)
    req = W.make_requests(cfg)
    words = C.words_tensor(O.compile_words(req.metas, req.lengths))
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda")
    a1 = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
    out1 = layer.forward(x, words, a1, offs).out.clone()
    a2 = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
    b2 = layer.forward(x, words, a2, offs, train=True)
    torch.cuda.synchronize()
    assert torch.equal(out1, b2.out)
    assert torch.equal(a1.token_rows, a2.token_rows) and torch.equal(a1.total, a2.total)
    # the saved projections reproduce the forward's h = silu(a) * b on a sample of rows
    ab = b2.ab[:64].double().cpu()
    I = cfg.inter
    h = torch.nn.functional.silu(ab[:, :I]) * ab[:, I:]
    oi = C.oracle_inputs(cfg)
    rows = b2.row_token[:64].cpu().numpy()
    e0 = 0  # the first rows belong to the lowest expert with rows
    while int(b2.expert_count[e0]) == 0:
        e0 += 1
    n0 = min(64, int(b2.expert_count[e0]))
    w13 = oi.w13_pub[e0] if e0 < cfg.n_pub else oi.w13_priv[e0 - cfg.n_pub]
    ref = oi.x[rows[:n0]] @ np.asarray(w13, np.float64).T
    assert C.rel_l2(ab[:n0].numpy(), ref) <= 1e-4
    assert torch.isfinite(h).all()


DS_SMALL = dict(tokens=400, requests=4, hidden=256, inter=128, n_pub=16, n_priv=8, top_k=4,
                n_shared=2, shared_inter=128)


@pytest.mark.parametrize("soft", [False, True], ids=["masked", "soft"])
def test_backward_pool_softmax_and_shared_experts(soft):
    """DeepSeek-shaped layer: softmax over the whole pool (the router gradient is dense
    over the pool), a logit bias, and two always-on shared experts (frozen, input gradient
    only)."""
    cfg = W.scaled_config(W.get_config("deepseek"), **DS_SMALL)
    log(f"backward deepseek-shaped {DS_SMALL} soft={soft}")
    oi = C.oracle_inputs(cfg)
    req = W.make_requests(cfg)
    words = O.compile_words(req.metas, req.lengths)
    rt, dout = oracle_route_and_dout(cfg, oi, words, soft)
    layer, Lw, b, g, _, _ = forward_backward(cfg, soft, dout)
    idx = b.topk_idx.view(cfg.tokens, cfg.top_k).cpu().numpy()
    keep = ~rt.near_tie
    assert np.array_equal(idx[keep], rt.idx[keep])
    ref = O.layer_backward(oi.x, oi.wr_pub, oi.wr_priv, oi.bias, stacked(oi.w13_pub, cfg.n_pub),
                           stacked(oi.w2_pub, cfg.n_pub), stacked(oi.w13_priv, cfg.n_priv),
                           stacked(oi.w2_priv, cfg.n_priv), words, cfg.top_k, C.np64(dout),
                           cfg.gate_mode, oi.w13_sh, oi.w2_sh, soft=soft)
    errs = {
        "dx": C.rel_l2(g.dx.cpu().numpy(), ref.dx),
        "dw13": C.rel_l2(g.dw13_priv.cpu().numpy(), ref.dw13_priv),
        "dw2": C.rel_l2(g.dw2_priv.cpu().numpy(), ref.dw2_priv),
        "dwr": C.rel_l2(g.dwr_priv.cpu().numpy(), ref.dwr_priv),
    }
    log(f"  rel_l2 {errs}")
    for k_, v in errs.items():
        assert v <= RTOL, (k_, v)
    # with pool gates every allowed token trains every private router row
    if not soft:
        assert np.all(np.abs(g.dwr_priv.cpu().numpy()).sum(axis=1) > 0)


def test_backward_deepseek_full_size_sampled_experts():
    """DeepSeek-shaped layer at full size (8192 tokens, 2 shared + 64 + 16 experts, top-6,
    pool softmax, bias): the weight gradients of two private experts against the oracle's
    SwiGLU backward on their rows."""
    cfg = W.get_config("deepseek")
    log("backward deepseek full size")
    oi = C.oracle_inputs(cfg)
    req = W.make_requests(cfg)
    words = O.compile_words(req.metas, req.lengths)
    rt, dout = oracle_route_and_dout(cfg, oi, words)
    layer, Lw, b, g, _, _ = forward_backward(cfg, False, dout)
    idx = b.topk_idx.view(cfg.tokens, cfg.top_k).cpu().numpy()
    keep = ~rt.near_tie
    assert np.array_equal(idx[keep], rt.idx[keep])
    dout64 = C.np64(dout)
    for p in (0, cfg.n_priv - 1):
        e = cfg.n_pub + p
        hit = rt.idx == e
        rows = np.nonzero(hit.any(axis=1))[0]
        slot = np.argmax(hit[rows], axis=1)
        gate = rt.gate[rows, slot].astype(np.float64)
        _, dW13, dW2 = O.swiglu_backward(oi.x[rows], oi.w13_priv[p], oi.w2_priv[p],
                                         gate[:, None] * dout64[rows])
        e13 = C.rel_l2(g.dw13_priv[p].cpu().numpy(), dW13)
        e2 = C.rel_l2(g.dw2_priv[p].cpu().numpy(), dW2)
        log(f"  private expert {p}: {len(rows)} rows, rel_l2 dw13 {e13:.2e} dw2 {e2:.2e}")
        assert e13 <= RTOL and e2 <= RTOL


def test_backward_deterministic_and_public_weights_untouched():
    cfg = W.scaled_config(W.get_config("qwen"), **SMALL[0])
    dout = W.make_dout(cfg)
    layer, Lw, b, g1, words, x = forward_backward(cfg, False, dout)
    fp_pub = P.fingerprint_tensors(Lw.wr_pub, Lw.w13_pub, Lw.w2_pub)
    snap = [t.clone() for t in (g1.dx, g1.dw13_priv, g1.dw2_priv, g1.dwr_priv)]
    g2 = layer.backward(x, dout.cuda(), b)
    torch.cuda.synchronize()
    for a_, b_ in zip(snap, (g2.dx, g2.dw13_priv, g2.dw2_priv, g2.dwr_priv)):
        assert torch.equal(a_, b_)
    assert torch.equal(P.fingerprint_tensors(Lw.wr_pub, Lw.w13_pub, Lw.w2_pub), fp_pub)


def test_backward_all_deny_forms_zero_private_gradient():
    cfg = W.scaled_config(W.get_config("qwen"), **SMALL[0])
    layer, Lw = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    T = cfg.tokens
    words = torch.zeros(T, dtype=torch.int32, device="cuda")
    audit = layer.audit_buffers(T, 1)
    b = layer.forward(x, words, audit, torch.tensor([0, T], device="cuda"))
    g = layer.grad_buffers(T)
    for t in (g.dw13_priv, g.dw2_priv, g.dwr_priv):
        t.fill_(float("nan"))
    layer.backward(x, W.make_dout(cfg, device="cuda"), b, g)
    torch.cuda.synchronize()
    assert not g.grad_rows.any()
    for t in (g.dw13_priv, g.dw2_priv, g.dwr_priv):
        assert not t.isnan().any() and not t.any()
    assert g.dx.abs().sum() > 0


def test_backward_qwen_full_size_sampled_experts():
    """Qwen-shaped layer (4096 tokens, 128 + 32 experts, top-8): the weight gradients of
    two private experts against the oracle's SwiGLU backward on their rows, and the row
    counts of every private expert against the oracle's route."""
    cfg = W.get_config("qwen")
    log("backward qwen full size")
    oi = C.oracle_inputs(cfg)
    req = W.make_requests(cfg)
    words = O.compile_words(req.metas, req.lengths)
    rt, dout = oracle_route_and_dout(cfg, oi, words)
    layer, Lw, b, g, _, _ = forward_backward(cfg, False, dout)
    idx = b.topk_idx.view(cfg.tokens, cfg.top_k).cpu().numpy()
    keep = ~rt.near_tie
    assert np.array_equal(idx[keep], rt.idx[keep])
    dout64 = C.np64(dout)
    for p in (0, cfg.n_priv - 1):
        e = cfg.n_pub + p
        hit = rt.idx == e
        rows = np.nonzero(hit.any(axis=1))[0]
        slot = np.argmax(hit[rows], axis=1)
        gate = rt.gate[rows, slot].astype(np.float64)
        _, dW13, dW2 = O.swiglu_backward(oi.x[rows], oi.w13_priv[p], oi.w2_priv[p],
                                         gate[:, None] * dout64[rows])
        e13 = C.rel_l2(g.dw13_priv[p].cpu().numpy(), dW13)
        e2 = C.rel_l2(g.dw2_priv[p].cpu().numpy(), dW2)
        log(f"  private expert {p}: {len(rows)} rows, rel_l2 dw13 {e13:.2e} dw2 {e2:.2e}")
        assert e13 <= RTOL and e2 <= RTOL
    if np.array_equal(idx, rt.idx):
        ref_rows = np.array([(rt.idx == cfg.n_pub + p).any(axis=1).sum() for p in range(cfg.n_priv)])
        assert np.array_equal(g.grad_rows.cpu().numpy(), ref_rows)


@pytest.mark.parametrize("n,rows,cols", [(1, 64, 64), (3, 128, 192), (5, 2048, 768)])
def test_transpose_experts(n, rows, cols):
    g = torch.Generator(device="cuda").manual_seed(rows + cols)
    src = torch.randn(n, rows, cols, device="cuda", generator=g).to(torch.bfloat16)
    dst = torch.empty(n, cols, rows, device="cuda", dtype=torch.bfloat16)
    P.pmpe_transpose_experts(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(dst.cpu(), src.cpu().transpose(1, 2))


@pytest.mark.parametrize("transposed", [True, False], ids=["nt", "transposing"])
def test_backward_152_row_expert_and_empty_experts(transposed):
    """The two cases the paper's FP8 preflight failed on: a reduction over an expert with
    exactly 152 rows (not a multiple of the 64-row K step) and experts with no rows (their
    gradients must be exactly zero). Planted route; private weight gradients against the
    oracle's SwiGLU backward on each expert's rows."""
    cfg = W.scaled_config(W.get_config("qwen"), tokens=400, requests=1, hidden=256, inter=128,
                          n_pub=16, n_priv=8, top_k=2)
    T, k = cfg.tokens, cfg.top_k
    rng = np.random.default_rng(7)
    idx = np.zeros((T, k), np.int64)
    for t in range(T):
        if t < 152:
            idx[t] = [3, 20]                       # private expert 4 (id 20): exactly 152 rows
        else:
            idx[t] = np.sort(rng.choice([0, 1, 2, 5, 6, 17, 18], 2, replace=False))
    gates = rng.random((T, k)).astype(np.float32)
    layer, Lw = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    b = layer.buffers(T)
    b.topk_idx.copy_(torch.from_numpy(idx.astype(np.int32).ravel()))
    b.topk_gate.copy_(torch.from_numpy(gates.ravel()))
    audit = layer.audit_buffers(T, 1)
    layer.dispatch(x, b)
    layer.expert_ffn(x, b, audit, train=True)
    dout = W.make_dout(cfg)
    g = layer.backward(x, dout.cuda(), b, transposed=transposed)
    torch.cuda.synchronize()
    count = b.expert_count.cpu().numpy()
    assert count[20] == 152
    oi = C.oracle_inputs(cfg)
    d64 = C.np64(dout)
    dw13 = g.dw13_priv.cpu().numpy()
    dw2 = g.dw2_priv.cpu().numpy()
    for p in range(cfg.n_priv):
        e = cfg.n_pub + p
        hit = idx == e
        rows = np.nonzero(hit.any(axis=1))[0]
        if len(rows) == 0:
            assert not dw13[p].any() and not dw2[p].any()
            assert not g.dwr_priv[p].any()
            continue
        slot = np.argmax(hit[rows], axis=1)
        gt = gates[rows, slot].astype(np.float64)
        _, r13, r2 = O.swiglu_backward(oi.x[rows], oi.w13_priv[p], oi.w2_priv[p], gt[:, None] * d64[rows])
        assert C.rel_l2(dw13[p], r13) <= RTOL and C.rel_l2(dw2[p], r2) <= RTOL, p
    assert np.isfinite(g.dx.cpu().numpy()).all()
    assert np.array_equal(g.grad_rows.cpu().numpy().astype(np.int64), count[cfg.n_pub:])
