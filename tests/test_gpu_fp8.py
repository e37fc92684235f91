"""fp8 (e4m3) expert weights with power-of-two row scales: the expert FFN gives bitwise the
same layer output and audit as the bf16 kernel run on the dequantised weights (the scales
are exact in fp32, every e4m3 value is a bf16 value), and matches the oracle on those
weights; denied requests never reach private fp8 weights (NULL private tensors)."""
import sys

import numpy as np
import pytest
import torch

import paper_2608_06690_amd as P
import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def fp8_layer(cfg, device="cuda"):
    """Device layer whose bf16 weights are the dequantised fp8 weights, plus the fp8 set."""
    Lw = W.make_layer(cfg, 0, device)
    parts = {}
    for name in ("w13_pub", "w2_pub", "w13_priv", "w2_priv"):
        q, sc, deq = W.quantize_fp8_rows(getattr(Lw, name))
        parts[name] = (q, sc)
        getattr(Lw, name).copy_(deq.to(torch.bfloat16))
    layer = P.PolicyMaskedMoE(C.make_desc(cfg), Lw.wr_pub, Lw.wr_priv, Lw.bias, Lw.w13_pub,
                              Lw.w2_pub, Lw.w13_priv, Lw.w2_priv)
    fp8 = (parts["w13_pub"][0], parts["w2_pub"][0], parts["w13_priv"][0], parts["w2_priv"][0],
           parts["w13_pub"][1], parts["w2_pub"][1], parts["w13_priv"][1], parts["w2_priv"][1])
    return layer, Lw, fp8


CASES = [("qwen", dict(tokens=512, requests=4, hidden=256, inter=128, n_pub=16, n_priv=8, top_k=4)),
         ("qwen", dict(tokens=4096, requests=8, hidden=256, inter=256, n_pub=16, n_priv=8, top_k=4)),
         ("qwen", {}), ("decode", {})]


@pytest.mark.parametrize("name,shape", CASES, ids=["small-tiles", "large-tiles", "qwen", "decode"])
def test_fp8_weights_equal_bf16_on_dequantised_weights(name, shape):
    cfg = W.scaled_config(W.get_config(name), **shape) if shape else W.get_config(name)
    log(f"fp8 weights {name} {shape}")
    layer, Lw, fp8 = fp8_layer(cfg)
    req = W.make_requests(cfg)
    words = C.words_tensor(O.compile_words(req.metas, req.lengths))
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda", dtype=torch.int32)
    a16 = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
    out16 = layer.forward(x, words, a16, offs).out.clone()
    a8 = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
    b8 = layer.forward_fp8(x, words, fp8, a8, offs)
    torch.cuda.synchronize()
    assert torch.equal(out16, b8.out)
    assert torch.equal(a16.token_rows, a8.token_rows) and torch.equal(a16.req_rows, a8.req_rows)
    assert int(b8.dev_status.item()) == 0


def test_fp8_layer_matches_oracle():
    cfg = W.scaled_config(W.get_config("qwen"), tokens=300, requests=3, hidden=256, inter=128,
                          n_pub=16, n_priv=8, top_k=4)
    layer, Lw, fp8 = fp8_layer(cfg)
    req = W.make_requests(cfg)
    words_l = O.compile_words(req.metas, req.lengths)
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda", dtype=torch.int32)
    a8 = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
    b8 = layer.forward_fp8(x, C.words_tensor(words_l), fp8, a8, offs)
    torch.cuda.synchronize()
    n = cfg.n_pub
    ref = O.layer_forward(C.np64(x), C.np64(Lw.wr_pub), C.np64(Lw.wr_priv), None,
                          C.np64(Lw.w13_pub), C.np64(Lw.w2_pub), C.np64(Lw.w13_priv),
                          C.np64(Lw.w2_priv), words_l, cfg.top_k, cfg.gate_mode)
    idx = b8.topk_idx.view(cfg.tokens, cfg.top_k).cpu().numpy()
    same = np.all(idx == ref.route.idx, axis=1)
    assert np.all(same | ref.route.near_tie)
    err = C.rel_l2(b8.out.double().cpu().numpy()[same], ref.out[same])
    log(f"  fp8 layer vs oracle rel_l2 {err:.2e}")
    assert err <= C.RTOL_BF16
    assert np.array_equal(a8.token_rows.cpu().numpy().view(np.uint32), ref.hook.rows)
    del n


def test_fp8_all_deny_with_null_private_weights():
    cfg = W.scaled_config(W.get_config("qwen"), tokens=512, requests=4, hidden=256, inter=128,
                          n_pub=16, n_priv=8, top_k=4)
    layer, Lw, fp8 = fp8_layer(cfg)
    T = cfg.tokens
    x = W.make_x(cfg, "cuda")
    deny = torch.zeros(T, dtype=torch.int32, device="cuda")
    offs = torch.tensor([0, T], device="cuda", dtype=torch.int32)
    a1 = layer.audit_buffers(T, 1)
    out1 = layer.forward_fp8(x, deny, fp8, a1, offs).out.clone()
    nulled = fp8[:2] + (None, None) + fp8[4:6] + (None, None)
    a2 = layer.audit_buffers(T, 1)
    b2 = layer.forward_fp8(x, deny, nulled, a2, offs)
    torch.cuda.synchronize()
    assert torch.equal(out1, b2.out)
    assert int(a2.total.item()) == 0 and int(b2.dev_status.item()) == 0
