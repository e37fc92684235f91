"""The private-only training step on the GPU: AdamW over private tensors against the
oracle (fp32 and bf16-with-master parameters, ragged lengths), and one whole step -
training forward, backward, optimizer - that changes the private parameters, leaves the
public fingerprint unchanged (G2 of Sec. 2.2; Sec. 3.2) and lowers the first-order loss."""
import sys

import numpy as np
import pytest
import torch

import paper_2608_06690_amd as P
import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C

pytestmark = pytest.mark.gpu

HP = dict(lr=1e-2, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("n", [1, 3, 4, 1021, 65536 + 5])
@pytest.mark.parametrize("bf16", [False, True])
def test_adamw_matches_oracle(n, bf16):
    log(f"adamw n={n} bf16={bf16}")
    g = torch.Generator().manual_seed(n)
    p0 = torch.randn(n, generator=g, dtype=torch.float64)
    if bf16:
        p0 = p0.to(torch.bfloat16).double()   # a representable starting point
    param = p0.to(torch.bfloat16 if bf16 else torch.float32).cuda()
    master = p0.float().cuda() if bf16 else None
    m = torch.zeros(n, dtype=torch.float32, device="cuda")
    v = torch.zeros_like(m)
    ref_p, ref_m, ref_v = p0.numpy(), np.zeros(n), np.zeros(n)
    for step in (1, 2, 3):
        grad = torch.randn(n, generator=g).float()
        P.pmpe_adamw(param, master, grad.cuda(), m, v, step, HP["lr"], HP["beta1"], HP["beta2"],
                     HP["eps"], HP["weight_decay"])
        ref_p, ref_m, ref_v = O.adamw_step(ref_p, grad.double().numpy(), ref_m, ref_v, step, **HP)
    torch.cuda.synchronize()
    got = (master if bf16 else param).double().cpu().numpy()
    assert C.rel_l2(got, ref_p) <= 1e-6
    assert C.rel_l2(m.double().cpu().numpy(), ref_m) <= 1e-6
    assert C.rel_l2(v.double().cpu().numpy(), ref_v) <= 1e-6
    if bf16:
        # the bf16 weight is the rounding of the master copy
        assert torch.equal(param, master.to(torch.bfloat16))
        assert C.rel_l2(param.double().cpu().numpy(), ref_p) <= C.RTOL_BF16


def test_private_training_step_keeps_public_fingerprint():
    cfg = W.scaled_config(W.get_config("qwen"), tokens=512, requests=4, hidden=256, inter=128,
                          n_pub=16, n_priv=8, top_k=4)
    layer, Lw = C.device_layer(cfg)
    req = W.make_requests(cfg)
    words = C.words_tensor(O.compile_words(req.metas, req.lengths))
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda", dtype=torch.int32)
    dout = W.make_dout(cfg, device="cuda")
    pub = [Lw.wr_pub, Lw.w13_pub, Lw.w2_pub]
    fp_pub = P.fingerprint_tensors(*pub)
    priv_before = [t.clone() for t in (Lw.wr_priv, Lw.w13_priv, Lw.w2_priv)]
    opt = P.PrivateAdamW(layer, lr=1e-3)

    def loss():
        a = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
        b = layer.forward(x, words, a, offs)
        return float((b.out.float() * dout.float()).sum())

    l0 = loss()
    for _ in range(2):
        a = layer.audit_buffers(cfg.tokens, len(req.offsets) - 1)
        b = layer.forward(x, words, a, offs, train=True)
        g = layer.backward(x, dout, b)
        opt.step(g)
    torch.cuda.synchronize()
    l1 = loss()
    log(f"  first-order loss {l0:.4f} -> {l1:.4f}")
    assert l1 < l0
    assert torch.equal(P.fingerprint_tensors(*pub), fp_pub)
    for before, now in zip(priv_before, (Lw.wr_priv, Lw.w13_priv, Lw.w2_priv)):
        assert not torch.equal(before, now)


def test_backward_after_step_uses_the_updated_private_weights():
    """The transposed private weights are kept between backward calls and remade by the
    optimizer step: the backward after a step equals the backward of a fresh layer object
    (which transposes the current weights itself), bitwise, and so does the backward after
    an in-place torch update of a private weight."""
    cfg = W.scaled_config(W.get_config("qwen"), tokens=512, requests=4, hidden=256, inter=128,
                          n_pub=16, n_priv=8, top_k=4)
    layer, Lw = C.device_layer(cfg)
    req = W.make_requests(cfg)
    words = C.words_tensor(O.compile_words(req.metas, req.lengths))
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda", dtype=torch.int32)
    dout = W.make_dout(cfg, device="cuda")
    opt = P.PrivateAdamW(layer, lr=1e-3)

    def grads(lay):
        a = lay.audit_buffers(cfg.tokens, len(req.offsets) - 1)
        b = lay.forward(x, words, a, offs, train=True)
        g = lay.backward(x, dout, b)
        torch.cuda.synchronize()
        return g, [t.clone() for t in (g.dx, g.dw13_priv, g.dw2_priv, g.dwr_priv)]

    def fresh():
        return P.PolicyMaskedMoE(layer.desc, Lw.wr_pub, Lw.wr_priv, Lw.bias, Lw.w13_pub, Lw.w2_pub,
                                 Lw.w13_priv, Lw.w2_priv)

    g, _ = grads(layer)
    opt.step(g)
    _, after_step = grads(layer)
    _, ref = grads(fresh())
    for a, r in zip(after_step, ref):
        assert torch.equal(a, r)
    log("  backward after an optimizer step equals a fresh layer's")
    with torch.no_grad():
        Lw.w2_priv.mul_(0.5)
    _, after_edit = grads(layer)
    _, ref = grads(fresh())
    for a, r in zip(after_edit, ref):
        assert torch.equal(a, r)
    # dW13 and dx flow through W2 (dh = W2^T u); dW2 = u h^T does not
    assert not torch.equal(after_edit[1], after_step[1]) and not torch.equal(after_edit[0], after_step[0])
