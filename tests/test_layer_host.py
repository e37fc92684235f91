"""Host-side bookkeeping of the layer object (no GPU): the transposed copies of the
private expert weights that the backward uses are made once, kept across backward
calls, and remade after an optimizer step, an in-place torch update or new tensors."""
import torch

import paper_2608_06690_amd as P
from paper_2608_06690_amd import _native as N
from paper_2608_06690_amd import layer as Lmod


def make_layer():
    H, I, npub, npriv = 16, 8, 3, 2
    desc = P.make_desc(H, 64, npub, npriv, 2)
    w = lambda *s: torch.randn(*s)  # noqa: E731
    return Lmod.PolicyMaskedMoE(desc, w(npub, H), w(npriv, H), None, w(npub, 2 * I, H), w(npub, H, I),
                                w(npriv, 2 * I, H), w(npriv, H, I))


def test_private_transposes_made_once_and_after_changes(monkeypatch):
    calls = []

    def transpose(src, dst, stream=None):
        calls.append(src.data_ptr())
        dst.copy_(src.transpose(1, 2))

    monkeypatch.setattr(N, "pmpe_transpose_experts", transpose)
    monkeypatch.setattr(N, "pmpe_adamw", lambda *a, **k: None)
    lay = make_layer()
    wt = lay.transposed_weights()
    assert len(calls) == 4  # public W2, W13 once; private W2, W13
    assert torch.equal(wt[2], lay.w2_priv.transpose(1, 2)) and torch.equal(wt[3], lay.w13_priv.transpose(1, 2))
    calls.clear()
    lay.transposed_weights()
    lay.transposed_weights()
    assert calls == []  # kept across backward calls
    # an in-place torch update of a private weight is seen through its version counter
    lay.w2_priv.mul_(2.0)
    wt = lay.transposed_weights()
    assert len(calls) == 2 and torch.equal(wt[2], lay.w2_priv.transpose(1, 2))
    calls.clear()
    # the optimizer step remakes them once (its kernel writes through a raw pointer)
    g = Lmod.GradBuffers(None, torch.zeros_like(lay.w13_priv), torch.zeros_like(lay.w2_priv),
                         torch.zeros_like(lay.wr_priv), None, None)
    opt = P.PrivateAdamW(lay)
    opt.step(g)
    assert len(calls) == 2
    calls.clear()
    lay.transposed_weights()
    assert calls == []
    # new private tensors
    lay.w13_priv = torch.randn_like(lay.w13_priv)
    wt = lay.transposed_weights()
    assert len(calls) == 2 and torch.equal(wt[3], lay.w13_priv.transpose(1, 2))
    # the public copies are never remade
    assert all(c not in calls for c in (lay.w2_pub.data_ptr(), lay.w13_pub.data_ptr()))
