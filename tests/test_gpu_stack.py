"""48-layer stack of Qwen3-30B-A3B-shaped policy-masked MoE layers (attention replaced by
identity): 16384 prefill tokens in 32 requests of 512, passes all allow / all deny /
all allow over the same inputs, h_{l+1} = bf16(h_l + MoE_l(h_l)), each layer with its
own seeded weights (48 x 1.51 GB on the device).

Checks: the private-row audit summed over all layers equals its closed form (allow:
48 * 16384 * 8 rows, 48 * 512 * 8 per request; deny: 0) and the audit is per token
exactly the route log's count; the recovery pass reproduces the first pass bitwise;
routing of layers 0, 23 and 47 equals the oracle's on the GPU's own layer input
(teacher-forced), and on layers 0 and 47 every agreeing token's layer output and every
one of its expert output rows match the oracle within the per-row bars (allow and deny
passes).
"""
import types
import sys

import numpy as np
import pytest
import torch

import paper_2608_06690_amd as P
import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C

pytestmark = pytest.mark.gpu

CHECK_LAYERS = (0, 23, 47)
FULL_LAYERS = (0, 47)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.timeout(900)
def test_stack_allow_deny_allow():
    cfg = W.get_config("stack")
    L, T, k = cfg.layers, cfg.tokens, cfg.top_k
    dev = "cuda"
    desc = C.make_desc(cfg)
    log(f"stack: generating {L} layers on the device")
    layers = []
    for ell in range(L):
        Lw = W.make_layer(cfg, ell, dev)
        layers.append(P.PolicyMaskedMoE(desc, Lw.wr_pub, Lw.wr_priv, Lw.bias, Lw.w13_pub, Lw.w2_pub,
                                        Lw.w13_priv, Lw.w2_priv))
    torch.cuda.synchronize()
    x0 = W.make_x(cfg, dev)
    bufs = layers[0].buffers(T)
    passes = []
    for p in range(3):
        req = W.make_requests(cfg, p)
        words = P.token_policy_words(req.metas, req.lengths, dev)
        req_off = P.request_offsets(req.lengths, dev)
        audit = layers[0].audit_buffers(T, cfg.requests)
        h = x0.clone()
        saved = {}
        route_rho = np.zeros(T, np.int64)
        for ell, layer in enumerate(layers):
            layer.route(h, words, bufs)
            layer.dispatch(h, bufs)
            layer.expert_ffn(h, bufs, audit)
            layer.combine(h, bufs)
            if ell in CHECK_LAYERS:
                rows = None
                if ell in FULL_LAYERS and p < 2:
                    rows = (bufs.token_row.view(T, k).cpu().numpy().astype(np.int64), bufs.y_perm.cpu().clone())
                saved[ell] = (h.cpu().clone(), bufs.topk_idx.view(T, k).cpu().numpy().astype(np.int64),
                              bufs.out.cpu().clone(), rows)
            route_rho += (bufs.topk_idx.view(T, k).cpu().numpy() >= cfg.n_pub).sum(1)
            h = (h.float() + bufs.out.float()).to(torch.bfloat16)
        layers[0].audit(T, bufs, audit, req_off)
        torch.cuda.synchronize()
        rows = audit.token_rows.cpu().numpy().view(np.uint32).astype(np.int64)
        tot = int(audit.total.item())
        req_rows = audit.req_rows.cpu().numpy()
        log(f"stack pass {p} ({req.kinds[0]}): private rows {tot}, violations {int(audit.violations.item())}")
        assert np.array_equal(rows, route_rho)          # executed rows == routed rows, per token
        if req.kinds[0] == "allow":
            assert tot == L * T * k == 6_291_456
            assert np.all(req_rows == L * cfg.req_len * k)
        else:
            assert tot == 0 and np.all(rows == 0)
        assert int(audit.violations.item()) == 0
        passes.append((h.cpu(), saved))
    # recovery reproduces the first allow pass bitwise
    assert torch.equal(passes[0][0], passes[2][0])
    for ell in CHECK_LAYERS:
        assert np.array_equal(passes[0][1][ell][1], passes[2][1][ell][1])
        assert torch.equal(passes[0][1][ell][2], passes[2][1][ell][2])
    del passes[2]
    # oracle: routing of the checked layers (teacher-forced); on layers 0 and 47 every
    # agreeing token's output and expert rows
    for p in (0, 1):
        req = W.make_requests(cfg, p)
        words_np = O.compile_words(req.metas, req.lengths)
        for ell in CHECK_LAYERS:
            h_in, idx, out, rows = passes[p][1][ell]
            wr_pub, wr_priv, _ = W.make_router(cfg, ell, "cpu")
            rt = O.route(C.np64(h_in), C.np64(wr_pub), C.np64(wr_priv), None, words_np, k)
            nt = rt.near_tie
            same = np.all(idx == rt.idx, axis=1)
            assert np.all(same | nt), f"layer {ell}: routing differs off near ties"
            log(f"stack pass {p} layer {ell}: routes agree on {int(same.sum())}/{T} (near ties {int(nt.sum())})")
            if ell in FULL_LAYERS:
                oi = C.oracle_inputs(cfg, ell, h_in)
                ref = O.layer_forward(oi.x, oi.wr_pub, oi.wr_priv, None, oi.w13_pub, oi.w2_pub,
                                      oi.w13_priv, oi.w2_priv, words_np, k, cfg.gate_mode)
                token_row, y_perm = rows
                d = types.SimpleNamespace(idx=idx, out=out, token_row=token_row, y_perm=y_perm)
                C.check_rows(cfg, d, ref, np.nonzero(same)[0], tag=f"stack pass {p} layer {ell}")
                del ref, oi
    del layers, bufs
    torch.cuda.empty_cache()
