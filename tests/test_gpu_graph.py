"""One layer pass (route, dispatch, expert FFN, combine, audit) captured as a HIP graph
replays the eager pass bit for bit.

The library's entry points launch kernels only (no allocation, no memset, no host
synchronisation; tile lists are built on the device), so a pass can be captured once and
replayed per batch. Every replay is checked against the eager pass, with eager work and
synchronisations between the replays, for the large-batch path (LDS-staged router, folded
dispatch count, 256x256 expert tiles) and the decode-sized path (register router,
single-workgroup dispatch, 64x128 tiles).
"""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C

pytestmark = pytest.mark.gpu

SHAPES = [
    dict(tokens=2113, requests=9, hidden=256, inter=128, n_pub=40, n_priv=12, top_k=4),
    dict(tokens=256, requests=8, hidden=256, inter=128, n_pub=32, n_priv=16, top_k=8),
]


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def one_pass(layer, x, words, req_off, audit, bufs, stream):
    layer.route(x, words, bufs, stream)
    layer.dispatch(x, bufs, stream)
    layer.expert_ffn(x, bufs, audit, stream)
    layer.combine(x, bufs, stream)
    layer.audit(x.shape[0], bufs, audit, req_off, stream)


def snapshot(bufs, audit):
    return {"out": bufs.out.cpu().clone(), "idx": bufs.topk_idx.cpu().clone(),
            "gate": bufs.topk_gate.cpu().clone(), "token_row": bufs.token_row.cpu().clone(),
            "rows": audit.token_rows.cpu().clone(), "req_rows": audit.req_rows.cpu().clone(),
            "total": int(audit.total.item()), "violations": int(audit.violations.item())}


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"T{s['tokens']}")
def test_layer_graph_replays_match_eager(shape):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    layer, _ = C.device_layer(cfg)
    x = W.make_x(cfg, "cuda")
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    req.lengths[-1] += cfg.tokens - sum(req.lengths)
    words = C.words_tensor(O.compile_words(req.metas, req.lengths))
    req_off = torch.tensor(req.offsets, device="cuda")
    audit = layer.audit_buffers(cfg.tokens, cfg.requests)
    bufs = layer.buffers(cfg.tokens)
    s = torch.cuda.current_stream()
    audit.zero_()
    one_pass(layer, x, words, req_off, audit, bufs, s)
    torch.cuda.synchronize()
    ref = snapshot(bufs, audit)
    # every allow token executes top_k private rows, no deny token any
    allow_tokens = sum(n for n, kind in zip(req.lengths, req.kinds) if kind == "allow")
    assert ref["total"] == cfg.top_k * allow_tokens and ref["violations"] == 0

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        one_pass(layer, x, words, req_off, audit, bufs, torch.cuda.current_stream())
    for rep in range(4):
        # eager work between replays: clear every output the pass writes or accumulates
        bufs.out.zero_()
        bufs.topk_idx.fill_(-1)
        bufs.token_row.fill_(-1)
        audit.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = snapshot(bufs, audit)
        log(f"T={cfg.tokens} replay {rep}: total={got['total']} violations={got['violations']}")
        for key in ("out", "idx", "gate", "token_row", "rows", "req_rows"):
            assert torch.equal(got[key], ref[key]), f"replay {rep}: {key} differs from the eager pass"
        assert got["total"] == ref["total"] and got["violations"] == ref["violations"]
