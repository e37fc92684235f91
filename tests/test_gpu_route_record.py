"""GPU route records (App. B.1 fifth step of the fail-closed procedure; App. B.2) against
the oracle's records of the same route, and reconciled against the independent
execution counters of the expert kernel: per request, the private slots in the route
log equal the private rows the expert kernel counted."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


CASES = [("tiny", {}, False), ("qwen", dict(tokens=512, requests=4, hidden=256, inter=128), False),
         ("qwen", dict(tokens=512, requests=4, hidden=256, inter=128), True),
         ("decode", {}, False), ("qwen", {}, False)]


@pytest.mark.parametrize("name,shape,soft", CASES,
                         ids=["tiny", "qwen-small", "qwen-small-soft", "decode", "qwen"])
def test_route_records_match_oracle_and_counters(name, shape, soft):
    cfg = W.scaled_config(W.get_config(name), **shape) if shape else W.get_config(name)
    log(f"route records {name} {shape} soft={soft}")
    layer, _ = C.device_layer(cfg, soft=soft)
    req = W.make_requests(cfg)
    words = O.compile_words(req.metas, req.lengths)
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda", dtype=torch.int32)
    d = C.run_device(layer, x, C.words_tensor(words), offs)
    b = layer.buffers(cfg.tokens)
    rec = layer.route_record(cfg.tokens, b, offs, layer=3)
    torch.cuda.synchronize()
    rec = rec.cpu().numpy().view(np.uint32)
    # the device's own route log, written out by the oracle's definition of a record
    ref = O.route_records(d.idx, d.allow, req.offsets, cfg.n_pub, 3)
    assert np.array_equal(rec, ref)
    # reconciliation with the expert kernel's counters (a separate code path)
    pop = np.array([bin(int(m)).count("1") for m in rec[:, 3]], np.int64)
    per_req = np.array([pop[a:e].sum() for a, e in zip(req.offsets[:-1], req.offsets[1:])])
    assert np.array_equal(per_req, d.req_rows.astype(np.int64))
    assert np.array_equal(pop, d.audit_rows)
    pool = rec[:, 0] >> 24
    if not soft:
        assert np.array_equal(pool, np.where(d.allow == 1, O.POOL_PRIVATE, O.POOL_PUBLIC))
    # and the oracle's own route gives the same records wherever the selections agree
    oi = C.oracle_inputs(cfg)
    rt = O.route(oi.x, oi.wr_pub, oi.wr_priv, oi.bias, words, cfg.top_k, cfg.gate_mode, soft=soft)
    same = np.all(d.idx == rt.idx, axis=1)
    ref_o = O.route_records(rt.idx, rt.allow, req.offsets, cfg.n_pub, 3)
    assert np.array_equal(rec[same], ref_o[same])
    assert np.all(same | rt.near_tie)
    log(f"  T={cfg.tokens} private slots={int(pop.sum())} mixed-pool tokens={int((pool == 2).sum())}")
