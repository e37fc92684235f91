"""GPU parity of the soft-routing control arm (Sec. 4.2, third row of the control
matrix; App. E): one router over the concatenated public and private pool, no mask.

The control is not a safe configuration; it exists to show what the mask prevents.
Checks: routes and outputs match the oracle's soft route; the execution audit counts
exactly the private rows executed, so deny tokens that reached private experts show up
as violations; the masked route of the same inputs reports none.
"""
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


def soft_check(cfg, req):
    words = O.compile_words(req.metas, req.lengths)
    offs = torch.tensor(req.offsets, device="cuda")
    x = W.make_x(cfg, "cuda")
    layer, _ = C.device_layer(cfg, soft=True)
    d = C.run_device(layer, x, C.words_tensor(words), offs)
    oi = C.oracle_inputs(cfg)
    ref = C.oracle_layer(cfg, oi, words, soft=True)
    stats = C.compare_routes(cfg, d, ref.route)
    C.check_dispatch_consistent(d, cfg.n_experts)
    same = np.all(d.idx == ref.route.idx, axis=1)
    # the audit counts executed private rows of the device's own route, token by token
    rho = (d.idx >= cfg.n_pub).sum(axis=1)
    assert np.array_equal(d.audit_rows, rho)
    assert np.array_equal(d.audit_rows[same], ref.hook.rows[same])
    taus = np.array([O.decode_word(w) for w in words])
    assert np.array_equal(d.allow, taus.astype(np.uint8))     # route log keeps the policy decision
    viol = int(((taus == 0) & (rho > 0)).sum())
    assert d.violations == viol
    if same.all():
        assert viol == O.audit(ref.hook.rows, ref.route.allow, req.offsets).deny_violations
    rtol = C.RTOL_BF16 if cfg.dtype == "bf16" else C.RTOL_F32
    err = C.rel_l2(d.out.to(torch.float64).numpy()[same], ref.out[same])
    log(f"soft {cfg.name}: T={cfg.tokens} E={cfg.n_experts} rel_l2={err:.3e} deny violations={viol} {stats}")
    assert err <= rtol
    # the masked route of the same inputs executes no private row for a deny token
    masked, _ = C.device_layer(cfg)
    dm = C.run_device(masked, x, C.words_tensor(words), offs)
    assert dm.violations == 0 and np.all(dm.audit_rows[taus == 0] == 0)
    return viol


def test_soft_router_tiny_fp32():
    cfg = W.get_config("tiny")
    soft_check(cfg, W.make_requests(cfg, 0))


@pytest.mark.parametrize("shape", [
    dict(tokens=300, requests=6, hidden=256, inter=192, n_pub=24, n_priv=12, top_k=4),
    dict(tokens=200, requests=4, hidden=256, inter=128, n_pub=200, n_priv=100, top_k=8),  # pool of 300
    # above 2048 tokens: the LDS-staged router, a ragged last tile, mixed-policy tiles
    dict(tokens=2150, requests=5, hidden=256, inter=128, n_pub=40, n_priv=12, top_k=4),
    dict(tokens=2200, requests=4, hidden=256, inter=128, n_pub=200, n_priv=100, top_k=8),  # pool of 300, large batch
], ids=["E36", "E300", "T2150", "T2200_E300"])
def test_soft_router_small_bf16_leaks_and_is_audited(shape):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    viol = soft_check(cfg, req)
    assert viol > 0   # without the mask some deny tokens reach private experts
