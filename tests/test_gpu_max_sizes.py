"""GPU parity at the largest sizes the layer descriptor accepts, against the CPU oracle.

* Both pools at their maximum (256 public + 256 private experts) with the largest top-k (16):
  the router ranks up to 256 keys per token (512 in the soft control arm), dispatch groups 512
  experts, the expert GEMMs schedule up to 513 groups, and the combine adds 16 slots (its
  generic path). Batches on both sides of the router's register/LDS switch (2048 tokens).
* The largest hidden size (16384): a 16384-long K loop in the router and in GEMM1, with a
  large-batch case on the LDS-staged router at hidden 4096.

Acceptance is the parity suite's (routing and audit bit-exact off near-ties, per-row and
aggregate output bars).
"""
import sys

import pytest

import workloads as W
from oracle import pmpe_oracle as O
from tests import pmpe_cases as C
from tests.test_gpu_parity import full_check
from tests.test_gpu_soft_router import soft_check

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def requests_for(cfg):
    req = W.alternating_requests(cfg.requests, cfg.tokens // cfg.requests)
    req.lengths[-1] += cfg.tokens - sum(req.lengths)
    return req


MAX_POOLS = [dict(tokens=300, requests=4, hidden=256, inter=128, n_pub=256, n_priv=256, top_k=16),
             dict(tokens=2300, requests=5, hidden=256, inter=128, n_pub=256, n_priv=256, top_k=16)]


@pytest.mark.parametrize("shape", MAX_POOLS, ids=lambda s: f"T{s['tokens']}")
def test_max_pools_and_top_k(shape):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    log(f"max pools: {shape}")
    layer, _ = C.device_layer(cfg)
    req = requests_for(cfg)
    full_check(cfg, layer, W.make_x(cfg, "cuda"), O.compile_words(req.metas, req.lengths), req)


@pytest.mark.parametrize("shape", MAX_POOLS, ids=lambda s: f"T{s['tokens']}")
def test_max_soft_pool(shape):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    log(f"max soft pool (512 experts): {shape}")
    soft_check(cfg, requests_for(cfg))


MAX_HIDDEN = [dict(tokens=96, requests=4, hidden=16384, inter=64, n_pub=16, n_priv=16, top_k=2),
              dict(tokens=2100, requests=5, hidden=4096, inter=128, n_pub=32, n_priv=16, top_k=4)]


@pytest.mark.parametrize("shape", MAX_HIDDEN, ids=lambda s: f"T{s['tokens']}_H{s['hidden']}")
def test_large_hidden(shape):
    cfg = W.scaled_config(W.get_config("qwen"), **shape)
    log(f"large hidden: {shape}")
    layer, _ = C.device_layer(cfg)
    req = requests_for(cfg)
    full_check(cfg, layer, W.make_x(cfg, "cuda"), O.compile_words(req.metas, req.lengths), req)
