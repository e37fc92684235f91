"""pmpe_dispatch on its own, bit-exact against the oracle's stable counting sort, on each
side of every dispatch path boundary: one workgroup (up to 8192 (token, slot) pairs), the
scatter blocks that recount every chunk's masks themselves (up to 128 chunks of 64 tokens),
and separate count and scatter launches (more chunks).

Expert choices are seeded and skewed (a Zipf-like draw over 160 experts, five of them never
drawn, so some experts get hundreds of rows and some none), distinct within a token and
ascending as the router writes them (or, in the repeated-id cases, with an id listed twice
in some tokens: only the first slot holding it gets a row); a few slots carry ids outside
[0, E), which must be neither counted nor given a row.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2608_06690_amd as P
from oracle import pmpe_oracle as O

pytestmark = pytest.mark.gpu

N_PUB, N_PRIV, K, H = 128, 32, 8, 256
E = N_PUB + N_PRIV


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def draw_idx(T, seed, repeats=False):
    rng = np.random.default_rng(seed)
    w = 1.0 / np.arange(1, E + 1) ** 1.1
    w = w[rng.permutation(E)]
    w[rng.choice(E, 5, replace=False)] = 0.0  # five experts no token selects
    w /= w.sum()
    idx = np.stack([np.sort(rng.choice(E, K, replace=False, p=w)) for _ in range(T)]).astype(np.int64)
    bad = rng.random(idx.shape) < 0.002  # out-of-range ids: not counted, no row
    idx[bad] = np.where(rng.random(int(bad.sum())) < 0.5, -1, E + 3)
    if repeats:  # some tokens list an expert twice: only the first slot gets a row
        for t in rng.choice(T, max(1, T // 50), replace=False):
            j = int(rng.integers(1, K))
            idx[t, j] = idx[t, int(rng.integers(0, j))]
    return idx


@pytest.mark.parametrize("repeats", [False, True], ids=["distinct", "repeated_ids"])
@pytest.mark.parametrize("T", [1024, 1025, 2113, 8192, 8256],
                         ids=["1024_one_workgroup", "1025_scatter_recount", "2113_scatter_recount",
                              "8192_128_chunks", "8256_129_chunks"])
def test_dispatch_matches_oracle(T, repeats):
    idx = draw_idx(T, seed=20260730 + T, repeats=repeats)
    desc = P.make_desc(H, 128, N_PUB, N_PRIV, K)
    ws = torch.empty(P.pmpe_workspace_bytes(desc, T), dtype=torch.uint8, device="cuda")
    dev_idx = torch.from_numpy(idx.astype(np.int32).reshape(-1)).cuda()
    count = torch.full((E,), -7, dtype=torch.int32, device="cuda")
    offset = torch.full((E + 1,), -7, dtype=torch.int32, device="cuda")
    row_token = torch.full((T * K,), -7, dtype=torch.int32, device="cuda")
    token_row = torch.full((T * K,), -7, dtype=torch.int32, device="cuda")
    log(f"dispatch T={T} pairs={T * K} out-of-range slots={int(((idx < 0) | (idx >= E)).sum())} "
        f"repeats={repeats}")
    P.pmpe_dispatch(desc, T, dev_idx, None, count, offset, row_token, token_row, None, ws)
    torch.cuda.synchronize()
    ref = O.dispatch(idx, E)
    n = int(ref.offset[E])
    assert np.array_equal(count.cpu().numpy(), ref.count)
    assert np.array_equal(offset.cpu().numpy(), ref.offset)
    assert np.array_equal(row_token.cpu().numpy()[:n], ref.row_token[:n])
    assert np.array_equal(token_row.cpu().numpy().reshape(T, K), ref.token_row)
    # the draw is skewed: an expert with more rows than a 256-row tile, and empty experts
    assert ref.count.max() > 256 and (ref.count == 0).sum() >= 5
    if repeats:  # a repeated id's later slot has no row, so fewer rows than valid slots
        valid = int(((idx >= 0) & (idx < E)).sum())
        assert n < valid and int((ref.token_row < 0).sum()) > int(((idx < 0) | (idx >= E)).sum())
