"""pmpe_dispatch_noalloc (the allocation-free variant of pmpe_dispatch, whose chunk masks and
bases live in the library's per-device scratch array) through the C ABI, against
pmpe_dispatch with a caller workspace on the same expert choices: bit-exact, on two calls
in a row, the second with a smaller batch (so the array still holds the first call's
masks), then the first size again; with and without the row gather. Also the size limit.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2608_06690_amd as P

pytestmark = pytest.mark.gpu

N_PUB, N_PRIV, K, H = 128, 32, 8, 256
E = N_PUB + N_PRIV


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def draw_idx(T, seed):
    rng = np.random.default_rng(seed)
    w = 1.0 / np.arange(1, E + 1) ** 1.1
    w = w[rng.permutation(E)]
    w /= w.sum()
    return np.stack([np.sort(rng.choice(E, K, replace=False, p=w)) for _ in range(T)]).astype(np.int64)


def outputs(T):
    f = lambda n: torch.full((n,), -7, dtype=torch.int32, device="cuda")  # noqa: E731
    return dict(count=f(E), offset=f(E + 1), row_token=f(T * K), token_row=f(T * K))


def run(T, idx, noalloc, gather):
    desc = P.make_desc(H, 128, N_PUB, N_PRIV, K)
    dev_idx = torch.from_numpy(idx.astype(np.int32).reshape(-1)).cuda()
    x = torch.randn(T, H, generator=torch.Generator().manual_seed(T)).to(torch.bfloat16).cuda()
    x_perm = torch.zeros(T * K, H, dtype=torch.bfloat16, device="cuda") if gather else None
    o = outputs(T)
    if noalloc:
        P.pmpe_dispatch_noalloc(desc, T, dev_idx, x, o["count"], o["offset"], o["row_token"],
                                o["token_row"], x_perm)
    else:
        ws = torch.empty(P.pmpe_workspace_bytes(desc, T), dtype=torch.uint8, device="cuda")
        P.pmpe_dispatch(desc, T, dev_idx, x, o["count"], o["offset"], o["row_token"], o["token_row"],
                        x_perm, ws)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in o.items()}
    if gather:
        res["x_perm"] = x_perm.view(torch.int16).cpu().numpy()
    return res


@pytest.mark.parametrize("gather", [False, True], ids=["no_gather", "gather"])
def test_noalloc_dispatch_equals_workspace_dispatch(gather):
    # 8256 tokens: separate count and scatter launches (129 chunks); 1025: the scatter blocks
    # recount the masks; 700: one workgroup
    for T in (8256, 1025, 700, 8256):
        idx = draw_idx(T, seed=T + 11)
        log(f"noalloc dispatch T={T} gather={gather}")
        a = run(T, idx, True, gather)
        b = run(T, idx, False, gather)
        n = int(b["offset"][E])
        assert n == T * K
        for key in ("count", "offset", "token_row"):
            assert np.array_equal(a[key], b[key]), key
        assert np.array_equal(a["row_token"][:n], b["row_token"][:n])
        if gather:
            assert np.array_equal(a["x_perm"], b["x_perm"])


def test_noalloc_dispatch_rejects_batches_beyond_its_scratch():
    desc = P.make_desc(H, 128, 256, 256, K)  # 512 experts: 12 bytes per (chunk, expert)
    T = 64 * (P.PMPE_NOALLOC_SCRATCH_BYTES // (512 * 12) + 1)
    o = outputs(T)
    idx = torch.zeros(T * K, dtype=torch.int32, device="cuda")
    with pytest.raises(P.PmpeError) as e:
        P.pmpe_dispatch_noalloc(desc, T, idx, None, o["count"], o["offset"], o["row_token"],
                                o["token_row"], None)
    assert e.value.status == P.PMPE_ERR_SCRATCH
    torch.cuda.synchronize()
    assert int(o["count"][0].item()) == -7  # nothing launched
