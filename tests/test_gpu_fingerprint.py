"""GPU parity of the weight fingerprint (SHA-256 tree, FIPS 180-4) against the oracle,
and the state discipline it supports: the frozen public weights keep their fingerprint
through forward passes and through updates of the private experts (Sec. 3.2 training and
checkpointing; Sec. 5.1; App. C.1)."""
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


def device_fp(data: torch.Tensor, nbytes=None) -> bytes:
    n = data.numel() * data.element_size() if nbytes is None else nbytes
    ws = torch.empty(max(P.pmpe_fingerprint_workspace_bytes(n), 1), dtype=torch.uint8, device="cuda")
    dig = torch.empty(32, dtype=torch.uint8, device="cuda")
    P.pmpe_fingerprint(data, dig, ws, nbytes=n)
    torch.cuda.synchronize()
    return bytes(dig.cpu().numpy())


def host_bytes(n, seed):
    return np.random.default_rng(seed).integers(0, 256, n, dtype=np.uint8)


SIZES = [0, 1, 3, 55, 56, 63, 64, 65, 119, 120, 1023, 1024, 1025, 2048 + 7, 16 * 1024,
         16 * 1024 + 1, 17 * 1024, 257 * 1024, 256 * 1024 + 1, (1 << 20) + 13]


@pytest.mark.parametrize("n", SIZES)
def test_fingerprint_matches_oracle(n):
    log(f"fingerprint n={n}")
    h = host_bytes(max(n, 1), n)[:n]
    d = torch.from_numpy(h.copy()).cuda() if n else torch.empty(16, dtype=torch.uint8, device="cuda")
    assert device_fp(d, n) == O.fingerprint(h.tobytes())


def test_fips_examples_on_device():
    for msg, hexd in [(b"abc", "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"),
                      (b"abcdbcdecdefdefgefghfghighijhijkijkljklmklmnlmnomnopnopq",
                       "248d6a61d20638b8e5c026930c3e6039a33ce45964ff2167f6ecedd419db06c1")]:
        d = torch.frombuffer(bytearray(msg), dtype=torch.uint8).cuda()
        assert device_fp(d).hex() == hexd


@pytest.mark.parametrize("shift,n", [(1, 1025), (3, 64 * 1024 + 5), (8, 4096), (15, 63)])
def test_unaligned_data_byte_path(shift, n):
    log(f"fingerprint unaligned shift={shift} n={n}")
    h = host_bytes(n + 64, 100 + shift)
    d = torch.from_numpy(h).cuda()[shift:shift + n]
    assert d.data_ptr() % 16 != 0
    assert device_fp(d, n) == O.fingerprint(h[shift:shift + n].tobytes())


def test_one_byte_change_changes_the_fingerprint():
    h = host_bytes(300_001, 7)
    d = torch.from_numpy(h.copy()).cuda()
    f0 = device_fp(d)
    d[123_457] ^= 1
    assert device_fp(d) != f0


def test_expert_weights_at_layer_size():
    """One layer's public expert weights (bf16 [n_pub, 2I, H] and [n_pub, H, I]) of the
    Qwen-shaped workload: the device tree equals the oracle's over the host copy."""
    cfg = W.get_config("qwen")
    Lw = W.make_layer(cfg, 0, "cuda")
    for name in ("w13_pub", "w2_pub"):
        t = getattr(Lw, name)
        log(f"fingerprint {name} {tuple(t.shape)} {t.numel() * t.element_size()} B")
        ref = O.fingerprint(t.cpu().contiguous().view(torch.uint8).numpy().tobytes())
        assert device_fp(t) == ref


def test_public_fingerprint_unchanged_by_forward_and_private_updates():
    cfg = W.get_config("tiny")
    layer, Lw = C.device_layer(cfg)
    pub = [Lw.wr_pub, Lw.w13_pub, Lw.w2_pub]
    f_pub = P.fingerprint_tensors(*pub)
    f_priv = P.fingerprint_tensors(Lw.wr_priv, Lw.w13_priv, Lw.w2_priv)
    torch.cuda.synchronize()
    ref = O.fingerprint_set([t.cpu().contiguous().view(torch.uint8).numpy().tobytes() for t in pub])
    assert bytes(f_pub.cpu().numpy()) == ref
    req = W.make_requests(cfg)
    words = O.compile_words(req.metas, req.lengths)
    x = W.make_x(cfg, "cuda")
    offs = torch.tensor(req.offsets, device="cuda")
    for _ in range(3):
        C.run_device(layer, x, C.words_tensor(words), offs)
    # a private-only update (what training changes) leaves the public fingerprint alone
    Lw.w13_priv.mul_(0.5)
    assert torch.equal(P.fingerprint_tensors(*pub), f_pub)
    assert not torch.equal(P.fingerprint_tensors(Lw.wr_priv, Lw.w13_priv, Lw.w2_priv), f_priv)
    # a public change does not
    Lw.w2_pub.view(-1)[5] += 1
    assert not torch.equal(P.fingerprint_tensors(*pub), f_pub)
