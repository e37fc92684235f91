"""C ABI checks that need no GPU: every symbol declared in include/pmpe.h is exported,
the binding's argument lists match the declarations, and host-side validation
returns the documented status before anything is launched."""
import ctypes
import os
import re

import pytest

import paper_2608_06690_amd as P
from paper_2608_06690_amd import _native as N

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "pmpe.h")


def declarations():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    decls = {}
    for m in re.finditer(r"\b(?:pmpe_status|size_t|const char\*|int32_t)\s+(pmpe_\w+)\s*\(([^)]*)\)\s*;", src):
        params = [p.strip() for p in m.group(2).split(",") if p.strip() and p.strip() != "void"]
        decls[m.group(1)] = params
    return decls


def test_header_declares_the_five_calls():
    d = declarations()
    for name in ["pmpe_route", "pmpe_dispatch", "pmpe_expert_ffn", "pmpe_combine", "pmpe_audit",
                 "pmpe_workspace_bytes", "pmpe_status_string", "pmpe_version", "pmpe_check_desc",
                 "pmpe_fingerprint", "pmpe_fingerprint_workspace_bytes"]:
        assert name in d, name


def test_every_declared_symbol_is_exported():
    lib = N.lib()
    for name in declarations():
        assert hasattr(lib, name), name
        assert isinstance(getattr(lib, name), ctypes._CFuncPtr)


def test_binding_argument_counts_match_header():
    lib = N.lib()
    for name, params in declarations().items():
        assert len(getattr(lib, name).argtypes) == len(params), name


def desc(**kw):
    base = dict(hidden=2048, inter=768, n_pub=128, n_priv=32, top_k=8)
    base.update(kw)
    return P.make_desc(**base)


def test_package_exports_descriptor_constants():
    for name in ["PMPE_BF16", "PMPE_F32", "PMPE_GATE_RENORM_TOPK", "PMPE_GATE_POOL_SOFTMAX",
                 "PMPE_ROUTE_MASKED", "PMPE_ROUTE_SOFT", "PMPE_POLICY_ALLOW", "PMPE_POLICY_DENY"]:
        assert hasattr(P, name), name
    d = P.make_desc(128, 64, 8, 8, 2, route_mode=P.PMPE_ROUTE_SOFT)
    assert d.route_mode == 1 and P.make_desc(128, 64, 8, 8, 2).route_mode == 0


def test_valid_descriptor_and_workspace():
    d = desc()
    assert P.pmpe_check_desc(d, 4096) == 0
    ws = P.pmpe_workspace_bytes(d, 4096)
    assert ws >= 4096 * 8 * 768 * 2          # the SwiGLU intermediate of every row
    assert P.pmpe_workspace_bytes(d, 0) >= 0


@pytest.mark.parametrize("kw,status", [
    (dict(top_k=9, n_priv=8), -3), (dict(top_k=129), -2), (dict(top_k=0), -2),
    (dict(hidden=100), -2), (dict(hidden=192), -2), (dict(inter=100), -2),
    (dict(n_pub=0), -2), (dict(n_pub=300), -2), (dict(n_priv=300), -2),
    (dict(n_shared=2, shared_inter=0), -2),
    (dict(hidden=16384, inter=65536), -2),                       # one expert's w13 >= 2^31 elements
    (dict(hidden=16384, inter=1024, n_shared=64, shared_inter=1024), -2),
])
def test_invalid_descriptor_codes(kw, status):
    d = desc(**kw)
    assert P.pmpe_check_desc(d, 16) == status
    assert P.pmpe_workspace_bytes(d, 16) == 0


def test_dtype_and_gate_mode_codes():
    d = desc()
    d.w_dtype = N.PMPE_F32
    assert P.pmpe_check_desc(d, 16) == -4
    d = desc()
    d.act_dtype = d.w_dtype = 7
    assert P.pmpe_check_desc(d, 16) == -4
    d = desc()
    d.gate_mode = 5
    assert P.pmpe_check_desc(d, 16) == -2
    d = desc()
    d.route_mode = 2
    assert P.pmpe_check_desc(d, 16) == -2
    d.route_mode = N.PMPE_ROUTE_SOFT
    assert P.pmpe_check_desc(d, 16) == 0
    assert P.pmpe_check_desc(desc(), -1) == -2
    # 32-bit byte offsets of the permuted rows: T*k*max(H, I) must stay below 2^31
    assert P.pmpe_check_desc(desc(hidden=8192, top_k=8), 32768) == -2
    assert P.pmpe_check_desc(desc(hidden=8192, top_k=8), 32767) == 0


def fake(addr):
    """A pointer-like stand-in: never dereferenced, validation fails before launch."""
    class F:
        def is_contiguous(self):
            return True

        def data_ptr(self):
            return addr
    return F()


def test_null_and_alignment_rejected_before_launch():
    d = desc()
    lib = N.lib()
    # NULL x
    st = lib.pmpe_route(ctypes.byref(d), 16, None, 0x1000, None, None, None, 0x2000, 0x3000, 0x4000,
                        None, None, 0x5000, 1 << 20, None)
    assert st == -1
    # route without workspace
    st = lib.pmpe_route(ctypes.byref(d), 16, 0x1000, 0x1000, None, None, None, 0x2000, 0x3000,
                        0x4000, None, None, None, 0, None)
    assert st == -6
    # misaligned x
    st = lib.pmpe_route(ctypes.byref(d), 16, 0x1004, 0x1000, None, None, None, 0x2000, 0x3000,
                        0x4000, None, None, 0x5000, 1 << 20, None)
    assert st == -5
    # soft-routing control without the private router rows
    ds = desc()
    ds.route_mode = N.PMPE_ROUTE_SOFT
    st = lib.pmpe_route(ctypes.byref(ds), 16, 0x1000, 0x1000, None, None, None, 0x2000, 0x3000,
                        0x4000, None, None, 0x5000, 1 << 20, None)
    assert st == -1
    # dispatch without workspace
    st = lib.pmpe_dispatch(ctypes.byref(d), 16, 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 0x6000,
                           None, None, 0, None)
    assert st == -6
    # expert ffn with a too small workspace
    st = lib.pmpe_expert_ffn(ctypes.byref(d), 16, 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 0x6000,
                             0x7000, None, None, None, None, None, 0x8000, 0x9000, None, None,
                             0xA000, 16, None)
    assert st == -6
    # shared experts requested but not given
    d2 = desc(n_shared=2, shared_inter=1408)
    st = lib.pmpe_combine(ctypes.byref(d2), 16, 0x1000, 0x2000, 0x3000, None, 0x4000, None)
    assert st == -1
    # audit: negative request count
    st = lib.pmpe_audit(ctypes.byref(d), 16, 0x1000, 0x2000, 0x3000, -1, 0x4000, 0x5000, 0x6000, None)
    assert st == -2


def test_backward_rejects_misaligned_outputs_before_launch():
    """A misaligned dx or gradient array is refused (PMPE_ERR_ALIGN) before any launch
    (dx is written in 16-byte vectors)."""
    d = desc()
    assert d.act_dtype == P.PMPE_BF16
    lib = N.lib()

    def call(dx=0x20000, dw13=0x21000, dw2=0x22000, dwr=0x23000):
        # x dout idx gate count offset row_token token_row y_perm wr_pub wr_priv w13_pub w2_pub
        # w13_priv w2_priv bias w13_sh w2_sh w2t_pub w13t_pub w2t_priv w13t_priv ab
        ins = [0x1000 * (i + 1) for i in range(15)] + [None, None, None, None, None, None, None, None]
        return lib.pmpe_backward(ctypes.byref(d), 16, *ins, dx, dw13, dw2, dwr, None, 0x30000, 1 << 30, None)

    assert call(dx=0x20004) == -5
    assert call(dw13=0x21008) == -5
    assert call(dw2=0x22004) == -5
    assert call(dwr=0x2300C) == -5
    assert call(dx=None) == -1


def test_fingerprint_workspace_and_validation():
    lib = N.lib()
    ws = P.pmpe_fingerprint_workspace_bytes
    # one leaf needs no workspace; n leaves need 32 n plus 32 ceil(n / 16), each rounded to 256
    assert ws(0) == 0 and ws(1) == 0 and ws(1024) == 0
    assert ws(1025) == 256 + 256
    n = 3 * 1024 * 1024 // 1024
    assert ws(3 * 1024 * 1024) == -(-32 * n // 256) * 256 + -(-32 * (-(-n // 16)) // 256) * 256
    assert ws((1 << 46) + 1) == 0
    assert P.PMPE_FP_LEAF_BYTES == 1024 and P.PMPE_FP_FANOUT == 16
    # NULL digest, NULL data with bytes, too large, misaligned digest, missing/short workspace
    assert lib.pmpe_fingerprint(0x1000, 16, None, None, 0, None) == -1
    assert lib.pmpe_fingerprint(None, 16, 0x2000, None, 0, None) == -1
    assert lib.pmpe_fingerprint(0x1000, (1 << 46) + 1, 0x2000, None, 0, None) == -2
    assert lib.pmpe_fingerprint(0x1000, 16, 0x2008, None, 0, None) == -5
    assert lib.pmpe_fingerprint(0x1000, 4096, 0x2000, None, 0, None) == -1
    assert lib.pmpe_fingerprint(0x1000, 4096, 0x2000, 0x3000, 16, None) == -6
    assert lib.pmpe_fingerprint(0x1000, 4096, 0x2000, 0x3008, 1 << 20, None) == -5


def test_zero_tokens_launch_nothing():
    d = desc()
    lib = N.lib()
    assert lib.pmpe_route(ctypes.byref(d), 0, 0x1000, 0x1000, None, None, None, 0x2000, 0x3000,
                          0x4000, None, None, None, 0, None) == 0
    assert lib.pmpe_combine(ctypes.byref(d), 0, 0x1000, 0x2000, 0x3000, None, 0x4000, None) == 0


def test_status_strings():
    for s in range(-8, 1):
        assert N.lib().pmpe_status_string(s).decode()
    assert P.pmpe_version() >= 10000


def test_policy_resolver_product_side():
    import workloads as W
    assert P.resolve_policy({"allow_private": True})
    for m in W.MALFORMED_META:
        assert not P.resolve_policy(m)
    w = P.token_policy_words([{"allow_private": True}, None], [2, 1])
    assert [int(v) & 0xFFFFFFFF for v in w] == [N.PMPE_POLICY_ALLOW] * 2 + [0]


def test_cache_tag_check_follows_the_oracle_rule():
    """The library's host-side cache-tag guard against the oracle's rule on every single
    field change, malformed decisions and missing tags."""
    from oracle import pmpe_oracle as O
    rev, fp = bytes(range(32)), bytes(range(100, 132))
    cases = [((1, rev, fp), (1, rev, fp)), ((0, rev, fp), (0, rev, fp)), ((1, rev, fp), (0, rev, fp)),
             ((2, rev, fp), (2, rev, fp)), ((0, rev, fp), (7, rev, fp))]
    for i in range(32):
        r2 = bytearray(rev); r2[i] ^= 0x40
        f2 = bytearray(fp); f2[i] ^= 0x01
        cases.append(((1, rev, fp), (1, bytes(r2), fp)))
        cases.append(((0, rev, fp), (0, rev, bytes(f2))))
    for c, r in cases:
        got = P.pmpe_cache_tag_check(P.make_cache_tag(*c), P.make_cache_tag(*r))
        assert got == O.cache_tag_ok(c, r), (c[0], r[0])
    assert not P.pmpe_cache_tag_check(None, P.make_cache_tag(1, rev, fp))
    assert not P.pmpe_cache_tag_check(P.make_cache_tag(1, rev, fp), None)


def test_route_record_validation():
    d = desc()
    lib = N.lib()
    assert lib.pmpe_route_record(ctypes.byref(d), 16, 70000, 0x1000, 0x2000, 0x3000, 1, 0x4000, None) == -2
    assert lib.pmpe_route_record(ctypes.byref(d), 16, 0, 0x1000, 0x2000, 0x3000, 0, 0x4000, None) == -2
    assert lib.pmpe_route_record(ctypes.byref(d), 16, 0, None, 0x2000, 0x3000, 1, 0x4000, None) == -1
    assert lib.pmpe_route_record(ctypes.byref(d), 16, 0, 0x1000, 0x2000, 0x3000, 1, 0x4008, None) == -5
    assert lib.pmpe_route_record(ctypes.byref(d), 0, 0, None, None, None, 0, None, None) == 0


def test_adamw_validation():
    lib = N.lib()
    a = (ctypes.c_float * 5)()
    ok = dict(lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, wd=0.0)
    call = lambda p, dt, master, n, step, b1=0.9, lr=1e-3: lib.pmpe_adamw(  # noqa: E731
        p, dt, master, 0x2000, 0x3000, 0x4000, n, step, lr, b1, 0.999, 1e-8, 0.0, None)
    assert call(0x1000, 2, None, 16, 1) == -4          # unknown dtype
    assert call(0x1000, 1, None, 16, 1) == -4          # bf16 without master
    assert call(0x1000, 0, 0x5000, 16, 1) == -4        # fp32 with master
    assert call(0x1000, 0, None, 16, 0) == -2          # step < 1
    assert call(0x1000, 0, None, 16, 1, b1=1.0) == -2  # beta out of range
    assert call(0x1000, 0, None, 16, 1, lr=float("nan")) == -2
    assert call(None, 0, None, 16, 1) == -1
    assert call(0x1004, 0, None, 16, 1) == -5
    assert call(None, 0, None, 0, 1) == 0              # nothing to do
    del a, ok


def test_fp8_entry_validation():
    lib = N.lib()
    d = desc()
    ptrs = [0x1000 * (i + 1) for i in range(17)]
    # bf16 weights through the fp8 entry: dtype error
    assert lib.pmpe_expert_ffn_fp8(ctypes.byref(d), 16, *ptrs, 0x20000, 1 << 20, None) == -4
    d8 = desc()
    d8.w_dtype = N.PMPE_FP8_E4M3
    # the bf16 entry refuses fp8 weights
    assert lib.pmpe_expert_ffn(ctypes.byref(d8), 16, *([0x1000] * 16), 0x20000, 1 << 20, None) == -4
    # shared experts are not supported with fp8 weights
    ds = desc(n_shared=2, shared_inter=256)
    ds.w_dtype = N.PMPE_FP8_E4M3
    assert lib.pmpe_expert_ffn_fp8(ctypes.byref(ds), 16, *ptrs, 0x20000, 1 << 20, None) == -2
    # private weights without their scales
    p2 = list(ptrs)
    p2[11] = None  # w13s_priv
    assert lib.pmpe_expert_ffn_fp8(ctypes.byref(d8), 16, *p2, 0x20000, 1 << 20, None) == -1
    # workspace too small
    assert lib.pmpe_expert_ffn_fp8(ctypes.byref(d8), 16, *ptrs, 0x20000, 16, None) == -6


def test_noalloc_dispatch_validation_before_the_device():
    """pmpe_dispatch_noalloc rejects a batch whose masks and chunk bases exceed its scratch
    array (PMPE_ERR_SCRATCH), a NULL output and a bad descriptor, all before it touches a
    device (these calls run with no GPU)."""
    lib = N.lib()
    d = desc(n_pub=256, n_priv=256)               # 512 experts: 12 bytes per (chunk, expert)
    chunks = N.PMPE_NOALLOC_SCRATCH_BYTES // (512 * 12)
    too_big = 64 * (chunks + 1)
    st = lib.pmpe_dispatch_noalloc(ctypes.byref(d), too_big, 0x1000, None, 0x3000, 0x4000, 0x5000,
                                   0x6000, None, None)
    assert st == N.PMPE_ERR_SCRATCH == -9
    assert "scratch" in lib.pmpe_status_string(-9).decode()
    st = lib.pmpe_dispatch_noalloc(ctypes.byref(d), 64, None, None, 0x3000, 0x4000, 0x5000, 0x6000,
                                   None, None)
    assert st == -1
    st = lib.pmpe_dispatch_noalloc(ctypes.byref(desc(top_k=0)), 64, 0x1000, None, 0x3000, 0x4000,
                                   0x5000, 0x6000, None, None)
    assert st == -2
    # the Qwen-shaped batches (160 experts) fit up to 69,888 tokens
    q = desc()
    assert (4096 + 63) // 64 * 160 * 12 <= N.PMPE_NOALLOC_SCRATCH_BYTES
    st = lib.pmpe_dispatch_noalloc(ctypes.byref(q), 64 * (N.PMPE_NOALLOC_SCRATCH_BYTES // (160 * 12) + 2),
                                   0x1000, None, 0x3000, 0x4000, 0x5000, 0x6000, None, None)
    assert st == -9
