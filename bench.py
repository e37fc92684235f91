"""Benchmark of the policy-masked MoE layer forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-decode]

A step is one pass of the whole layer (route, dispatch, expert FFN, combine, audit)
over the Qwen3-30B-A3B-shaped workload: 4096 tokens in 8 requests of 512 (4 allow,
4 deny), H 2048, I 768, 128 public + 32 private experts, top-8, bf16 experts, fp32
router; inputs synthetic and resident in HBM. Prints one JSON line.

Per-call times come from HIP events recorded on the stream the library launches on.
The roofline object describes pmpe_expert_ffn (the dominant call): its algorithmic
flops are 2 * 3 * H * I per (token, expert) pair. The CPU baseline is the CPU oracle
timed on a bounded sample of the same workload on this host's cores. The decode
object is the 256-request single-token workload, whose expert FFN is bound by HBM
reads of the touched experts' weights.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s (Qwen3-30B-A3B shape) + % MFMA peak; decode % HBM BW"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
# Integer VALU rate: 256 CUs x 64 lanes x 2.4 GHz, one 32-bit operation per lane per clock.
PEAK_VALU_OPS = 256 * 64 * 2.4e9
# SHA-256 needs about 1400 such operations per 64-byte block on CDNA4 (rotations and the
# two 3-input logic functions take one operation each, three-way xors and sums one each):
# 64 rounds x 14, 48 schedule words x 10, 8 state sums, 16 byte swaps.
SHA256_OPS_PER_BLOCK = 64 * 14 + 48 * 10 + 8 + 16
CALLS = ["route", "dispatch", "expert_ffn", "combine", "audit"]
COPY_BYTES = 1 << 30

# HBM traffic of one pmpe_expert_ffn call on the Qwen-shaped layer, from rocprofv3
# FETCH_SIZE and WRITE_SIZE (summed over its kernels, scaled by the counters' reading
# for a plain copy of known size). Keyed by the SHA-256 of the kernel sources the
# counters were taken on (the GEMM and its copy helper): any other source reports null.
FFN_TRAFFIC_BYTES = {
    "23d3c310a0ec016629cdb9c251d67b08d14b3f19f816719505763ac2b0edbf9c": 2_027_439_378,
}
FFN_SOURCES = ("ffn.hip", "lds_dma.h")


def ffn_source_hash():
    import hashlib
    h = hashlib.sha256()
    for name in FFN_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_06690_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-decode", action="store_true")
    p.add_argument("--no-fingerprint", action="store_true")
    p.add_argument("--no-backward", action="store_true")
    p.add_argument("--no-fp8", action="store_true")
    p.add_argument("--no-deepseek", action="store_true")
    p.add_argument("--stack", action="store_true",
                   help="also time the 48-layer stack (72.5 GB of weights, about a minute)")
    p.add_argument("--stack-only", action="store_true", help="only time the 48-layer stack")
    p.add_argument("--fp8-only", action="store_true", help="only time the fp8-weight variant")
    p.add_argument("--backward-only", action="store_true",
                   help="only time the private-only backward of the Qwen-shaped layer")
    p.add_argument("--vendor-gemm", action="store_true",
                   help="only time hipBLASLt on the same expert GEMM shapes (context)")
    p.add_argument("--fingerprint-only", action="store_true",
                   help="only time the public-weight fingerprint")
    p.add_argument("--cpu-sample", type=int, default=4096, help="tokens in the CPU-oracle sample")
    p.add_argument("--cpu-reps", type=int, default=3, help="timed repetitions of the CPU oracle")
    p.add_argument("--decode-only", action="store_true",
                   help="time only the decode workload (for a separate kernel profile)")
    p.add_argument("--all-deny", action="store_true",
                   help="run only the Qwen-shaped layer with every request denied (the expert FFN "
                        "must then read public expert weights only)")
    p.add_argument("--no-private-weights", action="store_true",
                   help="with --all-deny: pass NULL for every private tensor (router rows and "
                        "expert weights); the counters must read the same bytes as with them present")
    p.add_argument("--deepseek-only", action="store_true",
                   help="time only the DeepSeek-V2-Lite-shaped layer (for a separate kernel profile)")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="run only a plain 1 GiB device-to-device copy (counter calibration)")
    p.add_argument("--read-probe", action="store_true",
                   help="time only torch reductions that stream 0.9 GB from HBM once, L2/MALL "
                        "flushed before each (context for the decode rate: a plain read stream)")
    return p.parse_args()


def setup(cfg_name, device, all_deny=False, drop_private=False):
    import torch
    import workloads as W
    import paper_2608_06690_amd as P

    cfg = W.get_config(cfg_name)
    Lw = W.make_layer(cfg, 0, device)
    gm = P.PMPE_GATE_POOL_SOFTMAX if cfg.gate_mode == "pool_softmax" else P.PMPE_GATE_RENORM_TOPK
    desc = P.make_desc(cfg.hidden, cfg.inter, cfg.n_pub, cfg.n_priv, cfg.top_k, cfg.n_shared,
                       cfg.shared_inter, cfg.dtype == "bf16", gm)
    if drop_private:
        layer = P.PolicyMaskedMoE(desc, Lw.wr_pub, None, Lw.bias, Lw.w13_pub, Lw.w2_pub,
                                  None, None, Lw.w13_sh, Lw.w2_sh)
    else:
        layer = P.PolicyMaskedMoE(desc, Lw.wr_pub, Lw.wr_priv, Lw.bias, Lw.w13_pub, Lw.w2_pub,
                                  Lw.w13_priv, Lw.w2_priv, Lw.w13_sh, Lw.w2_sh)
    x = W.make_x(cfg, device)
    req = W.make_requests(cfg, 0)
    if all_deny:
        req = W.Requests(list(req.lengths), [dict(W.DENY_META) for _ in req.lengths],
                         ["deny"] * len(req.lengths))
    words = P.token_policy_words(req.metas, req.lengths, device)
    req_off = P.request_offsets(req.lengths, device)
    audit = layer.audit_buffers(cfg.tokens, len(req.lengths))
    bufs = layer.buffers(cfg.tokens)
    torch.cuda.synchronize()
    return cfg, layer, x, words, req_off, audit, bufs, req


def run_step(layer, x, words, req_off, audit, bufs, stream, events=None):
    """One layer pass; with `events` (6 events) records a boundary around every call."""
    T = x.shape[0]
    if events:
        events[0].record(stream)
    layer.route(x, words, bufs, stream)
    if events:
        events[1].record(stream)
    layer.dispatch(x, bufs, stream)
    if events:
        events[2].record(stream)
    layer.expert_ffn(x, bufs, audit, stream)
    if events:
        events[3].record(stream)
    layer.combine(x, bufs, stream)
    if events:
        events[4].record(stream)
    layer.audit(T, bufs, audit, req_off, stream)
    if events:
        events[5].record(stream)


def evict_caches(buf):
    """Push earlier data out of L2 and the MALL by reading `buf` (512 MiB, twice the MALL):
    a read leaves no dirty lines, so the timed pass that follows pays no write-back of the
    eviction traffic (a 512 MiB write left about 256 MB of dirty lines to drain)."""
    import torch
    v = buf.view(torch.int64)
    if not hasattr(evict_caches, "out") or evict_caches.out.device != v.device:
        evict_caches.out = torch.empty((), dtype=torch.int64, device=v.device)
    torch.sum(v, 0, out=evict_caches.out)


def time_layer(layer, x, words, req_off, audit, bufs, steps, warmup, flush=None):
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        audit.zero_()
        run_step(layer, x, words, req_off, audit, bufs, stream)
    torch.cuda.synchronize()
    # whole-step throughput: K back-to-back steps
    t0 = time.perf_counter()
    for _ in range(steps):
        run_step(layer, x, words, req_off, audit, bufs, stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # per-call durations from events on the launch stream
    per = {c: [] for c in CALLS}
    for _ in range(steps):
        if flush is not None:
            evict_caches(flush)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        run_step(layer, x, words, req_off, audit, bufs, stream, ev)
        torch.cuda.synchronize()
        for i, c in enumerate(CALLS):
            per[c].append(ev[i].elapsed_time(ev[i + 1]) * 1e3)  # us
    med = {c: sorted(v)[len(v) // 2] for c, v in per.items()}
    mean = {c: sum(v) / len(v) for c, v in per.items()}
    p10 = {c: sorted(v)[len(v) // 10] for c, v in per.items()}
    p90 = {c: sorted(v)[min(len(v) - 1, (9 * len(v)) // 10)] for c, v in per.items()}
    return wall / steps * 1e3, med, mean, p10, p90


def call_bytes(cfg, counts, T, any_allow, any_deny):
    """Algorithmic HBM bytes of each call of one layer pass (reads plus writes)."""
    H, k, E = cfg.hidden, cfg.top_k, cfg.n_pub + cfg.n_priv
    el = 2 if cfg.dtype == "bf16" else 4
    pairs = T * k
    touched = int((counts > 0).sum())
    return {
        # x, the permitted router rows, policy words; idx, gates, allow, kgap out
        "route": T * H * el + (cfg.n_pub * H * 4 if any_deny else 0)
                 + (cfg.n_priv * H * 4 if any_allow else 0) + T * 4 + pairs * 8 + T * 5,
        # idx in; counts, offsets, row_token, token_row out
        "dispatch": pairs * 4 + E * 8 + 4 + pairs * 8,
        # touched experts' weights once, x rows in, y rows out
        "expert_ffn": touched * 3 * H * cfg.inter * el + pairs * H * el * 2,
        # y rows, token_row and gates in; out
        "combine": pairs * H * el + pairs * 8 + T * H * el,
        # per-token counts and decisions in; per-request sums out
        "audit": T * 5 + (cfg.requests + 1) * 4 + cfg.requests * 8 + 12,
    }


def kernel_rates(nbytes, us):
    return {c: {"bytes": nbytes[c], "us": us[c], "gbs": nbytes[c] / (us[c] * 1e-6) / 1e9,
                "hbm_frac": nbytes[c] / (us[c] * 1e-6) / 1e9 / PEAK_HBM_GBS} for c in CALLS}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, req, n_sample, reps, min_seconds=10.0):
    """The CPU oracle on a bounded sample: n_sample tokens (half from allow requests,
    half from deny requests), routed and run through their experts; the median of at
    least `reps` timed repetitions, repeated until about `min_seconds` of CPU work."""
    import numpy as np
    import torch
    from oracle import pmpe_oracle as O
    import workloads as W

    torch.set_num_threads(len(os.sched_getaffinity(0)))
    words_all = O.compile_words(req.metas, req.lengths)
    rng = np.random.default_rng(0)
    allow_t = np.nonzero(words_all == O.ALLOW_WORD)[0]
    deny_t = np.nonzero(words_all != O.ALLOW_WORD)[0]
    toks = np.sort(np.concatenate([rng.choice(allow_t, n_sample // 2, replace=False),
                                   rng.choice(deny_t, n_sample - n_sample // 2, replace=False)]))
    x = W.make_x(cfg, "cpu")[torch.as_tensor(toks)].double().numpy()
    wr_pub, wr_priv, bias = (t.double().numpy() if t is not None else None for t in W.make_router(cfg))
    w13 = np.empty((cfg.n_experts, 2 * cfg.inter, cfg.hidden))
    w2 = np.empty((cfg.n_experts, cfg.hidden, cfg.inter))
    for e in range(cfg.n_experts):  # inputs resident before timing
        a, b = W.make_expert(cfg, 0, e, "cpu")
        w13[e] = a.double().numpy()
        w2[e] = b.double().numpy()
    words = words_all[toks]
    times = []
    while len(times) < reps or (sum(times) < min_seconds and len(times) < 50):
        t0 = time.perf_counter()
        res = O.layer_forward(x, wr_pub, wr_priv, bias, w13[:cfg.n_pub], w2[:cfg.n_pub],
                              w13[cfg.n_pub:], w2[cfg.n_pub:], words, cfg.top_k, cfg.gate_mode)
        O.audit(res.hook.rows, res.route.allow, [0, len(toks)])
        times.append(time.perf_counter() - t0)
    dt = sorted(times)[len(times) // 2]
    return {"value": len(toks) / dt, "unit": "tokens/s", "cores": torch.get_num_threads(),
            "kind": "oracle",
            "sample": f"{len(toks)} of the {cfg.tokens} tokens ({n_sample // 2} allow, "
                      f"{n_sample - n_sample // 2} deny), whole layer in fp64 numpy; median of "
                      f"{len(times)} runs, {dt:.2f} s each, {sum(times):.1f} s in all; "
                      f"CPU {cpu_model()}"}


def decode_bench(args, dev):
    """The decode workload: tokens/s and the expert FFN's HBM rate on the touched
    experts' weights (each read once per call), with L2/MALL flushed before each
    event-timed step."""
    import torch
    cfgd, layerd, xd, wd, rod, ad, bd, _ = setup("decode", dev)
    flush = torch.zeros(512 << 20, dtype=torch.uint8, device=dev)
    msd, medd, meand, p10d, p90d = time_layer(layerd, xd, wd, rod, ad, bd, args.steps, args.warmup, flush)
    counts = bd.expert_count.cpu()
    touched = int((counts > 0).sum())
    wb = touched * 3 * cfgd.hidden * cfgd.inter * 2
    gbs = wb / (meand["expert_ffn"] * 1e-6) / 1e9
    res = {"workload": "qwen3-30b-a3b-shaped decode layer, 256 requests x 1 token",
           "tokens_per_s": cfgd.tokens / (msd * 1e-3), "ms_per_step": msd,
           "experts_touched": touched, "weight_bytes": wb,
           "ffn_us_mean": meand["expert_ffn"], "ffn_hbm_gbs": gbs,
           "ffn_hbm_frac": gbs / PEAK_HBM_GBS, "calls_us_mean": meand,
           "calls_us_median": medd, "calls_us_p10": p10d, "calls_us_p90": p90d,
           "note": "L2/MALL flushed by reading a 512 MiB buffer before each event-timed step"}
    al = bd.allow.cpu()
    res["calls_hbm"] = kernel_rates(call_bytes(cfgd, counts, cfgd.tokens, bool(al.any()),
                                               bool((al == 0).any())), meand)
    del layerd, xd, bd, flush
    torch.cuda.empty_cache()
    return res


def deepseek_bench(args, dev):
    """The DeepSeek-V2-Lite-shaped layer (8192 tokens, 2 shared + 64 public + 16 private
    experts of intermediate 1408, top-6, pool softmax, N(0,1) logit bias): tokens/s and
    the expert FFN's MFMA fraction (routed and shared experts)."""
    import torch
    cfg, layer, x, words, req_off, audit, bufs, req = setup("deepseek", dev)
    ms, med, mean, p10, p90 = time_layer(layer, x, words, req_off, audit, bufs,
                                         max(10, args.steps // 2), args.warmup)
    pairs = cfg.tokens * cfg.top_k
    flop = 6 * cfg.hidden * (pairs * cfg.inter + cfg.tokens * cfg.n_shared * cfg.shared_inter)
    tf = flop / (mean["expert_ffn"] * 1e-6) / 1e12
    al = bufs.allow.cpu()
    counts = bufs.expert_count.cpu()
    res = {"workload": "deepseek-v2-lite-shaped layer, 16 requests x 512 tokens, allow/deny at 0.5",
           "tokens_per_s": cfg.tokens / (ms * 1e-3), "ms_per_step": ms,
           "experts_empty": int((counts == 0).sum()), "ffn_flop": flop, "ffn_us_mean": mean["expert_ffn"],
           "ffn_tflops": tf, "ffn_mfma_frac": tf / PEAK_BF16_TFLOPS, "calls_us_mean": mean,
           "calls_us_p10": p10, "calls_us_p90": p90,
           "calls_hbm": kernel_rates(call_bytes(cfg, counts, cfg.tokens, bool(al.any()),
                                                bool((al == 0).any())), mean)}
    del layer, x, bufs
    torch.cuda.empty_cache()
    return res


def stack_bench(args, dev):
    """The 48-layer Qwen-shaped stack (16384 tokens in 32 requests of 512, attention
    replaced by identity, h <- bf16(h + MoE(h)), independent weights per layer, 72.5 GB on
    the device): one all-allow and one all-deny pass, each timed whole after a warm-up
    pass, with the summed private-row audit."""
    import torch
    import workloads as W
    import paper_2608_06690_amd as P
    cfg = W.get_config("stack")
    L, T = cfg.layers, cfg.tokens
    desc = P.make_desc(cfg.hidden, cfg.inter, cfg.n_pub, cfg.n_priv, cfg.top_k)
    layers = []
    for ell in range(L):
        Lw = W.make_layer(cfg, ell, dev)
        layers.append(P.PolicyMaskedMoE(desc, Lw.wr_pub, Lw.wr_priv, Lw.bias, Lw.w13_pub, Lw.w2_pub,
                                        Lw.w13_priv, Lw.w2_priv))
    x0 = W.make_x(cfg, dev)
    bufs = layers[0].buffers(T)
    stream = torch.cuda.current_stream()
    flop_layer = T * cfg.top_k * 6 * cfg.hidden * cfg.inter
    res = {"workload": "48-layer qwen3-30b-a3b-shaped moe stack, 32 requests x 512 tokens",
           "layers": L, "tokens": T, "flop_per_pass": flop_layer * L}
    for p, kind in ((0, "allow"), (1, "deny")):
        req = W.make_requests(cfg, p)
        words = P.token_policy_words(req.metas, req.lengths, dev)
        req_off = P.request_offsets(req.lengths, dev)
        audit = layers[0].audit_buffers(T, cfg.requests)

        def one_pass(events=None):
            h = x0.clone()
            audit.zero_()
            for ell, layer in enumerate(layers):
                layer.route(h, words, bufs, stream)
                layer.dispatch(h, bufs, stream)
                if events:
                    events[ell][0].record(stream)
                layer.expert_ffn(h, bufs, audit, stream)
                if events:
                    events[ell][1].record(stream)
                layer.combine(h, bufs, stream)
                h = (h.float() + bufs.out.float()).to(torch.bfloat16)
            layers[0].audit(T, bufs, audit, req_off, stream)
            return h

        one_pass()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        one_pass()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(L)]
        one_pass(ev)
        torch.cuda.synchronize()
        ffn_us = sum(a.elapsed_time(b) for a, b in ev) * 1e3
        res[kind] = {"pass_ms": wall * 1e3, "layer_tokens_per_s": T * L / wall,
                     "ffn_us_per_layer": ffn_us / L,
                     "ffn_tflops": flop_layer * L / (ffn_us * 1e-6) / 1e12,
                     "ffn_mfma_frac": flop_layer * L / (ffn_us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS,
                     "private_rows_audited": int(audit.total.item()),
                     "private_rows_expected": L * T * cfg.top_k if kind == "allow" else 0,
                     "deny_violations": int(audit.violations.item())}
    del layers, bufs
    torch.cuda.empty_cache()
    return res


def fingerprint_bench(args, dev):
    """Fingerprint of one Qwen-shaped layer's public expert weights (w13 and w2, bf16):
    per-call time and the rate against the integer-VALU bound of SHA-256."""
    import torch
    import workloads as W
    import paper_2608_06690_amd as P
    cfg = W.get_config("qwen")
    Lw = W.make_layer(cfg, 0, dev)
    bufs = [Lw.w13_pub, Lw.w2_pub]
    nbytes = sum(t.numel() * t.element_size() for t in bufs)
    for _ in range(max(1, args.warmup // 2)):
        P.fingerprint_tensors(*bufs)
    torch.cuda.synchronize()
    reps = max(3, args.steps // 5)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        P.fingerprint_tensors(*bufs)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    gbs = nbytes / (us * 1e-6) / 1e9
    peak_gbs = PEAK_VALU_OPS / (SHA256_OPS_PER_BLOCK / 64) / 1e9
    del Lw, bufs
    torch.cuda.empty_cache()
    return {"workload": "public expert weights of one qwen3-30b-a3b-shaped layer (w13 + w2, bf16)",
            "bytes": nbytes, "us_per_call": us, "gbs": gbs, "bound": "alu",
            "peak_gbs": peak_gbs, "frac": gbs / peak_gbs, "reps": reps}


def backward_bench(args, dev):
    """Private-only backward of the Qwen-shaped layer (4 allow + 4 deny requests) after
    its forward: per-call time and the MFMA rate of its GEMM work."""
    import torch
    import workloads as W
    cfg, layer, x, words, req_off, audit, bufs, req = setup("qwen", dev)
    # training forward: keeps the gate and up projections for the backward
    layer.forward(x, words, audit, req_off, train=True)
    dout = W.make_dout(cfg, device=dev)
    g = layer.grad_buffers(cfg.tokens)
    for _ in range(max(1, args.warmup // 2)):
        layer.backward(x, dout, bufs, g)
    torch.cuda.synchronize()
    reps = max(5, args.steps // 2)
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        layer.backward(x, dout, bufs, g)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3)
    us = sum(times) / len(times)
    # one AdamW step over the private parameters (fp32 router rows; bf16 experts with fp32
    # master copies): read p, g, m, v and write p, m, v (+ the bf16 weight) per element
    import paper_2608_06690_amd as P
    opt = P.PrivateAdamW(layer, lr=1e-4)
    opt.step(g)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        opt.step(g)
    e1.record()
    torch.cuda.synchronize()
    opt_us = e0.elapsed_time(e1) * 1e3 / reps
    n_f32 = layer.wr_priv.numel()
    n_bf16 = layer.w13_priv.numel() + layer.w2_priv.numel()
    # the step also remakes the backward's transposed copies of the private experts
    # (read and write 2 bytes per bf16 weight), once per step instead of once per backward
    opt_bytes = 28 * n_f32 + 30 * n_bf16 + 4 * n_bf16
    counts = bufs.expert_count.cpu()
    R = cfg.tokens * cfg.top_k
    Rp = int(counts[cfg.n_pub:].sum())
    H, I = cfg.hidden, cfg.inter
    # algorithmic: dh (2 R H I) and row input gradients (4 R I H) over every row, weight
    # gradients (6 Rp H I) over the private rows (the gate and up projections come from
    # the training forward)
    alg = 6 * H * I * (R + Rp)
    executed = alg
    res = {"workload": "qwen3-30b-a3b-shaped layer backward, private experts and private "
                       "router rows trainable, 4 allow + 4 deny requests",
           "us_per_call": us, "us_p10": sorted(times)[len(times) // 10],
           "us_p90": sorted(times)[min(len(times) - 1, 9 * len(times) // 10)],
           "rows": R, "private_rows": Rp, "flop_algorithmic": alg, "flop_executed": executed,
           "tflops_algorithmic": alg / (us * 1e-6) / 1e12,
           "tflops_executed": executed / (us * 1e-6) / 1e12,
           "frac_algorithmic": alg / (us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, "reps": reps,
           "optimizer": {"kind": "AdamW over the private parameters only, then the transposed "
                                 "copies of the private expert weights that the backward uses",
                         "params": n_f32 + n_bf16, "us_per_step": opt_us, "bytes": opt_bytes,
                         "hbm_gbs": opt_bytes / (opt_us * 1e-6) / 1e9,
                         "hbm_frac": opt_bytes / (opt_us * 1e-6) / 1e9 / PEAK_HBM_GBS}}
    del layer, x, bufs, g, dout, opt
    torch.cuda.empty_cache()
    return res


def fp8_bench(args, dev):
    """Precision variant, not the bf16 metric: the expert FFN with fp8 (e4m3) weights and
    power-of-two row scales, on the Qwen-shaped prefill layer and the decode batch (L2/MALL
    flushed before each decode call)."""
    import torch
    import workloads as W
    import paper_2608_06690_amd as P
    res = {}
    for wl in ("qwen", "decode"):
        cfg, layer, x, words, req_off, audit, bufs, req = setup(wl, dev)
        parts = [W.quantize_fp8_rows(t)[:2] for t in (layer.w13_pub, layer.w2_pub, layer.w13_priv, layer.w2_priv)]
        fp8 = tuple(p[0] for p in parts) + tuple(p[1] for p in parts)
        d8 = P.make_desc(cfg.hidden, cfg.inter, cfg.n_pub, cfg.n_priv, cfg.top_k)
        d8.w_dtype = P.PMPE_FP8_E4M3
        layer.route(x, words, bufs)
        layer.dispatch(x, bufs)
        flush = torch.zeros(512 << 20, dtype=torch.uint8, device=dev) if wl == "decode" else None

        def call():
            P.pmpe_expert_ffn_fp8(d8, cfg.tokens, bufs.x_perm, x, bufs.expert_count,
                                  bufs.expert_offset, bufs.row_token, *fp8, bufs.y_perm,
                                  audit.token_rows, audit.priv_calls, bufs.dev_status, bufs.ws)

        for _ in range(3):
            call()
        torch.cuda.synchronize()
        times = []
        for _ in range(max(10, args.steps // 2)):
            if flush is not None:
                evict_caches(flush)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            call()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) * 1e3)
        us = sum(times) / len(times)
        counts = bufs.expert_count.cpu()
        touched = int((counts > 0).sum())
        wbytes = touched * 3 * cfg.hidden * cfg.inter  # one byte per weight
        flop = cfg.tokens * cfg.top_k * 6 * cfg.hidden * cfg.inter
        res[wl] = {"ffn_us_mean": us, "weight_bytes_fp8": wbytes,
                   "weight_gbs": wbytes / (us * 1e-6) / 1e9,
                   "weight_hbm_frac": wbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS,
                   "tflops": flop / (us * 1e-6) / 1e12,
                   "flushed": flush is not None}
        del layer, x, bufs, fp8, parts, flush
        torch.cuda.empty_cache()
    return {"kind": "fp8 e4m3 expert weights with power-of-two row scales (precision "
                    "variant; the metric line is bf16)", **res}


def vendor_gemm_bench(dev, reps=20):
    """Context only: hipBLASLt (torch.bmm) on the Qwen layer's per-expert GEMM shapes with
    uniform rows (128 per public expert, 512 per private expert), without the SwiGLU, the
    row gather, the ragged expert sizes or the audit that the expert FFN kernel fuses in.
    Weights are contiguous [E, K, N] tensors: bf16 batched products with a transposed view
    as the right operand are avoided (they have faulted the GPU)."""
    import torch
    H, I = 2048, 768

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    g = torch.Generator(device=dev).manual_seed(1)
    res = {}
    for name, E, R in (("public", 128, 128), ("private", 32, 512)):
        x = torch.randn(E, R, H, device=dev, dtype=torch.bfloat16, generator=g)
        hh = torch.randn(E, R, I, device=dev, dtype=torch.bfloat16, generator=g)
        w13 = torch.randn(E, H, 2 * I, device=dev, dtype=torch.bfloat16, generator=g).contiguous()
        w2 = torch.randn(E, I, H, device=dev, dtype=torch.bfloat16, generator=g).contiguous()
        o1 = torch.empty(E, R, 2 * I, device=dev, dtype=torch.bfloat16)
        o2 = torch.empty(E, R, H, device=dev, dtype=torch.bfloat16)
        g1 = timed(lambda: torch.bmm(x, w13, out=o1))
        g2 = timed(lambda: torch.bmm(hh, w2, out=o2))
        res[name] = {"experts": E, "rows_per_expert": R, "gemm1_us": g1, "gemm2_us": g2}
        del x, hh, w13, w2, o1, o2
        torch.cuda.empty_cache()
    total = sum(v["gemm1_us"] + v["gemm2_us"] for v in res.values())
    flop = 32768 * 6 * H * I
    return {"library": "hipBLASLt via torch.bmm", "pools": res, "total_us": total,
            "tflops": flop / (total * 1e-6) / 1e12}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the layer is single-GPU and no multi-GPU path is "
              f"built (asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    import torch
    import workloads as W

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        src = torch.ones(COPY_BYTES // 2, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 5
        print(json.dumps({"copy_bytes": COPY_BYTES, "copy_us": ms * 1e3,
                          "read_plus_write_gbs": 2 * COPY_BYTES / (ms * 1e-3) / 1e9}), flush=True)
        return
    if args.read_probe:
        # the decode workload's weight volume (96 experts x 9,437,184 bytes), read once
        nbytes = 96 * 3 * 2048 * 768 * 2
        src = torch.ones(nbytes // 2, dtype=torch.bfloat16, device=dev)
        flush = torch.zeros(512 << 20, dtype=torch.uint8, device=dev)
        out = {"bytes": nbytes}
        for name, fn in (("sum_bf16", lambda: src.sum(dtype=torch.float32)),
                         ("amax_bf16", lambda: src.amax())):
            ts = []
            for i in range(8):
                evict_caches(flush)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                fn()
                e1.record()
                torch.cuda.synchronize()
                if i >= 2:
                    ts.append(e0.elapsed_time(e1) * 1e3)
            us = sorted(ts)[len(ts) // 2]
            out[name] = {"us_median": us, "gbs": nbytes / (us * 1e-6) / 1e9,
                         "hbm_frac": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}
        print(json.dumps(out), flush=True)
        return
    if args.decode_only:
        print(json.dumps(decode_bench(args, dev)), flush=True)
        return
    if args.deepseek_only:
        print(json.dumps(deepseek_bench(args, dev)), flush=True)
        return
    if args.fp8_only:
        print(json.dumps(fp8_bench(args, dev)), flush=True)
        return
    if args.backward_only:
        print(json.dumps(backward_bench(args, dev)), flush=True)
        return
    if args.vendor_gemm:
        print(json.dumps(vendor_gemm_bench(dev)), flush=True)
        return
    if args.stack_only:
        print(json.dumps(stack_bench(args, dev)), flush=True)
        return
    if args.fingerprint_only:
        print(json.dumps(fingerprint_bench(args, dev)), flush=True)
        return
    if args.all_deny:
        cfg, layer, x, words, req_off, audit, bufs, req = setup("qwen", dev, all_deny=True,
                                                                drop_private=args.no_private_weights)
        ms, med, mean, p10, p90 = time_layer(layer, x, words, req_off, audit, bufs, args.steps, args.warmup)
        counts = bufs.expert_count.cpu()
        touched = int((counts > 0).sum())
        print(json.dumps({"workload": "qwen3-30b-a3b-shaped layer, 8 requests x 512 tokens, all denied",
                          "private_tensors": "NULL" if args.no_private_weights else "present",
                          "ms_per_step": ms, "private_rows_routed": int(counts[cfg.n_pub:].sum()),
                          "private_rows_executed": int(audit.total.item()),
                          "public_experts_touched": touched,
                          "public_weight_bytes": touched * 3 * cfg.hidden * cfg.inter * 2,
                          "calls_us_mean": mean}), flush=True)
        return
    cfg, layer, x, words, req_off, audit, bufs, req = setup("qwen", dev)
    ms, med, mean, p10, p90 = time_layer(layer, x, words, req_off, audit, bufs, args.steps, args.warmup)
    T = cfg.tokens
    pairs = T * cfg.top_k
    ffn_flop = pairs * 2 * 3 * cfg.hidden * cfg.inter
    w_bytes = cfg.n_experts * 3 * cfg.hidden * cfg.inter * 2
    ffn_us = mean["expert_ffn"]
    achieved = ffn_flop / (ffn_us * 1e-6) / 1e12
    ai = ffn_flop / w_bytes
    attainable = min(PEAK_BF16_TFLOPS, ai * PEAK_HBM_GBS / 1e3)
    out = {
        "metric": METRIC, "value": T / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "qwen3-30b-a3b-shaped policy-masked moe layer", "tokens": T,
                   "requests": cfg.requests, "hidden": cfg.hidden, "inter": cfg.inter,
                   "n_pub": cfg.n_pub, "n_priv": cfg.n_priv, "top_k": cfg.top_k,
                   "policy": "4 allow + 4 deny requests", "router": "fp32", "experts": "bf16"},
        "roofline": {"kernel": "pmpe_expert_ffn (gemm_bf16_kernel GEMM1 + GEMM2)",
                     "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": FFN_TRAFFIC_BYTES.get(ffn_source_hash()),
                     "flop_per_launch": ffn_flop, "avg_us": ffn_us,
                     "weight_bytes": w_bytes, "ai_flop_per_weight_byte": ai,
                     "attainable_tflops_at_hbm_peak": attainable,
                     "attainable_frac": achieved / attainable},
        "calls_us_mean": mean, "calls_us_median": med, "calls_us_p10": p10, "calls_us_p90": p90,
    }
    allow = bufs.allow.cpu()
    out["calls_hbm"] = kernel_rates(call_bytes(cfg, bufs.expert_count.cpu(), T, bool(allow.any()),
                                               bool((allow == 0).any())), mean)
    del layer, x, bufs
    torch.cuda.empty_cache()

    if not args.no_decode:
        out["decode"] = decode_bench(args, dev)
    if not args.no_deepseek:
        out["deepseek"] = deepseek_bench(args, dev)
    if args.stack:
        out["stack"] = stack_bench(args, dev)
    if not args.no_backward:
        out["backward"] = backward_bench(args, dev)
    if not args.no_fingerprint:
        out["fingerprint"] = fingerprint_bench(args, dev)
    if not args.no_fp8:
        out["fp8_weights"] = fp8_bench(args, dev)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, req, args.cpu_sample, args.cpu_reps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
