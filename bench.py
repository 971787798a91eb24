"""Benchmark of the WUSH-KV hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Headline workload (one GPU): large-batch decode attention over a 2-bit
WUSH-KV cache -- batch 64, 32 query / 8 kv heads, head_dim 128, ragged
contexts drawn uniformly from [16384, 32768] tokens, 4 sink + 128 recent
bf16 tokens and flushes of 8 -- the largest of the decode workloads that
fits one GPU.  The cache (about 0.94 GB of packed codes and parameters) is
filled by the library's own prefill appends from seeded synthetic keys and
values of the workload's distribution (Gaussian keys with 8 outlier
channels x10, RoPE theta 5e5; Gaussian values) and per-head transforms
T_K = Q diag(s) Q^T.  One step is one decode call: q~ = q^T T_K^-1, split-K
attention over the packed pages and the bf16 windows, and the split merge.

Reported value: algorithmic HBM bytes of a call (72 B per quantised
token-head, 512 B per bf16 window token-head, queries, transforms, outputs,
page table) over the call time, in GB/s: after W warm-up calls, one call
captured in a HIP graph and replayed K times back to back, bracketed by
device synchronisations (the same K calls launched from the host one by one
are reported beside it).  The roofline object
is the dominant kernel, decode_main_kernel, over at least 100 launches
stamped by HIP events on the launch stream.  The second half of the metric,
append throughput, is measured on the prefill workload (4 x 16384 new
tokens, QK-norm + RoPE theta 1e6 inputs, Student-t keys) and reported in
tokens/s; the Llama-3-8B-shaped decode step (append + attention + flush,
batch 8, 8192 tokens) and the other decode sizes are reported beside it.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
MALL_BYTES = 256 << 20


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU seconds (summed over threads) the oracle baseline runs for")
    ap.add_argument("--no-prefill", action="store_true", help="skip the append-throughput leg")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline leg")
    ap.add_argument("--prefill-only", action="store_true",
                    help="only run the append-throughput leg and print its JSON object")
    ap.add_argument("--no-scale", action="store_true",
                    help="skip the decode legs at the long-context and large-batch sizes")
    ap.add_argument("--wush-only", action="store_true",
                    help="only the transform-builder leg (all K/V heads of an 8B-shaped model)")
    ap.add_argument("--scale-only", action="store_true",
                    help="only run the long-context / large-batch decode legs")
    ap.add_argument("--chunk-only", action="store_true",
                    help="only the Llama-shaped step and chunk-attention legs")
    ap.add_argument("--headline-only", action="store_true",
                    help="only the large-batch decode headline (no oracle, no other legs)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 512 MiB device-to-device copy five times (a known-size "
                         "reference for the HBM byte counters) and exit")
    return ap.parse_args()


def profiled_traffic(summary, csrc, key="traffic_bytes_per_launch"):
    """HBM bytes per launch from a committed counter summary, or None when
    the kernel sources changed since the counters were taken (the summary
    records a sha256 prefix of each source it covers)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", summary)
    if not os.path.exists(path):
        return None
    fields = {}
    for ln in open(path):
        if ":" in ln and not ln.startswith(("|", " ", "#")):
            k_, v_ = ln.split(":", 1)
            fields[k_.strip()] = v_.strip()
    try:
        value = int(fields[key])
        want = dict(x.split("=") for x in fields["source_sha256_prefix"].split())
    except (KeyError, ValueError):
        return None
    for name, pre in want.items():
        with open(os.path.join(csrc, name), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest()[:len(pre)] != pre:
                return None
    return value


def copy_calibration():
    """A plain copy of known size: 512 MiB read and 512 MiB written per
    launch.  Profiling it with the same byte counters as the kernels gives
    the factor that turns counter readings into bytes."""
    import torch
    n = 512 << 20
    src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    assert torch.equal(dst[:4096], src[:4096])
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}), flush=True)


# ----------------------------------------------------------------- bytes

def decode_bytes(seq_len, quant_end, s_sink, n_kv, n_q, d, bits, page_tokens=64):
    """Algorithmic bytes one decode call must move."""
    per_q = 2 * d * bits // 8 + 8          # codes K+V and two fp16 (scale, zero) pairs
    per_w = 4 * d                          # bf16 K and V
    q_tok = w_tok = pages = 0
    for S, Q in zip(seq_len, quant_end):
        qe = min(max(Q, s_sink), S) if S > s_sink else S
        nq = max(0, qe - s_sink) if S > s_sink else 0
        q_tok += nq
        w_tok += S - nq
        pages += math.ceil(nq / page_tokens)
    B = len(seq_len)
    main = n_kv * (q_tok * per_q + w_tok * per_w)
    other = B * n_q * d * 2 + n_kv * d * d * 4 + B * n_q * d * 4 + B * pages * 4
    return main, other


def append_step_bytes(B, n_kv, d, bits, n_new, n_flushed):
    """One append call in which every sequence adds n_new tokens that stay in
    the bf16 ring and flushes n_flushed ring tokens into pages: bf16 K and V
    in, the window writes, the flushed tokens' ring reads and packed writes,
    and T_K once."""
    per_q = 2 * d * bits // 8 + 8
    per_seq_head = n_new * 4 * d + n_new * 4 * d + n_flushed * (4 * d + per_q)
    return B * n_kv * per_seq_head + n_kv * d * d * 2


def prefill_bytes(B, n_kv, d, bits, n_new, n_quant):
    """An append into an empty cache: bf16 K and V in, packed writes of the
    n_quant quantised tokens, bf16 writes of the rest, T_K once."""
    per_q = 2 * d * bits // 8 + 8
    per_seq_head = n_new * 4 * d + n_quant * per_q + (n_new - n_quant) * 4 * d
    return B * n_kv * per_seq_head + n_kv * d * d * 2


def window_quant_end(S, s_sink, s_keep, s_flush):
    """S_quant of a cache filled to S positions (window rule of Alg. 2,
    restated here for byte accounting; the kernels compute their own)."""
    start = s_sink
    return max(0, start + ((S - s_keep - start) // s_flush) * s_flush)


# ----------------------------------------------------------------- main

def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(every (sequence, kv head) pair is independent; see the design notes "
              "for how it would shard).  Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_38121_amd as wk
    from workloads import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.prefill_only:
        print(json.dumps(bench_prefill(torch, wk, synth, dev, args)), flush=True)
        return
    if args.scale_only:
        print(json.dumps(bench_decode_scale(torch, wk, synth, dev, args)), flush=True)
        return
    if args.wush_only:
        print(json.dumps(bench_wush(torch, wk, dev, args)), flush=True)
        return

    if args.chunk_only:
        _, state = bench_llama_step(torch, wk, synth, dev, args)
        print(json.dumps(bench_chunk(torch, wk, *state)), flush=True)
        return

    # ---- headline: large-batch decode (timed first, on a fresh device)
    head, sample = bench_bigbatch(torch, wk, synth, dev, args)
    extra = {}
    if not args.headline_only:
        # ---- the Llama-shaped decode step, append throughput, chunk
        # attention, the other decode sizes, the streaming-read reference
        # and the transform builder
        extra["llama8b_step"], state = bench_llama_step(torch, wk, synth, dev, args)
        if not args.no_prefill:
            extra["append"] = bench_prefill(torch, wk, synth, dev, args)
        if not args.no_scale:
            extra["chunk_attention"] = bench_chunk(torch, wk, *state)
            extra["decode_at_scale"] = bench_decode_scale(torch, wk, synth, dev, args)
        extra["stream_read"] = bench_stream_read(torch, wk, dev)
        if not args.no_scale:
            extra["wush_build"] = bench_wush(torch, wk, dev, args)
    cpu = None
    if not args.no_cpu and not args.headline_only:
        cpu = bench_oracle(sample, args.cpu_seconds)

    line = {
        "metric": "decode-attn achieved HBM GB/s (% of peak) on 2-bit cache; append tokens/s",
        "value": head["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": head["steps"],
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "pct_of_peak": round(100 * head["value"] / PEAK_HBM_GBS, 2),
        "config": head["config"],
        "call_us": head["call_us"],
        "roofline": head["roofline"],
        "cpu_baseline": cpu,
        "kernel_us": head["kernel_us"],
    }
    if "append" in extra and extra["append"] is not None:
        line["append_tokens_per_s"] = extra["append"]["tokens_per_s"]
    line.update(extra)
    print(json.dumps(line), flush=True)


def _pct(xs, q):
    return float(np.percentile(np.asarray(xs, np.float64), q))


def bench_bigbatch(torch, wk, synth, dev, args):
    """The headline: decode calls on the large-batch workload (batch 64,
    ragged 16384-32768 tokens, 2-bit).  The cache is filled by prefill
    appends (4096-token chunks) of seeded device-side keys and values with
    the workload's distribution: Gaussian keys with the workload's 8 outlier
    channels scaled x10, rotated by RoPE (theta 5e5) at their positions, and
    Gaussian values; T_K is the workload's per-head Q diag(s) Q^T.  K timed
    calls back to back after W warm-up calls; then at least 100 more calls
    with each kernel stamped by HIP events on the launch stream (median /
    p10 / p90 per launch).  Returns (result, the inputs of two sequences for
    the oracle baseline)."""
    name = "bigbatch"
    cfg = synth.CONFIGS[name]
    w = synth.Workload(cfg, seed=args.seed)
    B, H, NQ, D, BITS = cfg["batch"], cfg["n_kv"], cfg["n_q"], cfg["d"], cfg["bits"]
    lengths = w.lengths.astype(np.int64)
    cap = cfg["ctx"] + 64  # capacity and split plan: the workload's longest context + 64
    t0 = time.time()
    cache = wk.WushKVCache(B, H, D, BITS, cfg["s_sink"], cfg["s_keep"], cfg["s_flush"],
                           cfg["kappa_k"], cfg["kappa_v"], max_seq_len=cap, seed=args.seed,
                           device=dev)
    tk_bits, tinv = w.transform()
    as_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    tk = as_dev(tk_bits)
    tinv_d = torch.from_numpy(tinv).to(dev)
    table = torch.from_numpy(synth.rope_table(cfg["rope_theta"], D, cap)).to(dev)
    half = D // 2
    out_ch = torch.from_numpy(w.k_outlier_ch.astype(np.int64)).to(dev)
    gen = torch.Generator(device=dev).manual_seed(1000 + args.seed)
    # the oracle baseline's sample: every kv head of two sequences (the
    # shortest and the longest), their inputs copied out as they are made
    sample_seqs = [int(np.argmin(lengths)), int(np.argmax(lengths))]
    sample_k = {b: [] for b in sample_seqs}
    sample_v = {b: [] for b in sample_seqs}
    chunk = 4096
    done = np.zeros(B, np.int64)
    while (done < lengths).any():
        n = np.minimum(chunk, lengths - done)
        m = int(n.max())
        p0 = int(done[n > 0].min())  # every sequence still growing is at this position
        assert np.all(done[n > 0] == p0)
        x = torch.randn(B, m, H, D, generator=gen, device=dev)
        x[..., out_ch] *= float(cfg["outlier_scale"])
        cs = table[p0:p0 + m, :half][None, :, None, :]
        sn = table[p0:p0 + m, half:][None, :, None, :]
        x1, x2 = x[..., :half], x[..., half:]
        k = torch.cat([x1 * cs - x2 * sn, x2 * cs + x1 * sn], dim=-1).to(torch.bfloat16)
        v = torch.randn(B, m, H, D, generator=gen, device=dev).to(torch.bfloat16)
        wk.wushkv_append(cache, k, v, torch.from_numpy(n.astype(np.int32)).to(dev), tk)
        for b in sample_seqs:
            if n[b]:
                sample_k[b].append(k[b, :n[b]].contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
                sample_v[b].append(v[b, :n[b]].contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
        done += n
        del x, k, v
    torch.cuda.synchronize()
    seq = cache.seq_len.cpu().numpy()
    qe = cache.quant_end.cpu().numpy()
    assert np.array_equal(seq, lengths)
    main_b, other_b = decode_bytes(seq, qe, cfg["s_sink"], H, NQ, D, BITS)
    call_bytes = main_b + other_b
    q_bits = w.query(0)
    q = as_dev(q_bits)
    sm = 1.0 / math.sqrt(D)
    ws = torch.empty(wk.wushkv_decode_workspace_bytes(cache, NQ, cap), dtype=torch.uint8, device=dev)
    out = torch.empty(B, NQ, D, dtype=torch.float32, device=dev)
    cache_bytes = cache.pages.numel() + 2 * cache.win_k.numel() * 2
    log("%s: cache %.2f GB (pool), %d tokens, built in %.1fs" % (name, cache_bytes / 1e9, int(seq.sum()),
                                                                 time.time() - t0))
    assert cache_bytes >= 2 * MALL_BYTES  # one replica already defeats the Infinity Cache

    def call():
        wk.wushkv_decode_attention(cache, q, tinv_d, sm_scale=sm, max_seq_len=cap, out=out,
                                   workspace=ws)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    K = max(1, args.steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # K calls launched from the host back to back (for reference: at this
    # size the host's launch path, not the device, can set the pace)
    torch.cuda.synchronize()
    e0.record()
    for i in range(K):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms_eager = e0.elapsed_time(e1) / K
    # the timed steps: one call captured in a HIP graph, replayed K times
    g = torch.cuda.CUDAGraph()
    cap_stream = torch.cuda.Stream()
    cap_stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap_stream):
        with torch.cuda.graph(g, stream=cap_stream):
            call()
    torch.cuda.current_stream().wait_stream(cap_stream)
    torch.cuda.synchronize()
    g.replay()  # untimed: the capture itself ran nothing
    torch.cuda.synchronize()
    t_host = time.perf_counter()
    e0.record()
    for i in range(K):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    t_host = time.perf_counter() - t_host
    ms_call = e0.elapsed_time(e1) / K
    value = call_bytes / (ms_call * 1e-3) / 1e9
    log("%s decode: %d calls (graph replays), %.2f us per call (host clock %.2f us), %.1f GB/s "
        "(%.1f%% of 8 TB/s); launched from the host one by one %.2f us per call"
        % (name, K, ms_call * 1e3, t_host / K * 1e6, value, value / 80, ms_eager * 1e3))
    # the spread of single calls: at least 100 more, an event pair around each
    NC = max(K, 100)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * NC)]
    for i in range(NC):
        ev[2 * i].record()
        call()
        ev[2 * i + 1].record()
    torch.cuda.synchronize()
    per_call = [ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(NC)]

    # per-launch kernel durations: at least 100 calls, every kernel stamped
    NT = max(K, 100)
    wk.wushkv_timing_enable(4 * NT)
    for _ in range(NT):
        call()
    torch.cuda.synchronize()
    per = wk.wushkv_timing_launches()
    wk.wushkv_timing_enable(0)
    kern = {}
    for nm, ms in per:
        kern.setdefault(nm, []).append(ms * 1e3)
    main_us = kern["decode_main_kernel"]
    avg = float(np.mean(main_us))
    achieved = main_b / (avg * 1e-6) / 1e9
    log("decode_main_kernel: %d launches, avg %.2f us (median %.2f, p10 %.2f, p90 %.2f): %.1f GB/s, "
        "frac %.3f" % (len(main_us), avg, _pct(main_us, 50), _pct(main_us, 10), _pct(main_us, 90),
                       achieved, achieved / PEAK_HBM_GBS))
    res = {
        "value": round(value, 2),
        "steps": K,
        "ms_per_step": round(ms_call, 5),
        "call_us": {"mean": round(ms_call * 1e3, 3), "timed_as": "HIP graph of one call, replayed",
                    "host_launched_mean": round(ms_eager * 1e3, 3),
                    "single_calls": NC, "median": round(_pct(per_call, 50) * 1e3, 3),
                    "p10": round(_pct(per_call, 10) * 1e3, 3), "p90": round(_pct(per_call, 90) * 1e3, 3)},
        "config": {"workload": "large-batch decode: batch 64, 32 q / 8 kv heads, head_dim 128, "
                               "ragged ctx uniform in [16384, 32768], 2-bit keys+values",
                   "batch": B, "n_q_heads": NQ, "n_kv_heads": H, "head_dim": D, "bits": BITS,
                   "ctx_min": int(lengths.min()), "ctx_max": int(lengths.max()),
                   "tokens": int(seq.sum()), "s_sink": cfg["s_sink"], "s_keep": cfg["s_keep"],
                   "s_flush": cfg["s_flush"], "kappa_k": cfg["kappa_k"], "kappa_v": cfg["kappa_v"],
                   "bytes_per_call": int(call_bytes),
                   "step": "one wushkv_decode_attention call (q~ launch, main kernel, split merge)"},
        "roofline": {"bound": "hbm", "kernel": "decode_main_kernel",
                     "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": profiled_traffic("decode_main_kernel_bigbatch_2bit.md",
                                                 os.path.join(ROOT, "paper_2609_38121_amd", "csrc")),
                     "avg_us": round(avg, 3), "median_us": round(_pct(main_us, 50), 3),
                     "p10_us": round(_pct(main_us, 10), 3), "p90_us": round(_pct(main_us, 90), 3),
                     "launches": len(main_us), "bytes_per_launch": int(main_b),
                     "timing": "HIP start/stop events of each launch on its stream "
                               "(hipExtLaunchKernelGGL)"},
        "kernel_us": {nm: {"avg": round(float(np.mean(v_)), 3), "median": round(_pct(v_, 50), 3)}
                      for nm, v_ in kern.items()},
    }
    sample = {"cfg": cfg, "seqs": sample_seqs,
              "k": {b: np.concatenate(sample_k[b]) for b in sample_seqs},
              "v": {b: np.concatenate(sample_v[b]) for b in sample_seqs},
              "q": q_bits, "tk": tk_bits, "tinv": tinv, "lengths": lengths}
    del g, cache, ws, out
    torch.cuda.empty_cache()
    return res, sample


def bench_dequant(torch, wk, cache, B, H, D, bits, s_sink):
    """Reconstruction of stored entries (wushkv_dequant, Eq. (7)'s x =
    scale code + zero) of every quantised position of each sequence of a
    Llama-shaped cache: one launch per sequence, fp32 K and V out
    [kv heads][positions][d], the outputs rotated over four buffer pairs
    (beyond the 256 MB Infinity Cache).  Algorithmic bytes per launch: the
    codes and the two (scale, zero) pairs per token-head read (d bits / 4 +
    8 B: 72 B at d 128, 2 bits), 8 d B per token-head written; timed by the
    library's per-launch events."""
    qe = cache.quant_end.cpu().numpy()
    count = int(qe.min()) - s_sink
    outs = [(torch.empty((H, count, D), dtype=torch.float32, device=cache.device),
             torch.empty((H, count, D), dtype=torch.float32, device=cache.device)) for _ in range(4)]
    for b in range(B):
        wk.wushkv_dequant(cache, b, s_sink, count, *outs[b % 4])
    torch.cuda.synchronize()
    rounds = 4
    wk.wushkv_timing_enable(rounds * B + 8)
    for r in range(rounds):
        for b in range(B):
            wk.wushkv_dequant(cache, b, s_sink, count, *outs[(r * B + b) % 4])
    torch.cuda.synchronize()
    cnt, tot = wk.wushkv_timing_read("dequant_kernel")
    wk.wushkv_timing_enable(0)
    t = tot / cnt * 1e-3  # seconds per launch
    per_launch = H * count * (D * bits // 4 + 8 + 8 * D)
    ach = per_launch / t / 1e9
    del outs
    log("dequant: %d positions x %d kv heads per launch, %.1f us, %.1f GB/s" % (count, H, t * 1e6, ach))
    return {"positions_per_launch": count, "kv_heads": H, "launches": int(cnt),
            "roofline": {"bound": "hbm", "kernel": "dequant_kernel", "achieved": round(ach, 2),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                         "traffic": None, "avg_us": round(t * 1e6, 3), "bytes_per_launch": int(per_launch)}}


def bench_llama_step(torch, wk, synth, dev, args):
    """The Llama-3-8B-shaped decode layer (batch 8, 32 query / 8 kv heads,
    d 128, 8192-token context, 2-bit): one step appends one token per
    sequence (key transform, window routing, the flush when due) and decodes
    over the updated cache.  The cache is built by a prefill append and
    replicated past the 256 MB Infinity Cache; the step loop runs as a
    captured HIP graph.  Reported for the fused step (wushkv_decode_step,
    Alg. 2's order, two launches) and the separate calls, with the decode
    kernel's roofline at this size.  Returns (result dict, state for the
    chunk leg)."""
    steps = min(max(args.steps, 48), 400)
    cfg = synth.CONFIGS["llama8b"]
    w = synth.Workload(cfg, seed=args.seed)
    B, H, NQ, D, BITS = cfg["batch"], cfg["n_kv"], cfg["n_q"], cfg["d"], cfg["bits"]
    ctx = cfg["ctx"]
    as_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    # ---- build the cache by a prefill append of the context
    log("generating %d x %d tokens" % (B, ctx))
    t0 = time.time()
    k = np.stack([w.keys(b, 0, ctx) for b in range(B)])
    v = np.stack([w.values(b, 0, ctx) for b in range(B)])
    tk_bits, tinv = w.transform()
    log("  %.1fs" % (time.time() - t0))
    # capacity and split plan: every replica takes at most (warmup + 2
    # replica rounds + 2 steps + 128) / replicas + 17 tokens here, far below
    # 512 for steps <= 400
    max_seq = ctx + 512
    base = wk.WushKVCache(B, H, D, BITS, cfg["s_sink"], cfg["s_keep"], cfg["s_flush"],
                          cfg["kappa_k"], cfg["kappa_v"], max_seq_len=max_seq)
    tk = as_dev(tk_bits)
    tinv_d = torch.from_numpy(tinv).to(dev)
    wk.wushkv_append(base, as_dev(k), as_dev(v), torch.full((B,), ctx, dtype=torch.int32, device=dev), tk)
    torch.cuda.synchronize()
    del k, v
    dequant = bench_dequant(torch, wk, base, B, H, D, BITS, cfg["s_sink"])
    cache_bytes = base.pages.numel() + 2 * base.win_k.numel() * 2
    reps = max(1, math.ceil(2 * MALL_BYTES / cache_bytes))
    caches = [base] + [base.clone() for _ in range(reps - 1)]
    log("cache %.1f MB x %d replicas" % (cache_bytes / 1e6, reps))

    # per-step inputs: one new token per sequence and the decode query
    k1 = as_dev(np.stack([w.keys(b, ctx, 1) for b in range(B)]))
    v1 = as_dev(np.stack([w.values(b, ctx, 1) for b in range(B)]))
    q = as_dev(w.query(0))
    ones = torch.ones(B, dtype=torch.int32, device=dev)
    sm = 1.0 / math.sqrt(D)
    ws_bytes = wk.wushkv_decode_workspace_bytes(base, NQ, max_seq)
    work = [torch.empty(ws_bytes, dtype=torch.uint8, device=dev) for _ in range(reps)]
    outs = [torch.empty(B, NQ, D, dtype=torch.float32, device=dev) for _ in range(reps)]

    def step(i):
        r = i % reps
        wk.wushkv_append(caches[r], k1, v1, ones, tk, max_new=1)
        wk.wushkv_decode_attention(caches[r], q, tinv_d, sm_scale=sm, max_seq_len=max_seq,
                                   out=outs[r], workspace=work[r])

    def decode_only(i):
        r = i % reps
        wk.wushkv_decode_attention(caches[r], q, tinv_d, sm_scale=sm, max_seq_len=max_seq,
                                   out=outs[r], workspace=work[r])

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    done = args.warmup

    # lengths are the same for every sequence; track them on the host
    def lengths_at(step_index):
        """(S, S_quant) of the replica that step step_index runs on, after
        that step's append: prefill of ctx, then one token per visit."""
        S = ctx + step_index // reps + 1
        return S, quant_end_after(S)

    def quant_end_after(S):
        return window_quant_end(S, cfg["s_sink"], cfg["s_keep"], cfg["s_flush"])

    # ---- timed region, graph-captured steps
    log("capturing %d steps (one per replica) in a HIP graph" % reps)
    g = torch.cuda.CUDAGraph()
    cap_stream = torch.cuda.Stream()
    cap_stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap_stream):
        # replaying the graph runs steps done .. done + reps - 1 again and again;
        # capture itself must not run the kernels twice, so record only
        with torch.cuda.graph(g, stream=cap_stream):
            for i in range(reps):
                step(done + i)
    torch.cuda.current_stream().wait_stream(cap_stream)
    torch.cuda.synchronize()
    # the capture enqueued nothing; replays advance every replica by one
    # token; at least `steps` steps are timed (whole replays)
    n_rep = max(1, -(-steps // reps))
    K = n_rep * reps
    g.replay()  # one untimed replay (warm)
    torch.cuda.synchronize()
    done += reps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(n_rep):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_graph = e0.elapsed_time(e1) / K
    first_timed = done
    done += K

    # algorithmic bytes of the timed steps
    tot_main = tot_other = tot_app = 0
    for i in range(first_timed, first_timed + K):
        S, Q = lengths_at(i)
        main_b, other_b = decode_bytes([S] * B, [Q] * B, cfg["s_sink"], H, NQ, D, BITS)
        Q_prev = quant_end_after(S - 1)
        flushed = max(0, Q - max(Q_prev, cfg["s_sink"]))
        tot_main += main_b
        tot_other += other_b
        tot_app += append_step_bytes(B, H, D, BITS, 1, flushed)
    step_gbs = (tot_main + tot_other + tot_app) / K / (ms_graph * 1e-3) / 1e9
    log("graph step: %.2f us, %.1f GB/s" % (ms_graph * 1e3, step_gbs))

    # ---- eager steps with per-launch kernel timing (roofline of the decode
    # kernel): the library launches each kernel with a start/stop event pair
    # that the runtime stamps at that kernel's start and end
    wk.wushkv_timing_enable(8 * 64)
    KT = 64
    e0.record()
    for i in range(KT):
        step(done + i)
    e1.record()
    torch.cuda.synchronize()
    ms_eager = e0.elapsed_time(e1) / KT
    kernels = {}
    for name in ("decode_main_kernel", "decode_qt_kernel", "decode_combine_kernel",
                 "append_step_kernel", "append_kernel"):
        n, tot = wk.wushkv_timing_read(name)
        kernels[name] = (tot / n) if n else None
    wk.wushkv_timing_enable(0)
    main_sum = 0
    for i in range(done, done + KT):
        S, Q = lengths_at(i)
        main_b, _ = decode_bytes([S] * B, [Q] * B, cfg["s_sink"], H, NQ, D, BITS)
        main_sum += main_b
    done += KT
    main_per_launch = main_sum / KT
    t_main = kernels["decode_main_kernel"]
    achieved = main_per_launch / (t_main * 1e-3) / 1e9
    log("decode_main_kernel: %.2f us avg, %.1f GB/s (%.1f%% of 8 TB/s); eager step %.2f us"
        % (t_main * 1e3, achieved, 100 * achieved / PEAK_HBM_GBS, ms_eager * 1e3))

    # ---- decode call alone (graph), for context
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.stream(cap_stream):
        with torch.cuda.graph(g2, stream=cap_stream):
            for i in range(reps):
                decode_only(i)
    torch.cuda.synchronize()
    g2.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(n_rep):
        g2.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_dec = e0.elapsed_time(e1) / K
    dec_bytes = 0
    for r in range(reps):
        S = ctx + (done - r + reps - 1) // reps  # appends replica r has seen
        mb, ob = decode_bytes([S] * B, [quant_end_after(S)] * B, cfg["s_sink"], H, NQ, D, BITS)
        dec_bytes += mb + ob
        # the host-side bookkeeping must agree with the device counters
        assert int(caches[r].seq_len[0].item()) == S
        assert int(caches[r].quant_end[0].item()) == quant_end_after(S)
    dec_gbs = dec_bytes / reps / (ms_dec * 1e-3) / 1e9
    log("decode call (graph): %.2f us, %.1f GB/s" % (ms_dec * 1e3, dec_gbs))

    # ---- the fused step (wushkv_decode_step): the same append + decode in
    # Alg. 2's own order (the flush after the attention), two launches.  It
    # leaves a cache exactly as the separate calls do, so it continues on the
    # same replicas; its attention reads the positions its flush quantises
    # at bf16.
    k1s, v1s = k1[:, 0].contiguous(), v1[:, 0].contiguous()

    def fused(i):
        r = i % reps
        wk.wushkv_decode_step(caches[r], k1s, v1s, ones, tk, q, tinv_d, sm_scale=sm,
                              max_seq_len=max_seq, out=outs[r], workspace=work[r])

    g3 = torch.cuda.CUDAGraph()
    with torch.cuda.stream(cap_stream):
        with torch.cuda.graph(g3, stream=cap_stream):
            for i in range(reps):
                fused(done + i)
    torch.cuda.synchronize()
    g3.replay()
    torch.cuda.synchronize()
    done += reps
    e0.record()
    for _ in range(n_rep):
        g3.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_fused = e0.elapsed_time(e1) / K
    fz_bytes = 0
    for i in range(done, done + K):
        S, Q = lengths_at(i)
        Q_prev = quant_end_after(S - 1)
        main_b, other_b = decode_bytes([S] * B, [Q_prev] * B, cfg["s_sink"], H, NQ, D, BITS)
        flushed = max(0, Q - max(Q_prev, cfg["s_sink"]))
        fz_bytes += main_b + other_b + append_step_bytes(B, H, D, BITS, 1, flushed)
    done += K
    fused_gbs = fz_bytes / K / (ms_fused * 1e-3) / 1e9
    log("fused step (graph): %.2f us, %.1f GB/s" % (ms_fused * 1e3, fused_gbs))
    wk.wushkv_timing_enable(8 * 64)
    for i in range(64):
        fused(done + i)
    torch.cuda.synchronize()
    done += 64
    for name in ("step_finish_kernel",):
        n, tot = wk.wushkv_timing_read(name)
        kernels[name] = (tot / n) if n else None
    n, tot = wk.wushkv_timing_read("decode_main_kernel")
    kernels["decode_main_kernel (fused step)"] = (tot / n) if n else None
    wk.wushkv_timing_enable(0)
    for r in range(reps):
        S = ctx + (done - r + reps - 1) // reps
        assert int(caches[r].seq_len[0].item()) == S
        assert int(caches[r].quant_end[0].item()) == quant_end_after(S)

    fused = {
        "workload": "llama3-8b-layer-decode-2bit: batch 8, 32 q / 8 kv heads, d 128, ctx 8192, "
                    "4 sink + 128 recent, flush 8",
        "step": "append 1 token/seq + decode + flush in Alg. 2 order (wushkv_decode_step, "
                "2 launches), HIP graph over %d cache replicas" % reps,
        "us": round(ms_fused * 1e3, 3), "gbps": round(fused_gbs, 2), "steps": K,
        "split_step": {"calls": "wushkv_append then wushkv_decode_attention (3 launches)",
                       "us": round(ms_graph * 1e3, 3), "gbps": round(step_gbs, 2)},
        "roofline": {"bound": "hbm", "kernel": "decode_main_kernel",
                     "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": profiled_traffic("decode_main_kernel_llama8b_2bit.md",
                                                 os.path.join(ROOT, "paper_2609_38121_amd", "csrc")),
                     "avg_us": round(t_main * 1e3, 3),
                     "bytes_per_launch": int(main_per_launch)},
        "decode_call_gbps": round(dec_gbs, 2),
        "decode_call_us": round(ms_dec * 1e3, 3),
        "eager_step_us": round(ms_eager * 1e3, 3),
        "kernel_avg_us": {k_: (round(v_ * 1e3, 3) if v_ else None) for k_, v_ in kernels.items()},
        "dequant": dequant,
    }
    state = (caches, reps, k1, tk, tinv_d, B, NQ, D, max_seq, sm, cfg, lengths_at, done)
    return fused, state


def bench_prefill(torch, wk, synth, dev, args):
    """Append throughput on the prefill workload: 4 x 16384 new tokens, 8 kv
    heads, d 128, 2-bit.  The keys are given as projected: the append applies
    the headwise RMS normalisation and RoPE (theta 1e6) itself, then the key
    transform, the quantisation and the packing (the whole prefill path of
    that workload).  The same append on keys normalised and rotated by the
    input generator is reported beside it, and so is the fused append into a
    cache that uses the QuEST codec (Eq. (5)) instead of Eq. (7)."""
    cfg = synth.CONFIGS["prefill"]
    w = synth.Workload(cfg, seed=args.seed)
    B, H, D, BITS, n = cfg["batch"], cfg["n_kv"], cfg["d"], cfg["bits"], cfg["ctx"]
    log("prefill append: generating %d x %d tokens" % (B, n))
    as_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    k_raw = as_dev(np.stack([w.raw_keys(b, 0, n) for b in range(B)]))
    k = as_dev(np.stack([w.keys(b, 0, n) for b in range(B)]))
    v = as_dev(np.stack([w.values(b, 0, n) for b in range(B)]))
    tk_bits, _ = w.transform()
    tk = as_dev(tk_bits)
    cache = wk.WushKVCache(B, H, D, BITS, cfg["s_sink"], cfg["s_keep"], cfg["s_flush"],
                           cfg["kappa_k"], cfg["kappa_v"], max_seq_len=n)
    qcache = wk.WushKVCache(B, H, D, BITS, cfg["s_sink"], cfg["s_keep"], cfg["s_flush"],
                            cfg["kappa_k"], cfg["kappa_v"], max_seq_len=n, codec="quest")
    table = torch.from_numpy(synth.rope_table(cfg["rope_theta"], D, cache.max_pages * 64 + cfg["s_sink"])).to(dev)
    nn = torch.full((B,), n, dtype=torch.int32, device=dev)
    reps = 10
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # each timed call appends into its own empty cache replica, back to back
    # on the stream (no reset between calls), so that the time is the GPU's
    replicas = {"pclip": [cache] + [cache.clone() for _ in range(reps - 1)],
                "quest": [qcache] + [qcache.clone() for _ in range(reps - 1)]}
    calls = {
        "norm_rope": ("pclip", lambda c: wk.wushkv_append_norm_rope(c, k_raw, v, nn, tk, table,
                                                                    norm_eps=1e-6)),
        "prenormed": ("pclip", lambda c: wk.wushkv_append(c, k, v, nn, tk)),
        "quest": ("quest", lambda c: wk.wushkv_append_norm_rope(c, k_raw, v, nn, tk, table,
                                                                norm_eps=1e-6)),
    }

    def reset(cs):
        for c in cs:
            c.seq_len.zero_()
            c.quant_end.zero_()
        torch.cuda.synchronize()

    res = {}
    for name, (kind, call) in calls.items():
        cs = replicas[kind]
        times = []
        for rnd in range(3):
            reset(cs)
            e0.record()
            for c in cs:
                call(c)
            e1.record()
            torch.cuda.synchronize()
            if rnd >= 1:
                times.append(e0.elapsed_time(e1) / reps)
        # the same calls again, each kernel stamped by the library
        reset(cs)
        wk.wushkv_timing_enable(16 * reps)
        for c in cs:
            call(c)
        torch.cuda.synchronize()
        cnt, tot = wk.wushkv_timing_read("append_kernel")
        fcnt, ftot = wk.wushkv_timing_read("append_flush")
        ccnt, ctot = wk.wushkv_timing_read("append_commit")
        wk.wushkv_timing_enable(0)
        res[name] = (float(np.median(times)), tot / cnt, ftot / fcnt if fcnt else 0.0,
                     ctot / ccnt if ccnt else 0.0)
    tokens = B * n
    Q = int(cache.quant_end[0].item())
    n_quant = Q - cfg["s_sink"]
    byts = prefill_bytes(B, H, D, BITS, n, n_quant)
    table_bytes = n * D * 4  # the rotary table rows of the positions written
    out = None
    for name in ("norm_rope", "prenormed", "quest"):
        ms, t_kernel, t_flush, t_commit = res[name]
        b_ = byts + (table_bytes if name != "prenormed" else 0)
        ach = b_ / (t_kernel * 1e-3) / 1e9
        log("prefill append (%s): %.1f us/call, %.3g tokens/s, append_kernel %.1f us, %.1f GB/s "
            "(flush-only launch %.1f us, counter launch %.1f us)"
            % (name, ms * 1e3, tokens / (ms * 1e-3), t_kernel * 1e3, ach, t_flush * 1e3, t_commit * 1e3))
        tkey = {"norm_rope": "traffic_bytes_per_launch", "prenormed": "traffic_bytes_per_launch_prenormed",
                "quest": "traffic_bytes_per_launch_quest"}[name]
        traffic = profiled_traffic("append_kernel_prefill_4x16384_2bit.md",
                                   os.path.join(ROOT, "paper_2609_38121_amd", "csrc"), tkey)
        entry = {"tokens_per_s": round(tokens / (ms * 1e-3), 1), "ms_per_call": round(ms, 4),
                 "bytes_per_call": int(b_),
                 "roofline": {"bound": "hbm", "kernel": "append_kernel", "achieved": round(ach, 2),
                              "peak": PEAK_HBM_GBS, "unit": "GB/s",
                              "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": traffic,
                              "avg_us": round(t_kernel * 1e3, 3)},
                 "flush_launch_us": round(t_flush * 1e3, 3),
                 "counter_launch_us": round(t_commit * 1e3, 3),
                 "roofline_tokens_per_s": round(tokens / (b_ / (PEAK_HBM_GBS * 1e9)), 1)}
        if out is None:
            out = dict(entry, workload="prefill-append-4x16384-2bit, RMS norm + RoPE fused",
                       keys="projected (Student-t), normalised and rotated by the append")
        elif name == "prenormed":
            out["prenormed_keys"] = entry
        else:
            out["quest_codec"] = dict(entry, codec="QuEST, Eq. (5), alpha_2 = %.6f" % qcache.quest_alpha)
    return out


def bench_chunk(torch, wk, caches, reps, k1, tk, tinv, B, NQ, D, max_seq, sm, cfg, lengths_at,
                done, T=16, calls=24):
    """Chunk attention (Alg. 2 step 5 with S' = 16, causal inside the chunk)
    on the Llama-shaped caches: each replica first takes a 16-token chunk
    per sequence (one append), then the timed calls attend all 16 x 32
    query rows per sequence.  Reported: query tokens per second and the
    algorithmic bytes (the cache once, the queries and outputs) per second."""
    dev = k1.device
    gen = torch.Generator(device=dev).manual_seed(7)
    kc = torch.randn(B, T, k1.shape[2], D, generator=gen, device=dev).to(torch.bfloat16)
    vc = torch.randn(B, T, k1.shape[2], D, generator=gen, device=dev).to(torch.bfloat16)
    q = torch.randn(B, T, NQ, D, generator=gen, device=dev).to(torch.bfloat16)
    n = torch.full((B,), T, dtype=torch.int32, device=dev)
    for c in caches:
        wk.wushkv_append(c, kc, vc, n, tk)
    torch.cuda.synchronize()
    need = wk.wushkv_chunk_workspace_bytes(caches[0], NQ, T, max_seq)
    ws = [torch.empty(need, dtype=torch.uint8, device=dev) for _ in range(reps)]
    outs = [torch.empty(B, T, NQ, D, dtype=torch.float32, device=dev) for _ in range(reps)]
    call = lambda i: wk.wushkv_chunk_attention(caches[i % reps], q, tinv, n_tok=n, sm_scale=sm,
                                               max_seq_len=max_seq, out=outs[i % reps],
                                               workspace=ws[i % reps])
    for i in range(2 * reps):
        call(i)
    torch.cuda.synchronize()
    n_calls = max(calls, reps) // reps * reps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(n_calls):
        call(i)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / n_calls * 1e-3
    S = int(caches[0].seq_len[0].item())
    Q = int(caches[0].quant_end[0].item())
    main_b, other_b = decode_bytes([S] * B, [Q] * B, cfg["s_sink"], k1.shape[2], NQ, D, cfg["bits"])
    byts = main_b + other_b + (T - 1) * B * NQ * D * (2 + 4)  # the other 15 tokens' q and out
    log("chunk attention (16 tokens x %d sequences): %.1f us per call, %.3g query tokens/s, "
        "%.1f GB/s algorithmic" % (B, t * 1e6, B * T / t, byts / t / 1e9))
    return {"tokens_per_call": B * T, "call_us": round(t * 1e6, 2),
            "query_tokens_per_s": round(B * T / t, 1), "bytes_per_call": int(byts),
            "gbps_algorithmic": round(byts / t / 1e9, 1),
            "note": "16-token chunks on the 8192-token Llama-shaped cache; bytes_per_call counts "
                    "the cache once.  Two chunk tokens x 4 query heads make a group of 8 virtual "
                    "heads; a page workgroup takes the 64 query rows of all eight groups of a "
                    "sequence over its run, so each page leaves HBM once per call.  Launches: "
                    "q~ rows, the page runs, then the window slots merged with the runs"}


def bench_stream_read(torch, wk, dev, gib=2, reps=10):
    """The reference denominator (not a replacement for the nominal peak): a
    plain read of a 2 GiB buffer, eight times the Infinity Cache, by the
    library's read probe with 16-byte vector loads and with the 16-byte
    direct-to-LDS loads the decode kernel's pages use."""
    buf = torch.zeros(gib << 30, dtype=torch.uint8, device=dev)
    sink = torch.empty((gib << 30) // 65536, dtype=torch.int32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {"bytes": gib << 30}
    for mode, key in ((0, "vector_loads_gbps"), (1, "lds_dma_loads_gbps")):
        for _ in range(2):
            wk.wushkv_read_probe(buf, mode, sink)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            wk.wushkv_read_probe(buf, mode, sink)
        e1.record()
        torch.cuda.synchronize()
        gbs = (gib << 30) * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
        out[key] = round(gbs, 1)
    log("streaming read of %d GiB: %.1f GB/s (vector loads), %.1f GB/s (direct-to-LDS loads), "
        "%.0f%% / %.0f%% of 8 TB/s" % (gib, out["vector_loads_gbps"], out["lds_dma_loads_gbps"],
                                        out["vector_loads_gbps"] / 80, out["lds_dma_loads_gbps"] / 80))
    del buf
    return out


def bench_wush(torch, wk, dev, args, layers=32, heads=8, d=128, gamma=1e-2, reps=5):
    """The WUSH transform builder (Eq. (1)) for every key and value head of a
    Llama-3-8B-shaped model: 32 layers x 8 kv heads x 2 = 512 transforms of
    d = 128, with T^{-1}, from synthetic calibration statistics of the
    paper's form (M = K K^T of keys with outlier channels, H = 2 Q Q^T of
    queries with uneven channel scales; seeded device-side Gaussians).
    Reported: time per call, transforms per second, and the fp32 arithmetic
    rate against the vector peak, counting per transform 9 sweeps d^3 (each
    Jacobi sweep: d - 1 rounds of d / 2 column pairs, three length-d dot
    products and two rotated length-2d columns) plus 4 d^3 (two Cholesky
    factorisations, the triangular product and the inverse's product)."""
    count = layers * heads * 2
    n = 1024
    gen = torch.Generator(device=dev).manual_seed(args.seed + 11)
    K = torch.randn(count, d, n, generator=gen, device=dev)
    K[:, :8] *= 10.0
    Q = torch.randn(count, d, n, generator=gen, device=dev) * torch.linspace(0.3, 3.0, d, device=dev)[None, :, None]
    M = (K @ K.transpose(1, 2) / n).contiguous()
    Hh = (2.0 * Q @ Q.transpose(1, 2) / n).contiguous()
    M = 0.5 * (M + M.transpose(1, 2))
    Hh = (0.5 * (Hh + Hh.transpose(1, 2))).contiguous()
    M = M.contiguous()
    del K, Q
    T = torch.empty_like(M)
    Ti = torch.empty_like(M)
    sw = torch.empty(count, dtype=torch.int32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wk.wushkv_wush_transform(M, Hh, gamma, T, Ti, sweeps_out=sw)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0.record()
        wk.wushkv_wush_transform(M, Hh, gamma, T, Ti, sweeps_out=sw)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    ms = float(np.median(times))
    sweeps = sw.cpu().numpy()
    flops = float(np.sum(9.0 * sweeps * d ** 3 + 4.0 * d ** 3))
    tflops = flops / (ms * 1e-3) / 1e12
    log("wush build: %d transforms of d %d in %.3f ms (%.3g per s), sweeps %.1f mean, "
        "%.2f TFLOP/s fp32 (%.1f%% of vector peak)" % (count, d, ms, count / (ms * 1e-3),
                                                        sweeps.mean(), tflops, 100 * tflops / 157.3))
    return {"workload": "wush-transforms-llama3-8b-kv-heads (512 x d128, gamma 1e-2, with inverse)",
            "ms_per_call": round(ms, 4), "transforms_per_s": round(count / (ms * 1e-3), 1),
            "mean_sweeps": round(float(sweeps.mean()), 2),
            "roofline": {"bound": "alu", "achieved": round(tflops, 3), "peak": 157.3,
                         "unit": "TFLOP/s", "frac": round(tflops / 157.3, 4), "traffic": None}}


def bench_decode_scale(torch, wk, synth, dev, args, calls=24, names=("long2", "long4", "qwen32b")):
    """Decode calls alone on the long-context (131072 tokens, 2 and 4 bits,
    random page order) and Qwen3-32B-shaped (8 sequences of 8192 tokens, 64
    query heads on 8 kv heads) caches (the large-batch one is the headline).  The caches are filled by the library's own append from
    seeded device-side Gaussian keys and values (throughput does not depend
    on the values); lengths are the workloads' own.  Replicas are cycled so
    that the calls touch more than twice the 256 MB Infinity Cache."""
    out = {}
    for name in names:
        cfg = synth.CONFIGS[name]
        w = synth.Workload(cfg, seed=args.seed)
        B, H, NQ, D, BITS = cfg["batch"], cfg["n_kv"], cfg["n_q"], cfg["d"], cfg["bits"]
        lengths = w.lengths.astype(np.int64)
        cap = cfg["ctx"] + 64  # capacity and split plan (the full-size tests use the same)
        cache = wk.WushKVCache(B, H, D, BITS, cfg["s_sink"], cfg["s_keep"], cfg["s_flush"],
                               cfg["kappa_k"], cfg["kappa_v"], max_seq_len=cap,
                               page_order=cfg.get("page_order", "linear"),
                               pool_factor=cfg.get("pool_factor", 1.0), seed=args.seed, device=dev)
        gen = torch.Generator(device=dev).manual_seed(1000 + args.seed)
        tk = torch.eye(D, device=dev).expand(H, D, D).to(torch.bfloat16).contiguous()
        chunk = 4096
        done = np.zeros(B, np.int64)
        while (done < lengths).any():
            n = np.minimum(chunk, lengths - done)
            m = int(n.max())
            k = torch.randn(B, m, H, D, generator=gen, device=dev).to(torch.bfloat16)
            v = torch.randn(B, m, H, D, generator=gen, device=dev).to(torch.bfloat16)
            wk.wushkv_append(cache, k, v, torch.from_numpy(n.astype(np.int32)).to(dev), tk)
            done += n
        torch.cuda.synchronize()
        del k, v
        seq = cache.seq_len.cpu().numpy()
        qe = cache.quant_end.cpu().numpy()
        main_b, other_b = decode_bytes(seq, qe, cfg["s_sink"], H, NQ, D, BITS)
        cache_bytes = cache.pages.numel() + 2 * cache.win_k.numel() * 2
        reps = max(1, math.ceil(2 * MALL_BYTES / cache_bytes))
        caches = [cache] + [cache.clone() for _ in range(reps - 1)]
        q = torch.randn(B, NQ, D, generator=gen, device=dev).to(torch.bfloat16)
        tinv = torch.eye(D, device=dev).expand(H, D, D).contiguous()
        ws = [torch.empty(wk.wushkv_decode_workspace_bytes(cache, NQ, cap), dtype=torch.uint8,
                          device=dev) for _ in range(reps)]
        outs = [torch.empty(B, NQ, D, dtype=torch.float32, device=dev) for _ in range(reps)]
        call = lambda i: wk.wushkv_decode_attention(caches[i % reps], q, tinv, max_seq_len=cap,
                                                    out=outs[i % reps], workspace=ws[i % reps])
        for i in range(2 * reps):
            call(i)
        torch.cuda.synchronize()
        n_calls = max(calls, reps) // reps * reps
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(n_calls):
            call(i)
        e1.record()
        torch.cuda.synchronize()
        t_call = e0.elapsed_time(e1) / n_calls * 1e-3
        wk.wushkv_timing_enable(8 * n_calls)
        for i in range(n_calls):
            call(i)
        torch.cuda.synchronize()
        cnt, tot = wk.wushkv_timing_read("decode_main_kernel")
        wk.wushkv_timing_enable(0)
        t_main = tot / cnt * 1e-3
        ach = main_b / t_main / 1e9
        log("%s decode: call %.1f us (%.1f GB/s), decode_main_kernel %.1f us, %.1f GB/s (%.1f%% of "
            "8 TB/s), %d replicas" % (name, t_call * 1e6, (main_b + other_b) / t_call / 1e9,
                                      t_main * 1e6, ach, 100 * ach / PEAK_HBM_GBS, reps))
        out[name] = {"batch": B, "ctx_max": int(lengths.max()), "bits": BITS,
                     "tokens": int(seq.sum()), "bytes_per_call": int(main_b + other_b),
                     "call_us": round(t_call * 1e6, 2),
                     "call_gbps": round((main_b + other_b) / t_call / 1e9, 1),
                     "main_kernel_us": round(t_main * 1e6, 2),
                     "main_kernel_gbps": round(ach, 1),
                     "main_kernel_frac": round(ach / PEAK_HBM_GBS, 4), "replicas": reps}
        del caches, cache, ws, outs
        torch.cuda.empty_cache()
    return out


def bench_oracle(sample, budget_s):
    """The oracle as it stands, on the host cores, on a bounded sample of the
    headline workload: every kv head of two of its sequences (the shortest
    and the longest), with the same inputs the GPU cache was built from.
    The pairs' caches are filled by the oracle's own append (untimed); then
    decode passes -- each pair's query group attends over its whole cache,
    as the GPU call does -- run until about budget_s seconds of CPU (wall
    time times threads).  The pairs are spread over the host's threads by
    OpenMP (the pairs are independent; each pair's arithmetic is the serial
    oracle's); the same passes on one thread are reported beside it."""
    import oracle
    cfg = sample["cfg"]
    d, H, G = cfg["d"], cfg["n_kv"], cfg["n_q"] // cfg["n_kv"]
    sm = 1.0 / math.sqrt(d)
    pairs = [(b, h) for b in sample["seqs"] for h in range(H)]
    L = sample["lengths"]
    hs = oracle.HeadSet([int(L[b]) for b, _ in pairs], d, cfg["bits"], cfg["s_sink"], cfg["s_keep"],
                        cfg["s_flush"], cfg["kappa_k"], cfg["kappa_v"])
    t0 = time.time()
    threads = hs.append([np.ascontiguousarray(sample["k"][b][:, h]) for b, h in pairs],
                        [np.ascontiguousarray(sample["v"][b][:, h]) for b, h in pairs],
                        [sample["tk"][h] for _, h in pairs])
    log("oracle: %d (sequence, head) pairs filled in %.1fs on %d threads" % (len(pairs), time.time() - t0,
                                                                          threads))
    qs = [np.ascontiguousarray(sample["q"][b, h * G:(h + 1) * G]) for b, h in pairs]
    tinv = [sample["tinv"][h] for _, h in pairs]
    nbytes = 0
    for i in range(len(pairs)):
        main_b, other_b = decode_bytes([int(hs.seq_len[i])], [int(hs.quant_end[i])], cfg["s_sink"], 1,
                                       G, d, cfg["bits"])
        nbytes += main_b + other_b

    def run(nthreads, seconds_cpu, pick=None):
        sel = list(range(len(pairs))) if pick is None else pick
        sel_bytes = nbytes if pick is None else sum(
            sum(decode_bytes([int(hs.seq_len[i])], [int(hs.quant_end[i])], cfg["s_sink"], 1, G, d,
                             cfg["bits"])) for i in sel)
        passes, wall, used = 0, 0.0, 1
        while passes == 0 or wall * used < seconds_cpu:
            t = time.perf_counter()
            _, used = hs.decode(qs, tinv, sm, threads=nthreads, pairs=sel)
            wall += time.perf_counter() - t
            passes += 1
        return sel_bytes * passes / wall / 1e9, used, passes, wall

    gbs, used, passes, wall = run(0, budget_s)
    log("oracle decode: %d passes over %d pairs in %.2fs on %d threads -> %.4f GB/s"
        % (passes, len(pairs), wall, used, gbs))
    one = [0, H]  # one kv head of each sampled sequence
    gbs1, _, passes1, wall1 = run(1, min(budget_s, 6.0), pick=one)
    log("oracle decode, one thread: %d passes over %d pairs in %.2fs -> %.4f GB/s"
        % (passes1, len(one), wall1, gbs1))
    return {"value": round(gbs, 5), "unit": "GB/s", "cores": used, "kind": "oracle",
            "sample": "decode of every kv head (query group of %d heads each) of two sequences of the "
                      "headline workload (%d and %d tokens), %d passes, caches built by the oracle's "
                      "own append from the GPU run's inputs; OpenMP over the 16 (sequence, head) pairs"
                      % (G, int(L[sample["seqs"][0]]), int(L[sample["seqs"][1]]), passes),
            "cpu_count": os.cpu_count(), "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "single_thread": {"value": round(gbs1, 5), "unit": "GB/s",
                              "sample": "one kv head of each of the two sequences, %d passes" % passes1}}


if __name__ == "__main__":
    main()
