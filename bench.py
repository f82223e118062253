"""Benchmark: batch-1 MoE decode under expert offloading on one MI355X.

Default workload: the 32-layer Mixtral-8x7B-shaped stack (8 experts per
layer, top-2, d=4096, d_ff=14336, bf16 experts in pinned host memory), 4 HBM
expert slots per layer, LFU eviction (Table 2's setting), all 512 batch-1
decode tokens of the seeded synthetic stream (Zipf(1.1) concept skew,
Markov(0.6) persistence) from the warm start.  A step decodes the next chunk
of consecutive tokens through all 32 layers; the cache carries over between
steps, so the K timed steps together are one pass over the 512 tokens.  The
W warm-up steps are a separate pass over the first W chunks, after which the
cache is reset to the warm start.

Beside the headline the JSON line carries: comparison runs on stated token
prefixes (LRU at 4 slots, 2 and 6 slots under both policies, next-layer
prefetch of 2) and the one-layer Mixtral workload under LFU and LRU; hit
rates with Belady's MIN; trace analytics (per-layer hit rates, the paper's
per-layer activation histograms, repeat rates against random routing); the
decode FFN up kernel's HBM roofline (HIP events stamped by its dispatches in
the timed pass); the fetch kernel's host-link roofline against the best of a
DMA copy and a shader copy measured here; a streaming HBM read probe and a
bf16 MFMA probe; and the fp64 oracle timed on a bounded sample on the host
cores.

`--workload` selects another configuration (the one-layer workloads and the
64-expert stack keep one pass over their tokens per step).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode tokens/s per MoE stack at fixed cache slots; expert-FFN HBM GB/s; hit rate"
HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
PMC_SUMMARY = os.path.join(ROOT, "profiles", "ffn_up_mixtral_layer_pmc.json")

DESCRIPTIONS = {
    "tiny-stack": "tiny-stack: 2 MoE layers, 8 experts, top-2, d_model 256, d_ff 512 SwiGLU, fp32, "
                  "64 batch-1 decode tokens, 4 slots",
    "mixtral-layer": "mixtral-layer: 1 MoE layer, 8 experts, top-2, d_model 4096, d_ff 14336 SwiGLU, "
                     "bf16 experts in pinned host memory, 256 batch-1 decode tokens, 4 HBM slots, "
                     "Zipf(1.1)+Markov(0.6) routing skew",
    "mixtral-stack": "mixtral-stack: 32 Mixtral-shaped MoE layers (8 experts, top-2, d_model 4096, "
                     "d_ff 14336, bf16, 90 GB of experts in pinned host memory), batch-1 decode, "
                     "slots per layer swept",
    "mixtral-stack-prefetch": "mixtral-stack-prefetch: the 32-layer Mixtral-shaped stack, 4 slots, LFU, "
                              "next-layer speculative prefetch of up to 2 experts",
    "fine-grained": "fine-grained: 24 MoE layers, 64 experts, top-8, d_model 2048, d_ff 1408, bf16; "
                    "4096-token batched prefill then batch-1 decode; 16 slots, LFU + prefetch 2, Zipf(1.2)",
    "tiny-q2": "tiny-q2: 2 MoE layers, 8 experts, top-2, d_model 512, d_ff 1024, 2-bit group-16 experts, "
               "64 batch-1 decode tokens, 4 slots",
    "mixtral-layer-q2": "mixtral-layer-q2: the Mixtral-shaped layer with experts group-quantised as in the "
                        "paper's measured model (2-bit codes, groups of 16, fp16 scales, 8-bit zero codes: "
                        "77 MB per expert), 256 batch-1 decode tokens, 4 HBM slots, Zipf(1.1)+Markov(0.6)",
    "mixtral-stack-q2": "mixtral-stack-q2: 32 Mixtral-shaped layers, 2-bit group-16 experts (19.7 GB in "
                        "pinned host memory), 128 batch-1 decode tokens, 4 slots, LFU + next-layer prefetch 2",
}


def ffn_kernels(cfg):
    """Names of the decode FFN's up and down kernels for this model."""
    if cfg.dtype == "q2g16":
        return ("ffnq_up_lut_kernel" if cfg.d_model <= 4096 else "ffnq_up_kernel"), "ffnq_down_lut_kernel"
    return "ffn_up_kernel", "ffn_down_kernel"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def measure_link(torch, b, nbytes=1 << 30, reps=3):
    """Host-to-device link ceiling: the best of a 1 GiB pinned-to-HBM copy by
    the DMA engines (hipMemcpyAsync) and by the library's shader-copy probe
    (the fetch kernel's access pattern) at 64, 128 and 256 workgroups, over the
    same pinned buffer.  Returns {"best", "best_is", "sdma", "shader"} (GB/s)."""
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    sdma = 0.0
    for _ in range(reps):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src, non_blocking=True)
        e.record()
        e.synchronize()
        sdma = max(sdma, nbytes / (a.elapsed_time(e) * 1e-3) / 1e9)
    stream = torch.cuda.current_stream().cuda_stream
    shader = {wg: b.moe_probe_h2d_copy(src.data_ptr(), dst.data_ptr(), nbytes, wg, reps, stream)
              for wg in (64, 128, 256)}
    torch.cuda.synchronize()
    del src, dst
    best_wg = max(shader, key=shader.get)
    if shader[best_wg] > sdma:
        best, best_is = shader[best_wg], f"shader copy probe, {best_wg} workgroups, 1 GiB pinned -> HBM"
    else:
        best, best_is = sdma, "DMA copy (hipMemcpyAsync), 1 GiB pinned -> HBM"
    return {"best": best, "best_is": best_is, "sdma": round(sdma, 2),
            "shader": {str(k): round(v, 2) for k, v in shader.items()}}


def measure_mfma(torch, b):
    """bf16 matrix-core ceiling (TFLOP/s) of a register-only MFMA loop, for
    both bf16 instruction shapes."""
    stream = torch.cuda.current_stream().cuda_stream
    return {"v_mfma_f32_16x16x32_bf16": round(b.moe_probe_mfma_bf16(0, 4096, stream), 1),
            "v_mfma_f32_32x32x16_bf16": round(b.moe_probe_mfma_bf16(1, 2048, stream), 1)}


def measure_hbm_read(torch, b, nbytes=1 << 30, reps=20):
    """Streaming read rate (GB/s) of the library's HBM read probe over 1 GiB:
    what a kernel with nothing to do but read reaches on this device."""
    buf = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    gbps = b.moe_probe_hbm_read(buf.data_ptr(), nbytes, reps, torch.cuda.current_stream().cuda_stream)
    del buf
    return gbps


def measure_hbm_window(torch, b, nbytes, span=3 << 30, rounds=3):
    """One-shot read of `nbytes` by the same probe, one launch a window, the
    windows rotating over `span` bytes (well beyond the 256 MB MALL) so that
    every launch reads from HBM: what a single launch of that many bytes costs
    on this device, ramp and drain included.  Returns (median us, GB/s)."""
    nbytes -= nbytes % 4096
    span = max(span, 4 * nbytes)
    buf = torch.zeros(span, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream().cuda_stream
    us = []
    for _ in range(rounds):
        for i in range(span // nbytes):
            gbps = b.moe_probe_hbm_read(buf.data_ptr() + i * nbytes, nbytes, 1, stream)
            us.append(nbytes / gbps / 1e3)
    del buf
    us.sort()
    med = us[len(us) // 2]
    return med, nbytes / (med * 1e-6) / 1e9


def same_bytes_probe(torch, b, nbytes, kernel_us):
    med, gbps = measure_hbm_window(torch, b, nbytes)
    log(f"one-shot read of {nbytes} B: {med:.2f} us ({gbps:.1f} GB/s)")
    return {"bytes": nbytes, "median_us": round(med, 2), "gbps": round(gbps, 1),
            "roofline_kernel_frac_of_probe": round(med / kernel_us, 4) if kernel_us else None,
            "is": "the same probe reading the roofline kernel's bytes once per launch, launches rotating "
                  "over 3 GiB so each reads HBM; the ratio is probe time / kernel time"}


def calibrate_counters(torch, nbytes=512 << 20):
    """One plain device-to-device copy of known size (512 MiB read, 512 MiB
    written), so that hardware byte counters collected on this program can be
    scaled: factor = known bytes / counter reading of this copy."""
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def pmc_traffic():
    """Per-launch HBM bytes of ffn_up_kernel from the committed counter runs,
    or None when the kernel source changed since they were taken."""
    try:
        with open(PMC_SUMMARY) as f:
            s = json.load(f)
        with open(os.path.join(ROOT, s["source"]), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != s["source_sha256"]:
                return None
        return int(round(1024 * (s["fetch_kib"] * s["fetch_factor"] + s["write_kib"] * s["write_factor"])))
    except (OSError, KeyError, ValueError):
        return None


def run_steps(torch, b, moe, H0, H, n, timing, flags=0, prefill_tokens=0, batch=1):
    """n passes (reset, [prefill], decode all tokens, one at a time or
    `batch` at a time) at a MOE_TIMING_* level; returns seconds of decode,
    seconds of prefill, summed timing (None when off), summed per-layer
    statistics, the trace of the last pass and the prefill's share of the
    fetched bytes."""
    dec = pre = 0.0
    tim = None
    stats = None
    recs = None
    prefill_bytes = 0
    b.moe_cache_set_timing(moe.handle, timing)
    for _ in range(n):
        moe.reset()
        H.copy_(H0)
        torch.cuda.synchronize()
        if timing:
            b.moe_cache_read_timing(moe.handle)  # drop spans of the reset
        if prefill_tokens:
            t0 = time.perf_counter()
            moe.prefill(H[:prefill_tokens])
            moe.sync()
            torch.cuda.synchronize()
            pre += time.perf_counter() - t0
            prefill_bytes += sum(s["bytes_fetched"] for s in moe.stats())
        t0 = time.perf_counter()
        if batch > 1:
            moe.decode_batched(H[prefill_tokens:], batch)
        else:
            moe.decode(H[prefill_tokens:], flags=flags)
        moe.sync()
        torch.cuda.synchronize()
        dec += time.perf_counter() - t0
        if timing:
            t = b.moe_cache_read_timing(moe.handle)
            tim = t if tim is None else {k: tim[k] + t[k] for k in t}
        st = moe.stats()
        stats = st if stats is None else [{k: a[k] + c[k] for k in a} for a, c in zip(stats, st)]
        recs, _ = moe.trace_records()
    b.moe_cache_set_timing(moe.handle, b.MOE_TIMING_OFF)
    return dec, pre, tim, stats, recs, prefill_bytes


def cpu_baseline(cfg, store, gates_host, h0, max_tokens, slots, policy, budget_s):
    """The fp64 oracle (router, cache, SwiGLU FFN, residual) on the leading
    decode tokens of the same workload, one token at a time until `budget_s`
    seconds have passed (at least two tokens, at most `max_tokens`), timed on
    this host's cores.  Returns (tokens/s, tokens, seconds, threads)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import stack
    from oracle.cache import make_caches
    model = stack.Model(gates_host, lambda l, e: store.expert(l, e), cfg.d_model, cfg.d_ff, cfg.dtype,
                        keep=cfg.layers * cfg.experts * cfg.expert_bytes < (8 << 30))
    caches = make_caches(cfg.layers, cfg.experts, slots, policy)
    n = 0
    t0 = time.perf_counter()
    while n < max_tokens and (n < 2 or time.perf_counter() - t0 < budget_s):
        stack.decode_free(model, h0[n:n + 1].astype(np.float64), cfg.top_k, policy, slots, caches=caches)
        n += 1
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return n / dt, n, dt, threads


def summarize(cfg, r):
    """Throughput, hit rate, cache P/R and guess P/R of one (policy, slots) run."""
    from paper_2511_05814_amd import analysis
    acc = [x for x in r["recs"] if x[0] != 2]
    out = {
        "tokens_per_s": round(r["steps"] * cfg.tokens / r["dec"], 3),
        "hit_rate": round(analysis.hit_rate(acc), 4),
        "cache_precision_recall": [round(v, 4) for v in analysis.cache_precision_recall(acc, r["slots"])],
        "decode_bytes_fetched_per_step":
            (sum(s["bytes_fetched"] for s in r["stats"]) - r["prefill_bytes"]) // r["steps"],
    }
    if not r["flags"] and not r["pre"]:
        # Belady MIN on the same demand sequences from the same warm start:
        # the most hits any demand-fetching policy could have had
        out["belady_min_hit_rate"] = round(analysis.belady_hit_rate(acc, r["slots"]), 4)
    if cfg.layers > 1:
        out["per_layer_hit_rate"] = [round(v, 3) for v in analysis.per_layer_hit_rate(acc).values()]
    if r["flags"]:
        p, rc = analysis.guess_precision_recall(acc)
        out["guess_precision_recall"] = [round(p, 4), round(rc, 4)]
        out["transfer_precision"] = round(analysis.transfer_precision(acc), 4)
    if r["pre"]:
        out["prefill_tokens_per_s"] = round(r["steps"] * cfg.prefill_tokens / r["pre"], 1)
    return out


def batch_report(args, cfg, results, link):
    """JSON line of a batched-decode run: tokens/s, pair hit rate, link bytes,
    and the grouped GEMMs (which stream each routed expert's weights once per
    batch: HBM-bound at small batches)."""
    head = results[0]
    tim, steps = head["timing"], head["timing_steps"]  # passes the GEMM spans cover
    mb = cfg.matrix_bytes

    def rates(r):
        hits = sum(s["hits"] for s in r["stats"])
        misses = sum(s["misses"] for s in r["stats"])
        return {"tokens_per_s": round(r["steps"] * cfg.tokens / r["dec"], 3),
                "pair_hit_rate": round(hits / max(1, hits + misses), 4),
                "decode_bytes_fetched_per_step": sum(s["bytes_fetched"] for s in r["stats"]) // r["steps"]}

    # experts each batch routed tokens to (one batch record per expert; its
    # rank field holds the number of (token, rank) pairs), in the last pass
    used = sum(1 for x in head["recs"] if x[0] == 2 and x[3] > 0)
    up_bytes = used * 2 * mb
    down_bytes = used * mb
    up_s = tim["gemm_up_ms"] * 1e-3 / steps
    down_s = tim["gemm_down_ms"] * 1e-3 / steps
    up_gbps = up_bytes / up_s / 1e9 if up_s > 0 else None
    fetched = rates(head)["decode_bytes_fetched_per_step"]
    link_gbps = fetched / (head["dec"] / head["steps"]) / 1e9
    return {
        "metric": METRIC,
        "value": rates(head)["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * head["dec"] / head["steps"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": DESCRIPTIONS[args.workload] + f"; batched decode, {args.batch} tokens per step",
                   "weights_dtype": cfg.dtype, "policy": head["policy"], "slots": head["slots"],
                   "batch": args.batch, "decode_tokens_per_step": cfg.tokens},
        "runs": {f"{r['policy']}-s{r['slots']}": rates(r) for r in results},
        "roofline": {
            "kernel": "prefill_skinny_kernel<true>" if args.batch <= 32 else "prefill_gemm_kernel<true>",
            "bound": "hbm",
            "achieved": round(up_gbps, 1) if up_gbps else None, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(up_gbps / HBM_PEAK_GBPS, 4) if up_gbps else None, "traffic": None,
            "bytes_per_launch": up_bytes // max(1, tim["gemm_up_n"] // steps),
            "avg_launch_us": round(1e3 * tim["gemm_up_ms"] / max(1, tim["gemm_up_n"]), 2),
            "launches": tim["gemm_up_n"],
            "note": "weights of every routed expert (W1, W3) streamed once per batch",
        },
        "gemm_down": {"kernel": "prefill_skinny_kernel<false>" if args.batch <= 32 else "prefill_gemm_kernel<false>",
                      "achieved_gbps": round(down_bytes / down_s / 1e9, 1) if down_s > 0 else None,
                      "avg_launch_us": round(1e3 * tim["gemm_down_ms"] / max(1, tim["gemm_down_n"]), 2)},
        "experts_per_batch_layer": round(used / max(1, (cfg.tokens // args.batch) * cfg.layers), 3),
        "link": {"bytes_per_step": fetched, "achieved_over_decode_gbps": round(link_gbps, 2),
                 "peak": round(link, 2), "frac": round(link_gbps / link, 4)},
        "batch_layer_ms": round(tim["prefill_ms"] / max(1, tim["prefill_n"]), 3),
    }


# Stack workloads: the metric's own unit, tokens/s through a whole MoE stack.
STACK_WORKLOADS = ("mixtral-stack", "mixtral-stack-prefetch", "mixtral-stack-q2")
# comparison runs of the 32-layer stack: (policy, slots, speculate, token prefix)
STACK_COMPARISONS = {
    "mixtral-stack": [("lru", 4, False, 128), ("lfu", 2, False, 48), ("lru", 2, False, 48),
                      ("lfu", 6, False, 96), ("lru", 6, False, 96), ("lfu", 4, True, 64)],
    "mixtral-stack-prefetch": [("lfu", 4, False, 64)],
    "mixtral-stack-q2": [("lfu", 4, False, 64)],
}


def run_chunks(torch, b, moe, H0, H, steps, chunk, tokens, timing, flags=0):
    """One pass over the first `tokens` decode tokens from the warm start, in
    `steps` steps of `chunk` consecutive tokens (the last may be shorter), each
    through every layer; the cache carries over from step to step.  The
    region from the first step's start to the last step's end is timed with
    the device drained at both ends."""
    b.moe_cache_set_timing(moe.handle, timing)
    moe.reset()
    H.copy_(H0)
    torch.cuda.synchronize()
    if timing:
        b.moe_cache_read_timing(moe.handle)  # drop spans of the reset
    step_s = []
    t_start = time.perf_counter()
    for i in range(steps):
        a, z = i * chunk, min(tokens, (i + 1) * chunk)
        if a >= z:
            break
        t0 = time.perf_counter()
        moe.decode(H[a:z], flags=flags)
        moe.sync()
        torch.cuda.synchronize()
        step_s.append(time.perf_counter() - t0)
    total = time.perf_counter() - t_start
    tim = b.moe_cache_read_timing(moe.handle) if timing else None
    b.moe_cache_set_timing(moe.handle, b.MOE_TIMING_OFF)
    recs, dropped = moe.trace_records()
    if dropped:
        raise RuntimeError(f"trace ring overflowed ({dropped} records lost)")
    return {"total": total, "step_s": step_s, "tim": tim, "stats": moe.stats(), "recs": recs,
            "tokens": tokens}


def pass_summary(cfg, r, slots, flags):
    """Tokens/s, hit rate, cache and guess precision/recall of one pass."""
    from paper_2511_05814_amd import analysis
    acc = [x for x in r["recs"] if x[0] != 2]
    out = {"tokens": r["tokens"],
           "tokens_per_s": round(r["tokens"] / r["total"], 3),
           "hit_rate": round(analysis.hit_rate(acc), 4),
           "cache_precision_recall": [round(v, 4) for v in analysis.cache_precision_recall(acc, slots)],
           "bytes_fetched": sum(s["bytes_fetched"] for s in r["stats"])}
    if flags:
        p, rc = analysis.guess_precision_recall(acc)
        out["guess_precision_recall"] = [round(p, 4), round(rc, 4)]
        out["transfer_precision"] = round(analysis.transfer_precision(acc), 4)
    else:
        out["belady_min_hit_rate"] = round(analysis.belady_hit_rate(acc, slots), 4)
    return out


def layer_comparison(torch, b, offload, wl, fetch_mode):
    """The one-layer Mixtral-shaped workload (its own seed, 256 tokens, 4
    slots) under LFU and LRU: one pass each from the warm start."""
    cfg = wl.CONFIGS["mixtral-layer"]
    store = offload.HostStore(cfg)
    gates = offload.DeviceGates(cfg)
    H0 = torch.from_numpy(wl.hidden_states(cfg)).to("cuda")
    H = torch.empty_like(H0)
    out = {"workload": DESCRIPTIONS["mixtral-layer"]}
    try:
        for policy in ("lfu", "lru"):
            moe = offload.OffloadedMoE(cfg, store, gates, 4, policy, fetch_mode=fetch_mode)
            run_chunks(torch, b, moe, H0, H, 1, cfg.tokens, cfg.tokens, b.MOE_TIMING_OFF)  # warm-up pass
            r = run_chunks(torch, b, moe, H0, H, 1, cfg.tokens, cfg.tokens, b.MOE_TIMING_OFF)
            moe.close()
            out[f"{policy}-s4"] = pass_summary(cfg, r, 4, 0)
            log("mixtral-layer", policy, 4, f"{out[f'{policy}-s4']['tokens_per_s']:.2f} tok/s")
    finally:
        store.close()
    return out


def stack_main(args):
    """The metric's headline: batch-1 decode tokens/s through the whole
    32-layer stack at a fixed number of slots per layer (Table 2's setting:
    4 slots, Sec. 5.3), over every token of the workload from the warm start.
    Each step decodes the next chunk of consecutive tokens through all layers
    and the cache carries over between steps."""
    import math

    import torch

    from paper_2511_05814_amd import analysis
    from paper_2511_05814_amd import binding as b
    from paper_2511_05814_amd import offload, workload as wl

    cfg = wl.CONFIGS[args.workload]
    if args.prefetch_max >= 0:
        cfg = cfg.with_(prefetch_max=min(args.prefetch_max, cfg.top_k))
    if args.tokens:
        cfg = cfg.with_(tokens=min(args.tokens, cfg.tokens))
    if args.layers:
        cfg = cfg.with_(layers=min(args.layers, cfg.layers))
    fetch_mode = {"kernel": b.MOE_FETCH_KERNEL, "dma": b.MOE_FETCH_DMA, "split": b.MOE_FETCH_SPLIT}[args.fetch]
    slots = args.slots or 4
    if not cfg.top_k <= slots <= cfg.experts:
        sys.exit(f"--slots must lie in [top_k, experts] = [{cfg.top_k}, {cfg.experts}]")
    if args.host_store != "plain" and cfg.dtype != "bf16":
        sys.exit("a coded host store holds bf16 experts")
    steps = max(1, args.steps)
    chunk = math.ceil(cfg.tokens / steps)
    steps = math.ceil(cfg.tokens / chunk)  # every step decodes at least one token
    spec = cfg.prefetch_max > 0
    flags = b.MOE_PREFETCH_NEXT if spec else 0

    log("generating", cfg.name, "host store", cfg.layers * cfg.experts * cfg.expert_bytes / 1e9, "GB")
    t0 = time.perf_counter()
    store = offload.HostStore(cfg, fmt=args.host_store)
    gates = offload.DeviceGates(cfg)
    h0 = wl.hidden_states(cfg)
    log(f"inputs ready in {time.perf_counter() - t0:.1f}s ({store.distinct} distinct layers pinned)")
    link_info = measure_link(torch, b)
    link = link_info["best"]
    log(f"host link ceiling: {link:.2f} GB/s ({link_info['best_is']}; DMA {link_info['sdma']} GB/s)")
    hbm_probe = measure_hbm_read(torch, b)
    log(f"HBM read probe: {hbm_probe:.1f} GB/s")
    mfma = measure_mfma(torch, b)
    log("bf16 MFMA probe:", mfma)
    calibrate_counters(torch)

    H0 = torch.from_numpy(h0[:cfg.tokens]).to("cuda")
    H = torch.empty_like(H0)
    moe = offload.OffloadedMoE(cfg, store, gates, slots, "lfu", prefetch_max=cfg.prefetch_max if spec else 0,
                               fetch_mode=fetch_mode)
    if args.warmup:
        wt = min(cfg.tokens, args.warmup * chunk)
        w = run_chunks(torch, b, moe, H0, H, args.warmup, chunk, wt, b.MOE_TIMING_OFF, flags)
        log(f"warm-up: {args.warmup} steps, {wt} tokens, {wt / w['total']:.2f} tok/s")
    # timed pass: events on the decode FFN up launches only (the roofline kernel)
    head = run_chunks(torch, b, moe, H0, H, steps, chunk, cfg.tokens, b.MOE_TIMING_FFN_UP, flags)
    tokens_per_s = cfg.tokens / head["total"]
    log(f"lfu {slots} {'prefetch ' if spec else ''}{tokens_per_s:.3f} tok/s over {cfg.tokens} tokens "
        f"in {steps} steps of {chunk}")
    # every launch timed, on a prefix: kernel breakdown, copy time, overlap
    bd_tokens = max(1, min(cfg.tokens, args.breakdown_tokens))
    bd = run_chunks(torch, b, moe, H0, H, 1, bd_tokens, bd_tokens, b.MOE_TIMING_ALL, flags)
    moe.close()

    comparisons = {}
    if not args.lfu_only:
        for policy, s_, sp, prefix in STACK_COMPARISONS[args.workload]:
            if not cfg.top_k <= s_ <= cfg.experts:
                continue
            n = min(prefix, cfg.tokens)
            m = offload.OffloadedMoE(cfg, store, gates, s_, policy, prefetch_max=2 if sp else 0,
                                     fetch_mode=fetch_mode)
            r = run_chunks(torch, b, m, H0, H, 1, n, n, b.MOE_TIMING_OFF, b.MOE_PREFETCH_NEXT if sp else 0)
            m.close()
            key = f"{policy}-s{s_}" + ("-prefetch2" if sp else "")
            comparisons[key] = pass_summary(cfg, r, s_, sp)
            comparisons[key]["prefix"] = f"first {n} of the {cfg.tokens} tokens, one pass from the warm start"
            log(key, f"{comparisons[key]['tokens_per_s']:.3f} tok/s over {n} tokens")

    cpu = None
    if not args.no_cpu_baseline:
        cap = min(args.cpu_tokens, cfg.tokens) if args.cpu_tokens > 0 else cfg.tokens
        cpu = cpu_baseline(cfg, store, gates.host, h0, cap, slots, "lfu", args.cpu_seconds)
    aliased = store.aliased
    distinct = store.distinct
    store.close()
    layer_cmp = None
    if args.workload == "mixtral-stack" and not args.lfu_only and not args.no_layer_comparison:
        layer_cmp = layer_comparison(torch, b, offload, wl, fetch_mode)

    # ---- the report ---------------------------------------------------------
    K, d, dff, mb = cfg.top_k, cfg.d_model, cfg.d_ff, cfg.matrix_bytes
    up_bytes = K * 2 * mb + d * 4 + K * dff * 4
    down_bytes = K * mb + K * dff * 4 + d * 4
    ut = head["tim"]
    up_ms = ut["ffn_up_ms"] / ut["ffn_up_n"]
    up_gbps = up_bytes / (up_ms * 1e-3) / 1e9
    bt = bd["tim"]
    down_ms = bt["ffn_down_ms"] / max(1, bt["ffn_down_n"])
    down_gbps = down_bytes / (down_ms * 1e-3) / 1e9 if down_ms > 0 else None
    fetched = sum(s["bytes_fetched"] for s in head["stats"])
    bd_fetched = sum(s["bytes_fetched"] for s in bd["stats"])
    copy_ms = bt["fetch_ms"] + bt["pf_fetch_ms"]
    fetch_gbps = bd_fetched / (copy_ms * 1e-3) / 1e9 if copy_ms > 0 else None
    acc = [x for x in head["recs"] if x[0] != 2]
    headline = pass_summary(cfg, head, slots, flags)
    up_kernel, down_kernel = ffn_kernels(cfg)
    desc = (DESCRIPTIONS[args.workload]
            + f"; {cfg.tokens} batch-1 decode tokens from the warm start, {slots} HBM slots per layer, LFU"
            + (f", next-layer prefetch of up to {cfg.prefetch_max}" if spec else "")
            + f"; each step decodes {chunk} consecutive tokens through all {cfg.layers} layers and the "
              f"cache carries over between steps"
            + (f"; only the first {cfg.layers} layers" if args.layers else "")
            + (f"; the pinned store holds {distinct} distinct layers and layer l >= {distinct} reuses the "
               f"pages of layer l mod {distinct} (the driver pins about 70 GB at most): every miss still moves "
               f"a whole expert over the host link, only weight values repeat, gates are per layer"
               if aliased else ""))
    out = {
        "metric": METRIC,
        "value": round(tokens_per_s, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * head["total"] / steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": desc,
            "weights_dtype": cfg.dtype,
            "layers": cfg.layers,
            "policy": "lfu",
            "slots": slots,
            "speculative_prefetch": cfg.prefetch_max if spec else 0,
            "decode_tokens": cfg.tokens,
            "decode_tokens_per_step": chunk,
            "fetch": args.fetch,
            "host_store": args.host_store if args.host_store != "plain" else cfg.dtype,
        },
        "hit_rate": headline["hit_rate"],
        "headline_run": headline,
        "step_ms": {"min": round(1e3 * min(head["step_s"]), 1), "max": round(1e3 * max(head["step_s"]), 1),
                    "median": round(1e3 * sorted(head["step_s"])[len(head["step_s"]) // 2], 1)},
        "runs": comparisons,
        "roofline": {
            "kernel": up_kernel,
            "bound": "hbm",
            "achieved": round(up_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(up_gbps / HBM_PEAK_GBPS, 4),
            "traffic": pmc_traffic() if cfg.dtype == "bf16" else None,
            "bytes_per_launch": up_bytes,
            "avg_launch_us": round(up_ms * 1e3, 2),
            "launches": ut["ffn_up_n"],
            "note": "events stamped by every up launch of the timed pass; the step itself is bound by the "
                    "host link (link_roofline)",
        },
        "ffn_down": {"kernel": down_kernel, "achieved_gbps": round(down_gbps, 1) if down_gbps else None,
                     "frac": round(down_gbps / HBM_PEAK_GBPS, 4) if down_gbps else None,
                     "bytes_per_launch": down_bytes, "avg_launch_us": round(down_ms * 1e3, 2),
                     "reduce_avg_us": round(1e3 * bt["ffn_reduce_ms"] / max(1, bt["ffn_reduce_n"]), 2),
                     "from": f"the {bd_tokens}-token pass with every launch timed"},
        "hbm_read_probe": {"kernel": "hbm_read_probe_kernel", "gbps": round(hbm_probe, 1), "bytes": 1 << 30,
                           "roofline_kernel_frac_of_probe": round(up_gbps / hbm_probe, 4) if hbm_probe else None,
                           "same_bytes": same_bytes_probe(torch, b, up_bytes, up_ms * 1e3)},
        "mfma_bf16_probe_tflops": mfma,
        "link_roofline": {
            "kernel": "fetch_kernel",
            "bound": "host-link",
            "achieved": round(fetch_gbps, 2) if fetch_gbps else None,
            "peak": round(link, 2),
            "unit": "GB/s",
            "frac": round(fetch_gbps / link, 4) if fetch_gbps else None,
            "peak_is": link_info["best_is"],
            "probes_gbps": {"dma": link_info["sdma"], "shader_by_workgroups": link_info["shader"]},
            "achieved_is": f"bytes fetched / copy time of the {bd_tokens}-token pass with every launch timed",
            "bytes_fetched_timed_pass": fetched,
            "link_rate_over_timed_pass_gbps": round(fetched / head["total"] / 1e9, 2),
        },
        "router_us": round(1e3 * bt["router_ms"] / max(1, bt["router_n"]), 2),
    }
    ffn_bytes = cfg.tokens * cfg.layers * (up_bytes + down_bytes)
    link_s = fetched / (link * 1e9)
    hbm_s = ffn_bytes / (HBM_PEAK_GBPS * 1e9)
    out["step_roofline"] = {
        "bound_s": round(link_s + hbm_s, 3), "achieved_s": round(head["total"], 3),
        "frac": round((link_s + hbm_s) / head["total"], 4),
        "terms": "whole timed pass: its link bytes / link ceiling + FFN weight bytes / 8 TB/s (no overlap)",
        "overlap_bound_s": round(max(link_s, hbm_s), 3),
        "overlap_frac": round(max(link_s, hbm_s) / head["total"], 4),
    }
    bd_ms = 1e3 * bd["total"]
    out["copy_overlap"] = {
        "tokens": bd_tokens,
        "demand_copy_ms": round(bt["fetch_ms"], 2), "prefetch_copy_ms": round(bt["pf_fetch_ms"], 2),
        "compute_wait_ms": round(bt["wait_ms"], 2), "pass_ms": round(bd_ms, 2),
        "link_busy_frac": round(copy_ms / bd_ms, 4) if bd_ms > 0 else None,
        "hidden_copy_frac": round(max(0.0, 1.0 - bt["wait_ms"] / copy_ms), 4) if copy_ms > 0 else None,
        "definition": "hidden_copy_frac = 1 - compute wait / copy time: the share of the copy time "
                      "(demand + speculative) during which the compute stream was not waiting",
    }
    out["trace_analytics"] = analysis.report(acc, cfg.layers, cfg.experts, cfg.top_k)
    if layer_cmp:
        out["mixtral_layer_runs"] = layer_cmp
    if cpu is not None:
        tps, n, dt, thr = cpu
        out["cpu_baseline"] = {
            "value": round(tps, 4), "unit": "tokens/s", "cores": thr, "kind": "oracle",
            "sample": f"first {n} of the {cfg.tokens} decode tokens (a {args.cpu_seconds:g} s budget), fp64 router "
                      f"+ LFU cache + SwiGLU FFN through all {cfg.layers} layers from the warm start (bf16->fp64 "
                      f"widening of each used expert included), {dt:.1f} s"}
    print(json.dumps(out), flush=True)


def layer_main(args):
    """Workloads whose step is a whole pass over the token set from the warm
    start (the one-layer workloads, the 64-expert stack with its prefill,
    batched decode)."""
    import torch

    from paper_2511_05814_amd import binding as b
    from paper_2511_05814_amd import offload, workload as wl

    cfg = wl.CONFIGS[args.workload]
    if args.prefetch_max >= 0:
        cfg = cfg.with_(prefetch_max=min(args.prefetch_max, cfg.top_k))
    if args.tokens:
        cfg = cfg.with_(tokens=min(args.tokens, cfg.tokens))
    if args.layers:
        cfg = cfg.with_(layers=min(args.layers, cfg.layers))
    if args.prefill_tokens >= 0:
        cfg = cfg.with_(prefill_tokens=min(args.prefill_tokens, cfg.prefill_tokens))
    fetch_mode = {"kernel": b.MOE_FETCH_KERNEL, "dma": b.MOE_FETCH_DMA, "split": b.MOE_FETCH_SPLIT}[args.fetch]
    primary_slots = args.slots or (16 if cfg.experts == 64 else 4)
    if not cfg.top_k <= primary_slots <= cfg.experts:
        sys.exit(f"--slots must lie in [top_k, experts] = [{cfg.top_k}, {cfg.experts}]")
    if args.batch > 1 and cfg.dtype != "bf16":
        sys.exit("batched decode runs on bf16 experts (the grouped GEMMs use bf16 matrix cores)")
    if args.batch > 1 and cfg.prefill_tokens:
        sys.exit("batched decode is measured on the workloads without a prefill phase")
    # (policy, slots, speculate): the first entry is the timed headline run
    runs = [("lfu", primary_slots, cfg.prefetch_max > 0 and args.batch == 1)]
    if args.batch > 1:
        if not args.lfu_only:
            runs.append(("lru", primary_slots, False))
    elif not args.lfu_only:
        if args.workload in ("mixtral-layer", "tiny-stack", "mixtral-layer-q2", "tiny-q2"):
            runs += [("lru", primary_slots, False), ("lfu-aged:32", primary_slots, False)]
        elif args.workload == "mixtral-stack-q2":
            runs.append(("lfu", 4, False))
        elif args.workload == "mixtral-stack":
            runs += [("lru", 4, False)] + [(p, s, False) for s in (2, 6) for p in ("lru", "lfu")]
        elif args.workload == "mixtral-stack-prefetch":
            runs.append(("lfu", 4, False))
        elif args.workload == "fine-grained":
            runs.append(("lfu", 16, False))
    # store per run: the headline's, then (bf16 batch-1 decode on the plain
    # store) the headline's policy once more on each coded host store
    runs = [r + (args.host_store,) for r in runs]
    if args.host_store == "plain" and cfg.dtype == "bf16" and args.batch == 1 and not args.lfu_only:
        coded = ("packed", "entropy") if args.workload == "mixtral-layer" else ("entropy",)
        runs += [runs[0][:3] + (fmt,) for fmt in coded]

    log("generating", cfg.name, "host store", cfg.layers * cfg.experts * cfg.expert_bytes / 1e9, "GB")
    t0 = time.perf_counter()
    if args.host_store != "plain" and cfg.dtype != "bf16":
        sys.exit("a coded host store holds bf16 experts")
    store = offload.HostStore(cfg, fmt=args.host_store)
    gates = offload.DeviceGates(cfg)
    h0 = wl.hidden_states(cfg)
    log(f"inputs ready in {time.perf_counter() - t0:.1f}s")
    link_info = measure_link(torch, b)
    link = link_info["best"]
    log(f"host link ceiling: {link:.2f} GB/s ({link_info['best_is']})")
    hbm_probe = measure_hbm_read(torch, b)
    log(f"HBM read probe: {hbm_probe:.1f} GB/s")
    calibrate_counters(torch)

    H0 = torch.from_numpy(h0[:cfg.prefill_tokens + cfg.tokens]).to("cuda")
    H = torch.empty_like(H0)
    results = []
    cpu = None

    def time_oracle():
        """(all host threads, one thread) oracle timings; one thread only for
        the one- and two-layer workloads, on a quarter of the time budget."""
        if args.no_cpu_baseline:
            return None
        from threadpoolctl import threadpool_limits
        cap = min(args.cpu_tokens, cfg.tokens) if args.cpu_tokens > 0 else cfg.tokens
        full = cpu_baseline(cfg, store, gates.host, h0[cfg.prefill_tokens:], cap, primary_slots, "lfu",
                            args.cpu_seconds)
        one = None
        if cfg.layers <= 2:
            with threadpool_limits(limits=1):
                one = cpu_baseline(cfg, store, gates.host, h0[cfg.prefill_tokens:], cap, primary_slots, "lfu",
                                   args.cpu_seconds / 4)
        return full, one

    for i, (policy, slots, spec, fmt) in enumerate(runs):
        if fmt != store.fmt:
            if cpu is None:
                cpu = time_oracle()  # on the plain store's bytes, before it is released
            store.close()  # two stores at once could exceed the driver's pinning cap
            log(f"generating the {fmt} host store")
            store = offload.HostStore(cfg, fmt=fmt)
        flags = b.MOE_PREFETCH_NEXT if spec else 0
        moe = offload.OffloadedMoE(cfg, store, gates, slots, policy,
                                   prefetch_max=cfg.prefetch_max if spec else 0, fetch_mode=fetch_mode,
                                   max_prefill_tokens=max(cfg.prefill_tokens, args.batch if args.batch > 1 else 0))
        steps = args.steps if i == 0 else 1
        if i == 0 and args.warmup:
            run_steps(torch, b, moe, H0, H, args.warmup, b.MOE_TIMING_OFF, flags, cfg.prefill_tokens, args.batch)
        # timed passes: events on the decode FFN up launches only (the roofline
        # kernel); every other kernel's events cost GPU time that would show in
        # tokens/s, so the full breakdown comes from one more pass of the same
        # work (the headline run, and the coded-store runs for their rebuilds)
        dec, pre, up_tim, st, recs, pbytes = run_steps(torch, b, moe, H0, H, steps, b.MOE_TIMING_FFN_UP, flags,
                                                       cfg.prefill_tokens, args.batch)
        tim = up_tim
        if i == 0 or fmt != "plain":
            _, _, tim, _, _, _ = run_steps(torch, b, moe, H0, H, 1, b.MOE_TIMING_ALL, flags,
                                           cfg.prefill_tokens, args.batch)
            tim["ffn_up_ms"], tim["ffn_up_n"] = up_tim["ffn_up_ms"], up_tim["ffn_up_n"]
        results.append(dict(policy=policy, slots=slots, flags=flags, steps=steps, dec=dec, pre=pre,
                            prefill_bytes=pbytes, fmt=fmt, expert_stride=store.expert_stride,
                            timing=tim, timing_steps=1 if tim is not up_tim else steps, stats=st, recs=recs))
        log(policy, slots, "prefetch" if spec else "", f"{steps * cfg.tokens / dec:.2f} tok/s")
        moe.close()

    if args.batch > 1:
        print(json.dumps(batch_report(args, cfg, results, link)), flush=True)
        store.close()
        return

    head = results[0]
    K, d, dff, mb = cfg.top_k, cfg.d_model, cfg.d_ff, cfg.matrix_bytes
    tim = head["timing"]
    # algorithmic bytes per launch: the selected experts' weights plus the
    # activation vectors the kernel reads and writes
    up_bytes = K * 2 * mb + d * 4 + K * dff * 4
    down_bytes = K * mb + K * dff * 4 + d * 4
    up_ms = tim["ffn_up_ms"] / tim["ffn_up_n"]
    down_ms = tim["ffn_down_ms"] / tim["ffn_down_n"]
    up_gbps = up_bytes / (up_ms * 1e-3) / 1e9
    down_gbps = down_bytes / (down_ms * 1e-3) / 1e9
    fetched = sum(s["bytes_fetched"] for s in head["stats"]) - head["prefill_bytes"]  # decode only
    tsteps = head["timing_steps"]  # passes the breakdown spans cover
    copy_ms = (tim["fetch_ms"] + tim["pf_fetch_ms"]) / tsteps  # demand and speculative copies, per pass
    fetch_gbps = fetched / head["steps"] / (copy_ms * 1e-3) / 1e9 if copy_ms > 0 else None
    tokens_per_s = head["steps"] * cfg.tokens / head["dec"]
    traffic = pmc_traffic() if args.workload == "mixtral-layer" else None
    summary = {f"{r['policy']}-s{r['slots']}" + ("-prefetch" if r["flags"] else "")
               + (f"-{r['fmt']}" if r["fmt"] != head["fmt"] else ""): summarize(cfg, r)
               for r in results}

    out = {
        "metric": METRIC,
        "value": round(tokens_per_s, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * (head["dec"] + head["pre"]) / head["steps"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": DESCRIPTIONS[args.workload] + (f" (first {cfg.tokens} tokens)" if args.tokens else "")
                        + (f"; run with {head['slots']} slots per layer" if args.slots else "")
                        + (f"; first {cfg.layers} layers" if args.layers else "")
                        + (f"; {cfg.prefill_tokens}-token prefill" if args.prefill_tokens >= 0 else ""),
            "weights_dtype": cfg.dtype,
            "policy": head["policy"],
            "slots": head["slots"],
            "speculative_prefetch": cfg.prefetch_max if head["flags"] else 0,
            "decode_tokens_per_step": cfg.tokens,
            "prefill_tokens_per_step": cfg.prefill_tokens,
            "fetch": args.fetch,
            "host_store": ("bf16 coded losslessly (%s), %.2f bits a weight"
                           % (head["fmt"], 8 * head["expert_stride"] / cfg.expert_elems)
                           if head["fmt"] != "plain" else cfg.dtype),
        },
        "hit_rate": next(iter(summary.values()))["hit_rate"],
        "runs": summary,
        "ffn_hbm_gbps": round((up_bytes + down_bytes) / ((up_ms + down_ms) * 1e-3) / 1e9, 1),
        "roofline": {
            "kernel": ffn_kernels(cfg)[0],
            "bound": "hbm",
            "achieved": round(up_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(up_gbps / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "bytes_per_launch": up_bytes,
            "avg_launch_us": round(up_ms * 1e3, 2),
            "launches": tim["ffn_up_n"],
        },
        "ffn_down": {"kernel": ffn_kernels(cfg)[1],
                     "achieved_gbps": round(down_gbps, 1), "frac": round(down_gbps / HBM_PEAK_GBPS, 4),
                     "bytes_per_launch": down_bytes, "avg_launch_us": round(down_ms * 1e3, 2),
                     "reduce_avg_us": round(1e3 * tim["ffn_reduce_ms"] / max(1, tim["ffn_reduce_n"]), 2)},
        "hbm_read_probe": {
            "kernel": "hbm_read_probe_kernel",
            "gbps": round(hbm_probe, 1),
            "bytes": 1 << 30,
            "roofline_kernel_frac_of_probe": round(up_gbps / hbm_probe, 4) if hbm_probe else None,
            "is": "a streaming read with nothing else to do (one workgroup per CU, 8 16-byte loads in flight a lane)",
            "same_bytes": same_bytes_probe(torch, b, up_bytes, up_ms * 1e3),
        },
        "link_roofline": {
            "kernel": "fetch_kernel",
            "bound": "host-link",
            "achieved": round(fetch_gbps, 2) if fetch_gbps else None,
            "peak": round(link, 2),
            "unit": "GB/s",
            "frac": round(fetch_gbps / link, 4) if fetch_gbps else None,
            "peak_is": link_info["best_is"],
            "probes_gbps": {"dma": link_info["sdma"], "shader_by_workgroups": link_info["shader"]},
            "decode_bytes_fetched_per_step": fetched // head["steps"],
        },
        "router_us": round(1e3 * tim["router_ms"] / tim["router_n"], 2),
    }
    # the whole decode step against its two rooflines: the bytes this run
    # fetched over the host link at the measured link rate plus the selected
    # experts' weights streamed from HBM at peak
    ffn_step_bytes = cfg.tokens * cfg.layers * (up_bytes + down_bytes)
    bound_s = fetched / head["steps"] / (link * 1e9) + ffn_step_bytes / (HBM_PEAK_GBPS * 1e9)
    link_s = fetched / head["steps"] / (link * 1e9)
    hbm_s = ffn_step_bytes / (HBM_PEAK_GBPS * 1e9)
    step_s = head["dec"] / head["steps"]
    out["step_roofline"] = {"bound_ms_per_step": round(1e3 * bound_s, 3),
                            "achieved_ms_per_step": round(1e3 * step_s, 3),
                            "frac": round(bound_s / step_s, 4),
                            "terms": "link bytes / measured link + FFN weight bytes / 8 TB/s (no overlap)",
                            "overlap_bound_ms_per_step": round(1e3 * max(link_s, hbm_s), 3),
                            "overlap_frac": round(max(link_s, hbm_s) / step_s, 4)}
    # how the copies overlap the compute: the compute stream's wait between
    # each router and its FFN against the copy time (demand + speculative)
    dec_ms = 1e3 * head["dec"] / head["steps"]
    out["copy_overlap"] = {
        "demand_copy_ms_per_step": round(tim["fetch_ms"] / tsteps, 2),
        "prefetch_copy_ms_per_step": round(tim["pf_fetch_ms"] / tsteps, 2),
        "compute_wait_ms_per_step": round(tim["wait_ms"] / tsteps, 2),
        "link_busy_frac": round(copy_ms / dec_ms, 4) if not cfg.prefill_tokens else None,
        "hidden_copy_frac": round(max(0.0, 1.0 - tim["wait_ms"] / tsteps / copy_ms), 4) if copy_ms > 0 else None,
        "definition": "hidden_copy_frac = 1 - compute wait / copy time: the share of the copy time "
                      "(demand + speculative) during which the compute stream was not waiting",
    }
    # the kernels that rebuild bf16 experts from a coded host store
    rebuild = {"packed": "unpack_kernel", "entropy": "entropy_unpack_kernel"}
    for pk in results:
        if pk["fmt"] == "plain" or rebuild[pk["fmt"]] in out.get("unpack", {}):
            continue
        t = pk["timing"]
        out.setdefault("unpack", {})[rebuild[pk["fmt"]]] = {
            "run": "headline" if pk is head else f"{pk['fmt']} comparison run",
            "avg_launch_us": round(1e3 * t["unpack_ms"] / max(1, t["unpack_n"]), 2),
            "launches": t["unpack_n"], "bytes_per_expert_moved": pk["expert_stride"],
            "bytes_per_expert_rebuilt": cfg.expert_bytes}
    if cfg.prefill_tokens:
        mf = {"bound": "mfma", "unit": "TFLOP/s", "peak": MFMA_BF16_PEAK_TFLOPS,
              "gemm_launches": tim["gemm_up_n"] + tim["gemm_down_n"],
              "prefill_layer_ms": round(tim["prefill_ms"] / max(1, tim["prefill_n"]), 3)}
        for k in ("up", "down"):
            ms = tim[f"gemm_{k}_ms"]
            v = tim[f"gemm_{k}_flop"] / 1e12 / (ms * 1e-3) if ms else None
            mf[f"gemm_{k}_tflops"] = round(v, 1) if v else None
            mf[f"gemm_{k}_frac"] = round(v / MFMA_BF16_PEAK_TFLOPS, 4) if v else None
        out["prefill_mfma"] = mf

    if cpu is None:
        cpu = time_oracle()
    if cpu is not None:
        for key, res, budget in (("cpu_baseline", cpu[0], args.cpu_seconds),
                                 ("cpu_baseline_1thread", cpu[1], args.cpu_seconds / 4)):
            if res is None:
                continue
            tps, n, dt, thr = res
            out[key] = {"value": round(tps, 4), "unit": "tokens/s", "cores": thr, "kind": "oracle",
                        "sample": f"first {n} of the {cfg.tokens} decode tokens (a {budget:g} s budget), fp64 "
                                  f"router + LFU cache + SwiGLU FFN through all {cfg.layers} layers from the warm "
                                  f"start (bf16->fp64 widening included), {dt:.1f} s"}
    store.close()
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixtral-stack", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--cpu-tokens", type=int, default=0,
                    help="most decode tokens the fp64 oracle is timed on (0: the whole workload)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="time budget of the fp64 oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--fetch", choices=["split", "kernel", "dma"], default="split",
                    help="split: demand misses by the copy kernel, speculative prefetches by the DMA engines")
    ap.add_argument("--tokens", type=int, default=0,
                    help="decode only the first N tokens of the workload (profiling passes)")
    ap.add_argument("--lfu-only", action="store_true", help="skip the comparison runs")
    ap.add_argument("--layers", type=int, default=0, help="run only the first N layers of the workload")
    ap.add_argument("--prefill-tokens", type=int, default=-1,
                    help="prefill at most this many tokens (0: decode only)")
    ap.add_argument("--slots", type=int, default=0,
                    help="HBM slots per layer (default 4, 16 for the 64-expert workload; "
                         "slots = experts keeps every expert resident)")
    ap.add_argument("--host-store", choices=["plain", "packed", "entropy"], default="plain",
                    help="packed / entropy: bf16 experts coded losslessly in host memory (~12.25 / ~10.9 bits a "
                         "weight) and rebuilt on the GPU after each copy")
    ap.add_argument("--prefetch-max", type=int, default=-1,
                    help="override the workload's cap on next-layer experts prefetched per layer (0 turns "
                         "speculation off)")
    ap.add_argument("--batch", type=int, default=1,
                    help="decode B tokens per step through the batch path (bf16 experts; no speculation)")
    ap.add_argument("--breakdown-tokens", type=int, default=32,
                    help="stack workloads: tokens of the extra pass with every launch timed")
    ap.add_argument("--no-layer-comparison", action="store_true",
                    help="stack workloads: skip the one-layer Mixtral comparison runs")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the decode path runs on a single GPU with no collectives)", file=sys.stderr)
        sys.exit(2)
    if args.workload in STACK_WORKLOADS and args.batch == 1:
        stack_main(args)
    else:
        layer_main(args)


if __name__ == "__main__":
    main()
