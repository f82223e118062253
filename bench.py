"""Benchmark: batch-1 MoE decode under expert offloading on one MI355X.

Workload (one step): 256 batch-1 decode tokens through one Mixtral-8x7B-shaped
MoE layer (8 experts, top-2, d=4096, d_ff=14336, bf16 experts in pinned host
memory), 4 HBM expert slots, LFU eviction; seeded synthetic hidden states
with Zipf(1.1) concept skew and Markov(0.6) persistence.  Each step starts
from the same warm cache (experts 0..3 resident); the warm start and the
restore of the input hidden states are outside the timed region.

Prints one JSON line: decode tokens/s (LFU) and, alongside, LRU tokens/s,
hit rates, the FFN kernels' HBM roofline (event-timed inside the timed
region), the fetch kernel's host-link roofline against the H2D rate measured
here, and the fp64 oracle timed on a bounded sample on the host cores.
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

METRIC = "decode tokens/s per MoE stack at fixed cache slots; expert-FFN HBM GB/s; hit rate"
HBM_PEAK_GBPS = 8000.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def measure_link(torch, nbytes=1 << 30, reps=3):
    """Best pinned host -> HBM copy rate (GB/s) on a 1 GiB transfer."""
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    best = 0.0
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src, non_blocking=True)
        b.record()
        b.synchronize()
        best = max(best, nbytes / (a.elapsed_time(b) * 1e-3) / 1e9)
    del src, dst
    return best


def run_steps(torch, b, moe, H0, H, n, timing):
    """n decode passes over all tokens; returns (seconds, timing dict or None,
    layer-0 statistics summed over the passes)."""
    total = 0.0
    tim = None
    stats = None
    b.moe_cache_set_timing(moe.handle, bool(timing))
    for _ in range(n):
        moe.reset()
        H.copy_(H0)
        torch.cuda.synchronize()
        if timing:
            b.moe_cache_read_timing(moe.handle)  # drop spans of the reset
        t0 = time.perf_counter()
        moe.decode(H)
        moe.sync()
        torch.cuda.synchronize()
        total += time.perf_counter() - t0
        if timing:
            t = b.moe_cache_read_timing(moe.handle)
            tim = t if tim is None else {k: tim[k] + t[k] for k in t}
        st = moe.stats()[0]
        stats = st if stats is None else {k: stats[k] + st[k] for k in st}
    b.moe_cache_set_timing(moe.handle, False)
    return total, tim, stats


def cpu_baseline(cfg, store, gates_host, h0, tokens, slots, policy):
    """The fp64 oracle (router, cache, SwiGLU FFN, residual) on the first
    `tokens` tokens of the same workload, timed on this host's cores."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import stack
    from oracle.cache import make_caches
    model = stack.Model(gates_host, lambda l, e: store.expert(l, e), cfg.d_model, cfg.d_ff, cfg.dtype)
    caches = make_caches(cfg.layers, cfg.experts, slots, policy)
    t0 = time.perf_counter()
    stack.decode_free(model, h0[:tokens].astype(np.float64), cfg.top_k, policy, slots, caches=caches)
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return tokens / dt, dt, threads


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--cpu-tokens", type=int, default=8,
                    help="decode tokens the fp64 oracle is timed on (0: skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--fetch", choices=["kernel", "dma"], default="kernel")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the decode path runs on a single GPU with no collectives)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2511_05814_amd import binding as b
    from paper_2511_05814_amd import offload, workload as wl

    cfg = wl.CONFIGS["mixtral-layer"]
    slots = 4
    fetch_mode = b.MOE_FETCH_KERNEL if args.fetch == "kernel" else b.MOE_FETCH_DMA
    log("generating", cfg.name, "host store", cfg.layers * cfg.experts * cfg.expert_bytes / 1e9, "GB")
    t0 = time.perf_counter()
    store = offload.HostStore(cfg)
    gates = offload.DeviceGates(cfg)
    h0 = wl.hidden_states(cfg, cfg.tokens)
    log(f"inputs ready in {time.perf_counter() - t0:.1f}s")
    link = measure_link(torch)
    log(f"measured pinned H2D link: {link:.2f} GB/s")

    H0 = torch.from_numpy(h0).to("cuda")
    H = torch.empty_like(H0)
    results = {}
    for policy in ("lfu", "lru"):
        moe = offload.OffloadedMoE(cfg, store, gates, slots, policy, fetch_mode=fetch_mode)
        timed = args.steps if policy == "lfu" else 1
        run_steps(torch, b, moe, H0, H, args.warmup if policy == "lfu" else 0, False)
        secs, tim, st = run_steps(torch, b, moe, H0, H, timed, True)
        results[policy] = dict(secs=secs, steps=timed, timing=tim, stats=st)
        log(policy, f"{timed * cfg.tokens / secs:.1f} tok/s", "hits", st["hits"], "misses", st["misses"])
        moe.close()

    lfu = results["lfu"]
    K, d, dff, eb = cfg.top_k, cfg.d_model, cfg.d_ff, cfg.elem_bytes
    tim = lfu["timing"]
    # algorithmic bytes per launch: the selected experts' weights plus the
    # activation vectors the kernel reads and writes
    up_bytes = K * 2 * d * dff * eb + d * 4 + K * dff * 4
    down_bytes = K * d * dff * eb + K * dff * 4 + 2 * d * 4
    up_ms = tim["ffn_up_ms"] / tim["ffn_up_n"]
    down_ms = tim["ffn_down_ms"] / tim["ffn_down_n"]
    up_gbps = up_bytes / (up_ms * 1e-3) / 1e9
    down_gbps = down_bytes / (down_ms * 1e-3) / 1e9
    ffn_gbps = (up_bytes + down_bytes) / ((up_ms + down_ms) * 1e-3) / 1e9
    fetched = lfu["stats"]["bytes_fetched"]
    fetch_gbps = fetched / (tim["fetch_ms"] * 1e-3) / 1e9 if tim["fetch_ms"] > 0 else None
    tokens_per_s = lfu["steps"] * cfg.tokens / lfu["secs"]
    lru = results["lru"]

    out = {
        "metric": METRIC,
        "value": round(tokens_per_s, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * lfu["secs"] / lfu["steps"], 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "mixtral-layer: 1 MoE layer, 8 experts, top-2, d_model 4096, d_ff 14336 "
                        "SwiGLU, bf16 experts in pinned host memory, 256 batch-1 decode tokens, "
                        "4 HBM slots, LFU, Zipf(1.1)+Markov(0.6) routing skew",
            "weights_dtype": "bf16",
            "policy": "lfu",
            "slots": slots,
            "tokens_per_step": cfg.tokens,
            "fetch": args.fetch,
        },
        "hit_rate": round(lfu["stats"]["hits"] / (lfu["stats"]["lookups"] * K), 4),
        "lru": {"tokens_per_s": round(lru["steps"] * cfg.tokens / lru["secs"], 3),
                "hit_rate": round(lru["stats"]["hits"] / (lru["stats"]["lookups"] * K), 4)},
        "ffn_hbm_gbps": round(ffn_gbps, 1),
        "roofline": {
            "kernel": "ffn_up_kernel",
            "bound": "hbm",
            "achieved": round(up_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(up_gbps / HBM_PEAK_GBPS, 4),
            "traffic": None,
            "bytes_per_launch": up_bytes,
            "avg_launch_us": round(up_ms * 1e3, 2),
            "launches": tim["ffn_up_n"],
        },
        "ffn_down": {"achieved_gbps": round(down_gbps, 1), "frac": round(down_gbps / HBM_PEAK_GBPS, 4),
                     "bytes_per_launch": down_bytes, "avg_launch_us": round(down_ms * 1e3, 2)},
        "link_roofline": {
            "kernel": "fetch_kernel",
            "bound": "host-link",
            "achieved": round(fetch_gbps, 2) if fetch_gbps else None,
            "peak": round(link, 2),
            "unit": "GB/s",
            "frac": round(fetch_gbps / link, 4) if fetch_gbps else None,
            "peak_is": "best measured 1 GiB pinned H2D copy",
            "bytes_fetched_per_step": fetched // lfu["steps"],
            "misses_per_step": lfu["stats"]["misses"] // lfu["steps"],
        },
        "router_us": round(1e3 * tim["router_ms"] / tim["router_n"], 2),
    }

    if not args.no_cpu_baseline and args.cpu_tokens > 0:
        tps, dt, thr = cpu_baseline(cfg, store, gates.host, h0, args.cpu_tokens, slots, "lfu")
        out["cpu_baseline"] = {"value": round(tps, 4), "unit": "tokens/s", "cores": thr, "kind": "oracle",
                               "sample": f"first {args.cpu_tokens} of the 256 decode tokens, fp64 router + "
                                         f"cache + SwiGLU FFN (bf16->fp64 widening included), {dt:.1f}s"}
    store.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
