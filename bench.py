#!/usr/bin/env python3
"""Benchmark: prefix tokens/s per Re-Prefill layer step on one MI355X.

A step is one Re-Prefill layer of the hot path (chunk scoring, fp64 fold, top-k
selection, contiguous-span attention over the kept chunks plus the causal
suffix) through ``ckv_reprefill_layer``.  Steps cycle over the workload's layers,
each with its own seeded synthetic Q/K/V resident in HBM before timing starts.

Prints one JSON line.  Untimed diagnostic passes run first (they also bring
the GPU to its working clock): per-stage times from events between every
stage, the step time with no events, and the average time per layer when
layers share their set over Periods of 8 layers (Def. 4.2: one layer in eight
scores and selects) -- context only; the headline metric selects per layer.
Then W warm-up steps and the K timed steps, with no events at all: ``value``
and ``ms_per_step``.  Then the same K steps again on a context that times the
scoring kernel (the dominant kernel) by the kernel's own timestamps (from its
first workgroup's start to its last workgroup's end, 100 MHz realtime
counter), with nothing added between the launches: ``roofline`` is its
algorithmic flops per launch (2*S*Hq*n*d) over the average span,
``roofline.event_avg_us`` the kernel's average time between the HIP events of
the diagnostic pass (which include its dispatch), and
``roofline.trace_avg_us`` / ``frac_at_trace_avg`` the committed rocprofv3
kernel trace's duration of the kernel (dispatch to completion) and the
fraction of the peak at that duration.  ``roofline.traffic`` is the
kernel's HBM bytes per launch from the committed rocprofv3 counter summary
(FETCH_SIZE and WRITE_SIZE, each scaled by what the counter reads for a plain
copy of known size); it is null when the kernel's sources no longer match the
hash recorded with those counters.  ``cpu_baseline`` times the oracle (plain
C, fp64) on a bounded sample of the same workload on this host's cores, and
on one thread.  ``detail`` also holds the kept sets' reads against a store of
64-token blocks (the comparison systems' granularity, Sec. 3) and the
attention-guided cache's hit rates and host cost over a stream of requests on
the same prefix (Sec. 4.5).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefix tokens/sec per Re-Prefill layer step"
PERIOD = 8                  # layers per Period in the Period diagnostic (the paper's setting)
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 (matrix and vector)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def cpu_model() -> str:
    """The host CPU's model name (as lscpu reports it, from /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


SCORE_SOURCES = ("paper_2601_13631_amd/csrc/score.hip", "paper_2601_13631_amd/csrc/ckv_internal.h")


def score_source_hash() -> str:
    h = hashlib.sha256()
    for f in SCORE_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counter_traffic(workload: str):
    """HBM bytes per launch of score_bf16_kernel from the committed counter
    summary, or (None, reason) if there is none for this workload or the
    kernel's sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"score_bf16_kernel_{workload}_pmc.txt")
    if not os.path.exists(path):
        return None, "no counter summary for this workload"
    kv = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith((" ", "#")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != score_source_hash():
        return None, "kernel sources changed since the counters were taken"
    fetch = float(kv["fetch_size_kib_per_dispatch"]) * float(kv["fetch_scale"])
    write = float(kv["write_size_kib_per_dispatch"]) * float(kv["write_scale"])
    return (fetch + write) * 1024.0, os.path.relpath(path, ROOT)


def trace_avg_us(workload: str, kernel: str):
    """The kernel's average duration in the committed rocprofv3 kernel-trace
    summary of this workload (dispatch to completion), or None."""
    path = os.path.join(ROOT, "profiles", f"kernels_{workload}.txt")
    if not os.path.exists(path):
        return None, None
    with open(path) as fh:
        for line in fh:
            f = line.split()
            if len(f) == 4 and f[0] == kernel:
                return float(f[2]), os.path.relpath(path, ROOT)
    return None, None


def host_cache_requests(args, w, ckv, synth, np, torch, layers, stores, dims, k) -> dict:
    """Requests on the shared host-resident prefix (request r's queries from
    synth.request_queries), run layer by layer without a cache and with the
    attention-guided cache (Sec. 4.5) or its frequency-only foil attached, its
    GPU tier held in HBM slots: per request, time per layer and bytes over the
    host link."""
    L, m, R = len(layers), w.n_chunks, args.host_requests
    dev = torch.device("cuda:0")
    qs = [[torch.from_numpy(synth.request_queries(w, l, r)).view(torch.bfloat16).to(dev)
           for l in range(L)] for r in range(R)]
    gpu_slots = int(args.host_cache_frac * L * k)
    out = torch.empty_like(layers[0]["q"])
    res = {"requests": R, "layers": L, "gpu_slots": gpu_slots,
           "slot_bytes": 2 * w.chunk_size * w.n_kv_heads * w.head_dim * w.elem_bytes}
    for name, policy in (("none", None), ("attention", ckv.CACHE_ATTENTION),
                         ("attention_f_loads", ckv.CACHE_LOADS), ("lfu", ckv.CACHE_LFU)):
        ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
        cache = None
        if policy is not None:
            cache = ckv.Cache(L * m, gpu_slots, L * k, policy)
            ctx.attach_cache(cache)
        per = []
        for r in range(R):
            ctx.reset()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            sts = []
            for l in range(L):
                t = layers[l]
                sts.append(ctx.reprefill_layer(l, qs[r][l], t["k_suffix"], t["v_suffix"],
                                               t["k_prefix"], out, kv_host=stores[l],
                                               kv_host_next=stores[l + 1] if l + 1 < L else None))
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            per.append({"us_per_layer": round(dt * 1e6 / L, 1),
                         "host_link_mb_per_layer": round(sum(s_["bytes_prefetch"] + s_["bytes_demand"]
                                                             for s_ in sts) / L / 1e6, 2),
                         "cache_hit_pct": round(100.0 * sum(s_["cache_hits"] for s_ in sts) /
                                                (k * L), 2),
                         "cache_fill_mb_per_layer": round(sum(s_["bytes_cache_fill"] for s_ in sts)
                                                          / L / 1e6, 2)})
        ctx.reset()
        if cache is not None:
            ctx.attach_cache(None)
        ctx.close()
        if cache is not None:
            cache.close()
        res[name] = per
        log(f"requests, cache {name}: " + "; ".join(
            f"{p_['us_per_layer']} us/layer, {p_['host_link_mb_per_layer']} MB/layer" for p_ in per))
    return res


def host_store_run(args, w, ckv, synth, np, torch, host, layers, dims, k) -> dict:
    """The same layers with their chunks on storage: the chunk-major K/V of every
    layer written to one file under --host-store (flushed before timing), read
    by the storage tier's I/O threads with O_DIRECT (the page cache bypassed)
    into the pinned chunk pool and moved to HBM; with the cache attached the
    pool keeps the chunks of its GPU and CPU tiers.  Reports the file's raw read rate
    through the store, then per request the time per layer and the bytes read
    from the file, without and with the attention-guided cache."""
    L, m = len(layers), w.n_chunks
    span = 2 * w.chunk_size * w.n_kv_heads * w.head_dim * w.elem_bytes
    os.makedirs(args.host_store, exist_ok=True)
    path = os.path.join(args.host_store, f"{w.name}_kv.bin")
    with open(path, "wb") as f:
        for h in host:
            h.view(torch.uint8).numpy().tofile(f)
        f.flush()
        os.fsync(f.fileno())
    res = {"file_gib": round(L * m * span / 2**30, 2), "direct": True, "io_threads": args.io_threads,
           "period": args.host_period, "subperiod": args.host_subperiod}
    store = ckv.Store(path, L * m, span, args.io_threads, ckv.STORE_DIRECT)
    buf = torch.empty(m * span, dtype=torch.uint8).pin_memory()
    keys = np.arange(m, dtype=np.int64) + (L - 1) * m
    t0 = time.perf_counter()
    store.read(keys, buf)
    dt = time.perf_counter() - t0
    res["raw_read_gbs"] = round(m * span / dt / 1e9, 2)
    out = torch.empty_like(layers[0]["q"])
    for name, policy in (("none", None), ("attention", ckv.CACHE_ATTENTION)):
        ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
        if args.host_period > 1:
            ctx.set_period(args.host_period)
        ctx.set_subperiod(args.host_subperiod)
        cache = None
        if policy is not None:
            cache = ckv.Cache(L * m, int(args.host_cache_frac * L * k), L * k, policy)
            ctx.attach_cache(cache)
        ctx.attach_store(store)
        per = []
        for r in range(max(1, args.host_requests)):
            q = [layers[l]["q"] if r == 0 else
                 torch.from_numpy(synth.request_queries(w, l, r)).view(torch.bfloat16).to("cuda")
                 for l in range(L)]
            ctx.reset()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            sts = [ctx.reprefill_layer(l, q[l], layers[l]["k_suffix"], layers[l]["v_suffix"],
                                       layers[l]["k_prefix"], out) for l in range(L)]
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            read = sum(s_["bytes_storage"] for s_ in sts)
            link = sum(s_["bytes_prefetch"] + s_["bytes_demand"] for s_ in sts)
            per.append({"us_per_layer": round(dt * 1e6 / L, 1),
                        "store_mb_per_layer": round(read / L / 1e6, 2),
                        "store_gbs": round(read / dt / 1e9, 2),
                        "host_link_mb_per_layer": round(link / L / 1e6, 2),
                        "cache_hit_pct": round(100.0 * sum(s_["cache_hits"] for s_ in sts) / (k * L), 2)})
        ctx.reset()
        ctx.attach_store(None)
        if cache is not None:
            ctx.attach_cache(None)
            cache.close()
        ctx.close()
        res[name] = per
        log(f"store, cache {name}: " + "; ".join(
            f"{p_['us_per_layer']} us/layer, {p_['store_mb_per_layer']} MB/layer" for p_ in per))
    store.close()
    os.remove(path)
    return res


def period_sweep(args, w, ckv, torch, layers, stores, outs, dims, stream) -> dict:
    """Periods of --host-period layers with every layer's pinned store
    registered: a Period's first layer queues the copies of the whole Period
    (intra-period prefetch, Sec. 4.3.2) and its attention waits until the
    Period's first sp layers are in HBM (the SubPeriod gate), for sp in
    1, 2, 4, ... up to the Period.  Per sp: time per layer (host link
    included) over --host-reps passes, and the same without registration
    (one layer ahead) as the reference."""
    L = len(layers)
    res = {"period": args.host_period, "layers": L, "passes": max(1, args.host_reps)}

    def run(ctx):
        def one_pass():
            ctx.reset()
            for l in range(L):
                t = layers[l]
                ctx.reprefill_layer(l, t["q"], t["k_suffix"], t["v_suffix"], t["k_prefix"], outs[l],
                                    kv_host=stores[l],
                                    kv_host_next=stores[l + 1] if l + 1 < L else None, stream=stream)
        one_pass()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(res["passes"]):
            one_pass()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e6 / (res["passes"] * L)

    ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    ctx.set_period(args.host_period)
    res["one_layer_ahead_us_per_layer"] = round(run(ctx), 1)
    ctx.close()
    sp = 1
    while sp <= args.host_period:
        ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
        ctx.set_host_layers(stores[:L] + [stores[-1]] * (w.n_layers - L))
        ctx.set_period(args.host_period)
        ctx.set_subperiod(sp)
        res[f"sp{sp}_us_per_layer"] = round(run(ctx), 1)
        ctx.close()
        sp *= 2
    log("intra-period prefetch, Period " + str(args.host_period) + ": " +
        ", ".join(f"{k} {v}" for k, v in res.items() if k.endswith("per_layer")))
    return res


def host_resident(args, w, ckv, synth, np, torch) -> int:
    """Host-resident prefix (K/V of every layer in pinned host memory, a probe
    copy of K in HBM for scoring): per-layer steps in order, each fetching only
    its selected chunks over the host link (prefetched from the previous
    layer's set on a side stream, misses on demand).  The rate includes the
    host link, so it is reported in ``detail`` and ``value`` stays null."""
    L = min(args.host_layers, w.n_layers)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(0)
    log(f"generating {L} layers of {w.name}")
    host = synth.all_layers(w, layers=range(L), threads=min(16, os.cpu_count() or 1))
    stores = []
    for h in host:
        cm = synth.chunk_major(h["k_prefix"], h["v_prefix"], w.chunk_size)
        stores.append(torch.from_numpy(cm.reshape(-1)).view(torch.bfloat16).pin_memory())
        del h["v_prefix"]
        del cm

    def up(a):
        return torch.from_numpy(a).view(torch.bfloat16).to(dev)

    layers = [{k: up(v) for k, v in h.items()} for h in host]
    del host
    dims = ckv.make_dims(w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim,
                         w.chunk_size, ckv.DTYPE_BF16)
    ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, ckv.CTX_HOST_PREFIX)
    if args.host_period > 1:
        ctx.set_period(args.host_period)
    k = ctx.k
    outs = [torch.empty_like(l["q"]) for l in layers]
    stream = torch.cuda.current_stream()

    def one_pass(collect):
        ctx.reset()
        for l in range(L):
            t = layers[l]
            st = ctx.reprefill_layer(l, t["q"], t["k_suffix"], t["v_suffix"], t["k_prefix"], outs[l],
                                     kv_host=stores[l],
                                     kv_host_next=stores[l + 1] if l + 1 < L else None,
                                     stream=stream)
            if collect is not None:
                collect.append(st)

    log(f"warmup pass over {L} layers")
    one_pass(None)
    torch.cuda.synchronize()
    reps = max(1, args.host_reps)
    stats = []
    log(f"timing {reps} pass(es) over {L} layers")
    t0 = time.perf_counter()
    for _ in range(reps):
        one_pass(stats)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ctx.close()
    n = reps * L
    us = elapsed * 1e6 / n
    link = sum(s_["bytes_prefetch"] + s_["bytes_demand"] for s_ in stats)
    hits = sum(s_["hits"] for s_ in stats)
    later = [s_ for i, s_ in enumerate(stats) if i % L]
    log(f"{us:.1f} us per layer including the host link; {link / elapsed / 1e9:.1f} GB/s over it")
    sweep_detail = period_sweep(args, w, ckv, torch, layers, stores, outs, dims, stream) \
        if args.host_period > 1 and args.host_sweep else None
    cache_detail = host_cache_requests(args, w, ckv, synth, np, torch, layers, stores, dims, k) \
        if args.host_requests > 0 else None
    store_detail = host_store_run(args, w, ckv, synth, np, torch, stores, layers, dims, k) \
        if args.host_store else None
    line = {
        "metric": METRIC, "value": None, "unit": "tokens/s", "n_gpus": 1, "steps": n,
        "warmup": L, "ms_per_step": round(us * 1e-3, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded Q/K/V with planted heavy chunks; prefix K/V in pinned host "
                "memory, probe K in HBM",
        "config": {"workload": w.name, "layers": L, "n_prefix": w.n_prefix, "n_suffix": w.n_suffix,
                   "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "chunk_size": w.chunk_size, "keep_ratio": w.keep_ratio, "kept_chunks": k,
                   "gather": "host -> HBM slots, prefetch of the previous layer's set",
                   "period": args.host_period},
        "roofline": None, "cpu_baseline": None,
        "detail": {
            "note": "host-link-inclusive rate; value is reserved for HBM-resident inputs",
            "pcie_inclusive_prefix_tokens_per_s": round(w.n_prefix / (us * 1e-6), 1),
            "us_per_layer": round(us, 1),
            "stack_ms_layers_run": round(us * L * 1e-3, 3),
            "host_link_gbs": round(link / elapsed / 1e9, 2),
            "host_link_bytes_per_layer": round(link / n),
            "prefetch_hit_rate_after_first_layer": round(
                sum(s_["hits"] for s_ in later) / max(1, sum(s_["k"] for s_ in later)), 4),
            "hits_per_layer": round(hits / n, 1),
        },
    }
    if sweep_detail is not None:
        line["detail"]["intra_period_prefetch"] = sweep_detail
    if cache_detail is not None:
        line["detail"]["cache_requests"] = cache_detail
    if store_detail is not None:
        line["detail"]["storage_tier"] = store_detail
    print(json.dumps(line), flush=True)
    # every library object is closed above; the pinned stores and device
    # tensors are released here too, with the device idle, rather than by
    # interpreter and runtime teardown at exit
    del stores, layers, outs
    import gc
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if hasattr(torch._C, "_host_emptyCache"):
        torch._C._host_emptyCache()
    return 0


def io_sweep(args, ckv, synth, np, torch, dev) -> dict:
    """Untimed: read amplification of a 64-token block store against the chunk
    size, on the kept sets the GPU selects for the 64K-token workload at c = 8,
    16, 32 and 64 (Sec. 3's motivation; the block size of the comparison
    systems), over the first --io-layers layers of each."""
    res = {}
    for name in ("c4_qwen14b_64k_c8", "c4_qwen14b_64k_c16", "c4_qwen14b_64k_c32", "c4_qwen14b_64k_c64"):
        w = synth.WORKLOADS[name]
        dims = ckv.make_dims(w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim,
                             w.chunk_size, ckv.DTYPE_BF16)
        ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, 0)
        hs = synth.heavy_sets(w)
        tot = {"tokens_selected": 0, "runs": 0, "blocks": 0, "tokens_block": 0}
        for l in range(args.io_layers):
            t = {k_: torch.from_numpy(v).view(torch.bfloat16).to(dev)
                 for k_, v in synth.layer_tensors(w, l, hs[l]).items()}
            sel = torch.empty(ctx.k, dtype=torch.int32, device=dev)
            out = torch.empty_like(t["q"])
            ctx.reprefill_layer(l, t["q"], t["k_suffix"], t["v_suffix"], t["k_prefix"], out,
                                k_prefix=t["k_prefix"], v_prefix=t["v_prefix"], sel_idx=sel)
            torch.cuda.synchronize()
            for f, v in ckv.io_account(w.n_prefix, w.chunk_size, sel.cpu().numpy(), 64).items():
                tot[f] += v
            del t
        ctx.close()
        res[f"c{w.chunk_size}"] = {
            "kept_chunks": ctx.k, "tokens_contiguous": tot["tokens_selected"],
            "tokens_block_store": tot["tokens_block"],
            "block_store_read_amplification": round(tot["tokens_block"] / tot["tokens_selected"], 3),
            "contiguous_runs_per_layer": round(tot["runs"] / args.io_layers, 1)}
        log(f"io sweep c={w.chunk_size}: block store reads "
            f"{res[f'c{w.chunk_size}']['block_store_read_amplification']}x the kept tokens")
    return res


def tiers_detail(args, w, ckv, synth, np, torch, layers, dims, dev) -> dict:
    """Untimed: the layers' kept sets for several requests on the shared prefix
    (request r's queries from synth.request_queries), their reads against a
    64-token block store (Sec. 4.2; Sec. 3), and the attention-guided cache
    (Sec. 4.5) against its frequency-only foil over that request stream."""
    L, m, n, c = w.n_layers, w.n_chunks, w.n_prefix, w.chunk_size
    ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, 0)
    k = ctx.k
    out = torch.empty_like(layers[0]["q"])
    sels, scores = [], []
    for r in range(args.requests):
        for l in range(L):
            q = layers[l]["q"] if r == 0 else \
                torch.from_numpy(synth.request_queries(w, l, r)).view(torch.bfloat16).to(dev)
            A = torch.empty(m, dtype=torch.float64, device=dev)
            sel = torch.empty(k, dtype=torch.int32, device=dev)
            ctx.reprefill_layer(l, q, layers[l]["k_suffix"], layers[l]["v_suffix"],
                                layers[l]["k_prefix"], out, k_prefix=layers[l]["k_prefix"],
                                v_prefix=layers[l]["v_prefix"], chunk_scores=A, sel_idx=sel)
            sels.append(sel)
            scores.append(A)
    torch.cuda.synchronize()
    ctx.close()
    sels = [x.cpu().numpy() for x in sels]
    scores = [x.cpu().numpy() for x in scores]
    tot = {"tokens_selected": 0, "runs": 0, "blocks": 0, "tokens_block": 0}
    for sel in sels[:L]:
        for f, v in ckv.io_account(n, c, sel, 64).items():
            tot[f] += v
    io = {"layers": L, "block_tokens": 64, "tokens_contiguous": tot["tokens_selected"],
          "tokens_block_store": tot["tokens_block"],
          "contiguous_pct_of_block_store": round(100.0 * tot["tokens_selected"] /
                                                 tot["tokens_block"], 2),
          "block_store_read_amplification": round(tot["tokens_block"] / tot["tokens_selected"], 3),
          "contiguous_runs_per_layer": round(tot["runs"] / L, 1)}
    gpu_slots, cpu_slots = L * k // 2, L * k
    cache = {"requests": args.requests, "keys": "layer*m+chunk", "gpu_slots": gpu_slots,
             "cpu_slots": cpu_slots}
    # F counting uses (the library's reading), F counting loads into GPU or CPU
    # memory (the paper's wording read literally), and the frequency-only foil
    for name, policy in (("attention", ckv.CACHE_ATTENTION), ("attention_f_loads", ckv.CACHE_LOADS),
                         ("lfu", ckv.CACHE_LFU)):
        cm = ckv.Cache(L * m, gpu_slots, cpu_slots, policy)
        first = None
        t0 = time.perf_counter()
        for i, (sel, A) in enumerate(zip(sels, scores)):
            if i == L:
                _, first = cm.access([], [])
            cm.access((i % L) * m + sel.astype(np.int64), A[sel])
        host_s = time.perf_counter() - t0
        _, tot_c = cm.access([], [])
        cm.close()
        later = {f: tot_c[f] - (first[f] if first else 0) for f in ("hits_gpu", "hits_cpu", "misses")}
        used = sum(later.values())
        cache[name] = {"later_requests_gpu_hit_pct": round(100.0 * later["hits_gpu"] / used, 2) if used else None,
                       "later_requests_cpu_hit_pct": round(100.0 * later["hits_cpu"] / used, 2) if used else None,
                       "later_requests_miss_pct": round(100.0 * later["misses"] / used, 2) if used else None,
                       "host_us_per_layer": round(host_s * 1e6 / len(sels), 2)}
    return {"io_vs_64_token_blocks": io, "cache_manager": cache}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=560)
    ap.add_argument("--warmup", type=int, default=56)
    ap.add_argument("--workload", default="c3_qwen7b_32k")
    ap.add_argument("--materialize", action="store_true",
                    help="gather the kept chunks into compact buffers before attention")
    ap.add_argument("--cpu-layers", type=int, default=3, help="oracle layers in the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--host-layers", type=int, default=8,
                    help="host-resident workloads: layers per pass")
    ap.add_argument("--host-reps", type=int, default=3,
                    help="host-resident workloads: timed passes over those layers")
    ap.add_argument("--host-period", type=int, default=1,
                    help="host-resident workloads: layers per Period (Def. 4.2) in the timed passes")
    ap.add_argument("--host-requests", type=int, default=4,
                    help="host-resident workloads: requests on the shared prefix run without and "
                         "with a cache attached (0: skip)")
    ap.add_argument("--host-cache-frac", type=float, default=0.5,
                    help="host-resident workloads: cache GPU slots as a fraction of one request's "
                         "kept chunks over the layers run")
    ap.add_argument("--host-store", default="",
                    help="host-resident workloads: also run the layers from a file written in this "
                         "directory, read by the storage tier (O_DIRECT)")
    ap.add_argument("--io-threads", type=int, default=16, help="storage tier I/O threads")
    ap.add_argument("--host-sweep", action="store_true",
                    help="host-resident workloads with --host-period p > 1: also time intra-period "
                         "prefetch with the SubPeriod gate at 1, 2, 4, ... p layers")
    ap.add_argument("--host-subperiod", type=int, default=1,
                    help="storage tier: reads up to this many - 1 layers ahead inside a Period")
    ap.add_argument("--io-sweep", action="store_true",
                    help="also report block-store read amplification on the 64K-token workload "
                         "at chunk sizes 8, 16, 32 and 64")
    ap.add_argument("--io-layers", type=int, default=4, help="layers per chunk size in --io-sweep")
    ap.add_argument("--requests", type=int, default=4,
                    help="requests on the shared prefix in the read-accounting and cache diagnostic")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the method's per-layer path is measured on one MI355X)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2601_13631_amd as ckv
    import synth

    w = synth.WORKLOADS[args.workload]
    if w.host_resident:
        return host_resident(args, w, ckv, synth, np, torch)
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    L = w.n_layers
    log(f"generating {L} layers of {w.name}")
    t0 = time.time()
    host = synth.all_layers(w, threads=min(16, os.cpu_count() or 1))
    log(f"generated in {time.time() - t0:.1f}s; uploading")

    def up(a):
        t = torch.from_numpy(a)
        if a.dtype == np.uint16:
            t = t.view(torch.bfloat16)
        return t.to(dev)

    layers = [{k: up(v) for k, v in h.items()} for h in host]
    dims = ckv.make_dims(w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim,
                         w.chunk_size, ckv.DTYPE_F32 if w.dtype == "f32" else ckv.DTYPE_BF16)
    mat = ckv.CTX_MATERIALIZE if args.materialize else 0
    outs = [torch.empty_like(l["q"]) for l in layers]
    stream = torch.cuda.current_stream()

    def step(c, i: int) -> None:
        l = layers[i % L]
        c.reprefill_layer(i % L, l["q"], l["k_suffix"], l["v_suffix"], l["k_prefix"], outs[i % L],
                          k_prefix=l["k_prefix"], v_prefix=l["v_prefix"], stream=stream)

    def timed(c, n: int) -> float:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(n):
            step(c, i)
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    # untimed diagnostics first (they also bring the GPU to its working clock
    # before anything is timed): every stage bracketed by events, then the
    # step with no events at all, then layers sharing their set over Periods of
    # 8 layers (Def. 4.2, the paper's setting: one layer in eight scores and
    # selects, the others attend over its set)
    n_diag = max(4 * L, 112)
    diag = ckv.Context(dims, w.n_layers, w.keep_ratio, ckv.CTX_STAGE_TIMING | mat)
    for i in range(L):
        step(diag, i)
    torch.cuda.synchronize()
    diag.reset()
    for i in range(n_diag):
        step(diag, i)
    stage_ms, n_st = diag.stage_times()
    diag.close()
    per_layer = {s_: stage_ms[s_] / n_st for s_ in stage_ms}
    plain = ckv.Context(dims, w.n_layers, w.keep_ratio, mat)
    for i in range(L):
        step(plain, i)
    plain_us = timed(plain, n_diag) * 1e6 / n_diag
    plain.reset()
    plain.set_period(PERIOD)
    for i in range(L):
        step(plain, i)
    period_us = timed(plain, n_diag) * 1e6 / n_diag
    plain.close()
    log("diagnostic stages (us): " + ", ".join(f"{s_} {v * 1e3:.1f}" for s_, v in per_layer.items()) +
        f"; step without events {plain_us:.1f} us; with Periods of {PERIOD} layers "
        f"{period_us:.1f} us per layer")

    # the headline: W warm-up steps, then K timed steps with no events at all
    ctx = ckv.Context(dims, w.n_layers, w.keep_ratio, mat)
    k = ctx.k
    log(f"warmup {args.warmup} steps")
    for i in range(args.warmup):
        step(ctx, i)
    log(f"timing {args.steps} steps")
    elapsed = timed(ctx, args.steps)
    ctx.close()
    ms_per_step = elapsed * 1e3 / args.steps
    value = w.n_prefix * args.steps / elapsed
    # the same K steps again with the scoring kernel timed by its own
    # timestamps (first workgroup start to last workgroup end): the kernel's
    # average duration for the roofline
    sctx = ckv.Context(dims, w.n_layers, w.keep_ratio, ckv.CTX_SCORE_TIMING | mat)
    for i in range(args.warmup):
        step(sctx, i)
    torch.cuda.synchronize()
    sctx.reset()  # score times restart with the timed pass
    scored_elapsed = timed(sctx, args.steps)
    score_ms, n_timed = sctx.stage_times()
    sctx.close()
    assert n_timed == args.steps, (n_timed, args.steps)
    score_s = score_ms["score"] / n_timed * 1e-3
    log(f"{ms_per_step * 1e3:.1f} us/step; score kernel {score_s * 1e6:.1f} us "
        f"(timed pass: {scored_elapsed * 1e6 / args.steps:.1f} us/step; between events "
        f"{per_layer['score'] * 1e3:.1f} us)")

    # scoring: algorithmic flops per launch / average launch duration
    score_flops = 2.0 * w.n_suffix * w.n_q_heads * w.n_prefix * w.head_dim
    achieved = score_flops / score_s / 1e12
    traffic, traffic_src = counter_traffic(w.name) if w.dtype == "bf16" else (None, "fp32 kernel")
    roofline = {"kernel": "score_bf16_kernel" if w.dtype == "bf16" else "score_f32_kernel",
                "bound": "mfma", "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / (PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS), 4),
                "traffic": round(traffic) if traffic else None, "traffic_source": traffic_src,
                "flops_per_launch": score_flops, "avg_launch_us": round(score_s * 1e6, 2),
                "timing": ("kernel's own timestamps, first workgroup start to last workgroup end"
                           if w.dtype == "bf16" else "HIP events around the kernel"),
                "event_avg_us": round(per_layer["score"] * 1e3, 2)}
    # the committed kernel trace's duration of the same kernel (dispatch to
    # completion: it also holds the dispatch of the workgroups and the
    # end-of-kernel drain), and the fraction of the peak at that duration
    t_us, t_src = trace_avg_us(w.name, roofline["kernel"])
    if t_us:
        roofline.update({"trace_avg_us": t_us, "trace_source": t_src,
                         "frac_at_trace_avg": round(score_flops / (t_us * 1e-6) / 1e12 /
                                                    roofline["peak"], 4)})
    # attention and kept-chunk bytes, as context
    T = k * w.chunk_size
    attn_flops = 4.0 * w.head_dim * w.n_q_heads * (w.n_suffix * T + w.n_suffix * (w.n_suffix + 1) / 2)
    kept_bytes = 2 * T * w.n_kv_heads * w.head_dim * w.elem_bytes
    attn_s = per_layer["attn"] * 1e-3
    others = {
        "attn_tflops": round(attn_flops / attn_s / 1e12, 2),
        "attn_frac_mfma": round(attn_flops / attn_s / 1e12 / PEAK_BF16_TFLOPS, 4),
        "attn_kept_kv_gbs": round(kept_bytes / attn_s / 1e9, 1),
        "stage_us_per_layer": {s_: round(v * 1e3, 2) for s_, v in per_layer.items()},
        "stage_events_note": "diagnostic pass with events between all stages; each event adds a gap",
        "us_per_step_without_events": round(plain_us, 2),
        "us_per_step_scored_pass": round(scored_elapsed * 1e6 / args.steps, 2),
        "stack_ms_all_layers": round(ms_per_step * L, 4),
        f"period{PERIOD}_us_per_layer_without_events": round(period_us, 2),
        f"period{PERIOD}_prefix_tokens_per_s": round(w.n_prefix / (period_us * 1e-6), 1),
    }
    if w.dtype == "bf16" and args.requests > 0:
        others.update(tiers_detail(args, w, ckv, synth, np, torch, layers, dims, dev))
    if args.io_sweep:
        others["io_vs_64_token_blocks_by_chunk_size"] = io_sweep(args, ckv, synth, np, torch, dev)
    if args.materialize and per_layer["move"] > 0:
        others["gather_gbs"] = round(2 * kept_bytes / (per_layer["move"] * 1e-3) / 1e9, 1)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        s = oracle.Shape(w.n_prefix, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim,
                         w.chunk_size, oracle.F32 if w.dtype == "f32" else oracle.BF16)
        threads = os.cpu_count() or 1
        n_cpu = min(args.cpu_layers, L)
        log(f"oracle on {n_cpu} layer(s), {threads} threads")
        t0 = time.perf_counter()
        for l in range(n_cpu):
            h = host[l]
            oracle.reprefill_layer(s, w.keep_ratio, h["q"], h["k_prefix"], h["v_prefix"],
                                   h["k_suffix"], h["v_suffix"], threads=threads)
        cpu_s = time.perf_counter() - t0
        # one thread: the first layer with its first S/8 queries (the oracle's
        # work is linear in the number of queries: every query scores all n
        # prefix keys and attends over the kept chunks plus its causal suffix)
        S1 = max(1, w.n_suffix // 8)
        s1 = oracle.Shape(w.n_prefix, S1, w.n_q_heads, w.n_kv_heads, w.head_dim, w.chunk_size,
                          s.dtype)
        h = host[0]
        t0 = time.perf_counter()
        oracle.reprefill_layer(s1, w.keep_ratio, h["q"][:S1], h["k_prefix"], h["v_prefix"],
                               h["k_suffix"][:S1], h["v_suffix"][:S1], threads=1)
        one_s = time.perf_counter() - t0
        cpu = {"value": round(w.n_prefix * n_cpu / cpu_s, 1), "unit": "tokens/s", "cores": threads,
               "kind": "oracle",
               "sample": f"{n_cpu} full layer(s) of {w.name} (token importance, Eq. 1 pooling, "
                         f"top-k, sparse attention), fp64, {cpu_s:.1f}s",
               "cpu_model": cpu_model(),
               "one_thread": {"sample": f"layer 0 with its first {S1} of {w.n_suffix} queries, "
                                        f"1 thread, {one_s:.2f}s",
                              "est_s_per_layer": round(one_s * w.n_suffix / S1, 1),
                              "est_tokens_per_s": round(w.n_prefix * S1 / (one_s * w.n_suffix), 1)}}
        log(f"oracle {cpu_s:.1f}s on {threads} threads; one thread {one_s:.1f}s for {S1} queries")

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic: seeded Q/K/V with planted heavy chunks, HBM-resident",
        "config": {"workload": w.name, "layers": L, "n_prefix": w.n_prefix, "n_suffix": w.n_suffix,
                   "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "chunk_size": w.chunk_size, "keep_ratio": w.keep_ratio, "kept_chunks": k,
                   "gather": "materialized" if args.materialize else "in-place spans"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "detail": others,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
