#!/usr/bin/env python3
"""Benchmark of paged decode attention on one MI355X.

A step is one paged_decode_attention call (split kernel + merge kernel: the
whole hot path) over one batch of synthetic inputs already resident in HBM.
The default workload is the 70B-shaped long-context layer (batch 4, 64:8
heads, head_dim 128, 131072 cached tokens per sequence, page size 16): the
configuration that exercises many context splits and the log-sum-exp merge
and whose 2.15 GB of KV cannot sit in the 256 MB last-level cache.

Prints one JSON line.  ``value`` is achieved HBM bandwidth in GB/s computed
from the algorithmic bytes of the call (each live K and V element once, q,
out, page ids, lengths) over the measured time per call.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0   # MI355X HBM3E, 8 TB/s
METRIC = "paged decode attention µs/call + achieved HBM GB/s (% of MI355X peak), 1 GPU"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="long70b",
                    choices=["tiny", "llama8b", "batched", "long70b", "ragged", "window", "multiq", "gqa16",
                             "falcon3", "tokenpage", "prelude_qwen3_4b", "prelude_llama8b", "prelude_70b", "prelude_glm4",
                             "prelude_falcon3", "oproj_qwen3_4b", "oproj_llama8b", "oproj_70b",
                             "oproj_falcon3", "prelude_ragged", "oproj_ragged", "layer70b", "layer8b",
                             "layer_falcon3", "layer_ragged"])
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="budget of each oracle cpu_baseline sample (all cores, then one thread)")
    ap.add_argument("--compute-path", default="mfma", choices=["mfma", "valu"],
                    help="attention products on the matrix cores (default) or the vector-ALU variant "
                         "(the measured alternative; head_dim 128 and <= 8 columns per kv head)")
    ap.add_argument("--seed", type=int, default=None,
                    help="draw the attention workload with this seed instead of its own (same shapes; the "
                         "lengths come first, so two workloads of one length recipe then share lengths)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extra", default="batched,ragged,llama8b",
                    help="comma-separated workloads timed in the same run after the headline one and reported "
                         "under extra_workloads (with the default long70b headline only; '' for none)")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM traffic per launch (from rocprofv3 --pmc runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB device-to-device copy (known HBM traffic) "
                         "to calibrate rocprofv3 FETCH_SIZE / WRITE_SIZE")
    return ap.parse_args()


def copy_calibration(reps=5):
    """A plain copy of 1 GiB: reads 1 GiB and writes 1 GiB per launch."""
    import torch
    n = 1 << 29  # bf16 elements = 1 GiB
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read_per_launch": 2 * n, "bytes_written_per_launch": 2 * n,
                      "launches": reps}), flush=True)


def stream_read_reference(torch, pda, nbytes=1 << 31, reps=20):
    """Bandwidth of the library's plain streaming-read kernel (the attention
    kernel's loads, nothing else) over a 2 GiB buffer: the best median over a
    few launch shapes.  It is what a read-only kernel reaches on this GPU,
    the practical ceiling beside the 8 TB/s specification."""
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    best = None
    for unroll, bpc in ((16, 1), (8, 1), (8, 32)):
        for _ in range(3):
            pda.stream_read(buf, sink, unroll, bpc)
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record()
            pda.stream_read(buf, sink, unroll, bpc)
            a1.record()
            torch.cuda.synchronize()
            ts.append(a0.elapsed_time(a1))
        ts.sort()
        gbs = nbytes / (ts[len(ts) // 2] * 1e-3) / 1e9
        if best is None or gbs > best[0]:
            best = (gbs, unroll, bpc)
    del buf
    return {"gbs": round(best[0], 1), "bytes": nbytes, "unroll": best[1], "blocks_per_cu": best[2],
            "kernel": "stream_read_kernel (16-byte non-temporal buffer loads, read only)"}


def stream_read_same_size(torch, pda, nbytes, reps=24):
    """The library's streaming read over nbytes (the GEMV's own algorithmic
    bytes), cold: each launch reads another window of a 2 GiB buffer, as each
    GEMV call reads another copy of the weights.  Timed like the GEMV kernels
    (an event pair around each of back-to-back launches) over a few launch
    shapes, best median.  A read-only kernel of this size is the practical floor for the
    GEMV: at 20-50 MB the fixed costs of a launch (the first loads' latency,
    the last workgroups) are a large part of the time."""
    n = max(16 * 1024, (int(nbytes) // 1024) * 1024)
    total = 1 << 31
    buf = torch.empty(total, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    windows = max(2, total // n)
    best = None
    k = 0
    for unroll, bpc in ((16, 1), (8, 1), (4, 2), (8, 2)):
        for _ in range(3):
            pda.stream_read(buf[(k % windows) * n:(k % windows) * n + n], sink, unroll, bpc)
            k += 1
        torch.cuda.synchronize()
        # back to back, an event pair around each launch and one synchronize
        # at the end, as the library's own per-kernel events time the GEMV
        evs = []
        for _ in range(reps):
            view = buf[(k % windows) * n:(k % windows) * n + n]
            k += 1
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record()
            pda.stream_read(view, sink, unroll, bpc)
            a1.record()
            evs.append((a0, a1))
        torch.cuda.synchronize()
        ts = sorted(a0.elapsed_time(a1) for a0, a1 in evs)
        us = ts[len(ts) // 2] * 1e3
        if best is None or us < best[0]:
            best = (us, unroll, bpc)
    del buf
    return {"bytes": n, "us": round(best[0], 2), "gbs": round(n / (best[0] * 1e-6) / 1e9, 1),
            "unroll": best[1], "blocks_per_cu": best[2]}


def _host_cores():
    """CPU threads this process may use, at most 16 (one GPU's share of a host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


_POOL_JOB = None  # (work, items, budget, workers), set before the worker processes fork


def _pool_worker(i):
    """Cycle over items i, i + workers, ... (item i mod len(items) when there
    are more workers than items) for the budget; one BLAS thread."""
    from threadpoolctl import threadpool_limits
    work, items, budget_s, workers = _POOL_JOB
    share = items[i::workers] or [items[i % len(items)]]
    nbytes, count = 0, 0
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        deadline = t0 + budget_s
        while True:
            for item in share:
                nbytes += work(item)
                count += 1
                if time.perf_counter() >= deadline:
                    return nbytes, count, t0, time.perf_counter()


def _oracle_rate(work, items, budget_s, workers):
    """Bytes per second of `work(item) -> bytes` over `items`, cycled until the
    budget is spent, in `workers` processes forked from this one (1 = run here).
    Call it before anything in this process touches the GPU: the children are
    plain CPU processes."""
    global _POOL_JOB
    _POOL_JOB = (work, items, budget_s, workers)
    try:
        if workers == 1:
            parts = [_pool_worker(0)]
        else:
            import multiprocessing as mp
            with mp.get_context("fork").Pool(workers) as pool:
                parts = pool.map(_pool_worker, range(workers))
    finally:
        _POOL_JOB = None
    nbytes = sum(p[0] for p in parts)
    count = sum(p[1] for p in parts)
    dt = max(p[3] for p in parts) - min(p[2] for p in parts)  # first start to last end
    return nbytes / dt, count, dt


def cpu_baseline(w, budget_s):
    """Time the fp64 oracle on the same workload: (sequence, kv head) pairs
    (whole sequences for the masked variants) cycled until the budget is
    spent, on every host core (one process per core, each with one thread)
    and on one thread; report GB/s of algorithmic bytes processed."""
    import oracle
    import workloads as W
    variant = w.num_queries > 1 or w.window > 0
    g = w.num_q_heads // w.num_kv_heads
    d = w.head_dim
    rng = np.random.default_rng(0)
    if variant:
        q4 = w.q if w.q.ndim == 4 else w.q[:, None]
        items = list(range(w.batch))

        def work(b):
            oracle.attend_masked(q4[b:b + 1], w.k_cache, w.v_cache, w.block_table[b:b + 1],
                                 w.context_lens[b:b + 1], w.scale, w.window)
            L = int(w.context_lens[b])
            lo = W.window_start(L, w.num_queries, w.window)
            return (4 * d * w.num_kv_heads * (L - lo) + 4 * w.num_queries * w.num_q_heads * d
                    + 4 * ((L + w.page_size - 1) // w.page_size - lo // w.page_size) + 4)
        what = "sequences"
    else:
        items = [(b, kv) for b in range(w.batch) for kv in range(w.num_kv_heads)]

        def work(pair):
            oracle.attend_pairs(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens, w.scale, [pair])
            L = int(w.context_lens[pair[0]])
            return 4 * d * L + 4 * g * d + 4 * ((L + w.page_size - 1) // w.page_size) + 4
        what = "(sequence, kv head) pairs"
    rng.shuffle(items)
    whole = w.algorithmic_bytes()
    cores = _host_cores()
    rate, count, dt = _oracle_rate(work, items, budget_s, cores)
    rate1, count1, dt1 = _oracle_rate(work, items, budget_s, 1)
    return {
        "value": round(rate / 1e9, 4),
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"{count} {what} of the same workload ({len(items)} per call, cycled), {dt:.1f} s of fp64 "
                  f"numpy in {cores} processes of one thread each; host has {os.cpu_count()} logical cpus",
        "us_per_call_equiv": round(whole / rate * 1e6, 1),
        "single_thread": {"value": round(rate1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                          "sample": f"{count1} {what}, {dt1:.1f} s on one thread",
                          "us_per_call_equiv": round(whole / rate1 * 1e6, 1)},
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this path runs on one GPU; --gpus {args.gpus} is not supported "
              "(the kernel works on one GPU's share; sharding across GPUs is not built)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration()
        return
    if args.workload.startswith("prelude_"):
        prelude_main(args)
        return
    if args.workload.startswith("oproj_"):
        oproj_main(args)
        return
    if args.workload.startswith("layer"):
        layer_main(args)
        return

    import torch
    import workloads as W
    from paper_2606_07665_amd import binding as pda

    t_gen = time.perf_counter()
    w = W.make(args.workload, poison=False, seed=args.seed)
    print(f"[bench] generated {args.workload} in {time.perf_counter() - t_gen:.1f}s", file=sys.stderr, flush=True)
    cpu = None
    if not args.no_cpu_baseline:
        # before the GPU is touched: the all-cores leg forks worker processes
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_seconds)
        print(f"[bench] oracle: {cpu['value']} GB/s on {cpu['cores']} cores", file=sys.stderr, flush=True)
    pda.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    pda.set_option(pda.OPT_COMPUTE_PATH, 1 if args.compute_path == "valu" else 0)

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    q, k, v = bf(w.q), bf(w.k_cache), bf(w.v_cache)
    bt = torch.from_numpy(w.block_table).to(dev)
    lens = torch.from_numpy(w.context_lens).to(dev)
    out = torch.empty(tuple(w.q.shape), dtype=torch.bfloat16, device=dev)
    scale = float(w.scale)
    stream = torch.cuda.current_stream()

    variant = w.num_queries > 1 or w.window > 0
    if variant:
        if q.dim() == 3:
            q = q.unsqueeze(1).contiguous()
        out = torch.empty(tuple(q.shape), dtype=torch.bfloat16, device=dev)

    # Cache-resident workloads (KV well under the 256 MB last-level cache) are
    # timed cold: the calls rotate through replicas of the pool, > 1 GB in
    # all, each replica's page table pointing at its own copy.  The warm
    # figure (one replica, back to back) is reported beside it.
    kv_bytes = 2 * k.numel() * k.element_size()
    replicas = 1 if kv_bytes >= 512 * 2 ** 20 else -(-(1100 * 2 ** 20) // kv_bytes)
    warm_call_bt = bt
    if replicas > 1:
        n_pool = k.shape[0]
        k = k.repeat(replicas, 1, 1, 1)
        v = v.repeat(replicas, 1, 1, 1)
        bts = [torch.where(bt >= 0, bt + r * n_pool, bt) for r in range(replicas)]
    else:
        bts = [bt]
    it = [0]

    def call(table=None):
        t = bts[it[0] % replicas] if table is None else table
        it[0] += 1
        if variant:
            pda.paged_decode_attention_ext(q, k, v, t, lens, out, scale, window=w.window)
        else:
            pda.paged_decode_attention(q, k, v, t, lens, out, scale)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()

    # ---- timed region: exactly `steps` calls, events on the launch stream
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps

    # ---- per-call spread: an event pair around each call
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a0, a1 in pairs:
        a0.record(stream)
        call()
        a1.record(stream)
    torch.cuda.synchronize()
    per_call = sorted(a0.elapsed_time(a1) * 1e3 for a0, a1 in pairs)
    pct = {f"p{p_}": round(per_call[min(len(per_call) - 1, int(p_ / 100 * len(per_call)))], 2) for p_ in (10, 50, 90)}
    warm_us = None
    if replicas > 1:
        for _ in range(args.warmup):
            call(warm_call_bt)
        torch.cuda.synchronize()
        w0 = torch.cuda.Event(enable_timing=True)
        w1 = torch.cuda.Event(enable_timing=True)
        w0.record(stream)
        for _ in range(args.steps):
            call(warm_call_bt)
        w1.record(stream)
        torch.cuda.synchronize()
        warm_us = w0.elapsed_time(w1) / args.steps * 1e3

    # ---- per-kernel durations from HIP events the library records around each launch
    pda.profile_enable(True)
    for _ in range(args.steps):
        call()
    torch.cuda.synchronize()
    split_ms, merge_ms, n = pda.profile_read()
    pda.profile_enable(False)
    split_ms /= max(n, 1)
    merge_ms /= max(n, 1)

    # ---- hipGraph replay of 20 back-to-back calls (the paper's runtime replays graphs)
    graph_us = None
    if not args.no_graph:
        s = torch.cuda.Stream()
        pda.workspace_reserve(w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.page_size, w.max_pages,
                              stream=s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(20):
                call()
        g.replay()
        torch.cuda.synchronize()
        reps = max(1, args.steps // 20)
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record()
        for _ in range(reps):
            g.replay()
        g1.record()
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) / (reps * 20) * 1e3

    # ---- the KV append of the same decode step (alone, and append-then-attend)
    rng = np.random.default_rng(1234)
    kv_shape = (w.batch, w.num_kv_heads, w.head_dim)
    k_new = bf(W.f32_to_bf16_bits(rng.standard_normal(kv_shape, dtype=np.float32)))
    v_new = bf(W.f32_to_bf16_bits(rng.standard_normal(kv_shape, dtype=np.float32)))

    def timed(fn):
        for _ in range(5):
            fn()
        a0 = torch.cuda.Event(enable_timing=True)
        a1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a0.record(stream)
        for _ in range(args.steps):
            fn()
        a1.record(stream)
        torch.cuda.synchronize()
        return a0.elapsed_time(a1) / args.steps * 1e3

    append_us = timed(lambda: pda.kv_append(k_new, v_new, k, v, bt, lens))
    append_graph_us = None
    if not args.no_graph:
        # device-side cost without the host launch path: 20 appends in a graph
        ga = torch.cuda.CUDAGraph()
        with torch.cuda.graph(ga, stream=s):
            for _ in range(20):
                pda.kv_append(k_new, v_new, k, v, bt, lens)
        append_graph_us = timed(ga.replay) / 20
    append_attend_us = None
    if not variant:
        append_attend_us = timed(
            lambda: pda.paged_decode_attention_append(q, k_new, v_new, k, v, bt, lens, out, scale))
    append_bytes = 8 * w.batch * w.num_kv_heads * w.head_dim + 8 * w.batch

    stream_ref = stream_read_reference(torch, pda)
    nbytes = w.algorithmic_bytes()
    value = nbytes / (ms_per_step * 1e-3) / 1e9
    achieved = nbytes / (split_ms * 1e-3) / 1e9
    traffic_key = args.workload if args.compute_path == "mfma" else f"{args.workload}@valu"
    traffic = _attention_traffic(args.traffic, traffic_key)
    gpu_name = torch.cuda.get_device_name(0)
    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "us_per_call": round(ms_per_step * 1e3, 2),
        "us_per_call_spread": pct,
        "cold": {"kv_replicas": replicas,
                 "note": "calls rotate through KV replicas > 1 GB in all" if replicas > 1
                 else "KV larger than the last-level cache: every call is cold"},
        "warm_us_per_call": None if warm_us is None else round(warm_us, 2),
        "frac_of_peak": round(value / PEAK_HBM_GBS, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": args.workload,
            "batch": w.batch, "num_q_heads": w.num_q_heads, "num_kv_heads": w.num_kv_heads,
            "head_dim": w.head_dim, "page_size": w.page_size,
            "num_queries": w.num_queries, "window": w.window,
            "total_context_tokens": int(w.context_lens.astype(np.int64).sum()),
            "algorithmic_bytes": nbytes, "parallelism": "single GPU", "device": gpu_name,
            "compute_path": args.compute_path,
            "seed": args.seed if args.seed is not None else W.CONFIGS[args.workload].seed,
        },
        "kernels_ms": {"split": round(split_ms, 5), "merge": round(merge_ms, 5)},
        "graph_us_per_call": None if graph_us is None else round(graph_us, 2),
        "kv_append": {
            "us_per_call": round(append_us, 2), "bytes_per_call": append_bytes,
            "graph_us_per_call": None if append_graph_us is None else round(append_graph_us, 2),
            "append_then_attend_us_per_call": None if append_attend_us is None else round(append_attend_us, 2),
        },
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
            "kernel": "attn_kernel (online-softmax pass over the paged KV)" if args.compute_path == "mfma"
            else "attn_kernel, vector-ALU variant (online-softmax pass over the paged KV)",
            "frac_of_stream_read": round(achieved / stream_ref["gbs"], 4),
        },
        "stream_read": stream_ref,
    }
    if cpu is not None:
        res["cpu_baseline"] = cpu
    extra = [x for x in args.extra.split(",") if x] if args.workload == "long70b" and not variant else []
    if extra:
        del q, k, v, bt, lens, out, bts, warm_call_bt
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        res["extra_workloads"] = {name: extra_workload(name, args, torch, pda, stream_ref["gbs"]) for name in extra}
    print(json.dumps(res), flush=True)


def extra_workload(name, args, torch, pda, stream_gbs):
    """One more attention workload timed in the same run: `steps` calls
    between events on the launch stream after `warmup` calls, then the
    library's per-kernel events over another `steps` calls; a workload that
    fits in the last-level cache rotates over replicas and is also timed
    from a captured graph."""
    import workloads as W
    t_gen = time.perf_counter()
    w = W.make(name, poison=False)
    print(f"[bench] generated {name} in {time.perf_counter() - t_gen:.1f}s", file=sys.stderr, flush=True)
    dev = torch.device("cuda:0")

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    q, k, v = bf(w.q), bf(w.k_cache), bf(w.v_cache)
    bt = torch.from_numpy(w.block_table).to(dev)
    lens = torch.from_numpy(w.context_lens).to(dev)
    out = torch.empty(tuple(w.q.shape), dtype=torch.bfloat16, device=dev)
    scale = float(w.scale)
    stream = torch.cuda.current_stream()
    kv_bytes = 2 * k.numel() * k.element_size()
    # a workload that fits in the last-level cache (llama8b's single request)
    # is timed cold, as in main(): the calls rotate over > 1 GB of replicas
    replicas = 1 if kv_bytes >= 512 * 2 ** 20 else -(-(1100 * 2 ** 20) // kv_bytes)
    if replicas > 1:
        n_pool = k.shape[0]
        k = k.repeat(replicas, 1, 1, 1)
        v = v.repeat(replicas, 1, 1, 1)
        bts = [torch.where(bt >= 0, bt + r * n_pool, bt) for r in range(replicas)]
    else:
        bts = [bt]
    it = [0]

    def call():
        pda.paged_decode_attention(q, k, v, bts[it[0] % replicas], lens, out, scale)
        it[0] += 1

    for _ in range(args.warmup):
        call()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / args.steps * 1e3
    pda.profile_enable(True)
    for _ in range(args.steps):
        call()
    torch.cuda.synchronize()
    split_ms, merge_ms, n = pda.profile_read()
    pda.profile_enable(False)
    split_us = split_ms / max(n, 1) * 1e3
    merge_us = merge_ms / max(n, 1) * 1e3
    graph_us = None
    if replicas > 1 and not args.no_graph:
        # latency-bound: also from a captured graph of 20 calls (how a
        # serving loop replays a decode step)
        s = torch.cuda.Stream()
        pda.workspace_reserve(w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.page_size, w.max_pages,
                              stream=s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(20):
                call()
        g.replay()
        torch.cuda.synchronize()
        reps = max(1, args.steps // 20)
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record()
        for _ in range(reps):
            g.replay()
        g1.record()
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) / (reps * 20) * 1e3
        del g
    nbytes = w.algorithmic_bytes()
    achieved = nbytes / (split_us * 1e-6) / 1e9
    res = {
        "us_per_call": round(us, 2),
        "cold": {"kv_replicas": replicas} if replicas > 1 else None,
        "graph_us_per_call": None if graph_us is None else round(graph_us, 2),
        "gbs_per_call": round(nbytes / (us * 1e-6) / 1e9, 1),
        "frac_of_peak_per_call": round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
        "kernels_us": {"split": round(split_us, 2), "merge": round(merge_us, 2)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "frac_of_stream_read": round(achieved / stream_gbs, 4)},
        "config": {"batch": w.batch, "num_q_heads": w.num_q_heads, "num_kv_heads": w.num_kv_heads,
                   "head_dim": w.head_dim, "page_size": w.page_size,
                   "total_context_tokens": int(w.context_lens.astype(np.int64).sum()), "algorithmic_bytes": nbytes},
    }
    del q, k, v, bt, bts, lens, out
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def prelude_main(args):
    """The attention prelude (QKV GEMV + RoPE, optionally Q/K RMSNorm) of one
    decode step.  Weights are packed once; the timed calls cycle over enough
    copies of the layer's weights (>= 2 GB in all) that every call reads its
    weights from HBM, not from the 256 MB last-level cache, as a model's
    successive layers would."""
    import torch
    import workloads as W
    from paper_2606_07665_amd import binding as pda

    pda.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = W.make_prelude(args.workload)
    dev = torch.device("cuda:0")

    def bf(a):
        if a is None:
            return None
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    x, bias, qn, kn = bf(w.x), bf(w.bias), bf(w.q_norm), bf(w.k_norm)
    lens = torch.from_numpy(w.context_lens).to(dev)
    wp0 = pda.pack_weights(bf(w.w_qkv))
    wbytes = 2 * w.rows * w.hidden
    layers = max(1, -(-2_000_000_000 // wbytes))
    wps = [wp0] + [wp0.clone() for _ in range(layers - 1)]
    b, hq, hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    q = torch.empty((b, hq, d), dtype=torch.bfloat16, device=dev)
    k = torch.empty((b, hkv, d), dtype=torch.bfloat16, device=dev)
    v = torch.empty_like(k)
    stream = torch.cuda.current_stream()
    kw = dict(num_q_heads=hq, num_kv_heads=hkv, head_dim=d, rope_theta=float(w.theta), rotary_dim=w.rotary_dim,
              interleaved=w.interleaved, bias=bias, q_norm=qn, k_norm=kn, eps=float(w.eps))
    it = [0]

    def call():
        pda.attention_prelude(x, wps[it[0] % layers], lens, q, k, v, **kw)
        it[0] += 1

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps

    pda.profile_enable(True)
    for _ in range(args.steps):
        call()
    torch.cuda.synchronize()
    gemv_ms, epi_ms, n = pda.profile_read_prelude()
    pda.profile_enable(False)
    gemv_ms /= max(n, 1)
    epi_ms /= max(n, 1)

    graph_us = None
    if not args.no_graph:
        s = torch.cuda.Stream()
        pda.prelude_workspace_reserve(pda.prelude_dims(b, w.hidden, hq, hkv, d, w.rotary_dim, w.interleaved,
                                                       w.theta, w.eps), stream=s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for i in range(20):
                pda.attention_prelude(x, wps[i % layers], lens, q, k, v, **kw)
        g.replay()
        torch.cuda.synchronize()
        reps = max(1, args.steps // 20)
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record()
        for _ in range(reps):
            g.replay()
        g1.record()
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) / (reps * 20) * 1e3

    stream_ref = stream_read_reference(torch, pda)
    nbytes = w.algorithmic_bytes()
    gemv_bytes = 2 * w.rows * w.hidden + 2 * b * w.hidden     # weights once, x in
    same = stream_read_same_size(torch, pda, gemv_bytes)
    value = nbytes / (ms_per_step * 1e-3) / 1e9
    achieved = gemv_bytes / (gemv_ms * 1e-3) / 1e9
    traffic = None
    traffic = _gemv_traffic(args.workload)
    res = {
        "metric": "attention prelude (QKV GEMV + RoPE) µs/call + achieved HBM GB/s (% of MI355X peak), 1 GPU",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "us_per_call": round(ms_per_step * 1e3, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": args.workload, "batch": b, "hidden": w.hidden, "num_q_heads": hq, "num_kv_heads": hkv,
            "head_dim": d, "rotary_dim": w.rotary_dim, "interleaved": w.interleaved,
            "qk_norm": w.q_norm is not None, "bias": w.bias is not None, "weight_copies": layers,
            "algorithmic_bytes": nbytes, "parallelism": "single GPU", "device": torch.cuda.get_device_name(0),
        },
        "kernels_ms": {"gemv": round(gemv_ms, 5), "epilogue": round(epi_ms, 5)},
        "graph_us_per_call": None if graph_us is None else round(graph_us, 2),
        "roofline": {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
            "kernel": "gemv_kernel (packed-weight MFMA GEMV of the QKV projection)",
            "frac_of_stream_read": round(achieved / stream_ref["gbs"], 4),
            "frac_of_same_size_stream_read": round(achieved / same["gbs"], 4),
        },
        "stream_read": stream_ref,
        "same_size_stream_read": same,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = prelude_cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(res), flush=True)


def oproj_main(args):
    """The output projection + residual add + RMSNorm of one decode step, on
    cold weights (the calls cycle over >= 2 GB of weight copies)."""
    import torch
    import workloads as W
    from paper_2606_07665_amd import binding as pda

    pda.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = W.make_oproj(args.workload)
    dev = torch.device("cuda:0")

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    attn, res, nw = bf(w.attn), bf(w.residual), bf(w.norm_w)
    wp0 = pda.pack_weights(bf(w.w_o))
    wbytes = 2 * w.hidden * w.in_features
    layers = max(1, -(-2_000_000_000 // wbytes))
    wps = [wp0] + [wp0.clone() for _ in range(layers - 1)]
    z = torch.empty_like(res)
    h = torch.empty_like(res)
    stream = torch.cuda.current_stream()
    it = [0]

    def call(i=None):
        j = it[0] if i is None else i
        pda.o_proj_residual_norm(attn, wps[j % layers], res, nw, z, h, eps=float(w.eps))
        it[0] += 1

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps
    pda.profile_enable(True)
    for _ in range(args.steps):
        call()
    torch.cuda.synchronize()
    gemv_ms, epi_ms, n = pda.profile_read_o_proj()
    pda.profile_enable(False)
    gemv_ms /= max(n, 1)
    epi_ms /= max(n, 1)
    graph_us = None
    if not args.no_graph:
        s = torch.cuda.Stream()
        pda.o_proj_workspace_reserve(w.batch, w.in_features, w.hidden, stream=s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for i in range(20):
                call(i)
        g.replay()
        torch.cuda.synchronize()
        reps = max(1, args.steps // 20)
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record()
        for _ in range(reps):
            g.replay()
        g1.record()
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) / (reps * 20) * 1e3
    stream_ref = stream_read_reference(torch, pda)
    nbytes = w.algorithmic_bytes()
    gemv_bytes = wbytes + 2 * w.batch * w.in_features
    achieved = gemv_bytes / (gemv_ms * 1e-3) / 1e9
    same = stream_read_same_size(torch, pda, gemv_bytes)
    res_line = {
        "metric": "o_proj GEMV + residual + RMSNorm µs/call + achieved HBM GB/s (% of MI355X peak), 1 GPU",
        "value": round(nbytes / (ms_per_step * 1e-3) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "us_per_call": round(ms_per_step * 1e3, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": w.batch, "in_features": w.in_features, "hidden": w.hidden,
                   "weight_copies": layers, "algorithmic_bytes": nbytes, "parallelism": "single GPU",
                   "device": torch.cuda.get_device_name(0)},
        "kernels_ms": {"gemv": round(gemv_ms, 5), "epilogue": round(epi_ms, 5)},
        "graph_us_per_call": None if graph_us is None else round(graph_us, 2),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": _gemv_traffic(args.workload),
                     "kernel": "gemv_kernel (packed-weight MFMA GEMV of the output projection)",
                     "frac_of_stream_read": round(achieved / stream_ref["gbs"], 4),
                     "frac_of_same_size_stream_read": round(achieved / same["gbs"], 4)},
        "stream_read": stream_ref,
        "same_size_stream_read": same,
    }
    if not args.no_cpu_baseline:
        import oracle
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t0, calls = time.perf_counter(), 0
            while True:
                oracle.o_proj_residual_norm(w.attn, w.w_o, w.residual, w.norm_w, w.eps)
                calls += 1
                if time.perf_counter() - t0 >= args.cpu_seconds:
                    break
            dt = time.perf_counter() - t0
        res_line["cpu_baseline"] = {"value": round(nbytes * calls / dt / 1e9, 4), "unit": "GB/s", "cores": 1,
                                    "kind": "oracle",
                                    "sample": f"{calls} whole calls of the same workload, {dt:.1f} s fp64 numpy"}
    print(json.dumps(res_line), flush=True)


LAYERS = {
    # attention workload, prelude workload, o_proj workload of one decode step
    "layer70b": ("long70b", "prelude_70b", "oproj_70b"),
    "layer8b": ("batched", "prelude_llama8b", "oproj_llama8b"),
    "layer_falcon3": ("falcon3", "prelude_falcon3", "oproj_falcon3"),
    "layer_ragged": ("ragged", "prelude_ragged", "oproj_ragged"),
}


def layer_main(args):
    """One decode step of one transformer layer's attention block, as the
    paper's runtime replays it: the prelude (QKV projection, RoPE) writing k
    and v into the paged cache, paged decode attention over the advanced
    lengths, and the output projection with residual add and RMSNorm.  The
    lengths already count the new token.  Timed eagerly and as one captured
    graph per step; weights are cold (several layer copies)."""
    import torch
    import workloads as W
    from paper_2606_07665_amd import binding as pda

    pda.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    att_name, pre_name, op_name = LAYERS[args.workload]
    aw = W.make(att_name, poison=False)
    pw = W.make_prelude(pre_name)
    ow = W.make_oproj(op_name)
    assert pw.batch == aw.batch == ow.batch and pw.num_q_heads == aw.num_q_heads
    dev = torch.device("cuda:0")

    def bf(a):
        if a is None:
            return None
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    k, v = bf(aw.k_cache), bf(aw.v_cache)
    bt = torch.from_numpy(aw.block_table).to(dev)
    lens = torch.from_numpy(aw.context_lens).to(dev)
    x = bf(pw.x)
    wq0, wo0 = pda.pack_weights(bf(pw.w_qkv)), pda.pack_weights(bf(ow.w_o))
    layer_bytes = 2 * pw.rows * pw.hidden + 2 * ow.hidden * ow.in_features
    copies = max(1, -(-1_000_000_000 // layer_bytes))
    wqs = [wq0] + [wq0.clone() for _ in range(copies - 1)]
    wos = [wo0] + [wo0.clone() for _ in range(copies - 1)]
    b, hq, d = aw.batch, aw.num_q_heads, aw.head_dim
    q = torch.empty((b, hq, d), dtype=torch.bfloat16, device=dev)
    att = torch.empty_like(q)
    res = bf(ow.residual)
    nw = bf(ow.norm_w)
    z = torch.empty_like(res)
    h = torch.empty_like(res)
    pkw = dict(num_q_heads=hq, num_kv_heads=aw.num_kv_heads, head_dim=d, rope_theta=float(pw.theta),
               rotary_dim=pw.rotary_dim, interleaved=pw.interleaved, bias=bf(pw.bias), q_norm=bf(pw.q_norm),
               k_norm=bf(pw.k_norm), eps=float(pw.eps))
    scale = float(aw.scale)

    def step(i):
        pda.attention_prelude_append(x, wqs[i % copies], lens, q, k, v, bt, **pkw)
        pda.paged_decode_attention(q, k, v, bt, lens, att, scale)
        pda.o_proj_residual_norm(att.reshape(b, hq * d), wos[i % copies], res, nw, z, h, eps=float(ow.eps))

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(args.steps):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps

    graph_us = None
    if not args.no_graph:
        s = torch.cuda.Stream()
        pda.workspace_reserve(b, hq, aw.num_kv_heads, d, aw.page_size, aw.max_pages, stream=s)
        pda.prelude_workspace_reserve(pda.prelude_dims(b, pw.hidden, hq, aw.num_kv_heads, d, pw.rotary_dim,
                                                       pw.interleaved, pw.theta, pw.eps), stream=s)
        pda.o_proj_workspace_reserve(b, ow.in_features, ow.hidden, stream=s)
        graphs = []
        for i in range(copies):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                step(i)
            graphs.append(g)
        for g in graphs:
            g.replay()
        torch.cuda.synchronize()
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record()
        for i in range(args.steps):
            graphs[i % copies].replay()
        g1.record()
        torch.cuda.synchronize()
        graph_us = g0.elapsed_time(g1) / args.steps * 1e3

    nbytes = aw.algorithmic_bytes() + pw.algorithmic_bytes() + ow.algorithmic_bytes()
    res_line = {
        "metric": "one layer's attention block per decode step (prelude + paged attention + o_proj) µs/step "
                  "+ achieved HBM GB/s, 1 GPU",
        "value": round(nbytes / (ms_per_step * 1e-3) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "us_per_call": round(ms_per_step * 1e3, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "attention": att_name, "prelude": pre_name, "o_proj": op_name,
                   "weight_copies": copies, "algorithmic_bytes": nbytes, "parallelism": "single GPU",
                   "device": torch.cuda.get_device_name(0)},
        "graph_us_per_step": None if graph_us is None else round(graph_us, 2),
    }
    print(json.dumps(res_line), flush=True)


def prelude_cpu_baseline(w, budget_s):
    """The fp64 oracle prelude on the same workload, one thread, repeated
    until the budget is used."""
    import oracle
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=1)
    except Exception:  # pragma: no cover
        limiter = None
    calls = 0
    t0 = time.perf_counter()
    while True:
        oracle.prelude(w.x, w.w_qkv, w.num_q_heads, w.num_kv_heads, w.head_dim, w.context_lens, w.theta,
                       bias=w.bias, q_norm=w.q_norm, k_norm=w.k_norm, eps=w.eps, rotary_dim=w.rotary_dim,
                       interleaved=w.interleaved)
        calls += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    if limiter is not None and hasattr(limiter, "unregister"):
        limiter.unregister()
    return {
        "value": round(w.algorithmic_bytes() * calls / dt / 1e9, 4),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"{calls} whole calls of the same workload, {dt:.1f} s single-threaded fp64 numpy; "
                  f"host has {os.cpu_count()} logical cpus",
        "us_per_call_equiv": round(dt / calls * 1e6, 1),
    }


ATTENTION_SOURCES = ("pda_kernels.hip", "pda_internal.h")
GEMV_SOURCES = ("pda_gemv.hip", "pda_gemv.h")


def _attention_traffic(path, workload):
    """Calibrated HBM bytes per attention-kernel launch from a traffic file
    (profiles/traffic.json), or None when the attention source changed since
    the counters were taken or the workload was not profiled."""
    try:
        doc = json.load(open(path))
        t = doc.get(workload)
        if t and doc.get("kernel_source_sha") == _kernel_sha(ATTENTION_SOURCES):
            return t.get("bytes_per_launch")
    except Exception:
        pass
    return None


def _gemv_traffic(workload):
    """Calibrated HBM bytes per GEMV launch from profiles/traffic_gemv.json,
    or None when the GEMV source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic_gemv.json")
    try:
        t = json.load(open(path))
        if t.get("kernel_source_sha") == _kernel_sha(GEMV_SOURCES) and workload in t:
            return t[workload].get("bytes_per_launch")
    except Exception:
        pass
    return None


def _kernel_sha(files=ATTENTION_SOURCES):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_07665_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
