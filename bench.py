#!/usr/bin/env python3
"""One decode step of graph-segment attention on one MI355X, timed.

A step is the whole hot path over one batch of synthetic rollout-graph inputs already resident
in HBM: the GPU segment scheduler (group the branches sharing each segment, rank, chunk, build
the work list), the grouped segment attention kernel, and the log-sum-exp merge.  The default
workload is the merged-DAG rollout (64 prompts, 1024 branches, 7B attention shape).

Prints one JSON line: branch-tokens/s (one decode token per branch per step), the attention
kernel's achieved fraction of the HBM roofline counting unique K/V bytes, and the CPU oracle
timed on a bounded sample of the same workload.

--op extend times the multi-query variant instead (every branch of the merged-DAG rollout extends
a new step of --n-query tokens, all of them queries, causal inside the step): query-tokens/s and
the attention kernel's fraction of the bf16 MFMA roofline on the attention flops.  --op append
times storing one decode step's new K/V (one token per branch) into the page pool.  --op equiv
times equivalence detection (and beside it the graph suffix and the graph reward / dual-group
advantage) for one training batch's rollout states.

Timing: the K timed steps run without per-kernel events (ms_per_step, value); K further steps
time each kernel with HIP events (kernel_ms and the roofline): the attention and merge events are
bound to the kernels' own dispatches, so they span each kernel's execution, and the scheduler's
are recorded around its launches.

The default decode line also carries, under "configs", the same step timed on every other
configuration (tiny fp32 graph, 7B tree, 32B long reasoning, chain and equal-budget graph), with
the attention's fraction of the HBM roofline on unique K/V warm and with the memory-side cache
flushed, and under "decode_loop" the merged-DAG decode loop (append, grow, schedule, attend).
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "branch-tokens/s per decode step; % of HBM roofline on unique KV bytes"
COUNTERS_MD = os.path.join(ROOT, "profiles", "seg_attn_merged_dag_counters.md")
EXT_COUNTERS_MD = os.path.join(ROOT, "profiles", "seg_attn_extend_counters.md")
EQ_COUNTERS_MD = os.path.join(ROOT, "profiles", "equiv_classes_counters.md")
KERNEL_SRC = os.path.join(ROOT, "paper_2606_18954_amd", "csrc", "seg_attn.hip")
EQ_KERNEL_SRC = os.path.join(ROOT, "paper_2606_18954_amd", "csrc", "equiv.hip")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_hash(src=KERNEL_SRC):
    with open(src, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_counters(config, path=COUNTERS_MD, src=KERNEL_SRC):
    """HBM traffic and MFMA busy fraction from the committed rocprofv3 counter summary, only
    if it was taken on this exact kernel source and workload."""
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    kv = dict(re.findall(r"^- (\w+): (\S+)", txt, flags=re.M))
    if kv.get("kernel_source_sha256_16") != kernel_hash(src) or kv.get("workload") != config:
        return None
    return kv


def host_info():
    """The host the CPU oracle runs on: CPU model, cores available to this process, BLAS."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = []
    try:
        from threadpoolctl import threadpool_info
        blas = sorted({f"{i.get('internal_api', '?')} {i.get('version', '')}".strip()
                       for i in threadpool_info()})
    except Exception:
        pass
    return {"cpu_model": model, "cpus_available": len(os.sched_getaffinity(0)), "blas": blas}


def cpu_baseline(wl, n_sample):
    sys.path.insert(0, ROOT)
    from oracle import graphattn_oracle as O
    from paper_2606_18954_amd import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    g = wl.graph
    br = W.sample_branches(g, n_sample, seed=11)
    qb, pb = wl.q_bits(), wl.pool_bits()
    t0 = time.perf_counter()
    O.decode(qb, pb, g.seg_len, g.seg_page_offsets, g.seg_pages, g.path_offsets, g.path_segs,
             wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.dtype, branches=br)
    dt = time.perf_counter() - t0
    toks = sum(g.path_tokens(int(b)) for b in br)
    return {"value": len(br) / dt, "unit": "branch-tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{len(br)} seeded branches of the same workload ({toks} attended tokens), "
                      f"fp64 NumPy, {dt:.1f} s wall",
            "attended_tokens_per_s": toks / dt, "host": host_info()}


def timed_steps(torch, plan, step, steps, preroll=3):
    """Two timed regions of `steps` steps each on the launch stream.  The first has no
    per-kernel events (HIP event records between kernels lengthen a step by a few us each):
    it gives ms per step.  It starts behind `preroll` untimed steps, so that the GPU is already
    busy when its start event is recorded (after a synchronisation the first launch would
    otherwise wait for the host, and the clocks for the work).  The second turns on the
    library's kernel timing (HIP events bound to each attention and merge dispatch, recorded
    around each scheduler pass): it gives each kernel's average duration."""
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    for _ in range(preroll):
        step()
    ev0.record()
    for _ in range(steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    plan.profile(steps)
    for _ in range(steps):
        step()
    prof = plan.profile_read()
    plan.profile(0)
    attn_ms = prof.attn_ms / max(1, prof.runs)
    merge_ms = prof.merge_ms / max(1, prof.runs)
    sched_ms = prof.sched_ms / max(1, prof.schedules)
    log(f"timed {steps} steps: {ms:.4f} ms/step; {steps} more steps with kernel events: "
        f"attention {attn_ms:.4f} ms, merge {merge_ms:.4f} ms, scheduler {sched_ms:.4f} ms")
    return ms, attn_ms, merge_ms, sched_ms


def mall_flushed_attention(torch, plan, step, steps, dev):
    """Attention duration (the library's kernel events) with the memory-side cache (256 MB on
    MI355X) flushed before every step by reading a 512 MiB buffer (a read leaves no dirty lines
    for the attention kernel to write back); the read runs between steps, outside the kernel
    events."""
    junk = torch.ones(1 << 27, dtype=torch.float32, device=dev)
    plan.profile(steps)
    for _ in range(steps):
        junk.sum()
        step()
    prof = plan.profile_read()
    plan.profile(0)
    del junk
    torch.cuda.empty_cache()
    return prof.attn_ms / max(1, prof.runs)


def median_step_ms(torch, step, steps):
    """Median of per-step durations: one event pair around each step (the records between steps
    add a little to each; ms_per_step comes from the region without them)."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record()
        step()
        e1.record()
    torch.cuda.synchronize()
    d = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    return d[len(d) // 2] if len(d) % 2 else 0.5 * (d[len(d) // 2 - 1] + d[len(d) // 2])


def stream_copy_gbs(torch, dev, reps=10):
    """Bandwidth of a plain device copy (torch elementwise, 1 GiB read + 1 GiB written)."""
    a = torch.ones(1 << 29, dtype=torch.bfloat16, device=dev)
    b = torch.empty_like(a)
    torch.mul(a, 1.0, out=b)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        torch.mul(a, 1.0, out=b)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    torch.cuda.empty_cache()
    return 2.0 * (1 << 30) / (ms * 1e-3) / 1e9


def extend_flops(wl):
    """Attention flops of an extend step: 2 D per visible token for S = Q K^T and 2 D for O = P V,
    per query row and q-head; query i of branch b sees its path's other segments whole and
    len(last) - n_b + i + 1 tokens of the newest one."""
    g = wl.graph
    vis = 0
    for b in range(g.num_branches):
        n = int(wl.query_counts[b])
        L = g.path_tokens(b)
        vis += n * (L - n) + n * (n + 1) // 2
    return 4 * wl.head_dim * wl.num_q_heads * vis, vis


def cpu_baseline_extend(wl, n_sample):
    sys.path.insert(0, ROOT)
    import numpy as np
    from oracle import graphattn_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    g = wl.graph
    R = int(wl.query_counts.sum())
    rows = sorted(np.random.default_rng(11).choice(R, min(n_sample, R), replace=False).tolist())
    t0 = time.perf_counter()
    O.extend(wl.q_bits(), wl.pool_bits(), g.seg_len, g.seg_page_offsets, g.seg_pages,
             g.path_offsets, g.path_segs, wl.query_counts, wl.num_q_heads, wl.num_kv_heads,
             wl.head_dim, wl.dtype, rows=rows)
    dt = time.perf_counter() - t0
    return {"value": len(rows) / dt, "unit": "query-tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{len(rows)} seeded query rows of the same workload, fp64 NumPy, "
                      f"{dt:.1f} s wall"}


def calibrate_copy(torch, dev):
    """A plain elementwise copy of 1 GiB (bf16) three times: a kernel of known HBM traffic to
    scale the FETCH_SIZE / WRITE_SIZE counters against."""
    n = 1 << 29                                   # 1 GiB of bf16 read, 1 GiB written
    a = torch.ones(n, dtype=torch.bfloat16, device=dev)
    b = torch.empty_like(a)
    for _ in range(3):
        torch.mul(a, 1.0, out=b)
    torch.cuda.synchronize()
    log("copy calibration: 3 launches of a 1 GiB elementwise copy")
    del a, b
    torch.cuda.empty_cache()


def run_extend(args, torch, G, W):
    t0 = time.time()
    wl = W.config3_extend(n_query=args.n_query)
    g = wl.graph
    R = int(wl.query_counts.sum())
    log(f"workload {wl.name}: B={g.num_branches} rows={R} pages={g.num_pages} generated in "
        f"{time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    q, pool = wl.q.to(dev), wl.pool.to(dev)
    Hq, D = wl.num_q_heads, wl.head_dim
    out = torch.empty((R, Hq, D), dtype=q.dtype, device=dev)
    lse = torch.empty((R, Hq), dtype=torch.float32, device=dev)
    hg = G.HostGraph.from_graph(g)
    params = G.make_params(Hq, wl.num_kv_heads, D, g.num_pages, wl.dtype)
    plan = G.Plan(hg, params, query_counts=wl.query_counts)
    info = plan.info()

    def step():
        plan.schedule()
        plan.run(q, pool, out, lse)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ms, attn_ms, merge_ms, sched_ms = timed_steps(torch, plan, step, args.steps)
    flops, vis = extend_flops(wl)
    achieved = flops / (attn_ms * 1e-3) / 1e12
    ukv = wl.unique_kv_bytes()
    cnt = measured_counters("extend", EXT_COUNTERS_MD)
    traffic = None
    if cnt:
        traffic = float(cnt["fetch_bytes_per_launch"]) + float(cnt["write_bytes_per_launch"])
    res = {
        "metric": "query-tokens/s per extend step; % of bf16 MFMA roofline on attention flops",
        "value": R / (ms * 1e-3), "unit": "query-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) K/V/Q, seeded rollout graph)",
        "config": {"workload": wl.name, "branches": g.num_branches, "query_rows": R,
                   "n_query": args.n_query, "segments": g.num_segments,
                   "unique_tokens": g.unique_tokens(), "visible_token_pairs": vis,
                   "q_heads": Hq, "kv_heads": wl.num_kv_heads, "head_dim": D,
                   "page_tokens": 16, "chunk_pages": info.chunk_pages},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / MFMA_BF16_PEAK_TFLOPS,
                     "traffic": traffic},
        "kernel_ms": {"scheduler": sched_ms, "attention": attn_ms, "merge": merge_ms},
        "timing": "ms_per_step over the timed steps without per-kernel events, started behind "
                  "3 untimed steps so the GPU is busy at the start event; kernel_ms (and "
                  "the roofline) from as many further steps with HIP events bound to the attention "
                  "and merge dispatches (recorded around the scheduler)",
        "attention_flops": flops,
        "unique_kv_bytes": ukv,
        "unique_kv_hbm_frac": ukv / (attn_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
    }
    plan.close()
    del q, pool, out, lse
    torch.cuda.empty_cache()
    if args.calibrate_copy:
        calibrate_copy(torch, dev)
    if args.cpu_sample > 0:
        n = min(args.cpu_sample, 1024)
        log(f"timing the CPU oracle on {n} query rows")
        res["cpu_baseline"] = cpu_baseline_extend(wl, n)
    print(json.dumps(res), flush=True)


def run_append(args, torch, G, W):
    """One decode step's new K/V: the token of every branch of the merged-DAG rollout, stored
    at the next slot of its newest segment (a page of its own per branch).  A step is one call;
    the calls are timed replayed from a HIP graph (the call rate from Python is also given)."""
    import numpy as np
    wl = W.config3_merged_dag()
    g = wl.graph
    B, Hkv, D = g.num_branches, wl.num_kv_heads, wl.head_dim
    dev = torch.device("cuda:0")
    pool = wl.pool.to(dev)
    words = np.empty(B, dtype=np.int32)
    for b in range(B):
        s = int(g.path(b)[-1])
        t = int(g.seg_len[s]) % 16            # the slot after the segment's last token
        words[b] = int(g.seg_pages[g.seg_page_offsets[s + 1] - 1]) * 16 + t if t else -1
    keep = words >= 0
    gen = torch.Generator().manual_seed(7)
    kn = torch.randn((B, Hkv, D), generator=gen).to(torch.bfloat16).to(dev)
    vn = torch.randn((B, Hkv, D), generator=gen).to(torch.bfloat16).to(dev)
    wd = torch.from_numpy(words).to(dev)
    params = G.make_params(wl.num_q_heads, Hkv, D, g.num_pages, "bf16")
    for _ in range(args.warmup):
        G.kv_append(pool, kn, vn, wd, params)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        G.kv_append(pool, kn, vn, wd, params)
    ev1.record()
    torch.cuda.synchronize()
    host_ms = ev0.elapsed_time(ev1) / args.steps
    # Launched one by one from Python, the calls are spaced by the host; replayed from a HIP
    # graph (the calls captured back to back, no memsets) they run at the GPU's own pace.
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            for _ in range(args.steps):
                G.kv_append(pool, kn, vn, wd, params)
    torch.cuda.current_stream().wait_stream(side)
    graph.replay()
    torch.cuda.synchronize()
    ev0.record()
    graph.replay()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    log(f"append: {ms * 1e3:.2f} us per call replayed from a graph, {host_ms * 1e3:.2f} us per "
        f"call launched from Python")
    n = int(keep.sum())
    moved = n * Hkv * 2 * D * 2 * 2                 # read + written
    achieved = moved / (ms * 1e-3) / 1e9
    res = {
        "metric": "tokens/s stored per K/V append call; % of HBM roofline on bytes moved",
        "value": n / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "one decode step of the merged-DAG rollout (1024 branches, "
                               "28/4/128): one new token per branch", "tokens": n,
                   "padded_words": int(B - n)},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None},
        "ms_per_call_from_python": host_ms,
    }
    print(json.dumps(res), flush=True)


def measure_loop(torch, G, W, steps, warmup):
    """The decode loop on the merged-DAG rollout: every step stores one new token at the end of
    each newest segment (graphattn_kv_append), grows those segments by one token
    (graphattn_plan_set_lengths: the plan's chains rebuilt on the device), schedules and
    attends.  The page table gives every newest segment the pages it grows into; the pool gets
    those pages on top of the rollout's own.  Returns (workload, ms per step, host ms of one
    length update with the device idle, newest segments)."""
    import numpy as np
    wl = W.config3_merged_dag()
    g = wl.graph
    B, Hq, Hkv, D = g.num_branches, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    total = warmup + steps + 1
    newest = np.unique(np.array([int(g.path(b)[-1]) for b in range(B)]))
    S = g.num_segments
    lens = g.seg_len.astype(np.int32).copy()
    extra = np.zeros(S, dtype=np.int64)
    for s in newest:
        extra[s] = (int(lens[s]) + total + 15) // 16 - (int(lens[s]) + 15) // 16
    offs = np.zeros(S + 1, dtype=np.int64)
    np.cumsum((lens.astype(np.int64) + 15) // 16 + extra, out=offs[1:])
    pages = np.empty(int(offs[-1]), dtype=np.int32)
    nxt = g.num_pages
    for s in range(S):
        own = g.seg_pages[g.seg_page_offsets[s]:g.seg_page_offsets[s + 1]]
        pages[offs[s]:offs[s] + len(own)] = own
        pages[offs[s] + len(own):offs[s + 1]] = np.arange(nxt, nxt + extra[s], dtype=np.int32)
        nxt += int(extra[s])
    num_pages = nxt
    dev = torch.device("cuda:0")
    gen = torch.Generator().manual_seed(wl.seed + 29)
    pool = torch.cat([wl.pool, torch.randn((num_pages - g.num_pages, Hkv, 2, 16, D),
                                           generator=gen).to(wl.pool.dtype)]).to(dev)
    q = wl.q.to(dev)
    out = torch.empty((B, Hq, D), dtype=q.dtype, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    hg = G.HostGraph(lens.tolist(), offs, pages, g.path_offsets, g.path_segs)
    params = G.make_params(Hq, Hkv, D, num_pages, wl.dtype)
    plan = G.Plan(hg, params)
    n = len(newest)
    kn = torch.randn((n, Hkv, D), generator=gen).to(q.dtype).to(dev)
    vn = torch.randn((n, Hkv, D), generator=gen).to(q.dtype).to(dev)
    # slot words of every step's new tokens, uploaded once
    words = np.empty((total, n), dtype=np.int32)
    for k in range(total):
        t = lens[newest] + k
        words[k] = pages[offs[newest] + t // 16] * 16 + t % 16
    wd = torch.from_numpy(words).to(dev)
    cur = lens.copy()
    k = 0

    def step():
        nonlocal k
        G.kv_append(pool, kn, vn, wd[k], params)
        cur[newest] += 1
        plan.set_lengths(cur)
        plan.schedule()
        plan.run(q, pool, out, lse)
        k += 1

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # the length update's own host time, with the device idle (inside the loop the host waits
    # wherever the runtime's queue of submitted work is full, which is GPU time, not this call)
    host_s = []
    for _ in range(20):
        t0 = time.perf_counter()
        plan.set_lengths(cur)
        host_s.append(time.perf_counter() - t0)
        torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    set_ms = 1e3 * float(np.median(host_s))
    plan.close()
    del pool, q, out, lse
    torch.cuda.empty_cache()
    log(f"decode loop: {ms:.4f} ms per step (append {n} tokens, grow, schedule, attend); "
        f"length update {set_ms:.3f} ms on the host")
    return wl, ms, set_ms, int(n)


def run_loop(args, torch, G, W):
    wl, ms, set_ms, n = measure_loop(torch, G, W, args.steps, args.warmup)
    g = wl.graph
    B = g.num_branches
    res = {
        "metric": "branch-tokens/s per decode-loop step (append, grow, schedule, attend)",
        "value": B / (ms * 1e-3), "unit": "branch-tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": wl.name + ", decode loop", "branches": B,
                   "newest_segments": n, "q_heads": wl.num_q_heads, "kv_heads": wl.num_kv_heads,
                   "head_dim": wl.head_dim},
        "set_lengths_host_ms": set_ms,
    }
    print(json.dumps(res), flush=True)


def compared_pairs_count(parent):
    """Pairs the method compares: same prompt, neither an ancestor of the other.  A prompt with n
    states has n (n - 1) / 2 pairs, of which sum over states of (depth) are ancestor pairs."""
    import numpy as np
    N = len(parent)
    depth = np.zeros(N, dtype=np.int64)
    for v in range(N):
        depth[v] = 0 if parent[v] < 0 else depth[parent[v]] + 1
    roots = np.nonzero(parent < 0)[0].tolist() + [N]
    pairs = sum((b - a) * (b - a - 1) // 2 for a, b in zip(roots[:-1], roots[1:]))
    return pairs - int(depth.sum())


def run_equiv(args, torch, G, W):
    """Equivalence detection for one training batch's states: classes and edge similarities (the
    timed step); the graph suffix (it synchronises to size its output) and the graph reward and
    dual-group advantage timed on their own."""
    import numpy as np
    t0 = time.time()
    wl = W.equiv_batch()
    N, dim = wl.z.shape
    log(f"workload {wl.name} generated in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    z = wl.z.to(dev)
    f = G.Forest(wl.parent)
    labels = torch.empty(N, dtype=torch.int32, device=dev)
    esim = torch.empty(N, dtype=torch.float32, device=dev)
    for _ in range(args.warmup):
        f.classes(z, wl.kappa, labels, esim)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        f.classes(z, wl.kappa, labels, esim)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    # Graph reward and dual-group advantage on the same states (synthetic verifier outcomes).
    reward = torch.from_numpy(W.state_rewards(wl.parent, wl.seed)).to(dev)
    adv = f.advantages(labels, reward, esim, 0.7, 0.5)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        f.advantages(labels, reward, esim, 0.7, 0.5, out=adv)
    ev1.record()
    torch.cuda.synchronize()
    adv_ms = ev0.elapsed_time(ev1) / args.steps
    lab = labels.cpu().numpy()
    offs = torch.empty(N + 1, dtype=torch.int64, device=dev)
    total = f.suffix_total(labels, offs)
    states = torch.empty(max(1, total), dtype=torch.int32, device=dev)
    f.suffix(labels, offs, states)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        f.suffix(labels, offs, states)
    ev1.record()
    torch.cuda.synchronize()
    suffix_ms = ev0.elapsed_time(ev1) / args.steps
    log(f"timed {args.steps} steps: classes {ms:.4f} ms, graph suffix {suffix_ms:.4f} ms "
        f"(with its host synchronisation), reward and advantages {adv_ms:.4f} ms")
    zbytes = N * dim * 2
    pairs = compared_pairs_count(wl.parent)
    achieved = zbytes / (ms * 1e-3) / 1e9
    merged = int((lab != np.arange(N)).sum())
    cnt = measured_counters("equiv", EQ_COUNTERS_MD, EQ_KERNEL_SRC)
    traffic = None
    if cnt:
        traffic = float(cnt["fetch_bytes_per_launch"]) + float(cnt["write_bytes_per_launch"])
    res = {
        "metric": "rollout states/s classified per equivalence-detection call; % of HBM "
                  "roofline on embedding bytes",
        "value": N / (ms * 1e-3), "unit": "states/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded clustered N(0,1) embeddings, seeded state forest)",
        "config": {"workload": wl.name, "states": int(N), "dim": int(dim), "kappa": wl.kappa,
                   "compared_pairs": pairs, "classes": int(len(set(lab.tolist()))),
                   "merged_states": merged, "suffix_entries": total},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic},
        "compared_pair_tflops": pairs * 2 * dim / (ms * 1e-3) / 1e12,
        "kernel_ms": {"classes": ms, "graph_suffix": suffix_ms, "advantages": adv_ms},
    }
    f.close()
    if args.calibrate_copy:
        calibrate_copy(torch, dev)
    if args.cpu_sample > 0:
        from oracle import graphattn_oracle as O
        per = 205
        n = min(512, N // per)
        t1 = time.perf_counter()
        for p in range(n):
            a, b = p * per, (p + 1) * per
            sub = wl.parent[a:b].copy()
            sub[1:] -= a
            O.equivalence_classes(wl.z_bits()[a:b], "bf16", sub, wl.kappa)
        dt = time.perf_counter() - t1
        res["cpu_baseline"] = {"value": n * per / dt, "unit": "states/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{n} prompts ({n * per} states) of the same batch, "
                                         f"fp64 NumPy, {dt:.1f} s wall"}
    print(json.dumps(res), flush=True)


def other_config(torch, G, W, name, dev, steps):
    """One more configuration's decode step (schedule + attention + merge), timed like the main
    one on fewer steps: ms per step, each kernel's average duration from HIP events, the
    attention with the memory-side cache flushed before each step, and unique-K/V rates."""
    t0 = time.time()
    wl = W.CONFIGS[name]()
    g = wl.graph
    q, pool = wl.q.to(dev), wl.pool.to(dev)
    B, Hq, D = g.num_branches, wl.num_q_heads, wl.head_dim
    out = torch.empty((B, Hq, D), dtype=q.dtype, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    plan = G.Plan(G.HostGraph.from_graph(g), G.make_params(Hq, wl.num_kv_heads, D, g.num_pages,
                                                            wl.dtype))

    def step():
        plan.schedule()
        plan.run(q, pool, out, lse)

    for _ in range(3):
        step()
    torch.cuda.synchronize()
    ms, attn_ms, merge_ms, sched_ms = timed_steps(torch, plan, step, steps)
    cold_ms = mall_flushed_attention(torch, plan, step, steps, dev)
    plan.close()
    del q, pool, out, lse
    torch.cuda.empty_cache()
    ukv = wl.unique_kv_bytes()
    log(f"{name}: {ms:.4f} ms/step, attention {attn_ms:.4f} ms ({cold_ms:.4f} ms cold) "
        f"[{time.time() - t0:.1f} s]")
    return {"workload": wl.name, "dtype": wl.dtype, "branches": B,
            "unique_kv_bytes": ukv, "attended_tokens": g.attended_tokens(),
            "ms_per_step": ms, "branch_tokens_per_s": B / (ms * 1e-3),
            "kernel_ms": {"scheduler": sched_ms, "attention": attn_ms, "merge": merge_ms,
                          "attention_mall_flushed": cold_ms},
            "attention_unique_kv_frac": ukv / (attn_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "mall_flushed_frac": ukv / (cold_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "step_unique_kv_frac": ukv / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="c3",
                    choices=["c1", "c2", "c3", "c4", "c5chain", "c5graph"])
    ap.add_argument("--op", default="decode",
                    choices=["decode", "extend", "append", "equiv", "loop"])
    ap.add_argument("--n-query", type=int, default=16,
                    help="query tokens per branch for --op extend")
    ap.add_argument("--cpu-sample", type=int, default=1024,
                    help="branches the CPU oracle is timed on (0 skips it)")
    ap.add_argument("--all-configs", type=int, default=1,
                    help="decode only: also time the other configurations and the decode loop "
                         "(1, the default) and report them under configs / decode_loop")
    ap.add_argument("--other-steps", type=int, default=50,
                    help="timed steps per region for the other configurations")
    ap.add_argument("--cpu-configs", action="store_true",
                    help="decode only: also time the CPU oracle on a bounded seeded sample of "
                         "each other configuration (reported under cpu_configs; minutes of CPU "
                         "work, off by default)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (torch elementwise kernel) so HBM "
                         "counters can be scaled against a kernel of known traffic")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the design notes "
              "describe how prompts would be sharded across GPUs). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    sys.path.insert(0, ROOT)
    import torch
    from paper_2606_18954_amd import graphattn as G
    from paper_2606_18954_amd import workloads as W

    if args.op == "extend":
        return run_extend(args, torch, G, W)
    if args.op == "append":
        return run_append(args, torch, G, W)
    if args.op == "equiv":
        return run_equiv(args, torch, G, W)
    if args.op == "loop":
        return run_loop(args, torch, G, W)
    t0 = time.time()
    wl = W.CONFIGS[args.config]()
    g = wl.graph
    log(f"workload {wl.name}: B={g.num_branches} S={g.num_segments} pages={g.num_pages} "
        f"generated in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    q, pool = wl.q.to(dev), wl.pool.to(dev)
    B, Hq, D = g.num_branches, wl.num_q_heads, wl.head_dim
    out = torch.empty((B, Hq, D), dtype=q.dtype, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    hg = G.HostGraph.from_graph(g)
    params = G.make_params(Hq, wl.num_kv_heads, D, g.num_pages, wl.dtype)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    plan = G.Plan(hg, params)                       # host validation, chains, index upload
    torch.cuda.synchronize()
    plan_ms = (time.perf_counter() - t1) * 1e3
    info = plan.info()

    def step():
        plan.schedule()
        plan.run(q, pool, out, lse)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")
    ms, attn_ms, merge_ms, sched_ms = timed_steps(torch, plan, step, args.steps)
    cold_ms = mall_flushed_attention(torch, plan, step, args.steps, dev)
    med_ms = median_step_ms(torch, step, args.steps)
    copy_gbs = stream_copy_gbs(torch, dev)
    log(f"attention with the memory-side cache flushed before each step: {cold_ms:.4f} ms; "
        f"plain device copy: {copy_gbs:.0f} GB/s; plan creation {plan_ms:.1f} ms")

    ukv = wl.unique_kv_bytes()
    achieved = ukv / (attn_ms * 1e-3) / 1e9
    cnt = measured_counters(args.config)
    traffic = None
    mfma = None
    if cnt:
        traffic = float(cnt["fetch_bytes_per_launch"]) + float(cnt["write_bytes_per_launch"])
        mfma = float(cnt["mfma_busy_fraction"]) if "mfma_busy_fraction" in cnt else None
    res = {
        "metric": METRIC,
        "value": B / (ms * 1e-3),
        "unit": "branch-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) K/V/Q, seeded rollout graph)",
        "config": {"workload": wl.name, "branches": B, "segments": g.num_segments,
                   "unique_tokens": g.unique_tokens(), "attended_tokens": g.attended_tokens(),
                   "q_heads": Hq, "kv_heads": wl.num_kv_heads, "head_dim": D, "page_tokens": 16,
                   "chunk_pages": info.chunk_pages},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic},
        "kernel_ms": {"scheduler": sched_ms, "attention": attn_ms, "merge": merge_ms,
                      "attention_mall_flushed": cold_ms},
        "timing": "ms_per_step over the timed steps without per-kernel events, started behind "
                  "3 untimed steps so the GPU is busy at the start event; kernel_ms (and "
                  "the roofline) from as many further steps with HIP events bound to the attention "
                  "and merge dispatches (recorded around the scheduler); attention_mall_flushed "
                  "from as many more with a 512 MiB "
                  "read between steps",
        "mall_flushed_frac": ukv / (cold_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "ms_per_step_median": med_ms,
        "stream_copy_gbs": copy_gbs,
        "frac_of_stream_copy": achieved / copy_gbs,
        "plan_create_ms": plan_ms,
        "pcie_inclusive_branch_tokens_per_s": B / ((plan_ms + ms) * 1e-3),
        "unique_kv_bytes": ukv,
        "step_unique_kv_frac": ukv / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "attended_tokens_per_s": g.attended_tokens() / (ms * 1e-3),
        "mfma_busy_fraction": mfma,
    }
    plan.close()
    del q, pool, out, lse
    torch.cuda.empty_cache()
    if args.all_configs:
        res["configs"] = {}
        for name in ["c1", "c2", "c3", "c4", "c5chain", "c5graph"]:
            if name != args.config:
                res["configs"][name] = other_config(torch, G, W, name, dev, args.other_steps)
        _, loop_ms, set_ms, n = measure_loop(torch, G, W, args.other_steps, 3)
        res["decode_loop"] = {
            "workload": wl.name + ", decode loop" if args.config == "c3" else
                        "merged-DAG rollout decode loop",
            "ms_per_step": loop_ms, "branch_tokens_per_s": 1024 / (loop_ms * 1e-3),
            "newest_segments": n, "set_lengths_host_ms": set_ms,
            "what": "per step: append one token to each newest segment, grow them by one token "
                    "(length update), schedule, attend, merge"}
    if args.calibrate_copy:
        calibrate_copy(torch, dev)
    if args.cpu_sample > 0:
        log(f"timing the CPU oracle on {args.cpu_sample} branches")
        res["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample)
        log("CPU oracle done")
    if args.cpu_configs:
        # Branches per configuration: all of the small ones, a seeded sample of the long ones
        # (the oracle materialises each branch's whole context in fp64).
        sample = {"c1": 4, "c2": 128, "c3": 1024, "c4": 16, "c5chain": 32, "c5graph": 64}
        res["cpu_configs"] = {}
        for name in ["c1", "c2", "c3", "c4", "c5chain", "c5graph"]:
            if name == args.config:
                continue
            other = W.CONFIGS[name]()
            log(f"timing the CPU oracle on {name} ({sample[name]} branches)")
            res["cpu_configs"][name] = cpu_baseline(other, sample[name])
            del other
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
