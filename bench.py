#!/usr/bin/env python3
"""Benchmark of the MoE decode expert stage on one MI355X.

One step = one decode token through every MoE layer of the workload: router gating,
cache check + LRU update, SwiGLU FFN of cache-hit experts on the GPU, missed experts
on the host thread pool, post-fetch of missed experts into the cache, weighted
combine (Section III-A steps 1-3). Inputs (router weights, expert weights, AR(1)
hidden states) are synthetic and seeded; expert weights live in pinned host memory
(see build_world for the page-locked cap) and in the per-layer GPU expert cache (M of n experts per layer),
starting cold. The warmup steps fill the cache; the timed steps run the real LRU
trace, so they include host-side misses and post-fetch copies.

Prints one JSON line. `value` is MoE-stage tokens/s (all layers; attention is not
part of the stage). `roofline` is the gate/up/SiLU kernel (the largest share of the
weight stream) timed with HIP events on the compute stream over the timed steps,
against the MI355X HBM peak. `cpu_baseline` times the oracle (plain CPU reference)
on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def build_world(torch, moe, synth, wl, steps_total, seed, threads, pinned_gb, policy="lru", budget_gb=None,
                ways=None):
    """Device cache, pinned host experts, router weights and hidden states.

    Page-locked host memory is capped per process on the GPU hosts (64 GiB), below
    the full Mixtral/Phi/fine-grained expert sets (80-111 GB). The host copies of the
    experts therefore cover the first H layers, H = floor(pinned_gb / per-layer bytes),
    and layer l uses host layer l mod H (its router and its cache slots stay its own).
    """
    import numpy as np
    d, f, n, k, L, M = wl.d, wl.f, wl.n, wl.k, wl.L, (ways or wl.ways)
    stride = moe.slab_bytes(d, f)
    per_layer = n * stride
    H = max(1, min(L, int(pinned_gb * 2**30) // per_layer))
    t0 = time.perf_counter()
    hosts = [moe.PinnedBuffer(per_layer) for _ in range(H)]
    log(f"pinned host experts: {H} distinct layers x {per_layer / 1e9:.2f} GB in {time.perf_counter() - t0:.1f}s")
    tmp = torch.empty(3 * d * f, dtype=torch.bfloat16, device="cuda")
    for h in range(H):
        hview = torch.from_numpy(hosts[h].array)
        for e in range(n):
            synth.expert_slab_torch(synth.seed_for(seed, wl.name, "expert", h, e), d, f, wl.w_std, out=tmp)
            hview[e * stride: e * stride + 3 * d * f * 2].copy_(tmp.view(torch.uint8))
    del tmp
    log(f"expert weights drawn: {time.perf_counter() - t0:.1f}s")
    # The weights reached the pinned pages by DMA, so the CPU has never touched them; on
    # these hosts the first CPU access to each page is ~1 us (13x the steady-state FFN
    # time). Weights loaded from disk by the CPU would be touched already, so touch
    # every page once here, outside any timed region, from all host threads.
    from concurrent.futures import ThreadPoolExecutor
    chunks = [(hh, o) for hh in range(H) for o in range(0, per_layer, 1 << 28)]
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(lambda c: int(hosts[c[0]].array[c[1]:c[1] + (1 << 28):4096].sum()), chunks))
    log(f"host pages touched: {time.perf_counter() - t0:.1f}s")
    host_addrs = [hosts[l % H].ptr + e * stride for l in range(L) for e in range(n)]
    shared = None
    if wl.f_shared:
        sstride = moe.slab_bytes(d, wl.f_shared)
        shared = torch.zeros(L * sstride, dtype=torch.uint8, device="cuda")
        for l in range(L):
            t = shared[l * sstride: l * sstride + 3 * d * wl.f_shared * 2].view(torch.bfloat16)
            synth.expert_slab_torch(synth.seed_for(seed, wl.name, "shared", l, 0), d, wl.f_shared, wl.w_std, out=t)
    wr = torch.stack([synth.router_weights_torch(synth.seed_for(seed, wl.name, "router", l), n, d)
                      for l in range(L)]).contiguous()
    X = np.stack([synth.ar1_states(synth.seed_for(seed, wl.name, "states", l), steps_total, d) for l in range(L)])
    xd = torch.from_numpy(np.ascontiguousarray(X.transpose(1, 0, 2))).cuda()     # [T, L, d]
    covered = L
    if budget_gb is not None:   # Section III-B: slots S = budget / expert size, N = S / M covered layers
        _, covered = moe.cache_geometry(int(budget_gb * 1e9), stride, M, L)
    content = None
    if policy == "static":      # the "random" policy: a seeded uniform M-subset per layer, fixed
        content = [sorted(np.random.default_rng(synth.seed_for(seed, wl.name, "static-content", l))
                          .choice(n, M, replace=False).tolist()) for l in range(covered)]
    pool = torch.zeros(covered * M * stride, dtype=torch.uint8, device="cuda") if covered else None
    cache = moe.Cache(covered, n, M, k, policy=policy, static_content=content)
    hp = moe.HostPool(threads)
    rt = moe.Runtime(d, f, n, k, M, L, wr, pool, host_addrs, cache, hp, f_shared=wl.f_shared, shared_pool=shared)

    def fresh_runtime():
        """A new cold cache and runtime over the same weights (for a second measurement)."""
        c2 = moe.Cache(covered, n, M, k, policy=policy, static_content=content)
        return c2, moe.Runtime(d, f, n, k, M, L, wr, pool, host_addrs, c2, hp, f_shared=wl.f_shared,
                               shared_pool=shared)
    torch.cuda.synchronize()
    log(f"world ready in {time.perf_counter() - t0:.1f}s (device cache {0 if pool is None else pool.numel() / 1e9:.1f} GB, "
        f"{covered} of {L} layers covered, policy {policy})")
    return dict(hosts=hosts, H=H, wr=wr, X=X, xd=xd, pool=pool, shared=shared, cache=cache, hp=hp, rt=rt,
                stride=stride, covered=covered, policy=policy, fresh_runtime=fresh_runtime)


def cpu_baseline(wl, world, seed, budget_s, t_first):
    """The oracle (plain CPU reference) on a bounded sample of the same workload:
    consecutive tokens of layers 0, 1, ... (router, chosen experts, combine, LRU),
    until about budget_s seconds of CPU work; scaled to tokens/s over all layers."""
    import numpy as np
    import oracle
    from oracle import lru as olru
    wr = world["wr"].cpu().numpy()
    X = world["X"]
    hosts, H, stride = world["hosts"], world["H"], world["stride"]
    d, f, n, k, L = wl.d, wl.f, wl.n, wl.k, wl.L
    shared_np = None
    if wl.f_shared:
        sstride = moe_slab_bytes(d, wl.f_shared)
        shared_np = world["shared"].cpu().numpy()
    threads = oracle.get_threads()
    done, elapsed = 0, 0.0
    layers_used = set()
    T = X.shape[1]
    order = [(l, t) for l in range(L) for t in range(t_first, T)]
    cache = olru.LRUCache(L, wl.ways)
    for (l, t) in order:
        slabs = [hosts[l % H].array[e * stride:e * stride + 3 * d * f * 2].view(np.uint16) for e in range(n)]
        sh = None
        if shared_np is not None:
            sh = shared_np[l * sstride: l * sstride + 3 * d * wl.f_shared * 2].view(np.uint16)
        t0 = time.perf_counter()
        idx, w, out, gap = oracle.moe_token(X[l, t], wr[l], slabs, k, f, shared_slab=sh, f_shared=wl.f_shared)
        cache.access(l, list(idx))
        elapsed += time.perf_counter() - t0
        done += 1
        layers_used.add(l)
        if elapsed >= budget_s:
            break
    per_token_layer = elapsed / done
    # the same token-layers again on one thread, for a shorter budget
    oracle.set_threads(1)
    done1, elapsed1 = 0, 0.0
    try:
        for (l, t) in order[:done]:
            slabs = [hosts[l % H].array[e * stride:e * stride + 3 * d * f * 2].view(np.uint16) for e in range(n)]
            sh = None
            if shared_np is not None:
                sh = shared_np[l * sstride: l * sstride + 3 * d * wl.f_shared * 2].view(np.uint16)
            t0 = time.perf_counter()
            oracle.moe_token(X[l, t], wr[l], slabs, k, f, shared_slab=sh, f_shared=wl.f_shared)
            elapsed1 += time.perf_counter() - t0
            done1 += 1
            if elapsed1 >= budget_s / 4:
                break
    finally:
        oracle.set_threads(threads)
    return {
        "value": 1.0 / (per_token_layer * L), "unit": "tokens/s", "cores": threads, "kind": "oracle",
        "sample": (f"{done} token-layers (layers {min(layers_used)}-{max(layers_used)}, consecutive tokens from "
                   f"step {t_first}) through router + top-{k} SwiGLU experts + combine + LRU, "
                   f"{elapsed:.1f}s; scaled to {L} layers per token"),
        "ms_per_token_layer": per_token_layer * 1e3,
        "one_thread": {"tokens_per_s": 1.0 / (elapsed1 / done1 * L), "ms_per_token_layer": elapsed1 / done1 * 1e3,
                       "sample": f"the first {done1} of those token-layers, {elapsed1:.1f}s"},
        "host": host_info(),
    }


def host_info():
    """What the host that ran the oracle is: logical CPUs, the ones this process may use,
    the CPU model and whether it has AVX-512 (and its bf16 extension)."""
    model, flags = "unknown", set()
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name") and model == "unknown":
                    model = line.split(":", 1)[1].strip()
                elif line.startswith("flags") and not flags:
                    flags = set(line.split(":", 1)[1].split())
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"nproc": os.cpu_count(), "usable_cpus": usable, "cpu_model": model,
            "avx512f": "avx512f" in flags, "avx512_bf16": "avx512_bf16" in flags}


def host_sweep(moe, wl, world, threads_list=(1, 2, 4, 8, 16)):
    """Host expert path alone: one layer's k experts all missed (the CPU column of the
    paper's Table III), for several thread counts, nothing else running; both forms of
    the row dot product (fp32 widening; the AVX512_BF16 pair-dot where the CPU has it)."""
    import numpy as np
    d, f, k = wl.d, wl.f, wl.k
    stride = world["stride"]
    host = world["hosts"][0]
    slabs = [host.array[e * stride: e * stride + 3 * d * f * 2] for e in range(k)]
    x = world["X"][0, 0]
    w = np.full(k, 1.0 / k, np.float32)
    out = {}
    for dot in ("fp32", "bf16"):
        rows = {}
        for t in threads_list:
            pool = moe.HostPool(t)
            try:
                pool.set_dot(dot)
            except moe.MoeError:
                pool.close()
                break
            times = []
            for _ in range(5):
                t0 = time.perf_counter()
                pool.expert_ffn(x, slabs, w, d, f)
                times.append(time.perf_counter() - t0)
            pool.close()
            ms = sorted(times)[2] * 1e3
            rows[str(t)] = {"ms": round(ms, 2), "GB/s": round(k * 3 * d * f * 2 / (ms * 1e-3) / 1e9, 1)}
        if rows:
            out[dot] = rows
    return out


def hit_study(args, torch, moe, synth, wl):
    """Cache hit rates by policy and ways (the analog of the paper's Fig. on cache
    configurations and eviction policies, Section IV-D): the GPU router selects the
    experts of every AR(1) token of every layer, and the library's cache replays
    those selections under LRU, FIFO and a static random content. Also i.i.d. uniform
    selections, whose long-run rates must match the closed forms for every policy."""
    import math
    import numpy as np
    d, n, k, L, T = wl.d, wl.n, wl.k, wl.L, wl.T
    wr = torch.stack([synth.router_weights_torch(synth.seed_for(args.seed, wl.name, "router", l), n, d)
                      for l in range(L)]).contiguous()
    sel = np.empty((L, T, k), np.int32)
    for l in range(L):
        X = torch.from_numpy(synth.ar1_states(synth.seed_for(args.seed, wl.name, "states", l), T, d)).cuda()
        idx, _ = moe.router_topk(X, wr[l], k)
        sel[l] = idx.cpu().numpy()
    rng = np.random.default_rng(synth.seed_for(args.seed, wl.name, "subsets"))
    iid = np.stack([np.stack([rng.choice(n, k, replace=False) for _ in range(T)]) for _ in range(L)]).astype(np.int32)
    ways_list = sorted({m for m in (k, 2 * k, n // 4, n // 2, 3 * n // 4, wl.ways) if k <= m < n})

    def replay(trace, policy, M, warm):
        content = None
        if policy == "static":
            content = [sorted(np.random.default_rng(synth.seed_for(args.seed, wl.name, "static-content", l))
                              .choice(n, M, replace=False).tolist()) for l in range(L)]
        c = moe.Cache(L, n, M, k, policy=policy, static_content=content)
        anyh = allh = eh = ev = 0
        for t in range(T):
            for l in range(L):
                _, hits = c.lookup(l, trace[l, t])
                c.update(l, trace[l, t])
                if t >= warm:
                    anyh += bool(hits.any())
                    allh += bool(hits.all())
                    eh += int(hits.sum())
                    ev += 1
        return {"any_hit": round(anyh / ev, 4), "all_hit": round(allh / ev, 4), "expert_hit": round(eh / (ev * k), 4)}

    rows = []
    for M in ways_list:
        row = {"ways": M,
               "closed_form": {"any_hit": round(1 - math.comb(n - M, k) / math.comb(n, k), 4),
                               "all_hit": round(math.comb(M, k) / math.comb(n, k), 4)}}
        for policy in ("lru", "fifo", "static"):
            row[policy] = replay(sel, policy, M, warm=8)
            row["iid_" + policy] = replay(iid, policy, M, warm=8)
        rows.append(row)
        log(json.dumps(row))
    return {
        "metric": "expert-cache hit rate by policy and ways (router selections of AR(1) hidden states)",
        "value": next(r["lru"]["expert_hit"] for r in rows if r["ways"] == wl.ways) if wl.ways in ways_list else None,
        "unit": "fraction of selected experts found in the cache (LRU, the workload's ways)",
        "n_gpus": 1, "higher_is_better": True, "data": "synthetic",
        "config": {"workload": wl.desc, "experts": n, "top_k": k, "layers": L, "tokens": T,
                   "warm_tokens_excluded": 8, "events_per_row": L * (T - 8)},
        "rows": rows,
    }


def pcie_study(args, torch, moe, synth, wl):
    """Host-to-device expert copies (the transfer column of the paper's Table I and
    Table III): one expert slab from pinned memory on one stream, two slabs on two
    streams at once (two DMA engines, Section III-C), and one slab from pageable memory."""
    import numpy as np
    stride = moe.slab_bytes(wl.d, wl.f)
    payload = 3 * wl.d * wl.f * 2
    src = [torch.ones(payload, dtype=torch.uint8, pin_memory=True) for _ in range(2)]   # hipHostMalloc'd
    pageable = torch.ones(payload, dtype=torch.uint8)
    dst = torch.empty(2 * stride, dtype=torch.uint8, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()

    def timed(fn, reps=5):
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            ts.append(time.perf_counter() - t0)
        return sorted(ts)[len(ts) // 2]

    def one():
        with torch.cuda.stream(s1):
            dst[:payload].copy_(src[0], non_blocking=True)

    def two():
        with torch.cuda.stream(s1):
            dst[:payload].copy_(src[0], non_blocking=True)
        with torch.cuda.stream(s2):
            dst[stride:stride + payload].copy_(src[1], non_blocking=True)

    def page():
        dst[:payload].copy_(pageable)

    t1, t2, tp = timed(one), timed(two), timed(page, reps=3)
    res = {
        "metric": "host-to-device expert copy bandwidth (pinned, 1 and 2 streams; pageable)",
        "value": round(payload / t1 / 1e9, 2), "unit": "GB/s (one pinned slab, one stream)",
        "n_gpus": 1, "higher_is_better": True, "data": "synthetic",
        "config": {"workload": wl.desc, "slab_bytes": payload},
        "one_stream": {"ms": round(t1 * 1e3, 2), "GB/s": round(payload / t1 / 1e9, 2)},
        "two_streams": {"ms": round(t2 * 1e3, 2), "GB/s": round(2 * payload / t2 / 1e9, 2)},
        "pageable": {"ms": round(tp * 1e3, 2), "GB/s": round(payload / tp / 1e9, 2)},
    }
    log(json.dumps(res))
    return res


def small_batch_study(args, torch, moe, synth, wl):
    """Multi-token decode with every expert resident (T = 1..64 tokens per step): the
    grouped-GEMM path (prefill kernels at small T) against T single-token passes of the
    GEMV hit path and, for T <= 8, the multi-token GEMV path (each selected slab read once
    for all its tokens), per MoE layer. Not in the paper; it locates the crossovers
    between the decode and prefill kernels."""
    import numpy as np
    d, f, n, k = wl.d, wl.f, wl.n, wl.k
    L = 4                                   # distinct layers so weights are not reused from cache
    stride = moe.slab_bytes(d, f)
    pool = torch.empty(L * n * stride, dtype=torch.uint8, device="cuda")
    for l in range(L):
        for e in range(n):
            t = pool[(l * n + e) * stride:(l * n + e) * stride + 3 * d * f * 2].view(torch.bfloat16)
            synth.expert_slab_torch(synth.seed_for(args.seed, wl.name, "expert", l, e), d, f, wl.w_std, out=t)
    wr = torch.stack([synth.router_weights_torch(synth.seed_for(args.seed, wl.name, "router", l), n, d)
                      for l in range(L)]).contiguous()
    Tmax = 64
    X = torch.from_numpy(synth.iid_states(synth.seed_for(args.seed, wl.name, "prompt"), Tmax, d)).cuda()
    out = torch.empty((Tmax, d), device="cuda")
    ws = torch.empty(moe.prefill_workspace_bytes(d, f, n, k, Tmax), dtype=torch.uint8, device="cuda")
    # single-token GEMV path over resident experts: slot s of layer l holds expert s
    fws = torch.empty(moe.ffn_workspace_bytes(k, d, f), dtype=torch.uint8, device="cuda")
    idx = torch.empty((Tmax, k), dtype=torch.int32, device="cuda")
    wts = torch.empty((Tmax, k), dtype=torch.float32, device="cuda")
    y = torch.empty(d, device="cuda")
    tmax_tok = min(moe.MAX_TOKENS, 131072 // (4 * d))
    tws = torch.empty(moe.ffn_tokens_workspace_bytes(tmax_tok, k, d, f), dtype=torch.uint8, device="cuda")
    ytok = torch.empty((tmax_tok, d), device="cuda")

    def time_it(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    rows = []
    for T in (1, 2, 4, 8, 16, 32, 64):
        def grouped():
            for l in range(L):
                moe.prefill_forward(X[:T], wr[l], pool[l * n * stride:(l + 1) * n * stride], d, f, n, k, out[:T], ws)

        def gemv():
            for l in range(L):
                moe.router_topk(X[:T], wr[l], k, idx_out=idx[:T], w_out=wts[:T])
                for t in range(T):
                    moe.expert_ffn_hits(X[t], pool[l * n * stride:(l + 1) * n * stride], n, idx[t], wts[t], d, f, y,
                                        fws)
        def tokens():
            for l in range(L):
                moe.router_topk(X[:T], wr[l], k, idx_out=idx[:T], w_out=wts[:T])
                moe.expert_ffn_tokens(X[:T], pool[l * n * stride:(l + 1) * n * stride], n, idx[:T], wts[:T], d, f,
                                      ytok[:T], tws)
        g_us = time_it(grouped) / L
        v_us = time_it(gemv, reps=2 if T >= 16 else 5) / L
        t_us = time_it(tokens) / L if T <= tmax_tok else None
        # distinct experts per layer, averaged over the L timed layers (each reads its own)
        per_layer = []
        for l in range(L):
            moe.router_topk(X[:T], wr[l], k, idx_out=idx[:T], w_out=wts[:T])
            per_layer.append(int(np.unique(idx[:T].cpu().numpy()).size))
        touched = sum(per_layer) / L
        rows.append({"T": T, "grouped_us_per_layer": round(g_us, 1), "gemv_us_per_layer": round(v_us, 1),
                     "tokens_us_per_layer": None if t_us is None else round(t_us, 1),
                     "experts_touched": touched,
                     "grouped_weight_GBs": round(touched * 3 * d * f * 2 / (g_us * 1e-6) / 1e9, 1),
                     "tokens_weight_GBs": None if t_us is None else
                     round(touched * 3 * d * f * 2 / (t_us * 1e-6) / 1e9, 1)})
        log(json.dumps(rows[-1]))
    return {
        "metric": "multi-token decode, all experts resident: us per MoE layer, grouped GEMM vs per-token GEMV vs "
                  "multi-token GEMV",
        "value": None, "unit": "us per layer", "n_gpus": 1, "higher_is_better": False, "data": "synthetic",
        "config": {"workload": wl.desc, "layers_timed": L, "tokens": "i.i.d. N(0,1)"},
        "rows": rows,
    }


def _kernel_record(name):
    """A committed PMC record (profiles/<name>) if the kernel sources it lists still hash
    to the value it was taken on; else None."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", name)))
        # the kernel sources the counters were taken on, hashed in the listed order
        src = b"".join(open(os.path.join(ROOT, f), "rb").read() for f in rec["kernel_sources"])
    except (OSError, ValueError, KeyError, TypeError):
        return None
    if hashlib.sha256(src).hexdigest() != rec.get("kernel_sha256"):
        return None
    return rec


def geometry_sweep(args, torch, moe, synth, wl):
    """Cache geometry x host threads (Section III-B sizing, Section IV-C trade-off): for
    memory budgets (the paper's 24 GB card less 5 GB of non-expert weights, and the
    58-slot "(29,2)" configuration it discusses) and for full coverage at several ways,
    the decode loop runs with 1..16 host threads, every miss post-fetched, cold cache.
    Each point: a fresh cache and runtime over the same host experts and inputs."""
    import numpy as np
    d, f, n, k, L = wl.d, wl.f, wl.n, wl.k, wl.L
    steps_total = args.warmup + args.steps
    world = build_world(torch, moe, synth, wl, steps_total, args.seed, 1, args.pinned_gb)
    world["rt"].close()
    stride, xd = world["stride"], world["xd"]
    H = world["H"]
    host_addrs = [world["hosts"][l % H].ptr + e * stride for l in range(L) for e in range(n)]
    E = 3 * d * f * 2
    if wl.name == "mixtral":
        geoms = [(19.0, 2), (19.0, 4), (58 * E / 1e9, 2), (None, 2), (None, 4), (None, 6)]
    else:
        geoms = [(19.0, 4), (19.0, 6), (19.0, 8), (None, 4), (None, 6), (None, 8)]
    threads = [int(t) for t in args.sweep_threads.split(",")]
    streams = (torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream())
    out = torch.empty((2, L, d), dtype=torch.float32, device="cuda")
    hit = np.empty((L, k), np.uint8)
    rows = []
    for budget, M in geoms:
        if budget is None:
            covered, slots = L, L * M
        else:
            slots, covered = moe.cache_geometry(int(budget * 1e9), E, M, L)
        pool = torch.zeros(max(1, covered * M) * stride, dtype=torch.uint8, device="cuda") if covered else None
        for t in threads:
            cache = moe.Cache(covered, n, M, k)
            hp = moe.HostPool(t)
            rt = moe.Runtime(d, f, n, k, M, L, world["wr"], pool, host_addrs, cache, hp)
            for s in range(args.warmup):
                rt.decode_step(xd[s], out[s % 2], streams)
            torch.cuda.synchronize()
            rt.sync()
            rt.reset_stats()
            anyh = allh = 0
            t0 = time.perf_counter()
            for s in range(args.warmup, steps_total):
                rt.decode_step(xd[s], out[s % 2], streams, hit=hit)
                anyh += int(hit.any(axis=1).sum())
                allh += int(hit.all(axis=1).sum())
            torch.cuda.synchronize()
            rt.sync()
            dt = time.perf_counter() - t0
            st = rt.stats()
            K = args.steps
            sel = st["expert_hits"] + st["expert_misses"]
            row = {"budget_gb": None if budget is None else round(budget, 2), "ways": M, "slots": slots,
                   "covered_layers": covered, "host_threads": t, "tokens_per_s": round(K / dt, 2),
                   "expert_hit_rate": round(st["expert_hits"] / max(1, sel), 4),
                   "any_hit": round(anyh / (K * L), 4), "all_hit": round(allh / (K * L), 4),
                   "misses_per_token": round(st["expert_misses"] / K, 2),
                   "host_ffn_ms_per_token": round(st["host_ffn_ms"] / K, 2),
                   "fills_per_token": round(st["fills"] / K, 2)}
            log(json.dumps(row))
            rows.append(row)
            rt.close()
            cache.close()
            hp.close()
        del pool
        torch.cuda.empty_cache()
    return {
        "metric": "decode MoE-stage tokens/s by cache geometry and host threads",
        "value": None, "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True, "data": "synthetic",
        "config": {"workload": wl.desc, "expert_bytes": E, "warmup": args.warmup, "steps": args.steps,
                   "post_fetch": "every miss (Section III-A step 3); parity (waits)", "cache_start": "cold",
                   "host_expert_layers_distinct": H},
        "rows": rows,
    }


def measured_traffic(args, kernel, bytes_per_launch):
    """HBM bytes per launch of `kernel` (k_gate_up, k_down) for this run: the ratio of
    counted (rocprofv3 FETCH_SIZE/WRITE_SIZE, scaled by the copy calibration) to
    algorithmic bytes per launch in the committed record, taken on the current kernel
    source with the same workload and seed, times this run's algorithmic bytes per
    launch. None when no such record exists."""
    rec = _kernel_record("traffic.json")
    if rec is None or rec.get("workload") != args.workload or rec.get("seed") != args.seed or kernel not in rec:
        return None
    r = rec[kernel]["hbm_bytes_per_launch"] / rec[kernel]["algorithmic_bytes_per_launch"]
    return {"bytes_per_launch": round(r * bytes_per_launch), "ratio_to_algorithmic": round(r, 4)}


def read_stream_yardstick(torch, moe, buf, launch_bytes):
    """HBM read ceiling on this device: the library's plain nontemporal read stream over
    (i) as many bytes as one average k_gate_up launch reads and (ii) a long read, both from
    the device expert cache (event-timed on the launching stream, median of 20)."""
    total = buf.numel() * buf.element_size()
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = {}
    for name, nb in (("launch_size", launch_bytes), ("long", min(total, 8 << 30))):
        nb = int(min(nb, total)) // 16 * 16
        if nb <= 0:
            continue
        times = []
        for it in range(23):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            moe.read_stream(buf, nb, sink)
            e1.record()
            e1.synchronize()
            if it >= 3:
                times.append(e0.elapsed_time(e1))
        ms = sorted(times)[len(times) // 2]
        out[name] = {"bytes": nb, "us": round(ms * 1e3, 2), "gbs": round(nb / (ms * 1e-3) / 1e9, 1),
                     "frac": round(nb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    return out


def measured_prefill_traffic(d, f, n, k, T):
    """HBM bytes per prefill layer (the two grouped GEMMs and the gate/up tail combine)
    from the committed PMC record, if it was taken on the current kernel source at the
    same layer shape and prompt length."""
    rec = _kernel_record("traffic_prefill.json")
    if rec is None or rec.get("shape") != {"d": d, "f": f, "n": n, "k": k, "T": T}:
        return None
    return rec["hbm_bytes_per_layer"]


def prefill_pass(torch, moe, pool, wr, X, d, f, n, k, L, warmup, steps):
    """Prompt X [T, d] through layers 0..L-1 per step (layer l: slabs l*n .. l*n+n-1 of
    pool, router wr[l]), every expert resident; `warmup` untimed and `steps` timed steps.
    Time from events on the stream the library launches on (torch's current stream)."""
    T = X.shape[0]
    stride = moe.slab_bytes(d, f)
    out = torch.empty((T, d), device="cuda")
    ws = torch.empty(moe.prefill_workspace_bytes(d, f, n, k, T), dtype=torch.uint8, device="cuda")

    def step():
        for l in range(L):
            moe.prefill_forward(X, wr[l], pool[l * n * stride:(l + 1) * n * stride], d, f, n, k, out, ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t1 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t1
    per_layer_us = e0.elapsed_time(e1) * 1e3 / (steps * L)
    bytes_layer = n * 3 * d * f * 2.0
    flops_layer = 2.0 * 3 * d * f * T * k
    hbm = bytes_layer / (per_layer_us * 1e-6) / 1e9
    tf = flops_layer / (per_layer_us * 1e-6) / 1e12
    return {"tokens_per_s": round(T * steps / wall, 1), "ms_per_prompt": round(wall / steps * 1e3, 3),
            "us_per_layer": round(per_layer_us, 2), "hbm_gbs": round(hbm, 1),
            "hbm_frac": round(hbm / HBM_PEAK_GBS, 4), "mfma_tflops": round(tf, 1),
            "mfma_frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic_bytes_per_layer": measured_prefill_traffic(d, f, n, k, T)}


def bench_prefill(args, torch, moe, synth, wl):
    """One prompt of wl.T tokens through every layer, all experts resident in HBM
    (L x n slabs, layers visited in order so no slab is reused while cached)."""
    d, f, n, k, L, T = wl.d, wl.f, wl.n, wl.k, wl.L, wl.T
    stride = moe.slab_bytes(d, f)
    t0 = time.perf_counter()
    pool = torch.empty(L * n * stride, dtype=torch.uint8, device="cuda")
    for l in range(L):
        for e in range(n):
            off = (l * n + e) * stride
            t = pool[off: off + 3 * d * f * 2].view(torch.bfloat16)
            synth.expert_slab_torch(synth.seed_for(args.seed, wl.name, "expert", l, e), d, f, wl.w_std, out=t)
    wr = torch.stack([synth.router_weights_torch(synth.seed_for(args.seed, wl.name, "router", l), n, d)
                      for l in range(L)]).contiguous()
    X = torch.from_numpy(synth.iid_states(synth.seed_for(args.seed, wl.name, "prompt"), T, d)).cuda()
    torch.cuda.synchronize()
    log(f"prefill world ready in {time.perf_counter() - t0:.1f}s ({pool.numel() / 1e9:.1f} GB of experts in HBM)")
    r = prefill_pass(torch, moe, pool, wr, X, d, f, n, k, L, args.warmup, args.steps)
    return {
        "metric": "prefill MoE-layer tokens/s + achieved HBM GB/s (%peak), Mixtral-8x7B shape",
        "value": r["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": r["ms_per_prompt"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.desc, "d_model": d, "d_ffn": f, "experts": n, "top_k": k, "layers": L,
                   "prompt_tokens": T, "weights": "bf16, activations rounded to bf16, fp32 accumulate",
                   "parallelism": "single GPU"},
        "roofline": {"kernel": "prefill layer (router, grouping, grouped MFMA GEMMs, combine)", "bound": "hbm",
                     "achieved": r["hbm_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": r["hbm_frac"], "traffic": r["traffic_bytes_per_layer"],
                     "traffic_unit": "HBM bytes per layer of the grouped GEMMs (rocprofv3 FETCH_SIZE x2.0 + "
                                     "WRITE_SIZE, profiles/traffic_prefill.json)",
                     "mfma_tflops": r["mfma_tflops"], "mfma_peak_tflops": MFMA_BF16_PEAK_TFLOPS,
                     "mfma_frac": r["mfma_frac"], "us_per_layer": r["us_per_layer"]},
        "cpu_baseline": None,
    }


def all_resident_and_prefill(args, torch, moe, synth, wl, world, xd, tokens=64, prompts=4, prefill=True):
    """The GPU-bound regime on the same weights: every expert of every layer resident
    (a static cache holding all n experts; MI355X's HBM holds each workload's expert set),
    so each decode token runs router + hit FFN + reduce per layer with no host work and
    no copies. Timed once with the kernel timing events off (tokens/s) and once with
    them on (kernel rooflines). Then a 512-token prompt through the same resident
    layers (prefill: batched router, grouping, grouped MFMA GEMMs)."""
    d, f, n, k, L = wl.d, wl.f, wl.n, wl.k, wl.L
    stride = world["stride"]
    H = world["H"]
    host_addrs = [world["hosts"][l % H].ptr + e * stride for l in range(L) for e in range(n)]
    content = [list(range(n)) for _ in range(L)]
    pool = torch.empty(L * n * stride, dtype=torch.uint8, device="cuda")
    t0 = time.perf_counter()
    cache = moe.Cache(L, n, n, k, policy="static", static_content=content)
    rt = moe.Runtime(d, f, n, k, n, L, world["wr"], pool, host_addrs, cache, world["hp"], f_shared=wl.f_shared,
                     shared_pool=world["shared"])   # loads every slab
    torch.cuda.synchronize()
    log(f"all-resident world: {pool.numel() / 1e9:.1f} GB of experts loaded in {time.perf_counter() - t0:.1f}s")
    streams = (torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream())
    out = torch.empty((2, L, d), dtype=torch.float32, device="cuda")
    T = xd.shape[0]

    def run(t0_, count):
        for t in range(t0_, t0_ + count):
            rt.decode_step(xd[t % T], out[t % 2], streams)
        torch.cuda.synchronize()

    run(0, 4)
    rt.reset_stats()
    t1 = time.perf_counter()
    run(4, tokens)
    dt = time.perf_counter() - t1
    st = rt.stats()
    assert st["expert_misses"] == 0 and st["fills"] == 0
    rt.set_timing(True)
    run(4, tokens)
    st = rt.stats()
    rt.set_timing(False)
    rt.close()
    cache.close()
    alg_layer = k * 3 * d * f * 2 + n * d * 4 + 3 * d * wl.f_shared * 2
    us_layer = dt / (tokens * L) * 1e6
    gu = st["gate_up_bytes"] / (st["gate_up_ms"] * 1e-3) / 1e9
    dn = st["down_bytes"] / (st["down_ms"] * 1e-3) / 1e9
    res = {
        "what": f"every expert resident (static cache of all {n} experts per layer, no misses, no copies); "
                f"{tokens} tokens after 4 warm-up, timing events off; kernel figures from a second pass of "
                f"the same tokens with events on",
        "tokens_per_s": round(tokens / dt, 2), "ms_per_token": round(dt / tokens * 1e3, 3),
        "us_per_layer": round(us_layer, 2),
        "hbm_floor_us_per_layer": round(alg_layer / (HBM_PEAK_GBS * 1e3), 2),
        "frac_of_floor": round(alg_layer / (HBM_PEAK_GBS * 1e3) / us_layer, 4),
        "k_gate_up": {"avg_us": round(st["gate_up_ms"] / st["gate_up_launches"] * 1e3, 2),
                      "gbs": round(gu, 1), "frac": round(gu / HBM_PEAK_GBS, 4)},
        "k_down": {"avg_us": round(st["down_ms"] / st["down_launches"] * 1e3, 2),
                   "gbs": round(dn, 1), "frac": round(dn / HBM_PEAK_GBS, 4)},
        "hit_ffn_us_per_layer": round((st["gate_up_ms"] + st["down_ms"]) / st["gate_up_launches"] * 1e3, 2),
    }
    log(json.dumps(res))
    if not prefill:
        del pool
        torch.cuda.empty_cache()
        return res, None
    X = torch.from_numpy(synth.iid_states(synth.seed_for(args.seed, "prefill", "prompt"), 512, d)).cuda()
    pf = prefill_pass(torch, moe, pool, world["wr"], X, d, f, n, k, L, 2, prompts)
    pf["what"] = (f"one 512-token prompt (i.i.d. N(0,1)) through the {L} resident layers; 2 warm-up + {prompts} "
                  f"timed prompts; HBM fraction on the {n} expert slabs per layer, MFMA fraction of the bf16 "
                  f"dense peak")
    log(json.dumps(pf))
    del pool
    torch.cuda.empty_cache()
    return res, pf


def moe_slab_bytes(d, f):
    import paper_2512_16473_amd as moe
    return moe.slab_bytes(d, f)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="mixtral", choices=["mixtral", "phi", "fine", "tiny", "prefill"])
    ap.add_argument("--threads", type=int, default=0, help="host expert threads (0: OMP_NUM_THREADS or all cores)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--host-dot", default="auto", choices=["auto", "fp32", "bf16"],
                    help="form of the host path's dot products (bf16: AVX512_BF16 pair-dot)")
    ap.add_argument("--pinned-gb", type=float, default=56.0, help="page-locked host memory for expert copies (GiB)")
    ap.add_argument("--cpu-baseline-s", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-resident", action="store_true",
                    help="skip the all-resident decode sub-measurement (and the prefill one of the Mixtral line)")
    ap.add_argument("--policy", default="lru", choices=["lru", "fifo", "static"],
                    help="cache replacement policy (Section IV-D; the paper's is LRU)")
    ap.add_argument("--ways", type=int, default=0,
                    help="cache slots per layer (default: the workload's; = experts for an all-resident cache)")
    ap.add_argument("--budget-gb", type=float, default=None,
                    help="GPU memory for the expert cache (GB); layers past the covered ones run on the host")
    ap.add_argument("--fill-limit", type=int, default=0,
                    help="bounded post-fetch: at most this many expert slabs in flight (0: every miss fetched)")
    ap.add_argument("--nonblocking", action="store_true",
                    help="never wait for a post-fetch: experts whose copy has not landed run on the host")
    ap.add_argument("--hit-study", action="store_true",
                    help="only replay router selections through LRU/FIFO/static caches of several sizes")
    ap.add_argument("--pcie", action="store_true", help="only measure host-to-device expert copies")
    ap.add_argument("--small-batch", action="store_true",
                    help="only time multi-token decode (T = 1..64) with every expert resident")
    ap.add_argument("--sweep", action="store_true",
                    help="only run the cache-geometry x host-threads sweep (mixtral or phi)")
    ap.add_argument("--sweep-threads", default="1,2,4,8,16", help="host thread counts of --sweep")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB 5 times (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the decode expert stage has no multi-GPU path here "
              f"(--gpus {args.gpus} requested).", file=sys.stderr, flush=True)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2512_16473_amd as moe
    import synth

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        nbytes = args.copy_calibration << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": nbytes, "copy_calibration_bytes_written": nbytes}))
        return
    wl = synth.WORKLOADS[args.workload]
    if args.small_batch:
        print(json.dumps(small_batch_study(args, torch, moe, synth, wl)), flush=True)
        return
    if args.pcie:
        print(json.dumps(pcie_study(args, torch, moe, synth, wl)), flush=True)
        return
    if args.hit_study:
        print(json.dumps(hit_study(args, torch, moe, synth, wl)), flush=True)
        return
    if args.sweep:
        print(json.dumps(geometry_sweep(args, torch, moe, synth, wl)), flush=True)
        return
    if wl.prefill:
        print(json.dumps(bench_prefill(args, torch, moe, synth, wl)), flush=True)
        return
    steps_total = args.warmup + args.steps
    assert steps_total <= wl.T, f"at most {wl.T} decode steps in this workload"
    world = build_world(torch, moe, synth, wl, steps_total, args.seed, args.threads, args.pinned_gb,
                        policy=args.policy, budget_gb=args.budget_gb, ways=args.ways or None)
    rt, xd = world["rt"], world["xd"]
    world["hp"].set_dot(args.host_dot)
    rt.set_fill_limit(args.fill_limit)
    rt.set_nonblocking(args.nonblocking)
    L, k, d = wl.L, wl.k, wl.d
    out = torch.empty((2, L, d), dtype=torch.float32, device="cuda")
    streams = (torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream())
    idx = np.empty((L, k), np.int32)
    wts = np.empty((L, k), np.float32)
    hit = np.empty((L, k), np.uint8)

    for t in range(args.warmup):
        rt.decode_step(xd[t], out[t % 2], streams, idx, wts, hit)
    torch.cuda.synchronize()
    rt.sync()
    rt.reset_stats()
    rt.set_timing(True)

    torch.cuda.synchronize()
    rt.sync()
    t0 = time.perf_counter()
    for t in range(args.warmup, steps_total):
        rt.decode_step(xd[t], out[t % 2], streams, idx, wts, hit)
    torch.cuda.synchronize()
    rt.sync()
    t1 = time.perf_counter()
    st = rt.stats()
    rt.set_timing(False)

    K = args.steps
    dt = t1 - t0
    tok_s = K / dt
    gu_gbs = st["gate_up_bytes"] / (st["gate_up_ms"] * 1e-3) / 1e9 if st["gate_up_ms"] > 0 else 0.0
    hit_bytes = st["gate_up_bytes"] + st["down_bytes"]
    hit_ms = st["gate_up_ms"] + st["down_ms"]
    sel = st["expert_hits"] + st["expert_misses"]
    result = {
        "metric": "decode MoE-layer tokens/s + achieved HBM GB/s (%peak), Mixtral-8x7B shape",
        "value": round(tok_s, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(dt / K * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": wl.desc,
            "d_model": wl.d, "d_ffn": wl.f, "experts": wl.n, "top_k": wl.k, "layers": wl.L,
            "cache_ways": args.ways or wl.ways, "shared_d_ffn": wl.f_shared, "batch": 1,
            "weights": "bf16, fp32 accumulate", "cache_start": f"cold, {args.warmup} warmup tokens",
            "host_threads": world["hp"].threads, "host_dot": world["hp"].dot, "parallelism": "single GPU",
            "host_expert_layers_distinct": world["H"],
            "cache_policy": world["policy"], "covered_layers": world["covered"],
            "post_fetch": (f"at most {args.fill_limit} slabs in flight" if args.fill_limit
                           else "every miss (Section III-A step 3)")
                          + ("; non-blocking (in flight => host)" if args.nonblocking else "; parity (waits)"),
        },
        "roofline": {
            "kernel": "k_gate_up (W1/W3 rows + SiLU*mul)",
            "bound": "hbm",
            "achieved": round(gu_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gu_gbs / HBM_PEAK_GBS, 4),
            "traffic": None,
            "traffic_unit": "HBM bytes per launch: this run's algorithmic bytes per launch x the counted/algorithmic "
                            "ratio of rocprofv3 FETCH_SIZE x2.0 + WRITE_SIZE on the same kernel source, workload "
                            "and seed (profiles/traffic.json)",
            "launches": st["gate_up_launches"],
            "avg_us": round(st["gate_up_ms"] / max(1, st["gate_up_launches"]) * 1e3, 2),
            "bytes_per_launch": round(st["gate_up_bytes"] / max(1, st["gate_up_launches"])),
        },
        "hit_ffn": {
            "gbs": round(hit_bytes / (hit_ms * 1e-3) / 1e9, 1) if hit_ms > 0 else 0.0,
            "frac": round(hit_bytes / (hit_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if hit_ms > 0 else 0.0,
            "down_avg_us": round(st["down_ms"] / max(1, st["down_launches"]) * 1e3, 2),
            "down_gbs": round(st["down_bytes"] / (st["down_ms"] * 1e-3) / 1e9, 1) if st["down_ms"] > 0 else 0.0,
            "gpu_us_per_layer": round(hit_ms / max(1, st["gate_up_launches"]) * 1e3, 2),
        },
        "trace": {
            "expert_hit_rate": round(st["expert_hits"] / max(1, sel), 4),
            "misses_per_token": round(st["expert_misses"] / K, 3),
            "host_ffn_ms_per_token": round(st["host_ffn_ms"] / K, 3),
            "route_wait_ms_per_token": round(st["route_wait_ms"] / K, 3),
            "fills_per_token": round(st["fills"] / K, 3),
            "fills_skipped_per_token": round(st["fills_skipped"] / K, 3),
            "inflight_misses_per_token": round(st["inflight_misses"] / K, 3),
        },
    }
    for kern, key in (("k_gate_up", "roofline"), ("k_down", "hit_ffn")):
        bpl = (st["gate_up_bytes"] / max(1, st["gate_up_launches"]) if kern == "k_gate_up"
               else st["down_bytes"] / max(1, st["down_launches"]))
        tr = measured_traffic(args, kern, bpl)
        if kern == "k_gate_up":
            result["roofline"]["traffic"] = None if tr is None else tr["bytes_per_launch"]
            result["roofline"]["traffic_ratio"] = None if tr is None else tr["ratio_to_algorithmic"]
        else:
            result["hit_ffn"]["down_traffic_ratio"] = None if tr is None else tr["ratio_to_algorithmic"]
    log(json.dumps(result["trace"]), json.dumps(result["hit_ffn"]))
    if world["pool"] is not None and st["gate_up_launches"]:
        ys = read_stream_yardstick(torch, moe, world["pool"], result["roofline"]["bytes_per_launch"])
        if "launch_size" in ys:
            ys["k_gate_up_frac_of_launch_size_stream"] = round(gu_gbs / ys["launch_size"]["gbs"], 4)
        result["read_stream"] = ys
        log(json.dumps(ys))
    result["host_expert_layer"] = {
        "what": f"host FFN of one layer's {k} experts (all missed), alone, by thread count",
        "by_threads": host_sweep(moe, wl, world)}
    log(json.dumps(result["host_expert_layer"]))
    if args.fill_limit == 0 and not args.nonblocking and world["policy"] != "static" and world["covered"] > 0:
        # The same tokens once more, cold cache, with bounded post-fetch (at most two
        # slabs in flight): misses beyond that run on the host without being fetched.
        rt.close()
        world["cache"], rt2 = world["fresh_runtime"]()
        rt2.set_fill_limit(2)
        for t in range(args.warmup):
            rt2.decode_step(xd[t], out[t % 2], streams, idx, wts, hit)
        torch.cuda.synchronize()
        rt2.sync()
        rt2.reset_stats()
        t0 = time.perf_counter()
        for t in range(args.warmup, steps_total):
            rt2.decode_step(xd[t], out[t % 2], streams, idx, wts, hit)
        torch.cuda.synchronize()
        rt2.sync()
        dt2 = time.perf_counter() - t0
        s2 = rt2.stats()
        result["bounded_post_fetch"] = {
            "what": "same timed tokens, cold cache, at most 2 expert slabs in flight (misses beyond run on the host, "
                    "not fetched)",
            "tokens_per_s": round(K / dt2, 3), "ms_per_step": round(dt2 / K * 1e3, 3),
            "expert_hit_rate": round(s2["expert_hits"] / max(1, s2["expert_hits"] + s2["expert_misses"]), 4),
            "fills_per_token": round(s2["fills"] / K, 3), "fills_skipped_per_token": round(s2["fills_skipped"] / K, 3),
            "host_ffn_ms_per_token": round(s2["host_ffn_ms"] / K, 3)}
        log(json.dumps(result["bounded_post_fetch"]))
        rt = rt2
    if not args.no_resident and wl.name != "tiny":
        rt.close()
        result["all_resident"], pf = all_resident_and_prefill(args, torch, moe, synth, wl, world, xd,
                                                              prefill=wl.name == "mixtral")
        if pf is not None:
            result["prefill"] = pf
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, world, args.seed, args.cpu_baseline_s, args.warmup)
    else:
        result["cpu_baseline"] = None
    rt.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
