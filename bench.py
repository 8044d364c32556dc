#!/usr/bin/env python
"""Throughput of the LouisKV clustering-and-retrieval path on one MI355X.

One step is one full request pass of the long-input short-output workload
(li-so-32k: 32 layers x 8 KV heads = 256 slices, 32768 prompt tokens, 1024
clusters, 10 Lloyd iterations, bf16; then 128 decode steps with boundary test,
retrieval at boundaries (budget 2048), window store and sparse attention for
all layers):

  prefill   louiskv_cluster_prefill (k-means + cluster-packed K/V pool)
            (after the timed steps, the pipelined variant is timed apart:
            louiskv_cluster_prefill_pipelined, one layer's slices per chunk,
            each chunk's pool write overlapped with the next chunk's k-means)
  decode    128 x [boundary_check, retrieve_rows, segment_output,
                   sparse_decode_attn_rows]   (KV_critical as a pool row list)
            launched for all layers at once; the same loop with one launch
            sequence per layer (as a model runs) is timed apart

Inputs are seeded synthetic tensors already resident in HBM before timing.
Prints one JSON line: value = prompt keys clustered per second (the k-means
of louiskv_cluster_prefill: init, 10 x (assign + update) and the CSR/perm
build; the pool pack that follows in the same step is timed and reported
apart, as the paper overlaps it with the model's prefill); the decode
rate is reported alongside, and the decode rate with the gathered (copied)
KV_critical of louiskv_retrieve + louiskv_sparse_decode_attn after it;
`roofline` covers the dominant kernel (the MFMA k-means assignment), timed
with HIP events on the stream it runs on; `cpu_baseline` times the CPU oracle
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prompt keys clustered/s; retrieval+sparse-attn decode steps/s at 32K ctx"
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "kmeans_assign_traffic_li-so-32k.md")
ASSIGN_SOURCES = [os.path.join(ROOT, "paper_2510_11292_amd", "csrc", f) for f in ("kmeans.hip", "common.h")]
ATTN_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attention_traffic_li-so-32k.md")
ATTN_SOURCES = [os.path.join(ROOT, "paper_2510_11292_amd", "csrc", f) for f in ("decode.hip", "common.h")]


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def make_inputs(wl, device, layer_major: bool = False):
    """Seeded inputs of every (sequence, layer) group, sequence by sequence;
    with layer_major the groups are ordered layer by layer (all sequences of
    layer 0, then layer 1, ...) so that one layer of the batch is a contiguous
    run of slices."""
    import torch
    import synth
    t0 = time.time()
    if layer_major:
        groups = [(seq, layer) for layer in range(wl.n_layers) for seq in range(wl.batch)]
    else:
        groups = [(seq, layer) for seq in range(wl.batch) for layer in range(wl.n_layers)]
    data = synth.make_slices(wl, device, groups=groups)
    torch.cuda.synchronize()
    log(f"generated inputs for {data.n_slices} slices in {time.time() - t0:.1f}s")
    return data


def sources_sha256(paths) -> str:
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str, path: str = TRAFFIC_FILE, sources=ASSIGN_SOURCES):
    """HBM bytes per launch of a kernel from its committed counter summary
    (FETCH_SIZE + WRITE_SIZE, calibrated on a plain copy), or None when the
    summary is missing, covers another workload, or the kernel's sources have
    changed since the counters were taken."""
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].split(": ", 1)
                fields[k.strip()] = v.strip().strip("`")
    try:
        if fields.get("workload") != workload or fields.get("kernel_sources_sha256") != sources_sha256(sources):
            return None
        return float(fields["fetch_bytes_per_launch"]) + float(fields["write_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def time_attention(eng, wl, reps=20):
    """Average duration of louiskv_sparse_decode_attn on the engine's final
    decode state, timed with HIP events on the stream it is launched on."""
    import torch
    from paper_2510_11292_amd import louiskv as L
    c = eng.cfg
    t = c.gen_len - 1
    _, _, n_local, local_start = L.window_info(t, c.window, c.seg_len)
    q = torch.randn(c.n_groups, c.n_q_heads, c.head_dim, device=eng.device).to(eng.dtype)
    st = torch.cuda.current_stream()

    def launch():
        if eng.seg_state is not None:
            if eng.zero_copy:
                L.sparse_decode_attn_rows_seg(q, c.n_kv_heads, eng.k_pool, eng.v_pool, eng.sel_rows, eng.n_sel,
                                              eng.k_local, eng.v_local, eng.seg_state, t + 1, eng.out, eng.lse,
                                              workspace=eng.ws_attn, stream=st)
            else:
                L.sparse_decode_attn_seg(q, c.n_kv_heads, eng.k_buf, eng.v_buf, eng.n_sel, eng.k_local, eng.v_local,
                                         eng.seg_state, t + 1, eng.out, eng.lse, workspace=eng.ws_attn, stream=st)
        elif eng.zero_copy:
            L.sparse_decode_attn_rows(q, c.n_kv_heads, eng.k_pool, eng.v_pool, eng.sel_rows, eng.n_sel,
                                      eng.k_local, eng.v_local, local_start, n_local, eng.out, eng.lse,
                                      workspace=eng.ws_attn, stream=st)
        elif eng.delta:
            L.sparse_decode_attn_rows(q, c.n_kv_heads, eng.k_buf, eng.v_buf, eng.slot_list, eng.n_sel,
                                      eng.k_local, eng.v_local, local_start, n_local, eng.out, eng.lse,
                                      workspace=eng.ws_attn, stream=st)
        else:
            L.sparse_decode_attn(q, c.n_kv_heads, eng.k_buf, eng.v_buf, eng.n_sel, eng.k_local, eng.v_local,
                                 local_start, n_local, eng.out, eng.lse, workspace=eng.ws_attn, stream=st)
    for _ in range(3):
        launch()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(reps):
        launch()
    e1.record(st)
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) / reps / 1e3
    esz = eng.k_local.element_size()
    n_sel = int(eng.n_sel.sum())
    if eng.seg_state is not None:   # each slice's window from its first live token
        rows = n_sel + int((t + 1 - eng.seg_state[:, 1].long()).clamp(0, c.window).sum())
    else:
        rows = n_sel + c.n_slices * n_local
    nbytes = rows * 2 * c.head_dim * esz + 2 * c.n_groups * c.n_q_heads * c.head_dim * esz
    if eng.zero_copy:
        nbytes += 4 * n_sel            # the row list
    return sec, nbytes


def dense_decode_ms(wl, data, cfg, dtype, reps=2):
    """Decode loop with the dense KV_critical (louiskv_retrieve gathers every
    selected row, louiskv_sparse_decode_attn reads the copies), as one HIP
    graph after a fresh prefill; mean replay time in ms."""
    import torch
    from paper_2510_11292_amd.engine import LouisKVEngine
    eng = LouisKVEngine(cfg, dtype, "cuda", pool_on_host=wl.pool_on_host, zero_copy=False, delta=False)

    def decode_all():
        for t in range(wl.gen_len):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        decode_all()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    eng.t = 0
    with torch.cuda.graph(graph):
        decode_all()
    ms = 0.0
    for _ in range(reps):
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        ms += e0.elapsed_time(e1)
    del graph, eng
    torch.cuda.empty_cache()
    return ms / reps


def layer_by_layer_decode_ms(eng, data, wl, n_steps, reps=2, t0=0):
    """Decode steps t0 .. t0 + n_steps - 1 with every step run group by group
    (one launch sequence per layer of the batch, the order in which a model
    produces its queries), one HIP graph per decode step (as a serving loop
    captures its steps), replayed after a fresh prefill and the first t0 steps
    (one batched graph, untimed); mean ms of the timed steps."""
    import torch

    def one_step(t):
        # one launch sequence per layer: the batch's groups of a layer are contiguous
        eng.step_layer_by_layer(data.queries[t], data.gen_keys[t], data.gen_values[t], groups_per_launch=wl.batch)

    def advance():
        for t in range(t0):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        advance()
        for t in range(t0, t0 + n_steps):
            one_step(t)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    pre = None
    if t0 > 0:
        pre = torch.cuda.CUDAGraph()
        eng.t = 0
        with torch.cuda.graph(pre):
            advance()
    graphs = []
    eng.t = t0
    for t in range(t0, t0 + n_steps):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            one_step(t)
        graphs.append(g)
    ms = 0.0
    for _ in range(reps):
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
        if pre is not None:
            pre.replay()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for g in graphs:
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        ms += e0.elapsed_time(e1)
    del graphs, pre
    return ms / reps


def layer_roofline(attn_bytes: float, sec_per_step: float) -> dict:
    """HBM fraction of the layer-by-layer decode: the K/V rows one step
    attends to over all layers (the attention kernel's algorithmic bytes on
    the final state, the dominant traffic of a step) per measured step time."""
    achieved = attn_bytes / sec_per_step / 1e9
    return {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS, "bytes_per_step": attn_bytes, "us_per_step": sec_per_step * 1e6}


def layer_window(wl, n: int = 512):
    """The decode steps timed group by group: the last n of the generation,
    where the most evicted segments are units."""
    n = min(n, wl.gen_len)
    return wl.gen_len - n, n


def delta_fetch_rate(eng, data, wl) -> dict:
    """Host-link rate of the delta transfers: one louiskv_retrieve_delta with
    every group fired on the engine's final state, with an early query, so
    that many selected rows are new; bytes moved over the host link / time."""
    import torch
    from paper_2510_11292_amd import louiskv as L
    c = eng.cfg
    fire = torch.ones_like(eng.fire)
    fired = eng.fire
    eng.fire = fire
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_units = eng.n_units_before(c.gen_len - 1)
    e0.record()
    eng._retrieve_delta(data.queries[0], n_units, eng.seg_state)
    e1.record()
    torch.cuda.synchronize()
    moved = int(eng.n_fetched.sum()) * 2 * c.head_dim * eng.k_buf.element_size()
    sec = e0.elapsed_time(e1) / 1e3
    eng.fire = fired
    return {"delta_fetch_GBps": moved / sec / 1e9, "delta_fetch_bytes": moved, "delta_call_ms": sec * 1e3,
            "what": f"one {'louiskv_retrieve_cached' if eng.cached else 'louiskv_retrieve_delta'} (scores, "
                    f"selection, plan, fetch) with every group fired"}


def copy_calibration(mib: int):
    """A streaming copy kernel of a known size (outside the timed region): the
    reference for scaling the HBM byte counters.  torch.mul(x, 1) reads and
    writes `mib` MiB once each (a same-type copy_ would become a DMA transfer
    rather than a kernel)."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    log(f"copy calibration: 3 copy kernels of {mib} MiB")


def cpu_baseline(wl, data, budget_s: float):
    """The oracle on a bounded sample: k-means of the KV-head slices of one
    (sequence, layer) group (full iterations, until the time budget is used),
    then the decode loop of that group over the decode steps (until the budget
    is used), each scaled to the whole workload."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas_threads = 1

    def f64(t):
        return t.detach().float().cpu().numpy().astype(np.float64)

    H = wl.n_kv_heads
    bf16 = wl.dtype == "bf16"
    results = []
    t_km = 0.0
    for h in range(H):
        if results and t_km >= budget_s:
            break
        t0 = time.time()
        results.append(oracle.kmeans(f64(data.prompt_keys[h]), data.init_idx[h].cpu().numpy(), wl.n_iters, bf16))
        t_km += time.time() - t0
    km_slices = len(results)
    keys_per_s = km_slices * wl.prompt_len / t_km       # every slice costs the same
    # heads past the budget start decoding from one Lloyd iteration (same unit count and sizes scale)
    results += [oracle.kmeans(f64(data.prompt_keys[h]), data.init_idx[h].cpu().numpy(), 1, bf16)
                for h in range(km_slices, H)]

    # the same k-means on one core: two iterations of one slice, scaled to the
    # workload's iteration count (every iteration costs the same)
    keys_per_s_1 = None
    try:
        from threadpoolctl import threadpool_limits
        it1 = min(2, wl.n_iters)
        with threadpool_limits(limits=1):
            t0 = time.time()
            oracle.kmeans(f64(data.prompt_keys[0]), data.init_idx[0].cpu().numpy(), it1, bf16)
            t1 = time.time() - t0
        keys_per_s_1 = wl.prompt_len / (t1 * wl.n_iters / it1)
    except Exception:  # pragma: no cover
        pass
    st = oracle.prefill_state_from_kmeans([f64(data.prompt_keys[h]) for h in range(H)],
                                          [f64(data.prompt_values[h]) for h in range(H)], results)
    dec = oracle.GroupDecoder(st, wl.n_q_heads, wl.budget, wl.window, wl.seg_len, wl.tau, "anchor")
    t0 = time.time()
    n = 0
    while n < wl.gen_len and (time.time() - t0) < budget_s:
        dec.step(f64(data.queries[n, 0]), f64(data.gen_keys[n, :H]), f64(data.gen_values[n, :H]))
        n += 1
    t_dec = (time.time() - t0) / n          # one group, one step
    steps_per_s = 1.0 / (t_dec * wl.n_groups)
    return {
        "value": keys_per_s, "unit": "keys/s", "cores": int(blas_threads), "kind": "oracle",
        "decode_steps_per_s": steps_per_s, "value_1_core": keys_per_s_1,
        "sample": (f"k-means of {km_slices} of {wl.n_slices} slices ({wl.prompt_len} keys, C={wl.n_clusters}, "
                   f"{wl.n_iters} iterations) in {t_km:.1f}s, scaled linearly; decode: {n} of {wl.gen_len} steps "
                   f"of 1 of {wl.n_groups} layer groups in {t_dec * n:.1f}s, scaled by the group count; "
                   f"value_1_core: 2 iterations of one slice on one thread, scaled to {wl.n_iters}"),
        "host_cpus": len(os.sched_getaffinity(0)), "cpu": platform.processor() or platform.machine(),
    }


def host_link_rates(eng, data, mib: int = 256, reps: int = 4) -> dict:
    """Achievable host-link rates next to the path's own: pinned-memory DMA
    copies of `mib` MiB each way (hipMemcpyAsync through torch), and the
    zero-copy gather of louiskv_retrieve reading the selected rows of every
    slice from the host pool (all groups fired), in GB/s."""
    import torch
    from paper_2510_11292_amd import louiskv as L
    n = mib * (1 << 20)
    if hasattr(torch._C, "_host_emptyCache"):
        torch._C._host_emptyCache()   # pinned blocks of engines already freed
    host = torch.empty(n, dtype=torch.uint8).pin_memory()
    dev = torch.empty(n, dtype=torch.uint8, device=eng.device)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def rate(fn, nbytes):
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return nbytes * reps / (e0.elapsed_time(e1) / 1e3) / 1e9

    out = {"h2d_dma_GBps": rate(lambda: dev.copy_(host, non_blocking=True), n),
           "d2h_dma_GBps": rate(lambda: host.copy_(dev, non_blocking=True), n)}
    del host, dev
    c = eng.cfg
    kb = torch.empty(c.n_slices, c.budget, c.head_dim, dtype=eng.dtype, device=eng.device)
    vb = torch.empty_like(kb)
    su = torch.empty(c.n_slices, c.units_cap, dtype=torch.int32, device=eng.device)
    nsu = torch.empty(c.n_slices, dtype=torch.int32, device=eng.device)
    ns = torch.empty_like(nsu)
    ws = torch.empty(L.retrieve_workspace_size(c.n_slices, c.units_cap, c.budget), dtype=torch.uint8,
                     device=eng.device)
    q = data.queries[0]

    def gather():
        L.retrieve(q, c.n_kv_heads, eng.reps, eng.unit_start, eng.unit_size, c.n_clusters, eng.k_pool, eng.v_pool,
                   c.budget, su, nsu, ns, kb, vb, pool_on_host=True, workspace=ws)
    gather()
    torch.cuda.synchronize()
    moved = int(ns.sum()) * 2 * c.head_dim * kb.element_size()
    out["zero_copy_gather_GBps"] = rate(gather, moved)
    out["gather_bytes"] = moved
    del kb, vb, ws
    return out


def time_pipelined_prefill(eng, data, chunk: int, copy_engine: bool, reps: int = 3) -> float:
    """Mean ms of louiskv_cluster_prefill_pipelined over the engine's buffers
    (the clustering of each chunk of slices overlapped with the pool write of
    the previous one), after one untimed call."""
    import torch
    from paper_2510_11292_amd import louiskv as L
    c = eng.cfg
    S = c.n_slices
    chunk = max(1, min(chunk, S))
    dc = L.BF16 if eng.dtype == torch.bfloat16 else L.F32
    ws = torch.empty(L.cluster_prefill_pipelined_workspace_size(chunk, c.prompt_len, c.n_clusters, dc,
                                                                eng.pool_on_host, copy_engine),
                     dtype=torch.uint8, device=eng.device)
    events = [torch.cuda.Event() for _ in range(-(-S // chunk) + 1)]
    for e in events:
        e.record()
    copy_stream = torch.cuda.Stream()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    total = 0.0
    for i in range(reps + 1):
        t0.record()
        L.cluster_prefill_pipelined(data.prompt_keys, c.n_clusters, c.n_iters, data.init_idx, eng.reps,
                                    eng.unit_start, eng.unit_size, eng.assign, eng.perm, data.prompt_values,
                                    eng.k_pool, eng.v_pool, chunk, events, copy_stream,
                                    pool_on_host=eng.pool_on_host, copy_engine=copy_engine, workspace=ws)
        t1.record()
        torch.cuda.synchronize()
        if i > 0:
            total += t0.elapsed_time(t1)
    del ws
    return total / reps


def workload_pass(name: str, dev: str, layer_steps: int = 512) -> dict:
    """One stated timed pass of a workload other than the headline one, after
    one untimed pass: the clustering (keys/s and the assignment kernel's MFMA
    fraction, from HIP events on its stream), the decode loop as one HIP graph
    (steps/s), the attention kernel on the final state (GB/s and HBM
    fraction), the last `layer_steps` decode steps group by group (steps/s)
    and, for a host-resident pool, the host-link rates of the same run."""
    import torch
    import synth
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    from paper_2510_11292_amd import louiskv as L
    wl = synth.get_workload(name)
    t_start = time.time()
    # layer-major group order: a layer of the batch is one contiguous view
    data = make_inputs(wl, dev, layer_major=wl.batch > 1)
    cfg = config_from_workload(wl, mode=L.REF_ANCHOR)
    dtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    eng = LouisKVEngine(cfg, dtype, dev, pool_on_host=wl.pool_on_host)
    iters = wl.n_iters
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * iters)] for _ in range(2)]
    for evs in ev:
        for e in evs:
            e.record()
    ph = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(2)]

    def decode_all():
        for t in range(wl.gen_len):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
    # rows copied into KV_critical against rows selected over the fired slices
    # of the untimed pass (counted on the device)
    moved = torch.zeros(2, dtype=torch.int64, device=dev)

    def decode_all_counting():
        for t in range(wl.gen_len):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
            if eng.delta:
                fired = eng.fire.repeat_interleave(wl.n_kv_heads).bool()
                moved[0] += eng.n_fetched.sum()
                moved[1] += torch.where(fired, eng.n_sel, 0).sum()
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        decode_all_counting()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    eng.t = 0
    with torch.cuda.graph(graph):
        decode_all()
    for i in range(2):
        ph[i][0].record()
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx, iter_events=ev[i], pack_event=ph[i][3])
        ph[i][1].record()
        graph.replay()
        ph[i][2].record()
    torch.cuda.synchronize()
    t_cluster = ph[1][0].elapsed_time(ph[1][3]) / 1e3
    t_pre = ph[1][0].elapsed_time(ph[1][1]) / 1e3
    t_dec = ph[1][1].elapsed_time(ph[1][2]) / 1e3
    t_assign = sum(ev[1][2 * k].elapsed_time(ev[1][2 * k + 1]) for k in range(iters)) / iters / 1e3
    flops = 2.0 * wl.prompt_len * wl.n_clusters * wl.head_dim * wl.n_slices
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    t_attn, attn_bytes = time_attention(eng, wl)
    out = {
        "config": {"batch": wl.batch, "layers": wl.n_layers, "kv_heads": wl.n_kv_heads, "prompt_tokens":
                   wl.prompt_len, "clusters": wl.n_clusters, "decode_steps": wl.gen_len, "budget": wl.budget,
                   "dtype": wl.dtype, "pool": "pinned host" if wl.pool_on_host else "hbm"},
        "timed": "one pass (prefill + every decode step) after one untimed pass",
        "keys_per_s": wl.n_slices * wl.prompt_len / t_cluster,
        "cluster_ms": t_cluster * 1e3, "pool_pack_ms": (t_pre - t_cluster) * 1e3,
        "assign_roofline": {"achieved": flops / t_assign / 1e12, "peak": peak, "unit": "TFLOP/s",
                            "frac": flops / t_assign / 1e12 / peak, "avg_launch_ms": t_assign * 1e3,
                            "bound": "mfma", "dtype": wl.dtype},
        "decode_steps_per_s": wl.gen_len / t_dec,
        "attention_roofline": {"achieved": attn_bytes / t_attn / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                               "frac": attn_bytes / t_attn / 1e9 / PEAK_HBM_GBS, "avg_launch_us": t_attn * 1e6,
                               "bytes_per_launch": attn_bytes, "bound": "hbm",
                               "reads": "the pool rows of the selection (row list)" if eng.zero_copy else
                                        "the HBM KV_critical buffers (slot list)"},
    }
    del graph
    t0, n = layer_window(wl, layer_steps)
    lms = layer_by_layer_decode_ms(eng, data, wl, n, reps=1, t0=t0)
    out["decode_steps_per_s_layer_by_layer"] = n / (lms / 1e3)
    out["layer_by_layer_steps"] = f"steps {t0}..{t0 + n - 1} of {wl.gen_len}, one HIP graph per step"
    out["layer_by_layer_roofline"] = layer_roofline(attn_bytes, lms / 1e3 / n)
    if eng.pool_on_host:
        out["host_link"] = host_link_rates(eng, data)
        out["host_link"].update(delta_fetch_rate(eng, data, wl))
        mv = moved.tolist()
        out["host_link"].update({"kv_critical_rows": eng.cache_rows, "budget": wl.budget,
                                 "fetched_rows": mv[0], "selected_rows": mv[1],
                                 "fetched_fraction": mv[0] / max(mv[1], 1)})
    log(f"{name}: {out['keys_per_s']:.3g} keys/s (assign {out['assign_roofline']['frac']:.3f} of peak), decode "
        f"{out['decode_steps_per_s']:.0f} steps/s, layer by layer {out['decode_steps_per_s_layer_by_layer']:.0f}, "
        f"attention {out['attention_roofline']['achieved']:.0f} GB/s; {time.time() - t_start:.0f}s")
    del eng, data
    torch.cuda.empty_cache()
    if hasattr(torch._C, "_host_emptyCache"):
        torch._C._host_emptyCache()
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="li-so-32k")
    ap.add_argument("--mode", default="anchor", choices=["anchor", "prev"])
    ap.add_argument("--segments", default="fixed", choices=["fixed", "boundary"],
                    help="output segments: fixed runs (the workload's definition) or delimited by the boundaries")
    ap.add_argument("--cpu-budget-s", type=float, default=12.0,
                    help="seconds of oracle k-means, and again of oracle decode steps, in the CPU baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true", help="launch decode steps one by one (no HIP graph)")
    ap.add_argument("--prefill-chunk", type=int, default=0,
                    help="slices per chunk of the pipelined prefill that is timed after the run "
                         "(default: one layer's KV heads; -1 skips it)")
    ap.add_argument("--no-layer-by-layer", action="store_true",
                    help="skip the decode timing with one launch sequence per layer")
    ap.add_argument("--workloads", default="tiny-4k,si-lo-16k,li-lo-32k-b4,host-131k",
                    help="other workloads timed after the headline one, one pass each ('none' skips them)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after the run, copy this many MiB three times (counter calibration for profiles)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the LouisKV path is built and measured on a single MI355X "
              "(slices shard across GPUs with no communication except one boundary all-reduce per "
              "layer; see the design notes). Run with --gpus 1.", file=sys.stderr)
        return 2

    import torch
    import synth
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    from paper_2510_11292_amd import louiskv as L

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = "cuda"
    wl = synth.get_workload(args.workload)
    mode = L.REF_ANCHOR if args.mode == "anchor" else L.REF_PREV
    data = make_inputs(wl, dev)
    cfg = config_from_workload(wl, mode=mode, segments=args.segments,
                               allow_unit_overflow=args.segments == "boundary")
    dtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    eng = LouisKVEngine(cfg, dtype, dev, pool_on_host=wl.pool_on_host)

    total = args.warmup + args.steps
    iters = wl.n_iters
    assign_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * iters)] for _ in range(total)]
    for evs in assign_ev:          # create the underlying events before handing them to the library
        for e in evs:
            e.record()
    ph = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(total)]

    def decode_all():
        for t in range(wl.gen_len):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])

    # rows copied by the delta retrieval, against rows selected, over the
    # fired slices of one pass (counted on the device, eager pass only)
    moved = torch.zeros(2, dtype=torch.int64, device=dev)

    def decode_all_counting():
        for t in range(wl.gen_len):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
            if eng.delta:
                fired = eng.fire.repeat_interleave(wl.n_kv_heads).bool()
                moved[0] += eng.n_fetched.sum()
                moved[1] += torch.where(fired, eng.n_sel, 0).sum()

    graph = None
    if not args.eager:
        # capture the whole decode loop once; replays follow a fresh prefill
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            decode_all_counting()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        eng.t = 0
        with torch.cuda.graph(graph):
            decode_all()
        torch.cuda.synchronize()

    fires = []
    torch.cuda.synchronize()
    wall0 = None
    for i in range(total):
        if i == args.warmup:
            torch.cuda.synchronize()
            wall0 = time.perf_counter()
        ph[i][0].record()
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx, iter_events=assign_ev[i],
                    pack_event=ph[i][3])
        ph[i][1].record()
        if graph is not None:
            graph.replay()
        else:
            decode_all()
        ph[i][2].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0

    timed = range(args.warmup, total)
    t_pre = sum(ph[i][0].elapsed_time(ph[i][1]) for i in timed) / args.steps / 1e3
    t_cluster = sum(ph[i][0].elapsed_time(ph[i][3]) for i in timed) / args.steps / 1e3
    t_pack = t_pre - t_cluster
    t_dec = sum(ph[i][1].elapsed_time(ph[i][2]) for i in timed) / args.steps / 1e3
    t_assign = sum(assign_ev[i][2 * k].elapsed_time(assign_ev[i][2 * k + 1])
                   for i in timed for k in range(iters)) / (args.steps * iters) / 1e3
    flops_per_launch = 2.0 * wl.prompt_len * wl.n_clusters * wl.head_dim * wl.n_slices
    keys = wl.n_slices * wl.prompt_len
    ms_per_step = wall / args.steps * 1e3
    fire_rate = float(eng.fire.float().mean())  # last step's groups (informational)
    achieved = flops_per_launch / t_assign / 1e12
    t_attn, attn_bytes = time_attention(eng, wl)
    traffic = measured_traffic(wl.name)
    dense_ms = None
    if (eng.zero_copy or eng.delta) and not args.eager:
        dense_ms = dense_decode_ms(wl, data, cfg, dtype)
    layer_ms = layer_steps = layer_t0 = None
    if not args.eager and not args.no_layer_by_layer:
        layer_t0, layer_steps = layer_window(wl)
        if wl.batch > 1:
            # one launch sequence per layer needs the batch's groups of a
            # layer next to each other (the batched loop above runs faster
            # with the sequence-major order)
            del data
            torch.cuda.empty_cache()
            data = make_inputs(wl, dev, layer_major=True)
        layer_ms = layer_by_layer_decode_ms(eng, data, wl, layer_steps, t0=layer_t0)
        log(f"decode layer by layer: steps {layer_t0}..{layer_t0 + layer_steps - 1} in {layer_ms:.2f} ms "
            f"({layer_steps / (layer_ms / 1e3):.0f} steps/s)")
    link = None
    if eng.pool_on_host:
        link = host_link_rates(eng, data)
        log(f"host link: DMA {link['h2d_dma_GBps']:.1f} GB/s in, {link['d2h_dma_GBps']:.1f} GB/s out; "
            f"zero-copy gather of selected rows {link['zero_copy_gather_GBps']:.1f} GB/s")
    pipelined = None
    if args.prefill_chunk >= 0:
        chunk = args.prefill_chunk or wl.n_kv_heads
        pipelined = {"slices_per_chunk": chunk, "serial_ms": t_pre * 1e3}
        pipelined["overlapped_ms"] = time_pipelined_prefill(eng, data, chunk, True)
        if eng.pool_on_host:
            pipelined["pool_write"] = "copy engines (HBM staging, pitched copy)"
            pipelined["overlapped_ms_pack_kernel"] = time_pipelined_prefill(eng, data, chunk, False)
        else:
            pipelined["pool_write"] = "pack kernel on a second stream"
        log(f"prefill: serial {t_pre * 1e3:.2f} ms; pipelined over chunks of {chunk} slices "
            f"{pipelined['overlapped_ms']:.2f} ms"
            + (f" (pack kernel instead of copy engines: {pipelined['overlapped_ms_pack_kernel']:.2f} ms)"
               if eng.pool_on_host else ""))
    out = {
        "metric": METRIC,
        "value": keys / t_cluster,
        "unit": "keys/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name, "batch": wl.batch, "layers": wl.n_layers, "kv_heads": wl.n_kv_heads,
            "q_heads": wl.n_q_heads, "head_dim": wl.head_dim, "prompt_tokens": wl.prompt_len,
            "clusters": wl.n_clusters, "lloyd_iters": wl.n_iters, "decode_steps": wl.gen_len,
            "budget": wl.budget, "window": wl.window, "segment": wl.seg_len, "tau": wl.tau,
            "ref_mode": args.mode, "segments": args.segments,
            "decode_launch": "eager" if graph is None else "hip_graph",
            "kv_critical": ("pool row list (zero-copy)" if eng.zero_copy else
                            f"LRU cache of {eng.cache_rows} pool rows per slice" if eng.cached else
                            "last selection's pool rows (delta transfers)" if eng.delta else "gathered copy"),
        },
        "decode_steps_per_s": wl.gen_len / t_dec,
        "decode_steps_per_s_gathered_kv_critical": (wl.gen_len / (dense_ms / 1e3)) if dense_ms else None,
        "decode_steps_per_s_layer_by_layer": (layer_steps / (layer_ms / 1e3)) if layer_ms else None,
        "layer_by_layer_steps": (f"steps {layer_t0}..{layer_t0 + layer_steps - 1} of {wl.gen_len}, one HIP graph "
                                 f"per step, {wl.n_layers} launch sequences per step") if layer_ms else None,
        "layer_by_layer_roofline": (layer_roofline(attn_bytes, layer_ms / 1e3 / layer_steps)
                                    if layer_ms else None),
        "delta_rows_moved_per_selected": (float(moved[0]) / max(float(moved[1]), 1.0)) if eng.delta else None,
        "segment_overflow": eng.segment_overflow() if args.segments == "boundary" else None,
        "prefill_ms": t_pre * 1e3,
        "cluster_ms": t_cluster * 1e3,
        "pool_pack_ms": t_pack * 1e3,
        "decode_ms": t_dec * 1e3,
        "prefill_pipelined": pipelined,
        "host_link": link,
        "roofline": {
            "kernel": "kmeans_assign (bf16 MFMA, fused argmin)",
            "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
            "avg_launch_ms": t_assign * 1e3, "flops_per_launch": flops_per_launch,
        },
        "attention_roofline": {
            "kernel": ("sparse_decode_attn_rows" if (eng.zero_copy or eng.delta) else "sparse_decode_attn")
            + " (bf16 MFMA scores, all slices)", "bound": "hbm",
            "achieved": attn_bytes / t_attn / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": attn_bytes / t_attn / 1e9 / PEAK_HBM_GBS, "avg_launch_us": t_attn * 1e6,
            "bytes_per_launch": attn_bytes,
            "traffic": (measured_traffic(wl.name, ATTN_TRAFFIC_FILE, ATTN_SOURCES)
                        if eng.zero_copy and args.segments == "fixed" else None),
        },
    }
    log(f"clustering {t_cluster * 1e3:.2f} ms + pool pack {t_pack * 1e3:.2f} ms; decode {t_dec * 1e3:.2f} ms ({wl.gen_len / t_dec:.0f} steps/s), "
        f"assign {t_assign * 1e3:.3f} ms/launch = {achieved:.1f} TFLOP/s, last-step fire rate {fire_rate:.2f}")
    log(f"attention {t_attn * 1e6:.1f} us/launch = {attn_bytes / t_attn / 1e9:.0f} GB/s")
    if dense_ms:
        log(f"decode with the gathered KV_critical: {dense_ms:.2f} ms ({wl.gen_len / (dense_ms / 1e3):.0f} steps/s)")
    if args.copy_mib > 0:
        copy_calibration(args.copy_mib)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, data, args.cpu_budget_s)
    others = [w for w in args.workloads.split(",") if w and w != "none" and w != wl.name]
    if others:
        del eng, data
        torch.cuda.empty_cache()
        out["workloads"] = {w: workload_pass(w, dev) for w in others}
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
