"""Parity at the full workload sizes, in the launch configuration the benchmark
times: every slice of the workload runs on the GPU in one launch per call, and
sampled outputs are checked against the oracle one by one.

  k-means      li-so-32k, si-lo-16k, li-lo-32k-b4, host-131k: on sampled
               slices, the tenth assignment against the oracle's argmin from
               the GPU's ninth centroids (sampled keys), the tenth centroids
               and counts as exact means of that assignment, and the packed
               pool rows of sampled clusters.
  decode       every step of every group runs (all T steps); at sampled steps
               of two groups the step's outputs are recomputed by the oracle
               from the state the GPU held before the step: the boundary value
               and decision, the scores and the budgeted selection when the
               group fired, KV_critical (copied rows or the row list) against
               the pool rows of the selection,
               the local window and any evicted segment (mean and pool rows),
               and the attention output.
  layer by     li-so-32k, si-lo-16k, li-lo-32k-b4, host-131k: one launch sequence a
  layer        layer, as the benchmark runs it, step for step against the
               batched decode.
  graph        li-so-32k's 128-step decode loop as one HIP graph, as the
               benchmark times it, against the eager loop.
"""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import oracle  # noqa: E402
import synth  # noqa: E402
from parity_utils import REL, check_assignment, report, selection_matches, to64, to_np  # noqa: E402

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

DEV = "cuda"
LARGE = ["li-so-32k", "si-lo-16k", "li-lo-32k-b4", "host-131k"]


def _L():
    from paper_2510_11292_amd import louiskv
    louiskv.load_library()
    return louiskv


@pytest.mark.parametrize("name", LARGE)
def test_cluster_prefill_full_shape_sampled(name):
    L = _L()
    wl = synth.get_workload(name)
    S, P, C = wl.n_slices, wl.prompt_len, wl.n_clusters
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    keys = torch.empty(S, P, 128, dtype=dt, device=DEV)
    init = torch.empty(S, C, dtype=torch.int32)
    for s in range(S):
        grp, h = divmod(s, wl.n_kv_heads)
        seq, layer = divmod(grp, wl.n_layers)
        keys[s] = synth.slice_keys_values(wl, seq, layer, h, DEV, n_tokens=P)[0]
        init[s] = synth.init_indices(wl, seq, layer, h)
    init = init.to(DEV)
    outs = {}
    for iters in (wl.n_iters - 1, wl.n_iters):
        reps = torch.empty(S, C, 128, device=DEV)
        ustart = torch.empty(S, C, dtype=torch.int32, device=DEV)
        usize = torch.empty_like(ustart)
        assign = torch.empty(S, P, dtype=torch.int32, device=DEV)
        perm = torch.empty_like(assign)
        L.cluster_prefill(keys, C, iters, init, reps, ustart, usize, assign, perm)
        torch.cuda.synchronize()
        outs[iters] = (reps, assign, usize, ustart, perm)
    del perm
    rng = np.random.default_rng(0)
    n_sample = min(P, 2048)
    for s in (0, S // 3, S - 1):
        k64 = to64(keys[s])
        c9 = to64(outs[wl.n_iters - 1][0][s])
        reps10, z10, cnt10, st10, perm10 = (to_np(t[s]) for t in outs[wl.n_iters])
        sample = rng.choice(P, n_sample, replace=False)
        check_assignment(k64[sample], oracle.round_to_bf16(c9) if wl.dtype == "bf16" else c9, z10[sample])
        ref, cnt = oracle.kmeans_update(k64, z10, c9)
        assert np.array_equal(cnt10, cnt)
        assert np.array_equal(reps10.astype(np.float64), ref)
        # CSR of the assignment: members of each cluster in ascending token order
        assert np.array_equal(st10, np.concatenate([[0], np.cumsum(cnt)[:-1]]))
        for c in rng.choice(C, 8, replace=False):
            assert np.array_equal(perm10[st10[c]:st10[c] + cnt10[c]], np.flatnonzero(z10 == c))


def _check_step(eng, data, wl, t, gi, q_ref_before, stats):
    """Recompute decode step t of group gi with the oracle from the GPU's state."""
    L = _L()
    H, g, W, seg, C, P = wl.n_kv_heads, wl.group_size, wl.window, wl.seg_len, wl.n_clusters, wl.prompt_len
    scale = 1 / np.sqrt(128)
    q64 = to64(data.queries[t, gi])
    fire = bool(to_np(eng.fire)[gi])
    r = float(to_np(eng.r)[gi])
    if t == 0:
        assert fire
    else:
        r_ref = oracle.query_similarity(q64, q_ref_before)
        assert abs(r - r_ref) <= 1e-9 * max(1.0, abs(r_ref)), (t, gi, r, r_ref)
        if fire != oracle.boundary_fires(r_ref, wl.tau, False):
            assert abs(r_ref - wl.tau) <= REL * max(abs(r_ref), wl.tau), (t, gi, r_ref)
            stats["excused"] += 1
    n_units = eng.n_units_before(t)
    ev, nev, n_local, local_start = L.window_info(t, W, seg)
    for h in range(H):
        s = gi * H + h
        sizes = to_np(eng.unit_size[s, :n_units]).astype(np.int64)
        starts = to_np(eng.unit_start[s, :n_units]).astype(np.int64)
        got = to_np(eng.sel_units[s, :int(eng.n_sel_units[s])]).tolist()
        nsel = int(eng.n_sel[s])
        if fire:
            stats["fires"] += 1
            a = oracle.group_scores(q64[h * g:(h + 1) * g], to64(eng.reps[s, :n_units]), scale)
            np.testing.assert_allclose(to_np(eng.scores[s, :n_units]), a, rtol=1e-12, atol=1e-300)
            stats["excused"] += selection_matches(a, sizes, wl.budget, got)
            assert nsel == int(sizes[got].sum()) <= wl.budget
        # KV_critical holds the rows of the current selection, in rank order: as
        # copies (dense) or as the list of their pool rows (zero-copy)
        idx = [rr for u in got for rr in range(int(starts[u]), int(starts[u] + sizes[u]))]
        assert len(idx) == nsel
        rows = torch.as_tensor(idx, dtype=torch.long)
        kp = eng.k_pool[s].index_select(0, rows.to(eng.k_pool.device))
        vp = eng.v_pool[s].index_select(0, rows.to(eng.v_pool.device))
        if eng.zero_copy:
            assert to_np(eng.sel_rows[s, :nsel]).tolist() == idx
        elif eng.delta:
            _check_delta_slots(eng, s, nsel, idx)
        else:
            assert torch.equal(eng.k_buf[s, :nsel].cpu(), kp.cpu()) and torch.equal(eng.v_buf[s, :nsel].cpu(), vp.cpu())
        # local window after the append: tokens nev*seg .. t in their ring slots
        slots = [(local_start + i) % W for i in range(n_local)]
        toks = list(range(nev * seg, t + 1))
        assert torch.equal(eng.k_local[s, slots].cpu(), data.gen_keys[toks, s].cpu())
        assert torch.equal(eng.v_local[s, slots].cpu(), data.gen_values[toks, s].cpu())
        if ev >= 0:
            u = C + ev
            prow = P + ev * seg
            seg_keys = data.gen_keys[ev * seg:(ev + 1) * seg, s]
            assert int(eng.unit_start[s, u]) == prow and int(eng.unit_size[s, u]) == seg
            assert torch.equal(eng.k_pool[s, prow:prow + seg].cpu(), seg_keys.cpu())
            assert torch.equal(eng.v_pool[s, prow:prow + seg].cpu(),
                               data.gen_values[ev * seg:(ev + 1) * seg, s].cpu())
            assert np.array_equal(to64(eng.reps[s, u]), oracle.segment_mean(to64(seg_keys)))
        kk = np.concatenate([to64(kp), to64(eng.k_local[s, slots])])
        vv = np.concatenate([to64(vp), to64(eng.v_local[s, slots])])
        o, _ = oracle.attention(q64[h * g:(h + 1) * g], kk, vv, scale)
        err = np.abs(to64(eng.out[gi, h * g:(h + 1) * g]) - o).max()
        assert err <= 2e-3, (t, s, err)
    stats["checked"] += 1


def _check_delta_slots(eng, s, nsel, idx):
    """KV_critical as a cache of pool rows: the listed slots hold copies of
    exactly the selected pool rows (in slot order, not rank order)."""
    bslots = to_np(eng.slot_list[s, :nsel]).astype(np.int64)
    held = to_np(eng.buf_row[s])[bslots].astype(np.int64)
    assert len(set(bslots.tolist())) == nsel and sorted(held.tolist()) == sorted(idx)
    hi = torch.as_tensor(held, dtype=torch.long)
    bi = torch.as_tensor(bslots, dtype=torch.long)
    assert torch.equal(eng.k_buf[s].cpu()[bi], eng.k_pool[s].cpu()[hi])
    assert torch.equal(eng.v_buf[s].cpu()[bi], eng.v_pool[s].cpu()[hi])


def _sample_steps(wl):
    T, W, seg = wl.gen_len, wl.window, wl.seg_len
    base = {0, 1, 2, 3, W - 1, W, W + 1, W + seg, W + seg + 1, T // 2, T - 2, T - 1}
    return {t for t in base if 0 <= t < T}


# The engine's default retrieval (zero-copy rows for device pools, delta
# transfers into KV_critical for the host pool), plus the dense gather on the
# benchmark workload and on the host pool.
DECODE_CASES = [(n, None) for n in LARGE] + [("li-so-32k", "dense"), ("host-131k", "dense")]


@pytest.mark.parametrize("name,retrieval", DECODE_CASES)
def test_decode_full_shape_sampled(name, retrieval):
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    L = _L()
    wl = synth.get_workload(name)
    data = synth.make_slices(wl, DEV)
    cfg = config_from_workload(wl, mode=L.REF_ANCHOR)
    eng = LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, pool_on_host=wl.pool_on_host, keep_scores=True,
                        out_dtype=torch.float32, zero_copy=False if retrieval == "dense" else None,
                        delta=False if retrieval == "dense" else None)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    torch.cuda.synchronize()
    groups = (0, wl.n_groups - 1)
    # the pool holds each cluster's prompt K/V rows contiguously, members in token order
    rng = np.random.default_rng(1)
    for s in (0, wl.n_slices - 1):
        z = to_np(eng.assign[s])
        for c in rng.choice(wl.n_clusters, 4, replace=False):
            st, sz = int(eng.unit_start[s, c]), int(eng.unit_size[s, c])
            toks = torch.as_tensor(np.flatnonzero(z == c), dtype=torch.long, device=DEV)
            assert sz == toks.numel()
            assert torch.equal(eng.k_pool[s, st:st + sz].cpu(), data.prompt_keys[s].index_select(0, toks).cpu())
            assert torch.equal(eng.v_pool[s, st:st + sz].cpu(), data.prompt_values[s].index_select(0, toks).cpu())
    steps = _sample_steps(wl)
    fired_checks_left = {"mid": 3, "late": 3}
    last_fire = {gi: None for gi in groups}
    stats = dict(fires=0, excused=0, checked=0)
    for t in range(wl.gen_len):
        q_ref = {gi: (None if last_fire[gi] is None else to64(data.queries[last_fire[gi], gi])) for gi in groups}
        eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        fire = to_np(eng.fire)
        region = "mid" if wl.gen_len // 2 <= t < 3 * wl.gen_len // 4 else ("late" if t >= 3 * wl.gen_len // 4 else None)
        extra = region is not None and fired_checks_left[region] > 0 and bool(fire[groups[0]])
        if t in steps or extra:
            if extra:
                fired_checks_left[region] -= 1
            for gi in groups:
                _check_step(eng, data, wl, t, gi, q_ref[gi], stats)
        for gi in groups:
            if fire[gi]:
                last_fire[gi] = t
    assert stats["fires"] > 0
    assert stats["checked"] >= 2 * len(steps)
    report(f"full-shape decode {name}", stats, bound=max(3, stats["fires"] // 100),
           of="boundary and selection near-ties")


def _check_step_boundary(eng, data, wl, t, gi, q_ref_before, before, fires, stats):
    """Step t of group gi with boundary-delimited segments, recomputed from the
    GPU's state: the boundary, the scores and selection over the slice's own
    unit count, KV_critical, the window from its first live token, the segment
    that left (if any: the oldest tokens, a fired step or a full-length
    segment before it, mean and pool rows), and the attention output."""
    H, g, W, smax, P = wl.n_kv_heads, wl.group_size, wl.window, wl.seg_len, wl.prompt_len
    scale = 1 / np.sqrt(128)
    q64 = to64(data.queries[t, gi])
    fire = bool(to_np(eng.fire)[gi])
    if t == 0:
        assert fire
    else:
        r_ref = oracle.query_similarity(q64, q_ref_before)
        if fire != oracle.boundary_fires(r_ref, wl.tau, False):
            assert abs(r_ref - wl.tau) <= REL * max(abs(r_ref), wl.tau), (t, gi, r_ref)
            stats["excused"] += 1
    after = to_np(eng.seg_state[gi * H:(gi + 1) * H])
    for h in range(H):
        s = gi * H + h
        n_units, win0 = int(before[h, 0]), int(before[h, 1])
        assert after[h, 4] == 0
        sizes = to_np(eng.unit_size[s, :n_units]).astype(np.int64)
        starts = to_np(eng.unit_start[s, :n_units]).astype(np.int64)
        got = to_np(eng.sel_units[s, :int(eng.n_sel_units[s])]).tolist()
        nsel = int(eng.n_sel[s])
        if fire:
            stats["fires"] += 1
            a = oracle.group_scores(q64[h * g:(h + 1) * g], to64(eng.reps[s, :n_units]), scale)
            np.testing.assert_allclose(to_np(eng.scores[s, :n_units]), a, rtol=1e-12, atol=1e-300)
            stats["excused"] += selection_matches(a, sizes, wl.budget, got)
            assert nsel == int(sizes[got].sum()) <= wl.budget
        idx = [rr for u in got for rr in range(int(starts[u]), int(starts[u] + sizes[u]))]
        rows = torch.as_tensor(idx, dtype=torch.long)
        kp = eng.k_pool[s].index_select(0, rows.to(eng.k_pool.device))
        vp = eng.v_pool[s].index_select(0, rows.to(eng.v_pool.device))
        if eng.zero_copy:
            assert to_np(eng.sel_rows[s, :nsel]).tolist() == idx
        elif eng.delta:
            _check_delta_slots(eng, s, nsel, idx)
        else:
            assert torch.equal(eng.k_buf[s, :nsel].cpu(), kp.cpu()) and torch.equal(eng.v_buf[s, :nsel].cpu(), vp.cpu())
        n_after, win1 = int(after[h, 0]), int(after[h, 1])
        if n_after > n_units:
            assert n_after == n_units + 1 and t - win0 == W
            u = n_units
            a0, n = int(eng.unit_start[s, u]) - P, int(eng.unit_size[s, u])
            assert a0 == win0 and win1 == a0 + n and 1 <= n <= smax
            assert a0 == 0 or fires[gi][a0] or int(eng.unit_size[s, u - 1]) == smax
            seg_keys = data.gen_keys[a0:a0 + n, s]
            assert torch.equal(eng.k_pool[s, P + a0:P + a0 + n].cpu(), seg_keys.cpu())
            assert torch.equal(eng.v_pool[s, P + a0:P + a0 + n].cpu(), data.gen_values[a0:a0 + n, s].cpu())
            assert np.array_equal(to64(eng.reps[s, u]), oracle.segment_mean(to64(seg_keys)))
            stats["evictions"] += 1
        else:
            assert win1 == win0 and t - win0 < W
        slots = [j % W for j in range(win1, t + 1)]
        assert torch.equal(eng.k_local[s, slots].cpu(), data.gen_keys[win1:t + 1, s].cpu())
        assert torch.equal(eng.v_local[s, slots].cpu(), data.gen_values[win1:t + 1, s].cpu())
        kk = np.concatenate([to64(kp), to64(eng.k_local[s, slots])])
        vv = np.concatenate([to64(vp), to64(eng.v_local[s, slots])])
        o, _ = oracle.attention(q64[h * g:(h + 1) * g], kk, vv, scale)
        err = np.abs(to64(eng.out[gi, h * g:(h + 1) * g]) - o).max()
        assert err <= 2e-3, (t, s, err)
    stats["checked"] += 1


@pytest.mark.parametrize("name", ["si-lo-16k", "li-lo-32k-b4"])
def test_decode_full_shape_boundary_segments(name):
    """Every decode step of the full workload with boundary-delimited segments
    (segment cap = the workload's segment length); sampled steps of two groups,
    plus the first evictions, are recomputed from the GPU's state."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    L = _L()
    wl = synth.get_workload(name)
    data = synth.make_slices(wl, DEV)
    # 16K steps could evict more segments than a slice can score; the run
    # accepts that and then checks that no segment was dropped
    cfg = config_from_workload(wl, mode=L.REF_ANCHOR, segments="boundary", allow_unit_overflow=True)
    eng = LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, pool_on_host=wl.pool_on_host, keep_scores=True,
                        out_dtype=torch.float32)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    torch.cuda.synchronize()
    H = wl.n_kv_heads
    groups = (0, wl.n_groups - 1)
    steps = _sample_steps(wl) | set(range(wl.window, wl.window + 12))
    last_fire = {gi: None for gi in groups}
    fires = {gi: np.zeros(wl.gen_len, dtype=bool) for gi in groups}
    stats = dict(fires=0, excused=0, checked=0, evictions=0)
    for t in range(wl.gen_len):
        q_ref = {gi: (None if last_fire[gi] is None else to64(data.queries[last_fire[gi], gi])) for gi in groups}
        check = t in steps
        before = {gi: to_np(eng.seg_state[gi * H:(gi + 1) * H]) for gi in groups} if check else None
        eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        fire = to_np(eng.fire)
        for gi in groups:
            fires[gi][t] = bool(fire[gi])
        if check:
            for gi in groups:
                _check_step_boundary(eng, data, wl, t, gi, q_ref[gi], before[gi], fires, stats)
        for gi in groups:
            if fire[gi]:
                last_fire[gi] = t
    st = to_np(eng.seg_state)
    assert (st[:, 4] == 0).all() and not eng.segment_overflow()
    assert stats["fires"] > 0 and stats["evictions"] > 0
    assert stats["checked"] >= 2 * len(steps)
    report(f"full-shape boundary-segment decode {name}", stats, bound=max(3, stats["fires"] // 100),
           of="boundary and selection near-ties")


@pytest.mark.parametrize("name", ["li-so-32k", "host-131k"])
def test_pipelined_prefill_full_shape(name):
    """The pipelined prefill (one layer's slices per chunk, pool writes on a
    second stream; copy engines for the host pool) at full size against the
    one-pass prefill: unit tables, centroids and permutations of every slice
    identical, and the pool rows of sampled slices identical."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    L = _L()
    wl = synth.get_workload(name)
    data = synth.make_slices(wl, DEV)
    cfg = config_from_workload(wl)
    dt = data.prompt_keys.dtype
    eng = LouisKVEngine(cfg, dt, DEV, pool_on_host=wl.pool_on_host)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    torch.cuda.synchronize()
    names = ("reps", "unit_start", "unit_size", "assign", "perm")
    ref = {n: getattr(eng, n).clone() for n in names}
    sample = (0, wl.n_slices // 2 + 3, wl.n_slices - 1)
    ref_pool = [(eng.k_pool[s, :wl.prompt_len].clone(), eng.v_pool[s, :wl.prompt_len].clone()) for s in sample]
    for n in names:
        getattr(eng, n).zero_()
    for s in sample:
        eng.k_pool[s].zero_()
        eng.v_pool[s].zero_()
    chunk = wl.n_kv_heads
    events = [torch.cuda.Event() for _ in range(-(-wl.n_slices // chunk) + 1)]
    for e in events:
        e.record()
    ws = torch.empty(L.cluster_prefill_pipelined_workspace_size(chunk, wl.prompt_len, wl.n_clusters, L.BF16,
                                                                wl.pool_on_host, True), dtype=torch.uint8, device=DEV)
    print(f"pipelined prefill {name}: {wl.n_slices} slices in chunks of {chunk}", flush=True)
    L.cluster_prefill_pipelined(data.prompt_keys, wl.n_clusters, wl.n_iters, data.init_idx, eng.reps,
                                eng.unit_start, eng.unit_size, eng.assign, eng.perm, data.prompt_values, eng.k_pool,
                                eng.v_pool, chunk, events, torch.cuda.Stream(), pool_on_host=wl.pool_on_host,
                                copy_engine=True, workspace=ws)
    torch.cuda.synchronize()
    for n in names:
        assert torch.equal(getattr(eng, n), ref[n]), n
    for (kr, vr), s in zip(ref_pool, sample):
        assert torch.equal(eng.k_pool[s, :wl.prompt_len].cpu(), kr.cpu())
        assert torch.equal(eng.v_pool[s, :wl.prompt_len].cpu(), vr.cpu())


ABLATIONS = {
    "stride-5": dict(trigger="stride", stride=5),
    "pages-16": dict(index="pages", page_len=16),
    "per-head": dict(selection="per_head"),
}


@pytest.mark.parametrize("variant", sorted(ABLATIONS))
def test_ablation_baselines_full_shape_sampled(variant):
    """The ablation baselines on li-so-32k at full size (all 256 slices per
    launch; 2048 page units per slice for the page index, 1024 per-head lists
    for per-head selection): at sampled steps of two groups, the trigger, the
    scores and selection of every list against the oracle, the row lists and
    the attention output recomputed from the GPU's state."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    L = _L()
    wl = synth.get_workload("li-so-32k")
    data = synth.make_slices(wl, DEV)
    kw = ABLATIONS[variant]
    cfg = config_from_workload(wl, **kw)
    eng = LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, keep_scores=True, out_dtype=torch.float32)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    torch.cuda.synchronize()
    H, g, P, C = wl.n_kv_heads, wl.group_size, wl.prompt_len, cfg.n_clusters
    per_head = cfg.selection == "per_head"
    NL = H * g if per_head else H
    scale = 1 / np.sqrt(128)
    if cfg.index == "pages":
        assert C == P // 16
        for s in (0, wl.n_slices - 1):
            r, a, z = oracle.page_units(to64(data.prompt_keys[s]), 16)
            assert np.array_equal(to64(eng.reps[s, :C]), r)
            assert to_np(eng.unit_start[s, :C]).tolist() == a.tolist()
            assert torch.equal(eng.k_pool[s, :P], data.prompt_keys[s])
    groups = (0, wl.n_groups - 1)
    steps = {0, 1, 2, 5, 10, 37, 64, 100, wl.gen_len - 1}
    checked = fired = 0
    for t in range(wl.gen_len):
        eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        fire = to_np(eng.fire)
        if cfg.trigger == "stride":
            assert (fire == (1 if t % cfg.stride == 0 else 0)).all(), t
        if t not in steps:
            continue
        torch.cuda.synchronize()
        _, _, n_local, local_start = L.window_info(t, wl.window, wl.seg_len)
        slots = [(local_start + i) % wl.window for i in range(n_local)]
        n_units = eng.n_units_before(t)
        for gi in groups:
            q64 = to64(data.queries[t, gi])
            for li in range(NL):
                s_list = gi * NL + li
                h = li // g if per_head else li
                s = gi * H + h
                heads = slice(li, li + 1) if per_head else slice(h * g, (h + 1) * g)
                sizes = to_np(eng.unit_size[s, :n_units]).astype(np.int64)
                starts = to_np(eng.unit_start[s, :n_units]).astype(np.int64)
                got = to_np(eng.sel_units[s_list, :int(eng.n_sel_units[s_list])]).tolist()
                if fire[gi]:
                    fired += 1
                    a = oracle.group_scores(q64[heads], to64(eng.reps[s, :n_units]), scale)
                    np.testing.assert_allclose(to_np(eng.scores[s_list, :n_units]), a, rtol=1e-12, atol=1e-300)
                    selection_matches(a, sizes, wl.budget, got)
                idx = [rr for u in got for rr in range(int(starts[u]), int(starts[u] + sizes[u]))]
                nsel = int(eng.n_sel[s_list])
                assert nsel == len(idx) <= wl.budget
                assert to_np(eng.sel_rows[s_list, :nsel]).tolist() == idx
                rows = torch.as_tensor(idx, dtype=torch.long, device=DEV)
                kk = np.concatenate([to64(eng.k_pool[s].index_select(0, rows)), to64(eng.k_local[s, slots])])
                vv = np.concatenate([to64(eng.v_pool[s].index_select(0, rows)), to64(eng.v_local[s, slots])])
                o, _ = oracle.attention(q64[heads], kk, vv, scale)
                err = np.abs(to64(eng.out[gi, heads]) - o).max()
                assert err <= 2e-3, (variant, t, s_list, err)
                checked += 1
    assert checked >= len(steps) * 2 * NL and fired > 0


@pytest.mark.parametrize("name,start,n_steps", [("li-so-32k", 0, 128), ("si-lo-16k", 0, 512),
                                                 ("si-lo-16k", 15872, 512), ("li-lo-32k-b4", 0, 256),
                                                 ("li-lo-32k-b4", 15872, 512), ("host-131k", 0, 128),
                                                 ("host-131k", 7680, 128)])
def test_layer_by_layer_full_shape(name, start, n_steps):
    """The layer-by-layer decode in the configuration the benchmark times
    (full-size slices; one launch a layer, the batch's sequences of a layer
    together) against the batched decode of the same inputs, which
    test_decode_full_shape_sampled checks against the oracle: the same fires,
    unit tables, scores, selections and row lists (or cache slots) bit for
    bit at every step of the window, and the same attention outputs up to
    summation order.  Windows: all of li-so-32k's 128 steps; the first steps
    and the last 512 (or 128) of the long generations, the window the
    benchmark times, reached by running both engines batched (li-lo-32k-b4:
    a 1024-slice batched retrieval against 32-slice launches; host-131k: the
    pool in pinned host memory behind the LRU cache of pool rows)."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    _L()
    wl = synth.get_workload(name)
    steps = start + n_steps
    assert steps <= wl.gen_len
    # layer-major order: a layer's sequences are consecutive groups
    groups = [(b, l) for l in range(wl.n_layers) for b in range(wl.batch)]
    data = synth.make_slices(wl, DEV, groups=groups, gen_len=steps)
    cfg = config_from_workload(wl, gen_len=steps)
    engs = [LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, keep_scores=True, out_dtype=torch.float32,
                          pool_on_host=wl.pool_on_host) for _ in range(2)]
    for e in engs:
        e.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    a, b = engs
    for t in range(start):
        for e in engs:
            e.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
    fires = 0
    for t in range(start, steps):
        a.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        b.step_layer_by_layer(data.queries[t], data.gen_keys[t], data.gen_values[t], groups_per_launch=wl.batch)
        torch.cuda.synchronize()
        assert torch.equal(a.fire, b.fire), t
        fires += int(a.fire.sum())
        for f in ("n_sel", "n_sel_units", "sel_units", "unit_start", "unit_size", "reps"):
            assert torch.equal(getattr(a, f), getattr(b, f)), (t, f)
        if bool(a.fire.any()):
            assert torch.equal(a.scores, b.scores), t
        # the selection as pool rows, or as the cache's slots and their rows
        n = a.n_sel.long()
        listed = a.sel_rows if a.sel_rows is not None else a.slot_list
        other = b.sel_rows if b.sel_rows is not None else b.slot_list
        mask = torch.arange(listed.shape[1], device=DEV)[None, :] < n[:, None]
        assert torch.equal(torch.where(mask, listed, 0), torch.where(mask, other, 0)), t
        if a.sel_rows is None:
            for f in ("buf_row", "slot_step"):
                assert torch.equal(getattr(a, f), getattr(b, f)), (t, f)
        err = (a.out - b.out).abs().max().item()
        assert err <= 1e-5 * max(1.0, a.out.abs().max().item()), (t, err)
        assert (a.lse - b.lse).abs().max().item() <= 1e-5, t
    assert fires > 0


def test_decode_graph_full_shape():
    """The benchmark's batched decode of li-so-32k: the whole 128-step loop
    captured as one HIP graph and replayed after a fresh prefill, twice;
    after each replay the state (unit tables, index vectors, the last step's
    fires, selection, row list and reference queries) and the last step's
    attention output equal those of the same loop run eagerly, bit for bit."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    L = _L()
    wl = synth.get_workload("li-so-32k")
    data = synth.make_slices(wl, DEV)
    cfg = config_from_workload(wl, mode=L.REF_ANCHOR)
    engs = [LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, out_dtype=torch.float32) for _ in range(2)]
    a, b = engs

    def loop(e):
        for t in range(wl.gen_len):
            e.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
    a.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    loop(a)
    # b: one eager pass on a side stream (allocations, warm-up), then the capture
    b.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        loop(b)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    b.t = 0
    with torch.cuda.graph(graph):
        loop(b)
    names = ("reps", "unit_start", "unit_size", "fire", "n_sel", "n_sel_units", "sel_units", "q_ref", "out", "lse")
    for rep in range(2):
        b.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
        graph.replay()
        torch.cuda.synchronize()
        for f in names:
            assert torch.equal(getattr(a, f), getattr(b, f)), (rep, f)
        n = a.n_sel.long()
        mask = torch.arange(a.sel_rows.shape[1], device=DEV)[None, :] < n[:, None]
        assert torch.equal(torch.where(mask, a.sel_rows, 0), torch.where(mask, b.sel_rows, 0)), rep
