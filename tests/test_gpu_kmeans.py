"""Prefill k-means on the GPU (through the C ABI) against the CPU oracle."""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import oracle  # noqa: E402
import synth  # noqa: E402
from parity_utils import (check_assignment, check_kmeans_trajectory, check_rows_rel,  # noqa: E402
                          gpu_kmeans_states, report, to64, to_np)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _L():
    from paper_2510_11292_amd import louiskv
    return louiskv


def _keys(n_slices, n, dtype, seed, centres=None, scale=1.0):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    m = centres or max(1, n // 32)
    c = torch.randn(n_slices, m, 128, generator=g, device=DEV)
    z = torch.randint(0, m, (n_slices, n), generator=g, device=DEV)
    k = torch.gather(c, 1, z[..., None].expand(-1, -1, 128)) + 0.3 * torch.randn(n_slices, n, 128, generator=g,
                                                                                   device=DEV)
    k[..., :4] *= 8 * scale
    return k.to(dtype).contiguous()


def _init(n_slices, n, c, seed):
    g = torch.Generator()
    g.manual_seed(seed)
    return torch.stack([torch.randperm(n, generator=g)[:c] for _ in range(n_slices)]).to(torch.int32).to(DEV)


def _operand(c64, bf16):
    return oracle.round_to_bf16(c64) if bf16 else c64


CASES = [
    # (dtype, n_slices, n_tokens, n_clusters)
    (torch.float32, 8, 4096, 64),        # the tiny-4k workload shape
    (torch.bfloat16, 4, 4096, 128),
    (torch.bfloat16, 3, 5003, 77),       # ragged: neither tokens nor clusters fill a tile
    (torch.float32, 2, 777, 33),
    (torch.bfloat16, 2, 64, 64),         # C = N
    (torch.bfloat16, 2, 300, 1),         # C = 1
]


@pytest.mark.parametrize("dtype,S,N,C", CASES)
def test_assign_step(dtype, S, N, C):
    L = _L()
    keys = _keys(S, N, dtype, seed=N + C)
    init = _init(S, N, C, seed=C)
    cents = keys.float()[torch.arange(S, device=DEV)[:, None], init.long()].contiguous()
    z = torch.empty(S, N, dtype=torch.int32, device=DEV)
    L.kmeans_assign(keys, C, cents, z)
    torch.cuda.synchronize()
    k64, c64, zg = to64(keys), to64(cents), to_np(z)
    excused = 0
    for s in range(S):
        excused += check_assignment(k64[s], _operand(c64[s], dtype == torch.bfloat16), zg[s])
    report(f"k-means assign step {dtype}", dict(excused=excused), bound=max(2, S * N // 10000),
           of="assignment near-ties")


@pytest.mark.parametrize("dtype,S,N,C", CASES)
def test_update_step(dtype, S, N, C):
    L = _L()
    keys = _keys(S, N, dtype, seed=7 * N + C)
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    # leave some clusters empty: draw from the first half only when C > 2
    hi = C if C <= 2 else (C + 1) // 2
    z = torch.randint(0, hi, (S, N), generator=g, device=DEV, dtype=torch.int32)
    prev = torch.randn(S, C, 128, device=DEV)
    out = torch.empty_like(prev)
    counts = torch.empty(S, C, dtype=torch.int32, device=DEV)
    L.kmeans_update(keys, C, z, prev, out, counts)
    torch.cuda.synchronize()
    k64, zg, p64, o = to64(keys), to_np(z), to64(prev), to_np(out)
    for s in range(S):
        ref, cnt = oracle.kmeans_update(k64[s], zg[s], p64[s])
        assert np.array_equal(to_np(counts)[s], cnt)
        assert np.array_equal(o[s].astype(np.float64), ref), "centroids are not bit-exact"


@pytest.mark.parametrize("dtype,S,N,C", CASES[:4])
def test_cluster_prefill_step_locked(dtype, S, N, C):
    """Each Lloyd iteration checked against the oracle from the GPU's own
    previous centroids, then the fused prefill call against that chain."""
    L = _L()
    bf16 = dtype == torch.bfloat16
    keys = _keys(S, N, dtype, seed=11 * N + C)
    vals = _keys(S, N, dtype, seed=13 * N + C)
    init = _init(S, N, C, seed=N)
    iters = 10
    k64 = to64(keys)
    cents = keys.float()[torch.arange(S, device=DEV)[:, None], init.long()].contiguous()
    z = torch.empty(S, N, dtype=torch.int32, device=DEV)
    for it in range(iters):
        L.kmeans_assign(keys, C, cents, z)
        torch.cuda.synchronize()
        c64, zg = to64(cents), to_np(z)
        for s in range(S):
            check_assignment(k64[s], _operand(c64[s], bf16), zg[s])
        new = torch.empty_like(cents)
        L.kmeans_update(keys, C, z, cents, new)
        torch.cuda.synchronize()
        for s in range(S):
            ref, _ = oracle.kmeans_update(k64[s], zg[s], c64[s])
            assert np.array_equal(to64(new)[s], ref)
        cents = new

    cap = C + 5
    reps = torch.full((S, cap, 128), 7.0, device=DEV)
    ustart = torch.full((S, cap), -1, dtype=torch.int32, device=DEV)
    usize = torch.full((S, cap), -1, dtype=torch.int32, device=DEV)
    assign = torch.empty(S, N, dtype=torch.int32, device=DEV)
    perm = torch.empty(S, N, dtype=torch.int32, device=DEV)
    kp = torch.zeros(S, N + 9, 128, dtype=dtype, device=DEV)
    vp = torch.zeros_like(kp)
    L.cluster_prefill(keys, C, iters, init, reps, ustart, usize, assign, perm, values=vals, k_pool=kp, v_pool=vp)
    torch.cuda.synchronize()
    assert torch.equal(assign, z)
    assert torch.equal(reps[:, :C], cents)
    assert torch.all(reps[:, C:] == 7.0) and torch.all(ustart[:, C:] == -1)
    zg = to_np(z)
    for s in range(S):
        counts = np.bincount(zg[s], minlength=C)
        offs = np.concatenate([[0], np.cumsum(counts)[:-1]])
        assert np.array_equal(to_np(usize)[s, :C], counts)
        assert np.array_equal(to_np(ustart)[s, :C], offs)
        pr = np.argsort(zg[s], kind="stable")
        assert np.array_equal(to_np(perm)[s], pr)
        assert torch.equal(kp[s, :N], keys[s][torch.from_numpy(pr).to(DEV).long()])
        assert torch.equal(vp[s, :N], vals[s][torch.from_numpy(pr).to(DEV).long()])
        assert torch.all(kp[s, N:] == 0)


def test_cluster_prefill_matches_oracle_end_to_end():
    """The tiny-4k workload (fp32, 8 KV heads, P=4096, C=64, 10 iterations) run
    straight through on both sides."""
    L = _L()
    wl = synth.get_workload("tiny-4k")
    data = synth.make_slices(wl, DEV)
    S, P, C = data.n_slices, wl.prompt_len, wl.n_clusters
    reps = torch.empty(S, C, 128, device=DEV)
    ustart = torch.empty(S, C, dtype=torch.int32, device=DEV)
    usize = torch.empty_like(ustart)
    assign = torch.empty(S, P, dtype=torch.int32, device=DEV)
    perm = torch.empty_like(assign)
    L.cluster_prefill(data.prompt_keys, C, wl.n_iters, data.init_idx, reps, ustart, usize, assign, perm)
    torch.cuda.synchronize()
    k64 = to64(data.prompt_keys)
    states = gpu_kmeans_states(L, data.prompt_keys, data.init_idx, C)
    same = excused = 0
    for s in range(S):
        res = oracle.kmeans(k64[s], to_np(data.init_idx)[s], wl.n_iters, bf16_operand=False)
        if np.array_equal(res.z, to_np(assign)[s]):
            same += 1
            assert np.array_equal(to64(reps)[s], res.centroids)
            assert np.array_equal(to_np(perm)[s], res.perm)
        else:
            # the run left the oracle's: every iteration must be an exact
            # argmin and exact means up to excused near-ties
            excused += check_kmeans_trajectory(k64[s], to_np(data.init_idx)[s], wl.n_iters, False,
                                               lambda it: tuple(x[s] for x in states(it)))
    # the prefill call with n_iters = 10 is the same run as the states' tenth
    assert np.array_equal(states(wl.n_iters)[0], to_np(assign).astype(np.int64))
    report("k-means tiny-4k end to end", dict(slices_equal=same, excused=excused),
           bound=max(2, S * P * wl.n_iters // 10000), of="assignment near-ties")


def test_empty_cluster_keeps_centroid():
    L = _L()
    S, N, C = 2, 512, 8
    keys = _keys(S, N, torch.bfloat16, seed=5, centres=4)
    init = _init(S, N, C, seed=9)
    init[:, 5] = init[:, 2]          # duplicate start: cluster 5 loses every tie to 2
    reps = torch.empty(S, C, 128, device=DEV)
    ustart = torch.empty(S, C, dtype=torch.int32, device=DEV)
    usize = torch.empty_like(ustart)
    assign = torch.empty(S, N, dtype=torch.int32, device=DEV)
    perm = torch.empty_like(assign)
    L.cluster_prefill(keys, C, 1, init, reps, ustart, usize, assign, perm)
    torch.cuda.synchronize()
    for s in range(S):
        assert int(usize[s, 5]) == 0
        assert torch.equal(reps[s, 5], keys[s, int(init[s, 5])].float())
        res = oracle.kmeans(to64(keys)[s], to_np(init)[s], 1, bf16_operand=True)
        assert np.array_equal(to_np(assign)[s], res.z)
        assert np.array_equal(to64(reps)[s], res.centroids)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_pack_pool_writes_rows_in_perm_order(dtype):
    """louiskv_pack_pool: pool row r of a slice holds token perm[r] (entries
    clamped into [0, n_tokens)); rows past n_tokens are left alone."""
    L = _L()
    S, N, extra = 3, 300, 20
    g = torch.Generator(device=DEV).manual_seed(31)
    keys = torch.randn(S, N, 128, generator=g, device=DEV).to(dtype)
    values = torch.randn(S, N, 128, generator=g, device=DEV).to(dtype)
    perm = torch.stack([torch.randperm(N, generator=torch.Generator().manual_seed(s)) for s in range(S)])
    perm = perm.to(torch.int32).to(DEV)
    perm[1, 5] = -3
    perm[2, 7] = N + 7
    kp = torch.full((S, N + extra, 128), 5, dtype=dtype, device=DEV)
    vp = torch.full_like(kp, 6)
    L.pack_pool(keys, values, perm, kp, vp)
    torch.cuda.synchronize()
    idx = perm.clamp(0, N - 1).long()
    for s in range(S):
        assert torch.equal(kp[s, :N], keys[s, idx[s]])
        assert torch.equal(vp[s, :N], values[s, idx[s]])
        assert torch.all(kp[s, N:] == 5) and torch.all(vp[s, N:] == 6)


PIPELINE_CASES = [
    # (dtype, n_slices, n_tokens, n_clusters, slices_per_chunk, pool_on_host, copy_engine)
    (torch.float32, 8, 4096, 64, 3, False, True),     # ragged last chunk (3, 3, 2)
    (torch.bfloat16, 10, 5003, 77, 4, True, True),    # host pool through the copy engines
    (torch.bfloat16, 10, 5003, 77, 4, True, False),   # host pool written by the pack kernel
    (torch.bfloat16, 4, 4096, 128, 1, False, True),   # one slice per chunk
    (torch.bfloat16, 4, 4096, 128, 8, True, True),    # one chunk holds every slice
]


@pytest.mark.parametrize("dtype,S,N,C,chunk,host,copy_engine", PIPELINE_CASES)
def test_cluster_prefill_pipelined_equals_one_pass(dtype, S, N, C, chunk, host, copy_engine):
    """louiskv_cluster_prefill_pipelined gives the outputs and pool contents of
    louiskv_cluster_prefill bit for bit (the chunks are independent slices),
    leaves the pool rows past the prompt alone, and orders work enqueued on the
    calling stream after the whole pool write."""
    L = _L()
    keys = _keys(S, N, dtype, 700 + S)
    g = torch.Generator(device=DEV).manual_seed(701)
    values = torch.randn(S, N, 128, generator=g, device=DEV).to(dtype)
    init = _init(S, N, C, 702)
    cap, extra, iters = C + 5, 37, 4

    def outputs():
        return dict(reps=torch.zeros(S, cap, 128, device=DEV),
                    ustart=torch.zeros(S, cap, dtype=torch.int32, device=DEV),
                    usize=torch.zeros(S, cap, dtype=torch.int32, device=DEV),
                    assign=torch.zeros(S, N, dtype=torch.int32, device=DEV),
                    perm=torch.zeros(S, N, dtype=torch.int32, device=DEV))

    def pools():
        if host:
            kp = torch.full((S, N + extra, 128), 5, dtype=dtype).pin_memory()
            vp = torch.full((S, N + extra, 128), 6, dtype=dtype).pin_memory()
        else:
            kp = torch.full((S, N + extra, 128), 5, dtype=dtype, device=DEV)
            vp = torch.full((S, N + extra, 128), 6, dtype=dtype, device=DEV)
        return kp, vp

    ref = outputs()
    kr, vr = pools()
    L.cluster_prefill(keys, C, iters, init, ref["reps"], ref["ustart"], ref["usize"], ref["assign"], ref["perm"],
                      values=values, k_pool=kr, v_pool=vr, pool_on_host=host)
    torch.cuda.synchronize()

    out = outputs()
    kp, vp = pools()
    n_chunks = -(-S // min(chunk, S))
    events = [torch.cuda.Event() for _ in range(n_chunks + 1)]
    for e in events:
        e.record()
    copy_stream = torch.cuda.Stream()
    print(f"pipelined prefill dtype={dtype} S={S} N={N} C={C} chunk={chunk} host={host} "
          f"copy_engine={copy_engine}", flush=True)
    L.cluster_prefill_pipelined(keys, C, iters, init, out["reps"], out["ustart"], out["usize"], out["assign"],
                                out["perm"], values, kp, vp, chunk, events, copy_stream, pool_on_host=host,
                                copy_engine=copy_engine)
    # read the pools back with work on the calling stream, without a host sync
    k_seen = kp.to(DEV, non_blocking=True) if host else kp.clone()
    v_seen = vp.to(DEV, non_blocking=True) if host else vp.clone()
    torch.cuda.synchronize()
    for name in ref:
        assert torch.equal(out[name], ref[name]), name
    assert torch.equal(k_seen.cpu(), kr.cpu())
    assert torch.equal(v_seen.cpu(), vr.cpu())
    assert torch.all(k_seen[:, N:].cpu() == 5) and torch.all(v_seen[:, N:].cpu() == 6)
    # the one-pass prefill is checked against the oracle elsewhere; here one
    # slice again, directly: pool row r holds token perm[r]
    idx = ref["perm"][S - 1].long()
    assert torch.equal(k_seen[S - 1, :N], keys[S - 1, idx])
    assert torch.equal(v_seen[S - 1, :N], values[S - 1, idx])


@pytest.mark.parametrize("host", [True, False])
def test_cluster_prefill_pipelined_matches_oracle(host):
    """The pipelined prefill (chunks of one layer's slices, each chunk's pool
    write on a copy stream beside the next chunk's clustering) against the
    oracle directly: for every slice of two groups of a reduced host-131k
    workload, the oracle's k-means and cluster-by-cluster packing
    (prefill_state_from_kmeans) equal the GPU's centroids, unit table and pool,
    with any divergent run step-locked iteration by iteration through the
    pipelined call itself."""
    from parity_utils import check_prefill_against_state, oracle_prefill_state
    L = _L()
    wl = synth.get_workload("host-131k").replace(prompt_len=2048, n_clusters=64, name="host-131k")
    data = synth.make_slices(wl, DEV, groups=[(0, 0), (0, 1)], gen_len=1)
    S, N, C, H = data.n_slices, wl.prompt_len, wl.n_clusters, wl.n_kv_heads
    dt = data.prompt_keys.dtype

    def run(iters):
        reps = torch.zeros(S, C, 128, device=DEV)
        ustart = torch.zeros(S, C, dtype=torch.int32, device=DEV)
        usize = torch.zeros_like(ustart)
        assign = torch.zeros(S, N, dtype=torch.int32, device=DEV)
        perm = torch.zeros_like(assign)
        if host:
            kp = torch.zeros(S, N, 128, dtype=dt).pin_memory()
            vp = torch.zeros(S, N, 128, dtype=dt).pin_memory()
        else:
            kp = torch.zeros(S, N, 128, dtype=dt, device=DEV)
            vp = torch.zeros(S, N, 128, dtype=dt, device=DEV)
        events = [torch.cuda.Event() for _ in range(-(-S // H) + 1)]
        for e in events:
            e.record()
        L.cluster_prefill_pipelined(data.prompt_keys, C, iters, data.init_idx, reps, ustart, usize, assign, perm,
                                    data.prompt_values, kp, vp, H, events, torch.cuda.Stream(), pool_on_host=host,
                                    copy_engine=True)
        torch.cuda.synchronize()
        return reps, ustart, usize, assign, kp, vp

    reps, ustart, usize, assign, kp, vp = run(wl.n_iters)
    cache = {}

    def states(it):
        if it not in cache:
            r = run(it)
            cache[it] = (to_np(r[3]).astype(np.int64), to64(r[0]))
        return cache[it]
    k_excused = adopted = 0
    for gi in range(2):
        sl = slice(gi * H, (gi + 1) * H)
        st, ex, ad = oracle_prefill_state(to64(data.prompt_keys[sl]), to64(data.prompt_values[sl]),
                                          to_np(data.init_idx[sl]), wl.n_iters, True, to_np(assign[sl]),
                                          to64(reps[sl]), states, list(range(sl.start, sl.stop)))
        check_prefill_against_state(reps[sl], ustart[sl], usize[sl], kp[sl], vp[sl], st, N)
        k_excused += ex
        adopted += ad
    report(f"pipelined prefill vs oracle host={host}", dict(excused=k_excused, adopted=adopted),
           bound=max(2, S * N * wl.n_iters // 10000), of="assignment near-ties")
