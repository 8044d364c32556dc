"""Decode-stage calls on the GPU (through the C ABI) against the CPU oracle."""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(__file__))
import oracle  # noqa: E402
import synth  # noqa: E402
from parity_utils import (REL, check_prefill_against_state, check_rows_rel, gpu_kmeans_states,  # noqa: E402
                          oracle_prefill_state, report, selection_matches, to64, to_np)

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _L():
    from paper_2510_11292_amd import louiskv
    return louiskv


def _gen(seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return g


# ------------------------------------------------------------------ boundary

@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("mode", [0, 1])
def test_boundary_check(dtype, mode):
    L = _L()
    G, H = 64, 32
    g = _gen(1)
    base = torch.randn(G, H, 128, generator=g, device=DEV)
    q_ref0 = base.to(dtype)
    # a spread of similarities around tau: mix in noise of growing size
    noise = torch.randn(G, H, 128, generator=g, device=DEV) * torch.linspace(0, 1.5, G, device=DEV)[:, None, None]
    q = (base + noise).to(dtype)
    q[3] = q_ref0[3]                 # identical: r = 1
    q[4] = -q_ref0[4]                # opposite: r = -1
    q[5] = 0                         # zero query: r = 0
    for tau in (0.9, 0.5, 1.5, -1.5):
        q_ref = q_ref0.clone()
        fire = torch.empty(G, dtype=torch.uint8, device=DEV)
        r = torch.empty(G, dtype=torch.float64, device=DEV)
        L.boundary_check(q, q_ref, tau, mode, False, fire, r)
        torch.cuda.synchronize()
        q64, ref64 = to64(q), to64(q_ref0)
        for i in range(G):
            rr = oracle.query_similarity(q64[i], ref64[i])
            assert abs(float(r[i]) - rr) <= 1e-12, (i, float(r[i]), rr)
            want = oracle.boundary_fires(rr, tau, False)
            if bool(fire[i]) != want:
                assert abs(rr - tau) <= REL * max(abs(rr), abs(tau))
            expect_ref = q[i] if (mode == 0 or bool(fire[i])) else q_ref0[i]
            assert torch.equal(q_ref[i], expect_ref)
    # first step: everything fires, r is NaN, the reference is taken
    q_ref = torch.zeros_like(q)
    fire = torch.zeros(G, dtype=torch.uint8, device=DEV)
    r = torch.zeros(G, dtype=torch.float64, device=DEV)
    L.boundary_check(q, q_ref, 0.9, mode, True, fire, r)
    torch.cuda.synchronize()
    assert torch.all(fire == 1) and torch.all(torch.isnan(r)) and torch.equal(q_ref, q)


# ------------------------------------------------------------------ decode store

@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_segment_output_window_and_eviction(dtype):
    """Drive 300 steps of the store and compare the ring, the new units and the
    pool with the oracle's bookkeeping."""
    L = _L()
    S, W, seg, C, P, T = 6, 64, 16, 10, 40, 300
    g = _gen(2)
    keys = torch.randn(T, S, 128, generator=g, device=DEV).mul(3).to(dtype)
    vals = torch.randn(T, S, 128, generator=g, device=DEV).to(dtype)
    n_ev_total = (T - W + seg - 1) // seg
    cap = C + n_ev_total
    reps = torch.zeros(S, cap, 128, device=DEV)
    ustart = torch.zeros(S, cap, dtype=torch.int32, device=DEV)
    usize = torch.zeros_like(ustart)
    kl = torch.zeros(S, W, 128, dtype=dtype, device=DEV)
    vl = torch.zeros_like(kl)
    kp = torch.zeros(S, P + T, 128, dtype=dtype, device=DEV)
    vp = torch.zeros_like(kp)
    for t in range(T):
        L.segment_output(keys[t], vals[t], kl, vl, t, seg, reps, ustart, usize, C, kp, vp, P)
    torch.cuda.synchronize()
    ev, n_ev, n_local, start = L.window_info(T - 1, W, seg)
    assert n_ev == n_ev_total
    k64 = to64(keys)
    for e in range(n_ev):
        u = C + e
        assert torch.all(ustart[:, u] == P + e * seg) and torch.all(usize[:, u] == seg)
        for s in range(S):
            ref = oracle.segment_mean(k64[e * seg:(e + 1) * seg, s])
            assert np.array_equal(to64(reps[s, u]), ref)
        assert torch.equal(kp[:, P + e * seg:P + (e + 1) * seg], keys[e * seg:(e + 1) * seg].transpose(0, 1))
        assert torch.equal(vp[:, P + e * seg:P + (e + 1) * seg], vals[e * seg:(e + 1) * seg].transpose(0, 1))
    live = list(range(n_ev * seg, T))
    assert len(live) == n_local
    for i, tok in enumerate(live):
        slot = (start + i) % W
        assert slot == tok % W
        assert torch.equal(kl[:, slot], keys[tok]) and torch.equal(vl[:, slot], vals[tok])


# ------------------------------------------------------------------ retrieve

RETRIEVE_CASES = [
    # (dtype, n_groups, n_kv, g, n_units, budget, max unit size)
    (torch.bfloat16, 4, 8, 4, 1024, 2048, 64),
    (torch.float32, 2, 8, 4, 68, 512, 120),
    (torch.bfloat16, 3, 2, 8, 3000, 4096, 20),
    (torch.bfloat16, 2, 4, 1, 17, 100, 30),
    (torch.float32, 1, 8, 4, 50, 0, 10),          # zero budget: nothing selected
    (torch.bfloat16, 1, 8, 4, 64, 10 ** 6, 40),   # budget covers everything
    (torch.bfloat16, 2, 8, 4, 4348, 4096, 40),    # 131K-prompt unit count: 8192-entry sort
    (torch.float32, 2, 2, 3, 200, 300, 15),       # group size that is not a power of two
    (torch.bfloat16, 1, 8, 4, 1, 64, 40),         # a single unit
    (torch.bfloat16, 16, 8, 4, 300, 512, 20),     # 128 slices: the selection block computes its own logits
]


@pytest.mark.parametrize("dtype,G,H,g,U,B,maxsz", RETRIEVE_CASES)
def test_retrieve(dtype, G, H, g, U, B, maxsz):
    L = _L()
    S = G * H
    gen = _gen(U + B)
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).mul(2).to(dtype)
    reps = torch.randn(S, U + 3, 128, generator=gen, device=DEV)
    sizes = torch.randint(0, maxsz + 1, (S, U + 3), generator=gen, device=DEV, dtype=torch.int32)
    sizes[:, 0] = maxsz                                   # a big unit at a fixed place
    starts = torch.zeros_like(sizes)
    starts[:, 1:] = torch.cumsum(sizes, 1)[:, :-1].to(torch.int32)
    rows = int(sizes.sum(1).max()) + 5
    kp = torch.randn(S, rows, 128, generator=gen, device=DEV).to(dtype)
    vp = torch.randn(S, rows, 128, generator=gen, device=DEV).to(dtype)
    fire = (torch.arange(G, device=DEV) % 3 != 1).to(torch.uint8)
    bufrows = max(min(B, rows), 1)
    kb = torch.full((S, bufrows, 128), 9, dtype=dtype, device=DEV)
    vb = torch.full_like(kb, 9)
    sel = torch.full((S, U + 3), -1, dtype=torch.int32, device=DEV)
    nsu = torch.full((S,), -1, dtype=torch.int32, device=DEV)
    nsel = torch.full((S,), -1, dtype=torch.int32, device=DEV)
    scores = torch.zeros(S, U + 3, dtype=torch.float64, device=DEV)
    Bcall = min(B, bufrows) if B > 0 else 0
    L.retrieve(q, H, reps, starts, sizes, U, kp, vp, Bcall, sel, nsu, nsel, kb, vb, fire=fire, scores_out=scores)
    torch.cuda.synchronize()
    q64, r64, sz, st = to64(q), to64(reps), to_np(sizes), to_np(starts)
    for s in range(S):
        grp, h = divmod(s, H)
        if not fire[grp]:
            assert int(nsel[s]) == -1 and int(nsu[s]) == -1 and torch.all(kb[s] == 9)
            continue
        a = oracle.group_scores(q64[grp, h * g:(h + 1) * g], r64[s, :U], 1 / np.sqrt(128))
        np.testing.assert_allclose(to_np(scores[s, :U]), a, rtol=1e-12, atol=1e-300)
        got = to_np(sel[s, :int(nsu[s])]).tolist()
        selection_matches(a, sz[s, :U], Bcall, got)
        tot = int(sz[s, got].sum()) if got else 0
        assert int(nsel[s]) == tot <= max(Bcall, 0)
        ref_rows = oracle.gather_units(to64(kp[s]), st[s], sz[s], got)
        assert np.array_equal(to64(kb[s, :tot]), ref_rows)
        assert np.array_equal(to64(vb[s, :tot]), oracle.gather_units(to64(vp[s]), st[s], sz[s], got))


# ------------------------------------------------------------------ attention

ATTN_CASES = [
    # (dtype, out dtype, n_groups, n_kv, g, buf_rows, window, n_local, local_start)
    (torch.bfloat16, torch.float32, 4, 8, 4, 2048, 128, 128, 0),
    (torch.float32, torch.float32, 1, 8, 4, 512, 128, 97, 32),
    (torch.bfloat16, torch.bfloat16, 2, 8, 4, 300, 64, 10, 60),
    (torch.bfloat16, torch.float32, 2, 4, 8, 100, 32, 0, 0),
    (torch.float32, torch.float32, 3, 2, 1, 77, 16, 16, 5),
    (torch.bfloat16, torch.float32, 1, 8, 2, 4096, 128, 1, 127),
    # 256 slices and more: one block per slice writes the output directly
    (torch.bfloat16, torch.float32, 32, 8, 4, 2048, 128, 128, 17),
    (torch.bfloat16, torch.bfloat16, 32, 8, 4, 700, 128, 50, 100),
    (torch.float32, torch.float32, 64, 4, 4, 300, 64, 64, 3),
    (torch.bfloat16, torch.float32, 64, 4, 8, 500, 32, 32, 31),
    (torch.bfloat16, torch.float32, 40, 8, 4, 1000, 128, 0, 0),
    # one and two query heads a group in bf16 (matrix-core scores), split-KV and one block a slice
    (torch.bfloat16, torch.float32, 2, 8, 1, 600, 64, 64, 7),
    (torch.bfloat16, torch.bfloat16, 32, 8, 1, 300, 64, 20, 50),
    (torch.bfloat16, torch.float32, 32, 8, 2, 1000, 128, 128, 0),
]


@pytest.mark.parametrize("dtype,odt,G,H,g,BR,W,nl,ls", ATTN_CASES)
def test_sparse_decode_attn(dtype, odt, G, H, g, BR, W, nl, ls):
    L = _L()
    S = G * H
    gen = _gen(BR + W + nl)
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).mul(1.5).to(dtype)
    kb = torch.randn(S, BR, 128, generator=gen, device=DEV).mul(2).to(dtype)
    vb = torch.randn(S, BR, 128, generator=gen, device=DEV).to(dtype)
    kl = torch.randn(S, W, 128, generator=gen, device=DEV).mul(2).to(dtype)
    vl = torch.randn(S, W, 128, generator=gen, device=DEV).to(dtype)
    nsel = torch.randint(0, BR + 1, (S,), generator=gen, device=DEV, dtype=torch.int32)
    nsel[0] = BR
    nsel[-1] = 0
    out = torch.empty(G, H * g, 128, dtype=odt, device=DEV)
    lse = torch.empty(G, H * g, dtype=torch.float32, device=DEV)
    L.sparse_decode_attn(q, H, kb, vb, nsel, kl, vl, ls, nl, out, lse)
    torch.cuda.synchronize()
    q64 = to64(q)
    for s in range(S):
        grp, h = divmod(s, H)
        n = int(nsel[s])
        slots = [(ls + i) % W for i in range(nl)]
        kk = np.concatenate([to64(kb[s, :n]), to64(kl[s, slots])]) if slots else to64(kb[s, :n])
        vv = np.concatenate([to64(vb[s, :n]), to64(vl[s, slots])]) if slots else to64(vb[s, :n])
        o, l = oracle.attention(q64[grp, h * g:(h + 1) * g], kk, vv, 1 / np.sqrt(128))
        got = to64(out[grp, h * g:(h + 1) * g])
        if kk.shape[0] == 0:
            assert np.all(got == 0) and np.all(np.isneginf(to_np(lse[grp, h * g:(h + 1) * g])))
            continue
        if odt == torch.bfloat16:
            ref = oracle.round_to_bf16(o)
            ulp = np.abs(ref) * 2.0 ** -7 + 1e-30
            assert np.all(np.abs(got - ref) <= ulp + 1e-6)
        elif dtype == torch.float32:
            check_rows_rel(got, o, 1e-5, "fp32 attention")
        else:
            assert np.abs(got - o).max() <= 2e-3
        np.testing.assert_allclose(to64(lse[grp, h * g:(h + 1) * g]), l, rtol=1e-5, atol=1e-5)


@pytest.mark.parametrize("dtype,G,H,g,U,B,maxsz", RETRIEVE_CASES)
def test_retrieve_rows(dtype, G, H, g, U, B, maxsz):
    """Zero-copy retrieval: the same selection as a list of pool rows."""
    L = _L()
    S = G * H
    gen = _gen(U + B + 1)
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).mul(2).to(dtype)
    reps = torch.randn(S, U + 3, 128, generator=gen, device=DEV)
    sizes = torch.randint(0, maxsz + 1, (S, U + 3), generator=gen, device=DEV, dtype=torch.int32)
    starts = torch.zeros_like(sizes)
    starts[:, 1:] = torch.cumsum(sizes, 1)[:, :-1].to(torch.int32)
    rows_cap = int(sizes.sum(1).max()) + 5
    fire = (torch.arange(G, device=DEV) % 3 != 1).to(torch.uint8)
    Bcall = min(B, rows_cap) if B > 0 else 0
    sel_rows = torch.full((S, max(Bcall, 1)), -7, dtype=torch.int32, device=DEV)
    sel = torch.full((S, U + 3), -1, dtype=torch.int32, device=DEV)
    nsu = torch.full((S,), -1, dtype=torch.int32, device=DEV)
    nsel = torch.full((S,), -1, dtype=torch.int32, device=DEV)
    L.retrieve_rows(q, H, reps, starts, sizes, U, Bcall, sel, nsu, nsel, sel_rows, fire=fire)
    torch.cuda.synchronize()
    q64, r64, sz, st = to64(q), to64(reps), to_np(sizes), to_np(starts)
    for s in range(S):
        grp, h = divmod(s, H)
        if not fire[grp]:
            assert int(nsel[s]) == -1 and torch.all(sel_rows[s] == -7)
            continue
        a = oracle.group_scores(q64[grp, h * g:(h + 1) * g], r64[s, :U], 1 / np.sqrt(128))
        got = to_np(sel[s, :int(nsu[s])]).tolist()
        selection_matches(a, sz[s, :U], Bcall, got)
        idx = [r for u in got for r in range(int(st[s, u]), int(st[s, u] + sz[s, u]))]
        assert int(nsel[s]) == len(idx) <= max(Bcall, 0)
        assert to_np(sel_rows[s, :len(idx)]).tolist() == idx


@pytest.mark.parametrize("n_small", [200, 100])
def test_retrieve_rows_after_the_top_keys(n_small):
    """The selection's first search takes the 128 highest keys: with the
    best-scored n_small units one token each and the rest 100 (the budget
    holds about 25 units of the mean size, so that search runs) the 128 best
    all fit, so the full search decides (n_small = 200: 200 small units and
    18 large ones), or the prefix stops past them (n_small = 100: the budget
    stop falls inside the 128 at the 119th unit); either way the selection is
    the oracle's."""
    L = _L()
    G, H, g, U, B = 1, 8, 4, 1024, 2000
    S = G * H
    gen = _gen(U + B + n_small)
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).mul(2).to(torch.bfloat16)
    reps = torch.randn(S, U, 128, generator=gen, device=DEV)
    q64, r64 = to64(q), to64(reps)
    sizes = torch.full((S, U), 100, dtype=torch.int32)
    scores = []
    for s in range(S):
        a = oracle.group_scores(q64[0, s * g:(s + 1) * g], r64[s], 1 / np.sqrt(128))
        scores.append(a)
        sizes[s, torch.from_numpy(np.argsort(-a, kind="stable")[:n_small].copy())] = 1
    sizes = sizes.to(DEV)
    starts = torch.zeros_like(sizes)
    starts[:, 1:] = torch.cumsum(sizes, 1)[:, :-1].to(torch.int32)
    sel_rows = torch.full((S, B), -7, dtype=torch.int32, device=DEV)
    sel = torch.full((S, U), -1, dtype=torch.int32, device=DEV)
    nsu = torch.full((S,), -1, dtype=torch.int32, device=DEV)
    nsel = torch.full((S,), -1, dtype=torch.int32, device=DEV)
    fire = torch.ones(G, dtype=torch.uint8, device=DEV)
    L.retrieve_rows(q, H, reps, starts, sizes, U, B, sel, nsu, nsel, sel_rows, fire=fire)
    torch.cuda.synchronize()
    sz, st = to_np(sizes), to_np(starts)
    for s in range(S):
        got = to_np(sel[s, :int(nsu[s])]).tolist()
        selection_matches(scores[s], sz[s], B, got)
        assert len(got) == (218 if n_small == 200 else 119), (s, len(got))
        idx = [r for u in got for r in range(int(st[s, u]), int(st[s, u] + sz[s, u]))]
        assert int(nsel[s]) == len(idx) <= B
        assert to_np(sel_rows[s, :len(idx)]).tolist() == idx


@pytest.mark.parametrize("U,B", [(700, 2048), (1500, 2048), (8192, 8192)])
def test_retrieve_rows_same_for_every_block_size(U, B):
    """With more slices than compute units the retrieval runs 256-thread
    blocks (two to a compute unit), with fewer 512-thread ones, and the
    softmax sums keep one summation order: a call over more slices than the
    device has compute units and the same slices in calls of 32 (logits from
    their own kernel) give the same scores, selections and row lists bit for
    bit, and the oracle's selection (700 units: exponentials in registers;
    1500: in the workspace; 8192, the most units a slice may have, with a
    budget of about 270 of them: the radix search and the block sort)."""
    L = _L()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    H, g = 8, 4
    G = cus // H + 4
    S = G * H
    assert S > cus
    gen = _gen(U + S)
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).mul(2).to(torch.bfloat16)
    reps = torch.randn(S, U, 128, generator=gen, device=DEV)
    sizes = torch.randint(1, 60, (S, U), generator=gen, device=DEV, dtype=torch.int32)
    starts = torch.zeros_like(sizes)
    starts[:, 1:] = torch.cumsum(sizes, 1)[:, :-1].to(torch.int32)
    fire = (torch.arange(G, device=DEV) % 5 != 2).to(torch.uint8)

    def run(lo, hi):
        n = (hi - lo) * H
        out = (torch.full((n, B), -7, dtype=torch.int32, device=DEV),
               torch.full((n, U), -1, dtype=torch.int32, device=DEV),
               torch.full((n,), -1, dtype=torch.int32, device=DEV),
               torch.full((n,), -1, dtype=torch.int32, device=DEV),
               torch.full((n, U), -1.0, dtype=torch.float64, device=DEV))
        sl = slice(lo * H, hi * H)
        L.retrieve_rows(q[lo:hi], H, reps[sl], starts[sl], sizes[sl], U, B, out[1], out[2], out[3], out[0],
                        fire=fire[lo:hi], scores_out=out[4])
        return out

    big = run(0, G)
    parts = [run(lo, min(G, lo + 4)) for lo in range(0, G, 4)]
    torch.cuda.synchronize()
    for k, name in enumerate(("sel_rows", "sel_units", "n_sel_units", "n_sel", "scores")):
        assert torch.equal(big[k], torch.cat([p[k] for p in parts])), name
    q64, r64, sz = to64(q), to64(reps), to_np(sizes)
    for s in range(0, S, 7):
        grp, h = divmod(s, H)
        if not fire[grp]:
            assert int(big[3][s]) == -1
            continue
        a = oracle.group_scores(q64[grp, h * g:(h + 1) * g], r64[s], 1 / np.sqrt(128))
        np.testing.assert_allclose(to_np(big[4][s]), a, rtol=1e-12, atol=1e-300)
        selection_matches(a, sz[s], B, to_np(big[1][s, :int(big[2][s])]).tolist())


ROWS_ATTN_CASES = [
    # (dtype, out dtype, n_groups, n_kv, g, budget, pool rows, window, n_local, local_start)
    (torch.bfloat16, torch.float32, 32, 8, 4, 2048, 6000, 128, 128, 17),   # one block per slice
    (torch.bfloat16, torch.float32, 2, 8, 4, 700, 3000, 64, 40, 60),       # split-KV
    (torch.bfloat16, torch.bfloat16, 1, 8, 8, 300, 1000, 32, 32, 5),
    (torch.float32, torch.float32, 1, 8, 4, 512, 2000, 128, 97, 32),
    (torch.float32, torch.float32, 64, 4, 4, 300, 900, 64, 64, 3),
    (torch.bfloat16, torch.float32, 32, 8, 2, 1024, 3000, 128, 128, 0),
    (torch.bfloat16, torch.bfloat16, 2, 8, 1, 500, 2000, 64, 30, 10),
]


@pytest.mark.parametrize("dtype,odt,G,H,g,B,PR,W,nl,ls", ROWS_ATTN_CASES)
def test_sparse_decode_attn_rows(dtype, odt, G, H, g, B, PR, W, nl, ls):
    """Attention over listed pool rows (random rows, ragged counts, empty
    slices) then the local window, against the oracle on the same rows."""
    L = _L()
    S = G * H
    gen = _gen(B + PR + nl)
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).mul(1.5).to(dtype)
    kp = torch.randn(S, PR, 128, generator=gen, device=DEV).mul(2).to(dtype)
    vp = torch.randn(S, PR, 128, generator=gen, device=DEV).to(dtype)
    kl = torch.randn(S, W, 128, generator=gen, device=DEV).mul(2).to(dtype)
    vl = torch.randn(S, W, 128, generator=gen, device=DEV).to(dtype)
    rows = torch.stack([torch.randperm(PR, generator=torch.Generator().manual_seed(s))[:B] for s in range(S)])
    rows = rows.to(torch.int32).to(DEV)
    nsel = torch.randint(0, B + 1, (S,), generator=gen, device=DEV, dtype=torch.int32)
    nsel[0] = B
    nsel[-1] = 0
    out = torch.empty(G, H * g, 128, dtype=odt, device=DEV)
    lse = torch.empty(G, H * g, dtype=torch.float32, device=DEV)
    L.sparse_decode_attn_rows(q, H, kp, vp, rows, nsel, kl, vl, ls, nl, out, lse)
    torch.cuda.synchronize()
    q64 = to64(q)
    for s in range(S):
        grp, h = divmod(s, H)
        n = int(nsel[s])
        idx = rows[s, :n].long()
        slots = [(ls + i) % W for i in range(nl)]
        kk = np.concatenate([to64(kp[s, idx]), to64(kl[s, slots])])
        vv = np.concatenate([to64(vp[s, idx]), to64(vl[s, slots])])
        got = to64(out[grp, h * g:(h + 1) * g])
        if kk.shape[0] == 0:
            assert np.all(got == 0)
            continue
        o, l = oracle.attention(q64[grp, h * g:(h + 1) * g], kk, vv, 1 / np.sqrt(128))
        if odt == torch.bfloat16:
            ref = oracle.round_to_bf16(o)
            assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -7 + 1e-6)
        elif dtype == torch.float32:
            check_rows_rel(got, o, 1e-5, "fp32 attention over listed rows")
        else:
            assert np.abs(got - o).max() <= 2e-3
        np.testing.assert_allclose(to64(lse[grp, h * g:(h + 1) * g]), l, rtol=1e-5, atol=1e-5)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_split_kv_merge_repeats_on_one_workspace(dtype):
    """Split-KV attention keeps the chunk partials in the workspace between its
    two launches: repeated eager calls and graph replays on one workspace all
    write the output of a call with a fresh workspace (the output is poisoned
    with NaN before each call)."""
    L = _L()
    G, H, g, B, PR, W, nl, ls = 2, 8, 4, 700, 3000, 64, 40, 60
    S = G * H
    gen = _gen(4242)
    q = torch.randn(G, H * g, 128, generator=gen, device=DEV).to(dtype)
    kp = torch.randn(S, PR, 128, generator=gen, device=DEV).mul(2).to(dtype)
    vp = torch.randn(S, PR, 128, generator=gen, device=DEV).to(dtype)
    kl = torch.randn(S, W, 128, generator=gen, device=DEV).to(dtype)
    vl = torch.randn(S, W, 128, generator=gen, device=DEV).to(dtype)
    rows = torch.randint(0, PR, (S, B), generator=gen, device=DEV, dtype=torch.int32)
    nsel = torch.randint(0, B + 1, (S,), generator=gen, device=DEV, dtype=torch.int32)
    nsel[3] = 0
    wsb = L.sparse_decode_attn_rows_workspace_size(S, g, B, W)
    assert wsb > 0, "the case must split the rows over several blocks"
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    out = torch.empty(G, H * g, 128, dtype=torch.float32, device=DEV)
    lse = torch.empty(G, H * g, dtype=torch.float32, device=DEV)

    def call():
        L.sparse_decode_attn_rows(q, H, kp, vp, rows, nsel, kl, vl, ls, nl, out, lse, workspace=ws)

    results = []
    for _ in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        call()
        torch.cuda.synchronize()
        results.append((out.clone(), lse.clone()))
    # a fresh workspace gives the same result as the reused one
    ref_out = torch.empty_like(out)
    ref_lse = torch.empty_like(lse)
    L.sparse_decode_attn_rows(q, H, kp, vp, rows, nsel, kl, vl, ls, nl, ref_out, ref_lse)
    torch.cuda.synchronize()
    assert not torch.isnan(ref_out).any()
    for o, l in results:
        assert torch.equal(o, ref_out) and torch.equal(l, ref_lse)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for _ in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)


def test_sparse_decode_attn_rows_clamps_list_entries():
    """Entries outside [0, pool_rows) are clamped into the pool by the kernel."""
    L = _L()
    S, H, g, B, PR, W = 8, 8, 4, 64, 200, 32
    gen = _gen(99)
    q = torch.randn(1, H * g, 128, generator=gen, device=DEV).to(torch.bfloat16)
    kp = torch.randn(S, PR, 128, generator=gen, device=DEV).to(torch.bfloat16)
    vp = torch.randn(S, PR, 128, generator=gen, device=DEV).to(torch.bfloat16)
    kl = torch.zeros(S, W, 128, dtype=torch.bfloat16, device=DEV)
    rows = torch.randint(0, PR, (S, B), generator=gen, device=DEV, dtype=torch.int32)
    rows[:, 3] = -5
    rows[:, 9] = PR + 10
    nsel = torch.full((S,), B, dtype=torch.int32, device=DEV)
    out = torch.empty(1, H * g, 128, dtype=torch.float32, device=DEV)
    L.sparse_decode_attn_rows(q, H, kp, vp, rows, nsel, kl, kl, 0, 0, out)
    torch.cuda.synchronize()
    clamped = rows.clamp(0, PR - 1).long()
    q64 = to64(q)
    for s in range(S):
        o, _ = oracle.attention(q64[0, s * g:(s + 1) * g], to64(kp[s, clamped[s]]), to64(vp[s, clamped[s]]),
                                1 / np.sqrt(128))
        assert np.abs(to64(out[0, s * g:(s + 1) * g]) - o).max() <= 2e-3


# ------------------------------------------------------------------ whole decode loop

def _lru_model(buf_row, slot_step, rows, step):
    """The LRU policy of the cached KV_critical, written out: slots whose row
    is selected again keep it; the new rows, in selection order, go to the
    other slots with the smallest (last step, slot), taken in slot order."""
    buf_row, slot_step = buf_row.copy(), slot_step.copy()
    pos = {int(r): i for i, r in enumerate(buf_row) if r >= 0}
    new = []
    for r in rows:
        if r in pos:
            slot_step[pos[r]] = step
        else:
            new.append(r)
    cand = sorted((i for i in range(len(buf_row)) if slot_step[i] < step), key=lambda i: (slot_step[i], i))
    for r, i in zip(new, sorted(cand[:len(new)])):
        buf_row[i], slot_step[i] = r, step
    return buf_row, slot_step, [i for i in range(len(buf_row)) if slot_step[i] == step], len(new)


def _check_delta_buffers(eng, gi, H, before=None, t=None):
    """KV_critical kept as a cache of pool rows: the listed slots hold exactly
    the selected rows (as copies of their pool rows), every slot at most once;
    with an LRU cache, slots, steps and the fetch count follow the policy
    from the state before the step."""
    for h in range(H):
        s = gi * H + h
        n = int(eng.n_sel[s])
        slots = to_np(eng.slot_list[s, :n]).astype(np.int64)
        assert len(set(slots.tolist())) == n
        held = to_np(eng.buf_row[s])[slots].astype(np.int64)
        units = to_np(eng.sel_units[s, :int(eng.n_sel_units[s])])
        want = sorted(r for u in units for r in range(int(eng.unit_start[s, u]),
                                                       int(eng.unit_start[s, u]) + int(eng.unit_size[s, u])))
        assert sorted(held.tolist()) == want
        if eng.cached:
            rows = [r for u in units for r in range(int(eng.unit_start[s, u]),
                                                    int(eng.unit_start[s, u]) + int(eng.unit_size[s, u]))]
            b_row, b_step, lst, k = _lru_model(before[0][s], before[1][s], rows, t)
            assert np.array_equal(to_np(eng.buf_row[s]), b_row), (t, s)
            assert np.array_equal(to_np(eng.slot_step[s]), b_step), (t, s)
            assert slots.tolist() == lst and int(eng.n_fetched[s]) == k, (t, s)
        else:
            assert (to_np(eng.buf_row[s]) >= 0).sum() == n
        idx = torch.as_tensor(held, dtype=torch.long)
        assert torch.equal(eng.k_buf[s, torch.as_tensor(slots)].cpu(), eng.k_pool[s].cpu()[idx])
        assert torch.equal(eng.v_buf[s, torch.as_tensor(slots)].cpu(), eng.v_pool[s].cpu()[idx])


def _run_loop(wl, n_groups, steps, mode, pool_on_host=False, zero_copy=None, segments="fixed", delta=None,
              layer_by_layer=False, cache_rows=None, **ablation):
    """Prefill on the GPU, then `steps` decode steps on the GPU and in the
    oracle (started from the GPU's prefill state), step-locked.  With
    layer_by_layer each step runs group by group (one launch sequence per
    layer) through views of the engine's tensors."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    data = synth.make_slices(wl, DEV, groups=[(0, l) for l in range(n_groups)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=n_groups, mode=mode, gen_len=steps, segments=segments, **ablation)
    odt = torch.float32
    eng = LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, pool_on_host=pool_on_host, keep_scores=True,
                        out_dtype=odt, zero_copy=zero_copy, delta=delta, cache_rows=cache_rows)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    torch.cuda.synchronize()
    H, g = wl.n_kv_heads, wl.group_size
    C = cfg.n_clusters     # prompt units: clusters, or pages with index="pages"
    per_head = cfg.selection == "per_head"
    NL = H * g if per_head else H      # selection lists per group
    # the oracle's own prefill (k-means, then the pool packed cluster by
    # cluster, or the page index); the GPU's unit table and pool must equal it
    decs = []
    k_excused = adopted = 0
    bf16 = data.prompt_keys.dtype == torch.bfloat16
    states = gpu_kmeans_states(_L(), data.prompt_keys, data.init_idx, C) if cfg.index == "clusters" else None
    for gi in range(n_groups):
        sl = slice(gi * H, (gi + 1) * H)
        k64, v64 = to64(data.prompt_keys[sl]), to64(data.prompt_values[sl])
        if cfg.index == "pages":
            st = oracle.prefill_state_from_pages(k64, v64, cfg.page_len)
        else:
            st, ex, ad = oracle_prefill_state(k64, v64, to_np(data.init_idx[sl]), wl.n_iters, bf16,
                                              to_np(eng.assign[sl]), to64(eng.reps[sl, :C]), states,
                                              list(range(sl.start, sl.stop)))
            k_excused += ex
            adopted += ad
        check_prefill_against_state(eng.reps[sl], eng.unit_start[sl], eng.unit_size[sl], eng.k_pool[sl],
                                    eng.v_pool[sl], st, wl.prompt_len)
        decs.append(oracle.GroupDecoder(st, wl.n_q_heads, wl.budget, wl.window, wl.seg_len, wl.tau,
                                        "prev" if mode == 0 else "anchor", segments=segments,
                                        trigger=cfg.trigger, stride=cfg.stride, selection=cfg.selection))
    assert k_excused <= max(2, n_groups * H * wl.prompt_len * wl.n_iters // 10000), k_excused
    stats = dict(fires=0, excused=0, evictions=0, sizes=set(), fetched=0, selected=0)
    if layer_by_layer and pool_on_host:
        _require_interior_host_mapping(eng.k_pool, wl.n_kv_heads)
    for t in range(steps):
        before = (to_np(eng.buf_row), to_np(eng.slot_step)) if eng.cached else None
        if layer_by_layer:
            eng.step_layer_by_layer(data.queries[t], data.gen_keys[t], data.gen_values[t])
        else:
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        torch.cuda.synchronize()
        fire, r = to_np(eng.fire), to_np(eng.r)
        for gi, dec in enumerate(decs):
            q64 = to64(data.queries[t, gi])
            if cfg.trigger == "stride":
                want_fire = oracle.stride_fires(t + 1, cfg.stride)
                assert bool(fire[gi]) == want_fire, (t, gi)
            else:
                want_fire = t == 0 or oracle.boundary_fires(oracle.query_similarity(q64, dec.q_ref), wl.tau, False)
            if bool(fire[gi]) != want_fire:
                rr = oracle.query_similarity(q64, dec.q_ref)
                assert abs(rr - wl.tau) <= REL * max(abs(rr), wl.tau), (t, gi, rr)
                stats["excused"] += 1
            override = None
            if fire[gi]:
                stats["fires"] += 1
                override = []
                for li in range(NL):
                    s = gi * NL + li
                    h = li // g if per_head else li
                    got = to_np(eng.sel_units[s, :int(eng.n_sel_units[s])]).tolist()
                    heads = slice(li, li + 1) if per_head else slice(h * g, (h + 1) * g)
                    a = oracle.group_scores(q64[heads], np.asarray(dec.reps[h]), 1 / np.sqrt(128))
                    np.testing.assert_allclose(to_np(eng.scores[s, :len(a)]), a, rtol=1e-12, atol=1e-300)
                    stats["excused"] += selection_matches(a, dec.unit_size[h], wl.budget, got)
                    override.append(got)
            rec = dec.step(q64, to64(data.gen_keys[t, gi * H:(gi + 1) * H]),
                           to64(data.gen_values[t, gi * H:(gi + 1) * H]), fire_override=bool(fire[gi]),
                           select_override=override)
            assert to_np(eng.n_sel[gi * NL:(gi + 1) * NL]).tolist() == rec.n_sel
            if eng.delta and fire[gi]:
                _check_delta_buffers(eng, gi, H, before, t)
                stats["fetched"] += int(eng.n_fetched[gi * H:(gi + 1) * H].sum())
                stats["selected"] += int(eng.n_sel[gi * H:(gi + 1) * H].sum())
            got = to64(eng.out[gi])
            if data.prompt_keys.dtype == torch.float32:
                check_rows_rel(got, rec.out, 1e-5, f"step {t} attention")
            else:
                assert np.abs(got - rec.out).max() <= 2e-3, (t, np.abs(got - rec.out).max())
            if rec.evicted_unit is not None:
                u = rec.evicted_unit
                stats["evictions"] += 1
                stats["sizes"].add(dec.unit_size[0][u])
                for h in range(H):
                    assert np.array_equal(to64(eng.reps[gi * H + h, u]), dec.reps[h][u])
                    assert int(eng.unit_start[gi * H + h, u]) == dec.unit_start[h][u]
                    assert int(eng.unit_size[gi * H + h, u]) == dec.unit_size[h][u]
            if segments == "boundary":
                stt = to_np(eng.seg_state[gi * H:(gi + 1) * H])
                assert (stt[:, 0] == dec.n_units()).all(), (t, stt[:, 0], dec.n_units())
                assert (stt[:, 1] == dec.local[0][0][0]).all(), (t, stt[:, 1], dec.local[0][0][0])
                assert (stt[:, 4] == 0).all()
    stats["kmeans_excused"] = k_excused
    stats["kmeans_adopted"] = adopted
    report(f"decode loop {wl.name} groups={n_groups} steps={steps}", stats,
           bound=max(3, stats["fires"] // 100), of="boundary and selection near-ties")
    return stats


def test_decode_loop_tiny_workload_anchor():
    """The tiny-4k workload end to end (fp32, 256 decode steps, anchor mode)."""
    wl = synth.get_workload("tiny-4k")
    st = _run_loop(wl, 1, wl.gen_len, mode=1)
    assert st["fires"] > 20


def test_decode_loop_tiny_workload_prev():
    """PREV mode, with the dense (gathered) KV_critical."""
    wl = synth.get_workload("tiny-4k")
    st = _run_loop(wl, 1, wl.gen_len, mode=0, zero_copy=False)
    assert st["fires"] >= 1


@pytest.mark.parametrize("zero_copy", [True, False])
def test_decode_loop_bf16_with_evictions(zero_copy):
    """A bf16 reduction of the long-output shape: 2 groups, P=2048, C=64,
    300 steps so several segments are evicted and later retrieved; with
    KV_critical as a row list (zero-copy) and as gathered copies."""
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, name="si-lo-16k")
    st = _run_loop(wl, 2, 300, mode=1, zero_copy=zero_copy)
    assert st["fires"] > 40


@pytest.mark.parametrize("delta", [True, False])
def test_decode_loop_host_pool(delta):
    """The same reduction with the KV pool in pinned host memory: prefill packs
    into it, evictions append to it and retrieval copies from it over the
    host link, either every selected row (gather) or only the rows the
    previous selection did not hold (delta, the engine's default there)."""
    wl = synth.get_workload("host-131k").replace(prompt_len=2048, n_clusters=64, budget=512, name="host-131k")
    st = _run_loop(wl, 1, 200, mode=1, pool_on_host=True, delta=delta, cache_rows=wl.budget if delta else None)
    assert st["fires"] > 20
    if delta:
        assert 0 < st["fetched"] < st["selected"]


@pytest.mark.parametrize("segments,prompt,budget,cache", [("fixed", 2048, 512, 4 * 512),
                                                           ("boundary", 2048, 512, 4 * 512),
                                                           ("fixed", 4096, 1024, 36 * 1024)])
def test_decode_loop_host_pool_lru_cache(segments, prompt, budget, cache):
    """KV_critical as an LRU cache of pool rows over a pinned host pool (four
    budgets; and 36 K slots, more than the pool's rows, which takes the plan's
    longest register runs): oracle parity of every step, and slots, steps and
    fetch counts equal to the LRU policy written out in Python; the cache
    fetches fewer rows than the one-budget buffer on the same inputs."""
    wl = synth.get_workload("host-131k").replace(prompt_len=prompt, n_clusters=64, budget=budget, window=64,
                                                 seg_len=16, name="host-131k")
    st = _run_loop(wl, 1, 200, mode=1, pool_on_host=True, segments=segments, cache_rows=cache)
    assert st["fires"] > 20 and 0 < st["fetched"] < st["selected"]
    base = _run_loop(wl, 1, 200, mode=1, pool_on_host=True, segments=segments, cache_rows=wl.budget)
    print(f"fetched rows: LRU cache {st['fetched']}, one budget {base['fetched']}", flush=True)
    assert st["fetched"] < base["fetched"]


@pytest.mark.parametrize("cache", [10240, 16896])
def test_decode_loop_host_pool_lru_cache_evicting(cache):
    """The LRU cache smaller than the pool, at the sizes that take the plan's
    16- and 32-slot register runs (20 K-token prompt indexed by 16-token
    pages, 2048-token budget): slots, steps and fetch counts follow the
    policy at every step while rows are evicted, with oracle parity."""
    wl = synth.get_workload("host-131k").replace(prompt_len=20480, n_clusters=1280, budget=2048, name="host-131k")
    st = _run_loop(wl, 1, 120, mode=1, pool_on_host=True, cache_rows=cache, index="pages", page_len=16)
    assert st["fires"] > 15 and 0 < st["fetched"] < st["selected"]


def test_decode_loop_delta_device_pool():
    """Delta transfers over a pool in device memory (bf16 reduction with
    evictions, two groups)."""
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, name="si-lo-16k")
    st = _run_loop(wl, 2, 300, mode=1, zero_copy=False, delta=True)
    assert st["fires"] > 40 and 0 < st["fetched"] < st["selected"]


@pytest.mark.parametrize("zero_copy", [True, False])
def test_decode_loop_boundary_segments(zero_copy):
    """Boundary-delimited segments (anchor mode fires every few steps, so the
    segments are short and of varied length) on the bf16 long-output
    reduction: units, windows and attention step-locked with the oracle."""
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, window=64,
                                                 seg_len=16, name="si-lo-16k")
    st = _run_loop(wl, 2, 300, mode=1, zero_copy=zero_copy, segments="boundary")
    assert st["fires"] > 40 and st["evictions"] > 40 and len(st["sizes"]) >= 2


def test_decode_loop_boundary_segments_prev_fp32():
    """The tiny fp32 workload with boundary segments in previous-query mode:
    boundaries only at query jumps, so most segments end at the length cap."""
    wl = synth.get_workload("tiny-4k").replace(window=64, seg_len=12)
    st = _run_loop(wl, 1, wl.gen_len, mode=0, segments="boundary")
    assert st["evictions"] > 10 and 12 in st["sizes"]


def test_decode_loop_boundary_segments_host_pool():
    """Boundary segments with the pool in pinned host memory (gathered
    KV_critical over the host link)."""
    wl = synth.get_workload("host-131k").replace(prompt_len=2048, n_clusters=64, budget=512, window=64, seg_len=16,
                                                 name="host-131k")
    st = _run_loop(wl, 1, 200, mode=1, pool_on_host=True, segments="boundary")
    assert st["fires"] > 20 and st["evictions"] > 10


def _require_interior_host_mapping(pool, rows_per_view):
    """Group views of a pinned host pool hand the library interior pointers;
    check (a runtime query, no kernel) that the device address the runtime
    reports for one is the pool's device address plus the same offset."""
    import ctypes

    class Attr(ctypes.Structure):
        _fields_ = [("type", ctypes.c_int), ("device", ctypes.c_int), ("devicePointer", ctypes.c_void_p),
                    ("hostPointer", ctypes.c_void_p), ("isManaged", ctypes.c_int),
                    ("allocationFlags", ctypes.c_uint)]

    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipPointerGetAttributes.argtypes = [ctypes.POINTER(Attr), ctypes.c_void_p]
    a, b = Attr(), Attr()
    off = pool[rows_per_view].data_ptr() - pool.data_ptr()
    assert hip.hipPointerGetAttributes(ctypes.byref(a), ctypes.c_void_p(pool.data_ptr())) == 0
    assert hip.hipPointerGetAttributes(ctypes.byref(b), ctypes.c_void_p(pool.data_ptr() + off)) == 0
    assert a.devicePointer and b.devicePointer
    assert b.devicePointer - a.devicePointer == off, (hex(a.devicePointer), hex(b.devicePointer), off)


def test_decode_loop_layer_by_layer():
    """Each decode step run group by group (as a model runs its layers) over
    views of one engine's tensors: the same oracle parity as the batched step,
    with evictions (bf16 long-output reduction, three groups, zero-copy)."""
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, name="si-lo-16k")
    st = _run_loop(wl, 3, 300, mode=1, layer_by_layer=True)
    assert st["fires"] > 60 and st["evictions"] > 0


def test_decode_loop_layer_by_layer_boundary_delta():
    """Group-by-group steps with boundary segments and delta transfers over a
    device pool (per-slice segment state and buffer rows seen through views)."""
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, window=64,
                                                 seg_len=16, name="si-lo-16k")
    st = _run_loop(wl, 2, 200, mode=1, zero_copy=False, delta=True, segments="boundary", layer_by_layer=True)
    assert st["fires"] > 30 and st["evictions"] > 10 and 0 < st["fetched"] < st["selected"]


def test_decode_loop_layer_by_layer_device_lru_cache():
    """Group-by-group steps over a device pool with KV_critical as an LRU
    cache of three budgets (each view runs the four-launch cached decode
    step): oracle parity and the LRU policy at every step."""
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, name="si-lo-16k")
    st = _run_loop(wl, 2, 200, mode=1, zero_copy=False, delta=True, layer_by_layer=True, cache_rows=3 * 512)
    assert st["fires"] > 30 and 0 < st["fetched"] < st["selected"]


def test_decode_loop_layer_by_layer_host_pool():
    """Group-by-group steps with the pool in pinned host memory (delta
    transfers): each group's calls take pointers into the middle of the pool."""
    wl = synth.get_workload("host-131k").replace(prompt_len=2048, n_clusters=64, budget=512, name="host-131k")
    st = _run_loop(wl, 2, 160, mode=1, pool_on_host=True, layer_by_layer=True)
    assert st["fires"] > 20 and 0 < st["fetched"] < st["selected"]


def test_layer_by_layer_equals_batched_at_full_layer_count():
    """32 groups (one sequence of a 32-layer model; a reduced prompt so the
    run is short): steps run group by group give the batched steps' fires,
    selections and unit tables exactly, and the same attention outputs up to
    the summation order (one launch per layer splits each slice's rows over
    several blocks, the batched launch does not)."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=512, n_clusters=16, budget=128, name="si-lo-16k")
    G, steps = 32, 170
    data = synth.make_slices(wl, DEV, groups=[(0, l) for l in range(G)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=G, gen_len=steps)
    # batched; one group per launch; four groups per launch (a layer of a batch of four)
    engs = [LouisKVEngine(cfg, torch.bfloat16, DEV, out_dtype=torch.float32) for _ in range(3)]
    for e in engs:
        e.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    fires = 0
    for t in range(steps):
        engs[0].step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        engs[1].step_layer_by_layer(data.queries[t], data.gen_keys[t], data.gen_values[t])
        engs[2].step_layer_by_layer(data.queries[t], data.gen_keys[t], data.gen_values[t], groups_per_launch=4)
        torch.cuda.synchronize()
        a = engs[0]
        fires += int(a.fire.sum())
        for b in engs[1:]:
            assert torch.equal(a.fire, b.fire), t
            for name in ("n_sel", "n_sel_units", "sel_units", "unit_start", "unit_size", "reps"):
                assert torch.equal(getattr(a, name), getattr(b, name)), (t, name)
            for i in range(a.n_sel.shape[0]):
                n = int(a.n_sel[i])
                assert torch.equal(a.sel_rows[i, :n], b.sel_rows[i, :n]), (t, i)
            err = (a.out - b.out).abs().max().item()
            assert err <= 1e-5 * max(1.0, a.out.abs().max().item()), (t, err)
            assert (a.lse - b.lse).abs().max().item() <= 1e-5, t
    assert fires > G * steps // 8


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("host", [False, True])
def test_page_prefill_matches_oracle(dtype, host):
    """louiskv_page_prefill: page means bit-exact against the oracle's page
    index (ragged last page), unit tables exact, pool rows in token order and
    rows past the prompt untouched."""
    L = _L()
    S, N, P, extra = 3, 1000, 16, 9
    g = torch.Generator(device=DEV).manual_seed(51)
    keys = (torch.randn(S, N, 128, generator=g, device=DEV) * 2).to(dtype)
    values = torch.randn(S, N, 128, generator=g, device=DEV).to(dtype)
    n_pages = -(-N // P)
    cap = n_pages + 4
    reps = torch.full((S, cap, 128), 7.0, device=DEV)
    us = torch.full((S, cap), -5, dtype=torch.int32, device=DEV)
    uz = torch.full((S, cap), -5, dtype=torch.int32, device=DEV)
    if host:
        kp = torch.full((S, N + extra, 128), 3, dtype=dtype).pin_memory()
        vp = torch.full((S, N + extra, 128), 4, dtype=dtype).pin_memory()
    else:
        kp = torch.full((S, N + extra, 128), 3, dtype=dtype, device=DEV)
        vp = torch.full((S, N + extra, 128), 4, dtype=dtype, device=DEV)
    L.page_prefill(keys, P, reps, us, uz, values=values, k_pool=kp, v_pool=vp, pool_on_host=host)
    torch.cuda.synchronize()
    for sl in range(S):
        r, a, z = oracle.page_units(to64(keys[sl]), P)
        assert np.array_equal(to64(reps[sl, :n_pages]), r)
        assert to_np(us[sl, :n_pages]).tolist() == a.tolist() and to_np(uz[sl, :n_pages]).tolist() == z.tolist()
    assert torch.all(reps[:, n_pages:] == 7.0) and torch.all(us[:, n_pages:] == -5)
    assert torch.equal(kp[:, :N].cpu(), keys.cpu()) and torch.equal(vp[:, :N].cpu(), values.cpu())
    assert torch.all(kp[:, N:].cpu() == 3) and torch.all(vp[:, N:].cpu() == 4)


def test_fire_every():
    """louiskv_fire_every sets every group's flag on multiples of the stride."""
    L = _L()
    fire = torch.full((37,), 9, dtype=torch.uint8, device=DEV)
    for step in range(12):
        L.fire_every(fire, step, 5)
        torch.cuda.synchronize()
        assert torch.all(fire == (1 if step % 5 == 0 else 0)), step


def _ablation_wl():
    return synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, name="si-lo-16k")


def test_decode_loop_stride_trigger():
    """Fixed-stride trigger (a retrieval every 5 steps) through the decode
    loop, step-locked with the oracle (bf16 reduction with evictions)."""
    st = _run_loop(_ablation_wl(), 2, 200, mode=1, trigger="stride", stride=5)
    assert st["fires"] == 2 * 40 and st["evictions"] > 0


def test_decode_loop_page_index():
    """Page-level index (16-token pages of the prompt in place of clusters)
    through the decode loop with the gathered KV_critical."""
    st = _run_loop(_ablation_wl(), 2, 200, mode=1, zero_copy=False, index="pages", page_len=16)
    assert st["fires"] > 30


def test_decode_loop_per_head_selection():
    """Per-head selection (each of the four query heads of a KV head ranks
    and selects alone) step-locked with the oracle, bf16 (matrix-core
    attention over one head per list)."""
    st = _run_loop(_ablation_wl(), 2, 200, mode=1, selection="per_head")
    assert st["fires"] > 30 and st["evictions"] > 0


def test_decode_loop_per_head_selection_fp32():
    """Per-head selection on the tiny fp32 workload (vector attention path)."""
    wl = synth.get_workload("tiny-4k")
    st = _run_loop(wl, 1, 160, mode=1, selection="per_head")
    assert st["fires"] > 10


@pytest.mark.parametrize("case", ["bf16-zero-copy", "fp32-gather", "bf16-host-delta"])
def test_fused_prologue_equals_separate_calls(case):
    """louiskv_decode_prologue (boundary test and store in one launch, before
    the retrieval) leaves every output and every piece of state exactly as
    louiskv_boundary_check and louiskv_segment_output called around it do,
    through evictions."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    if case == "fp32-gather":
        wl = synth.get_workload("tiny-4k").replace(window=64, seg_len=16)
        kw = dict(zero_copy=False)
        host = False
    elif case == "bf16-host-delta":
        wl = synth.get_workload("host-131k").replace(prompt_len=2048, n_clusters=64, budget=512, name="host-131k")
        kw = {}
        host = True
    else:
        wl = _ablation_wl()
        kw = {}
        host = False
    steps = 200
    G = 2 if wl.n_layers > 1 else 1
    data = synth.make_slices(wl, DEV, groups=[(0, l) for l in range(G)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=G, gen_len=steps)
    dt = data.prompt_keys.dtype
    a = LouisKVEngine(cfg, dt, DEV, pool_on_host=host, out_dtype=torch.float32, fuse_prologue=True, **kw)
    b = LouisKVEngine(cfg, dt, DEV, pool_on_host=host, out_dtype=torch.float32, fuse_prologue=False, **kw)
    for e in (a, b):
        e.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    names = ["fire", "r", "q_ref", "k_local", "v_local", "reps", "unit_start", "unit_size", "n_sel", "out", "lse"]
    names += ["sel_rows"] if a.zero_copy else ["k_buf", "v_buf"]
    fires = 0
    for t in range(steps):
        for e in (a, b):
            e.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        torch.cuda.synchronize()
        fires += int(a.fire.sum())
        for n in names:
            x, y = getattr(a, n), getattr(b, n)
            assert torch.equal(x, y) or (n == "r" and t == 0), (t, n)
    # pool rows written so far: the prompt and the evicted segments (the rest
    # of both pools is uninitialised memory)
    L = _L()
    rows = cfg.prompt_len + L.window_info(steps - 1, cfg.window, cfg.seg_len)[1] * cfg.seg_len
    assert rows > cfg.prompt_len
    assert torch.equal(a.k_pool[:, :rows].cpu(), b.k_pool[:, :rows].cpu())
    assert torch.equal(a.v_pool[:, :rows].cpu(), b.v_pool[:, :rows].cpu())
    assert fires > 10


@pytest.mark.parametrize("case", ["zero-copy", "boundary-segments", "host-delta", "host-lru-cache"])
def test_decode_graph_replays_match_eager(case):
    """The decode loop captured once as a HIP graph (as the benchmark runs it)
    and replayed three times, each after a fresh eager prefill and with eager
    work and synchronisations between the replays, gives at every step the
    outputs and selection sizes of the eager loop."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    host = case.startswith("host")
    if host:
        wl = synth.get_workload("host-131k").replace(prompt_len=2048, n_clusters=64, budget=512, name="host-131k")
    else:
        wl = _ablation_wl()
    seg = dict(segments="boundary", window=64, seg_len=16) if case == "boundary-segments" else {}
    steps, G = 160, 2
    data = synth.make_slices(wl, DEV, groups=[(0, l) for l in range(G)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=G, gen_len=steps, **seg)
    eng = LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, pool_on_host=host, out_dtype=torch.float32,
                        cache_rows=3 * wl.budget if case == "host-lru-cache" else wl.budget)
    hist = torch.zeros(steps, *eng.out.shape, device=DEV)
    hist_n = torch.zeros(steps, *eng.n_sel.shape, dtype=torch.int32, device=DEV)

    def loop():
        for t in range(steps):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
            hist[t].copy_(eng.out)
            hist_n[t].copy_(eng.n_sel)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    loop()
    torch.cuda.synchronize()
    ref, ref_n = hist.clone(), hist_n.clone()
    assert int((ref_n > 0).sum()) > 0
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    eng.t = 0
    with torch.cuda.graph(graph):
        loop()
    for rep in range(3):
        hist.zero_()
        hist_n.zero_()
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
        torch.cuda.synchronize()
        print(f"graph replay {rep} ({case})", flush=True)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(hist, ref), (case, rep)
        assert torch.equal(hist_n, ref_n), (case, rep)
    del graph


def test_host_pool_flag_rejects_device_memory():
    """pool_on_host=1 with device tensors is refused on the host, before any launch."""
    L = _L()
    from paper_2510_11292_amd.louiskv import LouisKVError
    S, U, B = 8, 16, 64
    q = torch.zeros(1, 32, 128, dtype=torch.bfloat16, device=DEV)
    reps = torch.zeros(S, U, 128, device=DEV)
    sizes = torch.full((S, U), 4, dtype=torch.int32, device=DEV)
    starts = (torch.arange(U, dtype=torch.int32, device=DEV) * 4).repeat(S, 1)
    kp = torch.zeros(S, 4 * U, 128, dtype=torch.bfloat16, device=DEV)
    kb = torch.full((S, B, 128), 7, dtype=torch.bfloat16, device=DEV)
    sel = torch.zeros(S, U, dtype=torch.int32, device=DEV)
    nsu = torch.full((S,), -5, dtype=torch.int32, device=DEV)
    nsel = torch.full((S,), -5, dtype=torch.int32, device=DEV)
    with pytest.raises(LouisKVError) as ei:
        L.retrieve(q, 8, reps, starts, sizes, U, kp, kp, B, sel, nsu, nsel, kb, kb.clone(), pool_on_host=True)
    assert ei.value.status == 4
    torch.cuda.synchronize()
    assert torch.all(nsel == -5) and torch.all(kb == 7)


@pytest.mark.parametrize("case", ["bf16-anchor", "bf16-prev", "fp32-anchor", "bf16-anchor-hostcache",
                                  "fp32-prev-hostcache", "bf16-anchor-g8", "bf16-prev-g1-hostcache", "bf16-prev-g2",
                                  "bf16-anchor-g1-b100", "bf16-anchor-n8", "bf16-prev-g8-n8",
                                  "bf16-anchor-h4-b4096-n1"])
def test_decode_step_equals_stage_calls(case):
    """louiskv_decode_step (boundary, store, retrieval and attention of a step
    in one launch in bf16, whose attention blocks wait for a fired slice's
    selection blocks, and in two launches in fp32; blocks of a slice hand over
    through the workspace) against the stage calls it replaces, every step of
    a run with evictions: decisions, r, reference queries, scores, selections,
    row lists, unit tables, window and pool equal bit for bit; the attention
    output and lse too in fp32 (same chunks, same merge arithmetic), within
    1e-5 in bf16 (the step splits each slice's rows into smaller chunks).
    Group sizes 1, 2, 4 and 8; b100: a 100-row budget, so that the selected
    rows and the window share an attention chunk; n8: 8 groups (64 slices),
    so that a slice gets 4 blocks of 160 rows and a wave several tiles;
    h4-b4096-n1: one group of 4 slices with a 4096-row budget, 32 blocks of
    144 rows a slice.  The arrival counters, ready
    flags and status word in the workspace are zero after every step.  hostcache:
    louiskv_decode_step_cached over a pinned host pool with an LRU cache of
    four budgets against the stage calls with the same cache (buffer rows,
    slot steps, slot lists, fetch counts and cached rows equal too)."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    dname, mname = case.split("-")[:2]
    cached = case.endswith("hostcache")
    gsize = next((int(p[1:]) for p in case.split("-") if p[0] == "g" and p[1:].isdigit()), None)
    bsize = next((int(p[1:]) for p in case.split("-") if p[0] == "b" and p[1:].isdigit()), None)
    ngroups = next((int(p[1:]) for p in case.split("-") if p[0] == "n" and p[1:].isdigit()), None)
    nkv = next((int(p[1:]) for p in case.split("-") if p[0] == "h" and p[1:].isdigit()), None)
    mode = _L().REF_PREV if mname == "prev" else _L().REF_ANCHOR
    if dname == "bf16":
        wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, name="si-lo-16k")
        n_groups, steps = ngroups or 2, 300
    else:
        wl = synth.get_workload("tiny-4k")
        n_groups, steps = 1, 256
    if gsize is not None:   # other query-group sizes: 8 KV heads, g query heads each
        wl = wl.replace(n_q_heads=wl.n_kv_heads * gsize)
    if bsize is not None:   # a budget whose rows and the window's split into ragged attention chunks
        wl = wl.replace(budget=bsize)
    if nkv is not None:     # fewer KV heads, a longer prompt for the larger budget
        g = wl.n_q_heads // wl.n_kv_heads
        wl = wl.replace(n_kv_heads=nkv, n_q_heads=nkv * g, prompt_len=8192, n_clusters=256)
    data = synth.make_slices(wl, DEV, groups=[(0, l) for l in range(n_groups)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=n_groups, mode=mode, gen_len=steps)
    dt = data.prompt_keys.dtype
    kw = dict(pool_on_host=True, cache_rows=4 * wl.budget) if cached else {}
    a = LouisKVEngine(cfg, dt, DEV, out_dtype=torch.float32, keep_scores=True, fused_step=False, **kw)
    b = LouisKVEngine(cfg, dt, DEV, out_dtype=torch.float32, keep_scores=True, fused_step=True, **kw)
    assert b._use_fused_step() and (b._fused_cached == cached)
    for e in (a, b):
        e.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    S = cfg.n_slices
    fires = evictions = 0
    for t in range(steps):
        a.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        b.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        torch.cuda.synchronize()
        assert torch.equal(a.fire, b.fire), t
        assert torch.equal(a.r.view(torch.int64), b.r.view(torch.int64)), t
        for name in ("q_ref", "n_sel", "n_sel_units", "scores", "reps", "unit_start", "unit_size", "k_local",
                     "v_local"):
            assert torch.equal(getattr(a, name), getattr(b, name)), (t, name)
        written = wl.prompt_len + _L().window_info(t, wl.window, wl.seg_len)[1] * wl.seg_len   # pool rows so far
        assert torch.equal(a.k_pool[:, :written], b.k_pool[:, :written]), t
        assert torch.equal(a.v_pool[:, :written], b.v_pool[:, :written]), t
        for i in range(S):
            assert torch.equal(a.sel_units[i, :int(a.n_sel_units[i])], b.sel_units[i, :int(b.n_sel_units[i])]), (t, i)
            if cached:
                n = int(b.n_sel[i])
                assert torch.equal(a.slot_list[i, :n], b.slot_list[i, :n]), (t, i)
                sl = b.slot_list[i, :n].long()
                assert torch.equal(a.k_buf[i, sl], b.k_buf[i, sl]) and torch.equal(a.v_buf[i, sl], b.v_buf[i, sl])
            else:
                assert torch.equal(a.sel_rows[i, :int(a.n_sel[i])], b.sel_rows[i, :int(b.n_sel[i])]), (t, i)
        if cached:
            for name in ("buf_row", "slot_step"):
                assert torch.equal(getattr(a, name), getattr(b, name)), (t, name)
            fired = a.fire.repeat_interleave(cfg.n_kv_heads).bool()
            assert torch.equal(torch.where(fired, a.n_fetched, 0), torch.where(fired, b.n_fetched, 0)), t
        if dname == "fp32":
            assert torch.equal(a.out, b.out) and torch.equal(a.lse, b.lse), t
        else:
            err = (a.out - b.out).abs().max().item()
            assert err <= 1e-5 * max(1.0, a.out.abs().max().item()), (t, err)
            assert (a.lse - b.lse).abs().max().item() <= 1e-5, t
        assert int(b.ws_step[:256 * (4 * S + 1)].view(torch.int32).abs().sum()) == 0, t
        fires += int(a.fire.sum())
        evictions += int(_L().window_info(t, wl.window, wl.seg_len)[0] >= 0)
    print(f"[decode step] {case}: {steps} steps, {fires} group fires, {evictions} evictions", flush=True)
    assert fires >= (2 if mname == "prev" else 20) and evictions > 2


def test_decode_step_wait_is_bounded(monkeypatch):
    """The one-launch step's wait for a fired slice's selection is bounded:
    with the bound forced down to one poll (LOUISKV_STEP_SPIN_LIMIT=1) the
    blocks of the first step, which always fires, give up at once (the
    selection of 1024 units takes far longer than a poll), the launch
    completes, and the workspace's status word reports the time-out.  That
    step's outputs are undefined; with the workspace zeroed and the default
    bound the next steps equal the stage calls again and leave the status
    word at zero."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=8192, n_clusters=1024, budget=2048, name="si-lo-16k")
    steps = 6
    data = synth.make_slices(wl, DEV, groups=[(0, 0)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=1, gen_len=steps)
    S = cfg.n_slices
    status_at = 256 * 4 * S   # byte offset of the status word (after 4 S counters/flags 256 bytes apart)
    a = LouisKVEngine(cfg, torch.bfloat16, DEV, out_dtype=torch.float32, fused_step=False)
    b = LouisKVEngine(cfg, torch.bfloat16, DEV, out_dtype=torch.float32, fused_step=True)
    for e in (a, b):
        e.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    monkeypatch.setenv("LOUISKV_STEP_SPIN_LIMIT", "1")
    print("[bounded wait] step 0 with a one-poll bound", flush=True)
    b.step(data.queries[0], data.gen_keys[0], data.gen_values[0])
    torch.cuda.synchronize()
    assert int(b.ws_step[status_at:status_at + 4].view(torch.int32)) == 1
    monkeypatch.delenv("LOUISKV_STEP_SPIN_LIMIT")
    # start both engines again from the same state, b with a cleared workspace
    for e in (a, b):
        e.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    b.ws_step.zero_()
    for t in range(steps):
        a.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        b.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        torch.cuda.synchronize()
        assert torch.equal(a.n_sel, b.n_sel) and torch.equal(a.sel_units, b.sel_units), t
        err = (a.out - b.out).abs().max().item()
        assert err <= 1e-5 * max(1.0, a.out.abs().max().item()), (t, err)
        assert int(b.ws_step[:status_at + 4].view(torch.int32).abs().sum()) == 0, t


@pytest.mark.parametrize("case", ["host-delta", "fused-device"])
def test_layer_by_layer_step_graphs_match_eager(case):
    """The group-by-group decode captured as one HIP graph per step (as the
    benchmark times it) and replayed twice after fresh prefills equals the
    eager group-by-group loop: over a pinned host pool with the default LRU
    cache of pool rows (interior pointers of the pool resolved per group view
    at capture time, the decode step baked into each graph),
    and over a device pool, where each view runs the one-launch decode step
    whose workspace counters and flags must return to zero on every replay."""
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    host = case.startswith("host")
    if host:
        wl = synth.get_workload("host-131k").replace(prompt_len=2048, n_clusters=64, budget=512, name="host-131k")
    else:
        wl = synth.get_workload("si-lo-16k").replace(prompt_len=2048, n_clusters=64, budget=512, name="si-lo-16k")
    steps, G = 96, 2
    data = synth.make_slices(wl, DEV, groups=[(0, l) for l in range(G)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=G, gen_len=steps)
    eng = LouisKVEngine(cfg, data.prompt_keys.dtype, DEV, pool_on_host=host, out_dtype=torch.float32)
    # each view runs the fused step: one launch over a device pool, four
    # with the LRU cache over the host pool
    assert eng.group_view(0)._use_fused_step() and eng.group_view(0)._fused_cached == host
    hist = torch.zeros(steps, *eng.out.shape, device=DEV)
    hist_n = torch.zeros(steps, *eng.n_sel.shape, dtype=torch.int32, device=DEV)

    def one_step(t):
        eng.step_layer_by_layer(data.queries[t], data.gen_keys[t], data.gen_values[t])
        hist[t].copy_(eng.out)
        hist_n[t].copy_(eng.n_sel)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    for t in range(steps):
        one_step(t)
    torch.cuda.synchronize()
    ref, ref_n = hist.clone(), hist_n.clone()
    assert int((ref_n > 0).sum()) > 0
    graphs = []
    eng.t = 0
    for t in range(steps):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            one_step(t)
        graphs.append(g)
    print(f"captured {len(graphs)} step graphs ({case})", flush=True)
    for rep in range(2):
        hist.zero_()
        hist_n.zero_()
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
        torch.cuda.synchronize()
        for g in graphs:
            g.replay()
        torch.cuda.synchronize()
        print(f"step-graph replay {rep} ({case})", flush=True)
        assert torch.equal(hist, ref), (case, rep)
        assert torch.equal(hist_n, ref_n), (case, rep)
        assert all(int(w[:256 * (4 * cfg.n_kv_heads + 1)].view(torch.int32).abs().sum()) == 0
                   for w in eng._view_ws_step.values())
    del graphs


def test_boundary_segment_overflow_is_reported():
    """Boundary-delimited segments with every step firing (tau > 1): each
    token is a segment of its own, so after W + (8192 - C) steps the unit
    table (8192 units, the most a retrieval scores) is full.  The engine
    refuses the configuration unless told to accept dropped segments; with
    that, segments keep becoming units while there is room (the flag stays
    clear and the unit count grows by one per step) and the first one that
    does not fit raises the overflow flag, which segment_overflow() reports."""
    from paper_2510_11292_amd.engine import LouisKVEngine, MAX_UNITS, config_from_workload
    wl = synth.get_workload("si-lo-16k").replace(prompt_len=256, n_clusters=32, budget=64, window=64, seg_len=16,
                                                 tau=1.5, name="si-lo-16k")
    full_at = wl.window + (MAX_UNITS - wl.n_clusters)      # first step whose segment finds no room
    steps = full_at + 24
    data = synth.make_slices(wl, DEV, groups=[(0, 0)], gen_len=steps)
    cfg = config_from_workload(wl, n_groups=1, gen_len=steps, segments="boundary")
    with pytest.raises(ValueError, match="allow_unit_overflow"):
        LouisKVEngine(cfg, torch.bfloat16, DEV)
    cfg = config_from_workload(wl, n_groups=1, gen_len=steps, segments="boundary", allow_unit_overflow=True)
    assert cfg.units_cap == MAX_UNITS
    eng = LouisKVEngine(cfg, torch.bfloat16, DEV, out_dtype=torch.float32)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    for t in range(steps):
        eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        if t in (full_at - 1, full_at):
            torch.cuda.synchronize()
            n_units = to_np(eng.seg_state[:, 0])
            if t == full_at - 1:
                assert (n_units == MAX_UNITS).all() and not eng.segment_overflow(), (t, n_units)
            else:
                assert eng.segment_overflow(), t
    torch.cuda.synchronize()
    assert bool(eng.fire.all()) and eng.segment_overflow()
    print(f"[overflow] unit table full at step {full_at - 1}; overflow reported from step {full_at}", flush=True)
