"""Pins of the CPU oracle to facts outside itself.

Each pin takes the oracle namespace as an argument so the mutation tests can
run it against copies with a planted mistake and check that it fails.  The
facts come from the mathematics of each step and from independent library
routines: brute-force enumeration, closed forms, scikit-learn's Lloyd
iteration, scipy's softmax, torch's scaled-dot-product attention and bf16
conversion, and invariants of the definitions in the paper.
"""
from __future__ import annotations

import itertools

import numpy as np
import torch

RNG = np.random.default_rng


def _direct_sqdist(k, c):
    return ((k[:, None, :] - c[None, :, :]) ** 2).sum(-1)


# --------------------------------------------------------------------------- rounding

def pin_bf16_rounding(orc):
    """round_to_bf16 agrees with torch's float32 -> bfloat16 conversion."""
    rng = RNG(1)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * 10.0,
        rng.standard_normal(2000).astype(np.float32) * 1e-30,
        # exact halfway cases between two bf16 values, both parities
        (np.arange(1, 200, dtype=np.uint32) << np.uint32(16) | np.uint32(0x8000)).view(np.float32),
        np.array([0.0, -0.0, 1.0, -3.5, 65504.0, 3.0e38], dtype=np.float32),
    ]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = orc.round_to_bf16(x)
    assert np.array_equal(got, ref), "bf16 rounding differs from torch"
    assert np.array_equal(orc.round_to_f32(np.float64(1) + 2.0 ** -30), np.float64(1.0))


# --------------------------------------------------------------------------- k-means

def pin_squared_distances(orc):
    rng = RNG(2)
    k = rng.standard_normal((37, 9)) * 3
    c = rng.standard_normal((5, 9))
    assert np.allclose(orc.squared_distances(k, c), _direct_sqdist(k, c), rtol=1e-12, atol=1e-10)


def pin_assign_nearest(orc):
    """Each key goes to its nearest centroid by direct distance; ties -> lowest id."""
    rng = RNG(3)
    k = rng.standard_normal((300, 16))
    c = rng.standard_normal((12, 16))
    c[7] = c[3]            # exact duplicate: index 3 must win every tie
    z = orc.kmeans_assign(k, c)
    d = _direct_sqdist(k, c)
    assert np.array_equal(z, np.argmin(d, axis=1))
    assert not np.any(z == 7)
    # a key exactly between two centroids goes to the lower index
    c2 = np.array([[1.0, 0.0], [-1.0, 0.0]])
    assert orc.kmeans_assign(np.array([[0.0, 5.0]]), c2)[0] == 0
    assert orc.kmeans_assign(np.array([[0.0, 5.0]]), c2[::-1].copy())[0] == 0


def pin_kmeans_bruteforce(orc):
    """Lloyd's result is a local optimum no better than the global optimum found
    by enumerating every assignment; on separated data from a good start it is
    the global optimum."""
    rng = RNG(4)
    for trial in range(12):
        n, c = 7, 3
        centres = rng.standard_normal((c, 3)) * (8.0 if trial % 2 == 0 else 0.7)
        lab = rng.integers(0, c, n)
        lab[:c] = np.arange(c)
        k = centres[lab] + 0.3 * rng.standard_normal((n, 3))
        init = np.arange(c) if trial % 2 == 0 else rng.permutation(n)[:c]
        res = orc.kmeans(k, init, n_iters=20, bf16_operand=False)
        cost = orc.clustering_cost(k, res.z, res.centroids)
        best = np.inf
        for a in itertools.product(range(c), repeat=n):
            a = np.asarray(a)
            tot = 0.0
            for j in range(c):
                m = k[a == j]
                if len(m):
                    tot += ((m - m.mean(0)) ** 2).sum()
            best = min(best, tot)
        assert cost >= best - 1e-4 * (1 + best)
        if trial % 2 == 0:
            assert abs(cost - best) <= 1e-4 * (1 + best), (cost, best)
        # centroids are the float32-rounded means of their members
        for j in range(c):
            m = k[res.z == j]
            if len(m):
                assert np.allclose(res.centroids[j], m.mean(0), rtol=1e-6, atol=1e-6)


def pin_kmeans_special_cases(orc):
    rng = RNG(5)
    k = (rng.standard_normal((50, 8)) * 2).astype(np.float32).astype(np.float64)
    # one cluster: the centroid is the global mean
    res = orc.kmeans(k, [13], n_iters=3, bf16_operand=False)
    assert np.array_equal(res.z, np.zeros(50))
    assert np.array_equal(res.centroids[0], np.mean(k, axis=0).astype(np.float32).astype(np.float64))
    # as many clusters as keys with the identity start: identity assignment, cost 0
    res = orc.kmeans(k, np.arange(50), n_iters=2, bf16_operand=False)
    assert np.array_equal(res.z, np.arange(50))
    assert orc.clustering_cost(k, res.z, res.centroids) == 0.0
    assert np.array_equal(res.perm, np.arange(50))
    assert np.array_equal(res.offsets, np.arange(51))


def pin_kmeans_empty_cluster(orc):
    """Duplicate initial centroids: in the first assignment the higher copy
    loses every tie, so its cluster is empty and it keeps its centroid."""
    rng = RNG(6)
    k = rng.standard_normal((40, 4))
    init = [5, 9, 5]
    res = orc.kmeans(k, init, n_iters=1, bf16_operand=False)
    assert res.counts[2] == 0 and res.counts[0] > 0
    assert np.array_equal(res.centroids[2], k[5])
    assert not np.array_equal(res.centroids[0], k[5])
    assert res.offsets[2] == res.offsets[3]
    z, prev = res.z, res.centroids
    c2, counts = orc.kmeans_update(k, np.where(z == 1, 0, z), prev)
    assert counts[1] == 0 and np.array_equal(c2[1], prev[1])


def pin_kmeans_monotone_and_sklearn(orc):
    """Cost never increases (float32-rounded means change it by rounding only)
    and the iteration matches scikit-learn's Lloyd from the same start."""
    from sklearn.cluster import KMeans
    rng = RNG(7)
    m = 6
    centres = rng.standard_normal((m, 12)) * 4
    lab = rng.integers(0, m, 600)
    k = centres[lab] + rng.standard_normal((600, 12))
    init = rng.permutation(600)[:m]
    res = orc.kmeans(k, init, n_iters=15, bf16_operand=False, keep_history=True)
    costs = np.array(res.costs)
    assert np.all(np.diff(costs) <= 1e-6 * costs[:-1]), costs
    sk = KMeans(n_clusters=m, init=k[init], n_init=1, max_iter=15, tol=0.0,
                algorithm="lloyd").fit(k)
    assert np.array_equal(sk.labels_, res.z)
    assert np.allclose(sk.cluster_centers_, res.centroids, rtol=1e-6, atol=1e-6)
    # CSR outputs: perm groups token ids by cluster, ascending inside
    for j in range(m):
        members = res.perm[res.offsets[j]:res.offsets[j + 1]]
        assert np.array_equal(members, np.flatnonzero(res.z == j))


def pin_kmeans_bf16_operand(orc):
    """With the bf16 operand, each assignment is exact against the bf16
    rounding of the previous float32 centroids."""
    rng = RNG(8)
    k = torch.from_numpy(rng.standard_normal((400, 32)) * 2).to(torch.bfloat16).double().numpy()
    init = rng.permutation(400)[:10]
    res = orc.kmeans(k, init, n_iters=3, bf16_operand=True, keep_history=True)
    prev = res.history[-2]
    chat = torch.from_numpy(prev.astype(np.float32)).to(torch.bfloat16).double().numpy()
    assert np.array_equal(res.z, np.argmin(_direct_sqdist(k, chat), axis=1))


# --------------------------------------------------------------------------- segments, boundary

def pin_segment_mean(orc):
    rng = RNG(9)
    rows = rng.standard_normal((32, 128)).astype(np.float32)
    assert np.array_equal(orc.segment_mean(rows), np.mean(rows.astype(np.float64), axis=0).astype(np.float32))


def pin_boundary_closed_forms(orc):
    rng = RNG(10)
    q = rng.standard_normal((32, 128))
    assert abs(orc.query_similarity(q, q) - 1.0) < 1e-12
    assert abs(orc.query_similarity(q, 3.0 * q) - 1.0) < 1e-12
    assert abs(orc.query_similarity(-q, q) + 1.0) < 1e-12
    # orthogonal heads
    a = np.zeros((4, 8)); b = np.zeros((4, 8))
    a[:, 0] = 1.0; b[:, 1] = 2.0
    assert orc.query_similarity(a, b) == 0.0
    # the mean runs over heads: half identical, half opposite -> 0
    h = q.copy(); h[16:] *= -1
    assert abs(orc.query_similarity(q, h)) < 1e-12
    # one head off by angle theta, the rest identical
    th = 0.3
    u = np.zeros((2, 2)); v = np.zeros((2, 2))
    u[:, 0] = 1.0; v[0, 0] = 1.0; v[1] = [np.cos(th), np.sin(th)]
    assert abs(orc.query_similarity(u, v) - (1 + np.cos(th)) / 2) < 1e-12
    # zero-norm query: cosine taken as 0
    assert orc.query_similarity(np.zeros((1, 4)), np.ones((1, 4))) == 0.0
    # threshold rule: strict "<", first step always fires
    assert orc.boundary_fires(0.5, 0.9, False) and not orc.boundary_fires(0.9, 0.9, False)
    assert orc.boundary_fires(0.99, 0.9, True)
    assert orc.boundary_fires(1.0, 1.01, False) and not orc.boundary_fires(-1.0, -1.01, False)


# --------------------------------------------------------------------------- scoring and selection

def pin_group_scores(orc):
    from scipy.special import softmax
    rng = RNG(11)
    q = rng.standard_normal((4, 128)) * 3
    reps = rng.standard_normal((300, 128))
    s = 1 / np.sqrt(128)
    a = orc.group_scores(q, reps, s)
    assert abs(a.sum() - 1.0) < 1e-12 and np.all(a > 0)
    ref = np.mean([softmax(q[j] @ reps.T * s) for j in range(4)], axis=0)
    assert np.allclose(a, ref, rtol=1e-12, atol=1e-15)
    t = torch.softmax(torch.from_numpy(q) @ torch.from_numpy(reps).T * s, dim=1).mean(0).numpy()
    assert np.allclose(a, t, rtol=1e-12, atol=1e-15)
    # one query head: the ranking is the ranking of the raw dot products
    a1 = orc.group_scores(q[:1], reps, s)
    assert np.array_equal(np.argsort(-a1, kind="stable"), np.argsort(-(reps @ q[0]), kind="stable"))
    # permuting the units permutes the scores
    p = rng.permutation(300)
    assert np.allclose(orc.group_scores(q, reps[p], s), a[p], rtol=1e-12, atol=1e-15)
    # a unit's score grows with its alignment to the queries: the unit equal to
    # the mean query direction scaled up ranks first
    reps2 = reps.copy()
    reps2[17] = q.sum(0) / np.linalg.norm(q.sum(0)) * 40
    assert int(np.argmax(orc.group_scores(q, reps2, s))) == 17


def _select_by_sort(scores, size, budget):
    order = np.lexsort((np.arange(len(scores)), -np.asarray(scores)))
    csum = np.cumsum(np.asarray(size)[order])
    n = int(np.searchsorted(csum, budget, side="right"))
    return [int(u) for u in order[:n]], int(csum[n - 1]) if n else 0


def pin_select_budget(orc):
    rng = RNG(12)
    for trial in range(200):
        u = int(rng.integers(1, 60))
        scores = rng.random(u)
        if trial % 3 == 0:
            scores = np.round(scores * 4) / 4          # many exact ties
        size = rng.integers(1, 40, u)
        budget = int(rng.integers(0, 400))
        got, tot = orc.select_budget(scores, size, budget)
        ref, rtot = _select_by_sort(scores, size, budget)
        assert got == ref and tot == rtot
        assert tot <= budget and tot == int(np.sum(size[got])) if got else tot == 0
        if len(got) < u:
            order = sorted(range(u), key=lambda x: (-scores[x], x))
            assert tot + size[order[len(got)]] > budget
    # budget covering everything selects every unit, in rank order
    scores = np.array([0.1, 0.5, 0.5, 0.3]); size = np.array([3, 4, 5, 6])
    assert orc.select_budget(scores, size, 100) == ([1, 2, 3, 0], 18)
    # top unit larger than the budget: nothing
    assert orc.select_budget(scores, size, 3) == ([], 0)
    assert orc.select_budget(scores, size, 9) == ([1, 2], 9)


def pin_gather(orc):
    pool = np.arange(40, dtype=np.float64).reshape(20, 2)
    rows = orc.gather_units(pool, [0, 5, 12], [5, 7, 8], [2, 0])
    assert np.array_equal(rows[:, 0] / 2, np.r_[12:20, 0:5])


# --------------------------------------------------------------------------- attention

def pin_attention(orc):
    rng = RNG(13)
    q = rng.standard_normal((4, 64))
    k = rng.standard_normal((90, 64)) * 2
    v = rng.standard_normal((90, 64))
    s = 1 / 8.0
    o, lse = orc.attention(q, k, v, s)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, :, None, :], torch.from_numpy(k)[None, None].expand(1, 4, 90, 64),
        torch.from_numpy(v)[None, None].expand(1, 4, 90, 64), scale=s)[0, :, 0].numpy()
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-12)
    w = np.exp((q @ k.T) * s - lse[:, None])
    assert np.allclose(w.sum(1), 1.0, atol=1e-12)
    o1, l1 = orc.attention(q, k[:1], v[:1], s)
    assert np.allclose(o1, np.repeat(v[:1], 4, 0), atol=1e-15)
    assert np.allclose(l1, (q @ k[0]) * s)
    oe, le = orc.attention(q, k[:0], v[:0], s)
    assert np.all(oe == 0) and np.all(np.isneginf(le))


ALL_PINS = [
    pin_bf16_rounding, pin_squared_distances, pin_assign_nearest,
    pin_kmeans_bruteforce, pin_kmeans_special_cases, pin_kmeans_empty_cluster,
    pin_kmeans_monotone_and_sklearn, pin_kmeans_bf16_operand, pin_segment_mean,
    pin_boundary_closed_forms, pin_group_scores, pin_select_budget, pin_gather,
    pin_attention,
]


# --------------------------------------------------------------------------- decode driver

def _tiny_group(seed, p=96, t=80, c=8, h_kv=2, g=2, d=16):
    rng = RNG(seed)
    pk = rng.standard_normal((h_kv, p, d)) * 2
    pv = rng.standard_normal((h_kv, p, d))
    gk = rng.standard_normal((t, h_kv, d)) * 2
    gv = rng.standard_normal((t, h_kv, d))
    q = rng.standard_normal((t, h_kv * g, d))
    return pk, pv, gk, gv, q


def _prefill(orc, pk, pv, c):
    res = [orc.kmeans(pk[h], np.arange(c) * 3, n_iters=3, bf16_operand=False) for h in range(pk.shape[0])]
    return orc.prefill_state_from_kmeans(pk, pv, res)


def pin_decode_dense_special_case(orc):
    """Always firing with an unbounded budget gives dense attention over every
    token so far, except the segment evicted at that very step (it left the
    window after this step's retrieval, as in Algorithm 1's order)."""
    pk, pv, gk, gv, q = _tiny_group(20)
    h_kv, p, d = pk.shape
    g = q.shape[1] // h_kv
    dec = orc.GroupDecoder(_prefill(orc, pk, pv, 8), n_q_heads=q.shape[1], budget=10 ** 9,
                           window=32, seg_len=8, tau=1.5, mode="prev")
    s = 1 / np.sqrt(d)
    evictions = 0
    for t in range(q.shape[0]):
        rec = dec.step(q[t], gk[t], gv[t])
        assert rec.fire
        gone = set()
        if rec.evicted_unit is not None:
            evictions += 1
            e = rec.evicted_unit - 8
            gone = set(range(8 * e, 8 * e + 8))
        keep = [j for j in range(t + 1) if j not in gone]
        for h in range(h_kv):
            kk = torch.from_numpy(np.concatenate([pk[h], gk[keep, h]]))
            vv = torch.from_numpy(np.concatenate([pv[h], gv[keep, h]]))
            qq = torch.from_numpy(q[t, h * g:(h + 1) * g])
            ref = torch.nn.functional.scaled_dot_product_attention(
                qq[None, :, None, :], kk[None, None].expand(1, g, -1, -1),
                vv[None, None].expand(1, g, -1, -1), scale=s)[0, :, 0].numpy()
            assert np.allclose(rec.out[h * g:(h + 1) * g], ref, rtol=1e-10, atol=1e-12)
    assert evictions == (q.shape[0] - 32 + 7) // 8


def pin_decode_frozen_and_schedule(orc):
    """tau below -1 fires only at t = 1, so KV_critical never changes; segments
    leave the window at t = W+1, W+1+s, ... and their index vector is the mean
    of exactly those generated keys, stored at pool row P + first token."""
    pk, pv, gk, gv, q = _tiny_group(21)
    h_kv, p, d = pk.shape
    dec = orc.GroupDecoder(_prefill(orc, pk, pv, 8), n_q_heads=q.shape[1], budget=40,
                           window=32, seg_len=8, tau=-1.5, mode="anchor")
    first_sel = None
    ev_steps = []
    for t in range(q.shape[0]):
        rec = dec.step(q[t], gk[t], gv[t])
        assert rec.fire == (t == 0)
        if t == 0:
            first_sel = [list(x) for x in rec.sel_units]
            n0 = rec.n_sel
            assert all(0 < n <= 40 for n in n0)
        assert dec.crit_units == first_sel and rec.n_sel == n0
        if rec.evicted_unit is not None:
            ev_steps.append(t + 1)
    assert ev_steps == list(range(33, q.shape[0] + 1, 8))
    for e in range(len(ev_steps)):
        for h in range(h_kv):
            u = 8 + e
            assert dec.unit_start[h][u] == p + 8 * e and dec.unit_size[h][u] == 8
            ref = gk[8 * e:8 * e + 8, h].mean(0).astype(np.float32)
            assert np.array_equal(dec.reps[h][u], ref)
            assert np.array_equal(np.asarray(dec.k_pool[h])[p + 8 * e:p + 8 * e + 8], gk[8 * e:8 * e + 8, h])


def pin_decode_boundary_modes(orc):
    """On the synthetic query process, the previous-query mode fires exactly at
    the query jumps (a fresh query is nearly orthogonal to the last one, an
    AR(1) step keeps cosine ~0.97); the anchor mode also fires once the drift
    since the last boundary drops the cosine under 0.9 (every ~4 steps)."""
    import synth
    wl = synth.tiny_workload(prompt_len=128, n_clusters=8, gen_len=600, n_iters=2,
                             budget=64, window=32)
    data = synth.make_slices(wl, "cpu", groups=[(0, 0)])
    jumps = synth.jump_steps(wl, 0).numpy()
    pk = data.prompt_keys.double().numpy()
    pv = data.prompt_values.double().numpy()
    rates = {}
    for mode in ("prev", "anchor"):
        res = [orc.kmeans(pk[h], data.init_idx[h].numpy(), 2, False) for h in range(8)]
        dec = orc.GroupDecoder(orc.prefill_state_from_kmeans(pk, pv, res), 32, wl.budget,
                               wl.window, wl.seg_len, wl.tau, mode)
        fires = []
        for t in range(wl.gen_len):
            rec = dec.step(data.queries[t, 0].double().numpy(), data.gen_keys[t].double().numpy(),
                           data.gen_values[t].double().numpy())
            fires.append(rec.fire)
        fires = np.array(fires)
        rates[mode] = fires.mean()
        if mode == "prev":
            assert np.array_equal(fires, jumps)
    assert 0.18 < rates["anchor"] < 0.35, rates


def pin_decode_boundary_segments(orc):
    """Boundary-delimited segments.  (1) When only the first step fires, the
    segments are the seg_len-token runs of the fixed scheme, so the two
    decoders agree step for step.  (2) When every step fires, every segment is
    one token: from step W+1 on each step evicts the token W steps back, as a
    unit of size 1 whose index vector is that key.  (3) For an arbitrary fire
    pattern the evicted units tile the generated tokens in order, none is
    longer than seg_len, each starts at a fired step or right after a unit of
    exactly seg_len tokens, the window never holds more than W tokens, a
    segment leaves exactly when the window held W tokens before the step, and
    every index vector is the mean of its unit's rows."""
    pk, pv, gk, gv, q = _tiny_group(22, t=120)
    h_kv, p, d = pk.shape
    # (1)
    a = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 40, 32, 8, -1.5, "anchor")
    b = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 40, 32, 8, -1.5, "anchor", segments="boundary")
    for t in range(q.shape[0]):
        ra, rb = a.step(q[t], gk[t], gv[t]), b.step(q[t], gk[t], gv[t])
        assert ra.evicted_unit == rb.evicted_unit and np.array_equal(ra.out, rb.out)
    assert a.unit_size == b.unit_size and a.unit_start == b.unit_start
    # (2)
    dec = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 40, 16, 4, 1.5, "prev", segments="boundary")
    for t in range(q.shape[0]):
        rec = dec.step(q[t], gk[t], gv[t])
        assert rec.fire
        if t < 16:
            assert rec.evicted_unit is None
        else:
            u = rec.evicted_unit
            assert u == 8 + t - 16
            for h in range(h_kv):
                assert dec.unit_size[h][u] == 1 and dec.unit_start[h][u] == p + t - 16
                assert np.array_equal(dec.reps[h][u], gk[t - 16, h].astype(np.float32))
    # (3)
    rng = RNG(23)
    W, smax = 24, 5
    fires = rng.random(q.shape[0]) < 0.3
    dec = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 40, W, smax, 0.9, "anchor", segments="boundary")
    for t in range(q.shape[0]):
        before = len(dec.local[0])
        rec = dec.step(q[t], gk[t], gv[t], fire_override=bool(fires[t]) or t == 0)
        assert len(dec.local[0]) <= W
        assert (rec.evicted_unit is not None) == (before == W)
        left = dec.unit_size[0][rec.evicted_unit] if rec.evicted_unit is not None else 0
        assert len(dec.local[0]) == before - left + 1
    for h in range(h_kv):
        starts, sizes = dec.unit_start[h][8:], dec.unit_size[h][8:]
        assert starts[0] == p and all(x + n == y for x, n, y in zip(starts, sizes, starts[1:]))
        assert all(1 <= n <= smax for n in sizes)
        for i, (st, n) in enumerate(zip(starts, sizes)):
            g0 = st - p
            assert g0 == 0 or fires[g0] or sizes[i - 1] == smax
            assert np.array_equal(dec.reps[h][8 + i], gk[g0:g0 + n, h].mean(0).astype(np.float32))
        assert starts[-1] + sizes[-1] - p + len(dec.local[h]) == q.shape[0]


def pin_page_units(orc):
    """Pages are consecutive runs of page_len tokens (the last one ragged),
    each indexed by its mean key (numpy's mean, rounded to float32); one page
    of every token is the global mean, pages of one token are the keys; the
    page-level prefill keeps the prompt in token order, so always firing with
    an unbounded budget is dense attention."""
    rng = RNG(41)
    k = rng.standard_normal((50, 8)) * 3
    reps, starts, sizes = orc.page_units(k, 16)
    assert starts.tolist() == [0, 16, 32, 48] and sizes.tolist() == [16, 16, 16, 2]
    for i, (a, z) in enumerate(zip(starts, sizes)):
        np.testing.assert_allclose(reps[i], np.mean(k[a:a + z], axis=0), rtol=1e-7, atol=0)
        assert np.array_equal(reps[i], reps[i].astype(np.float32))
    one, _, sz = orc.page_units(k, 50)
    assert sz.tolist() == [50]
    np.testing.assert_allclose(one[0], k.mean(0), rtol=1e-7, atol=0)
    single, st1, sz1 = orc.page_units(k, 1)
    assert np.array_equal(single, k.astype(np.float32)) and st1.tolist() == list(range(50))
    big, _, szb = orc.page_units(k, 64)
    assert szb.tolist() == [50]
    # decode over pages: dense when every step fires with an unbounded budget
    pk, pv, gk, gv, q = _tiny_group(43)
    h_kv, p, d = pk.shape
    g = q.shape[1] // h_kv
    st = orc.prefill_state_from_pages(pk, pv, 16)
    assert all(np.array_equal(st.k_pool[h], pk[h]) for h in range(h_kv))
    dec = orc.GroupDecoder(st, q.shape[1], budget=10 ** 9, window=64, seg_len=16, tau=1.5, mode="prev")
    s = 1 / np.sqrt(d)
    for t in range(40):
        rec = dec.step(q[t], gk[t], gv[t])
        for h in range(h_kv):
            kk = torch.from_numpy(np.concatenate([pk[h], gk[:t + 1, h]]))
            vv = torch.from_numpy(np.concatenate([pv[h], gv[:t + 1, h]]))
            qq = torch.from_numpy(q[t, h * g:(h + 1) * g])
            ref = torch.nn.functional.scaled_dot_product_attention(
                qq[None, :, None, :], kk[None, None].expand(1, g, -1, -1),
                vv[None, None].expand(1, g, -1, -1), scale=s)[0, :, 0].numpy()
            assert np.allclose(rec.out[h * g:(h + 1) * g], ref, rtol=1e-10, atol=1e-12)


def pin_decode_stride_trigger(orc):
    """The fixed-stride trigger fires at steps 1, 1 + s, 1 + 2s, ... whatever
    the queries do; stride 1 behaves as a boundary test that always fires and
    a stride past the last step as one that never fires after the first."""
    pk, pv, gk, gv, q = _tiny_group(44, t=60)
    st = _prefill(orc, pk, pv, 8)
    dec = orc.GroupDecoder(st, q.shape[1], 40, 32, 8, 0.9, "anchor", trigger="stride", stride=5)
    fired = [dec.step(q[t], gk[t], gv[t]).fire for t in range(q.shape[0])]
    assert [t for t, f in enumerate(fired) if f] == list(range(0, q.shape[0], 5))
    for stride, tau in ((1, 1.5), (1000, -2.0)):
        a = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 40, 32, 8, 0.9, "anchor", trigger="stride",
                             stride=stride)
        b = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 40, 32, 8, tau, "anchor")
        for t in range(q.shape[0]):
            ra, rb = a.step(q[t], gk[t], gv[t]), b.step(q[t], gk[t], gv[t])
            assert ra.fire == rb.fire and ra.sel_units == rb.sel_units
            assert np.array_equal(ra.out, rb.out)


def pin_decode_per_head(orc):
    """Per-head selection: each query head's units are the budget prefix of
    the ranking by its own softmax (scipy's, over its logits); with one query
    head per KV head it is the group-consistent selection; with the heads of
    a group given equal queries every head takes the group's selection; with
    an unbounded budget every head attends to everything, as the group does."""
    from scipy.special import softmax
    pk, pv, gk, gv, q = _tiny_group(45, t=50)
    h_kv, p, d = pk.shape
    g = q.shape[1] // h_kv
    s = 1 / np.sqrt(d)
    # rankings of the units that exist before each step (its eviction comes
    # after its retrieval)
    dec = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 30, 32, 8, 1.5, "prev", selection="per_head")
    for t in range(q.shape[0]):
        reps_now = [np.asarray(r).copy() for r in dec.reps]
        sizes_now = [list(z) for z in dec.unit_size]
        rec = dec.step(q[t], gk[t], gv[t])
        assert len(rec.sel_units) == h_kv * g
        for li in range(h_kv * g):
            h = li // g
            a = softmax(q[t, li] @ reps_now[h].T * s)
            assert rec.sel_units[li] == _select_by_sort(a, sizes_now[h], 30)[0]
    heads_differ = any(len(set(map(tuple, rec.sel_units[h * g:(h + 1) * g]))) > 1 for h in range(h_kv))
    assert heads_differ
    # one query head per KV head
    q1 = q[:, ::g]
    a = orc.GroupDecoder(_prefill(orc, pk, pv, 8), h_kv, 30, 32, 8, 0.9, "anchor", selection="per_head")
    b = orc.GroupDecoder(_prefill(orc, pk, pv, 8), h_kv, 30, 32, 8, 0.9, "anchor")
    for t in range(q.shape[0]):
        ra, rb = a.step(q1[t], gk[t], gv[t]), b.step(q1[t], gk[t], gv[t])
        assert ra.fire == rb.fire and ra.sel_units == rb.sel_units and np.array_equal(ra.out, rb.out)
    # equal queries within each group
    qe = np.repeat(q[:, ::g], g, axis=1)
    a = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 30, 32, 8, 0.9, "anchor", selection="per_head")
    b = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 30, 32, 8, 0.9, "anchor")
    for t in range(q.shape[0]):
        ra, rb = a.step(qe[t], gk[t], gv[t]), b.step(qe[t], gk[t], gv[t])
        if rb.fire:
            assert ra.sel_units == [u for u in rb.sel_units for _ in range(g)]
        assert np.allclose(ra.out, rb.out, rtol=1e-12, atol=1e-14)
    # unbounded budget
    a = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 10 ** 9, 32, 8, 1.5, "prev", selection="per_head")
    b = orc.GroupDecoder(_prefill(orc, pk, pv, 8), q.shape[1], 10 ** 9, 32, 8, 1.5, "prev")
    for t in range(q.shape[0]):
        ra, rb = a.step(q[t], gk[t], gv[t]), b.step(q[t], gk[t], gv[t])
        assert np.allclose(ra.out, rb.out, rtol=1e-10, atol=1e-12)


def pin_prefill_pool_packing(orc):
    """The unified pool after prefill (Section 4.2, Fig. 4, Algorithm 1's
    prompt offload): each cluster is one contiguous run of pool rows holding
    exactly the prompt tokens the final assignment gives it, in ascending
    token order, for keys and values alike; the runs follow cluster order and
    tile the prompt; a run's index vector is the mean of its rows.  A decode
    step whose budget takes a strict subset of the clusters attends to
    exactly the member tokens of the chosen clusters plus the window, checked
    with torch SDPA over those tokens taken from the unpermuted prompt."""
    rng = RNG(47)
    h_kv, p, d, c, g = 2, 120, 8, 6, 2
    pk = rng.standard_normal((h_kv, p, d)) * 2
    pv = rng.standard_normal((h_kv, p, d))
    res = [orc.kmeans(pk[h], rng.permutation(p)[:c], n_iters=4, bf16_operand=False) for h in range(h_kv)]
    st = orc.prefill_state_from_kmeans(pk, pv, res)
    for h in range(h_kv):
        z = np.asarray(res[h].z)
        start = 0
        for cl in range(c):
            members = np.flatnonzero(z == cl)
            n = members.size
            assert int(st.unit_start[h][cl]) == start and int(st.unit_size[h][cl]) == n, (h, cl)
            assert np.array_equal(np.asarray(st.k_pool[h])[start:start + n], pk[h][members])
            assert np.array_equal(np.asarray(st.v_pool[h])[start:start + n], pv[h][members])
            if n:
                assert np.allclose(st.reps[h][cl], pk[h][members].mean(0), rtol=1e-6, atol=1e-6)
            start += n
        assert start == p
    # a partial selection attends to the member tokens of the chosen clusters
    gk = rng.standard_normal((3, h_kv, d)) * 2
    gv = rng.standard_normal((3, h_kv, d))
    q = rng.standard_normal((3, h_kv * g, d))
    dec = orc.GroupDecoder(st, h_kv * g, budget=p // 2, window=16, seg_len=4, tau=1.5, mode="prev")
    s = 1 / np.sqrt(d)
    for t in range(3):
        rec = dec.step(q[t], gk[t], gv[t])
        assert all(0 < n < p for n in rec.n_sel)
        for h in range(h_kv):
            toks = np.flatnonzero(np.isin(np.asarray(res[h].z), rec.sel_units[h]))
            assert toks.size == rec.n_sel[h]
            kk = torch.from_numpy(np.concatenate([pk[h][toks], gk[:t + 1, h]]))
            vv = torch.from_numpy(np.concatenate([pv[h][toks], gv[:t + 1, h]]))
            qq = torch.from_numpy(q[t, h * g:(h + 1) * g])
            ref = torch.nn.functional.scaled_dot_product_attention(
                qq[None, :, None, :], kk[None, None].expand(1, g, -1, -1),
                vv[None, None].expand(1, g, -1, -1), scale=s)[0, :, 0].numpy()
            assert np.allclose(rec.out[h * g:(h + 1) * g], ref, rtol=1e-10, atol=1e-12)


DECODE_PINS = [pin_prefill_pool_packing, pin_decode_dense_special_case, pin_decode_frozen_and_schedule, pin_decode_boundary_modes,
               pin_decode_boundary_segments, pin_page_units, pin_decode_stride_trigger, pin_decode_per_head]
ALL_PINS = ALL_PINS + DECODE_PINS
