"""Comparison helpers for the HIP path against the CPU oracle.

Integer results (assignments, permutations, unit tables, boundary decisions,
selected units and rows) must match exactly, except where the float64
quantity that decides them is a near-tie.  Near-tie bands (relative 1e-6):
  assignment  |D_a - D_b| <= 1e-6 * (||k||^2 + max(||c_a||^2, ||c_b||^2)), the
              error scale of an fp32-accumulated expanded distance;
  boundary    |r - tau| <= 1e-6 * max(|r|, |tau|);
  scores      |A_a - A_b| <= 1e-6 * max(A_a, A_b).
Where the two sides differ inside a band, the checker adopts the GPU's
choice so the runs do not diverge afterwards.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle

REL = 1e-6


def to64(t) -> np.ndarray:
    if isinstance(t, np.ndarray):
        return t.astype(np.float64)
    return t.detach().float().cpu().numpy().astype(np.float64)


def to_np(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def check_assignment(keys, operand, z_gpu, z_ref=None):
    """z_gpu must be an exact argmin of ||k - operand_c||^2 up to the band.

    Returns the number of keys whose choice differs from the oracle's but lies
    inside the band.  Raises AssertionError otherwise.
    """
    k = np.asarray(keys, dtype=np.float64)
    c = np.asarray(operand, dtype=np.float64)
    z_gpu = np.asarray(z_gpu, dtype=np.int64)
    if z_ref is None:
        z_ref = oracle.kmeans_assign(k, c)
    bad = np.flatnonzero(z_gpu != z_ref)
    if bad.size == 0:
        return 0
    kk = k[bad]
    a, b = z_gpu[bad], z_ref[bad]
    assert np.all((a >= 0) & (a < c.shape[0])), "assignment out of range"
    da = ((kk - c[a]) ** 2).sum(1)
    db = ((kk - c[b]) ** 2).sum(1)
    scale = (kk * kk).sum(1) + np.maximum((c[a] ** 2).sum(1), (c[b] ** 2).sum(1))
    gap = np.abs(da - db)
    worst = int(np.argmax(gap / scale))
    assert np.all(gap <= REL * scale), (
        f"{bad.size} assignments differ; worst key {bad[worst]}: gpu {a[worst]} ({da[worst]!r}) vs oracle "
        f"{b[worst]} ({db[worst]!r}), relative gap {gap[worst] / scale[worst]:.3e}")
    return int(bad.size)


def check_rows_rel(got, ref, rel, what):
    """Per row: max |got - ref| <= rel * max |ref| (rows along the last axis)."""
    g = np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    err = np.abs(g - r).max(axis=-1)
    scale = np.maximum(np.abs(r).max(axis=-1), 1e-30)
    bad = err > rel * scale
    assert not np.any(bad), f"{what}: {int(bad.sum())} rows off, worst {float((err / scale).max()):.3e}"


def selection_matches(scores_ref, sizes, budget, sel_gpu):
    """The GPU's selected units are a valid budgeted selection for the oracle's
    scores: the prefix stop (Section 3.1, Algorithm 1 Retrieve) applied to a
    ranking that differs from the oracle's only by reordering units whose
    scores lie within the band.  That holds when

      - the units are distinct and in range, and their sizes total <= budget;
      - the list is in descending score order up to the band;
      - no unselected unit outscores a selected one beyond the band;
      - the list is maximal: unless every unit is taken, some unselected unit
        tied (within the band) with the best unselected one does not fit in
        what the budget leaves, so the prefix stop had to end there.

    A list cut short by one unit with a clear score gap fails the last rule.
    Returns True when the list differs from the oracle's (a near-tie excused),
    False when it is identical; raises AssertionError otherwise."""
    ref, _ = oracle.select_budget(scores_ref, sizes, budget)
    sel = [int(u) for u in sel_gpu]
    if sel == ref:
        return False
    s = np.asarray(scores_ref, dtype=np.float64)
    size = np.asarray(sizes, dtype=np.int64)
    n_units = s.shape[0]
    assert all(0 <= u < n_units for u in sel), f"selected unit out of range: {sel}"
    assert len(set(sel)) == len(sel), f"a unit is selected twice: {sel}"
    tot = int(size[sel].sum()) if sel else 0
    assert tot <= budget, f"selection holds {tot} tokens > budget {budget}"

    def within(a, b):            # a >= b up to the band (scores are positive)
        return a >= b - REL * max(a, b)

    sv = s[sel]
    if sv.size > 1:
        suffix_max = np.maximum.accumulate(sv[::-1])[::-1]
        for i in range(sv.size - 1):
            assert within(sv[i], suffix_max[i + 1]), (
                f"rank order broken at {i}: unit {sel[i]} ({sv[i]!r}) before a unit scoring {suffix_max[i + 1]!r}")
    rest = np.setdiff1d(np.arange(n_units), np.asarray(sel, dtype=np.int64))
    if rest.size:
        best = float(s[rest].max())
        if sv.size:
            assert within(float(sv.min()), best), (
                f"unselected unit {int(rest[np.argmax(s[rest])])} ({best!r}) outscores selected "
                f"{sel[int(np.argmin(sv))]} ({float(sv.min())!r})")
        tied = rest[[within(float(x), best) for x in s[rest]]]
        assert np.any(tot + size[tied] > budget), (
            f"selection stops early: {len(sel)} units, {tot} tokens, but the next unit (one of {tied.tolist()[:8]}, "
            f"score {best!r}) fits budget {budget}; the oracle takes {len(ref)} units")
    return True


def check_kmeans_trajectory(keys, init_idx, n_iters, bf16_operand, gpu_state):
    """Step-lock a whole k-means run with the oracle (Section 4.2; Algorithm 1
    KMeans / ComputeCentroid).  gpu_state(it) gives the GPU's (assignment [N],
    centroids [C][d]) after `it` Lloyd iterations of the same slice.  At every
    iteration the GPU's assignment must be an exact argmin to the operand of
    its previous centroids up to the assignment band, and its centroids the
    exact means of that assignment (empty clusters unchanged): so a run that
    ends away from the oracle's can only have left it at an excused near-tie.
    Returns the number of excused keys summed over iterations."""
    k = np.asarray(keys, dtype=np.float64)
    prev = k[np.asarray(init_idx, dtype=np.int64)]
    excused = 0
    for it in range(1, n_iters + 1):
        z, c = gpu_state(it)
        operand = oracle.round_to_bf16(prev) if bf16_operand else prev
        excused += check_assignment(k, operand, z)
        ref, _ = oracle.kmeans_update(k, np.asarray(z, dtype=np.int64), prev)
        c = np.asarray(c, dtype=np.float64)
        if not np.array_equal(c, ref):
            check_rows_rel(c, ref, 1e-5, f"iteration {it}: centroids as means of the assignment")
        prev = c
    return excused


def gpu_kmeans_states(L, keys, init_idx, n_clusters):
    """A callable it -> (assignments [S][N], centroids [S][C][d]) as numpy:
    the GPU's clustering of every slice after `it` Lloyd iterations, from
    louiskv_cluster_prefill run with n_iters = it (cached per it)."""
    cache = {}

    def state(it):
        if it not in cache:
            S, N, d = keys.shape
            reps = torch.empty(S, n_clusters, d, dtype=torch.float32, device=keys.device)
            ustart = torch.empty(S, n_clusters, dtype=torch.int32, device=keys.device)
            usize = torch.empty_like(ustart)
            z = torch.empty(S, N, dtype=torch.int32, device=keys.device)
            perm = torch.empty_like(z)
            L.cluster_prefill(keys, n_clusters, it, init_idx, reps, ustart, usize, z, perm)
            torch.cuda.synchronize()
            cache[it] = (to_np(z).astype(np.int64), to64(reps))
        return cache[it]
    return state


def oracle_prefill_state(keys64, values64, init_idx, n_iters, bf16_operand, z_gpu, c_gpu,
                         gpu_states=None, slice_ids=None):
    """The oracle's prefill for the KV heads of one group: k-means of each
    slice, then the pool packed cluster by cluster (prefill_state_from_kmeans).
    Where a slice's final GPU assignment differs from the oracle's, the GPU's
    whole run is step-locked with check_kmeans_trajectory (gpu_states(it)
    gives every slice's state after it iterations; slice_ids maps the
    group's heads to those slices) and its clustering is adopted.  Returns
    (state, keys excused over all iterations, slices adopted)."""
    results, excused, adopted = [], 0, 0
    for h in range(len(keys64)):
        init = np.asarray(init_idx[h], dtype=np.int64)
        res = oracle.kmeans(keys64[h], init, n_iters, bf16_operand)
        z = np.asarray(z_gpu[h], dtype=np.int64)
        if not np.array_equal(res.z, z):
            assert gpu_states is not None, f"head {h}: the final assignment differs from the oracle's"
            sid = h if slice_ids is None else slice_ids[h]
            excused += check_kmeans_trajectory(keys64[h], init, n_iters, bf16_operand,
                                               lambda it: tuple(x[sid] for x in gpu_states(it)))
            res = oracle.kmeans_finish(z, c_gpu[h])
            adopted += 1
        elif not np.array_equal(np.asarray(c_gpu[h], dtype=np.float64), res.centroids):
            check_rows_rel(c_gpu[h], res.centroids, 1e-5, f"head {h} centroids")
        results.append(res)
    return oracle.prefill_state_from_kmeans(keys64, values64, results), excused, adopted


def check_prefill_against_state(reps, unit_start, unit_size, k_pool, v_pool, st, n_prompt):
    """The GPU's unit table and packed pool rows of one group equal the
    oracle's prefill state (index vectors bit for bit or within 1e-5 per row,
    integer tables and pool rows exactly)."""
    for h in range(len(st.reps)):
        n_units = len(st.unit_size[h])
        r = to64(reps[h, :n_units])
        if not np.array_equal(r, np.asarray(st.reps[h], dtype=np.float64)):
            check_rows_rel(r, st.reps[h], 1e-5, f"head {h} index vectors")
        assert np.array_equal(to_np(unit_start[h, :n_units]).astype(np.int64), np.asarray(st.unit_start[h])), h
        assert np.array_equal(to_np(unit_size[h, :n_units]).astype(np.int64), np.asarray(st.unit_size[h])), h
        assert np.array_equal(to64(k_pool[h, :n_prompt]), np.asarray(st.k_pool[h], dtype=np.float64)), h
        assert np.array_equal(to64(v_pool[h, :n_prompt]), np.asarray(st.v_pool[h], dtype=np.float64)), h


def report(name, stats, bound=None, of=None):
    """Print a test's excused near-tie counts (and fail past a bound)."""
    print(f"[parity] {name}: " + ", ".join(f"{k}={v}" for k, v in stats.items() if not isinstance(v, set)),
          flush=True)
    if bound is not None:
        assert stats["excused"] <= bound, f"{name}: {stats['excused']} excused near-ties > bound {bound} ({of})"
