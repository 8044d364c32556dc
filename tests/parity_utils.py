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
    """The GPU's selected units equal the oracle's, or differ only by the order
    of units whose oracle scores are within the band (then every prefix rule
    still holds).  Returns True if an excuse was used."""
    ref, _ = oracle.select_budget(scores_ref, sizes, budget)
    sel_gpu = [int(u) for u in sel_gpu]
    if sel_gpu == ref:
        return False
    s = np.asarray(scores_ref, dtype=np.float64)
    # the GPU's list must be a valid ranking prefix up to near-ties
    for i in range(len(sel_gpu) - 1):
        a, b = sel_gpu[i], sel_gpu[i + 1]
        assert s[a] >= s[b] - REL * max(s[a], s[b]), f"rank order broken at {i}"
    n = min(len(sel_gpu), len(ref))
    for i in range(n):
        if sel_gpu[i] != ref[i]:
            a, b = sel_gpu[i], ref[i]
            assert abs(s[a] - s[b]) <= REL * max(s[a], s[b]), (
                f"selection differs at rank {i}: gpu {a} ({s[a]!r}) vs oracle {b} ({s[b]!r})")
    tot = int(np.sum(np.asarray(sizes)[sel_gpu])) if sel_gpu else 0
    assert tot <= budget
    return True
