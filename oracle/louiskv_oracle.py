"""Step functions of the LouisKV path, in plain NumPy float64.

TEST INFRASTRUCTURE ONLY (see the package docstring): a slow, obviously
correct reference.  Every input is widened exactly to float64; results that
the path stores in a narrower type are rounded once, where the path stores
them, by the helpers below.  Paper references are to "LouisKV: Efficient KV
Cache Retrieval for Long Input-Output Sequences" (arXiv 2510.11292).

Readings of points the paper leaves open are stated where they are used:
squared Euclidean k-means with a mean update, the bf16 rounding of the
centroid operand, lowest-index tie-breaks, prefix-stop budgeting, a cosine
with a clamped denominator.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


# ---------------------------------------------------------------------------
# rounding helpers
# ---------------------------------------------------------------------------

def round_to_f32(x) -> np.ndarray:
    """Round to the nearest float32 (ties to even), returned as float64."""
    return np.asarray(x, dtype=F64).astype(np.float32).astype(F64)


def round_to_bf16(x) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), as float64.

    bfloat16 keeps the top 16 bits of a float32.  Adding 0x7FFF plus the lowest
    kept bit before truncating the low 16 bits rounds to nearest with ties to
    even.  NaN inputs are not handled (the path never produces them).
    """
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    keep_lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + keep_lsb) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).astype(F64)


# ---------------------------------------------------------------------------
# prefill: k-means clustering of the prompt keys (Section 4.2, Algorithm 1
# store_cache prefill branch)
# ---------------------------------------------------------------------------

def squared_distances(keys, centroids) -> np.ndarray:
    """D[i, c] = ||k_i - c_c||^2 for every key and centroid, in float64.

    Uses the identity ||k - c||^2 = ||k||^2 - 2 k.c + ||c||^2 so the cross
    term is one matrix product; the tests check it against the direct form.
    """
    k = np.asarray(keys, dtype=F64)
    c = np.asarray(centroids, dtype=F64)
    kk = np.einsum("nd,nd->n", k, k)[:, None]
    cc = np.einsum("cd,cd->c", c, c)[None, :]
    return kk - 2.0 * (k @ c.T) + cc


def kmeans_assign(keys, centroids, chunk: int = 8192) -> np.ndarray:
    """z_i = argmin_c ||k_i - c_c||^2, ties to the lowest centroid index.

    Section 4.2 groups similar key vectors with k-means; similarity is read as
    squared Euclidean distance, the metric whose minimiser is the mean used as
    the centroid.  np.argmin returns the first minimum, i.e. the lowest index.
    """
    k = np.asarray(keys, dtype=F64)
    n = k.shape[0]
    z = np.empty(n, dtype=np.int64)
    for s in range(0, n, chunk):
        z[s:s + chunk] = np.argmin(squared_distances(k[s:s + chunk], centroids), axis=1)
    return z


def kmeans_update(keys, z, prev_centroids) -> Tuple[np.ndarray, np.ndarray]:
    """Centroid = mean of the keys assigned to it (Section 4.2 ComputeCentroid).

    The sum is taken in float64 and the mean rounded once to float32.  A
    cluster with no member keeps its previous centroid.  Returns (centroids as
    float64 holding float32 values, member counts).
    """
    k = np.asarray(keys, dtype=F64)
    z = np.asarray(z, dtype=np.int64)
    prev = np.asarray(prev_centroids, dtype=F64)
    n_clusters = prev.shape[0]
    counts = np.bincount(z, minlength=n_clusters)
    sums = np.zeros_like(prev)
    np.add.at(sums, z, k)
    out = prev.copy()
    nz = counts > 0
    out[nz] = round_to_f32(sums[nz] / counts[nz][:, None])
    return out, counts


def clustering_cost(keys, z, centroids) -> float:
    """Sum over keys of the squared distance to the assigned centroid."""
    k = np.asarray(keys, dtype=F64)
    c = np.asarray(centroids, dtype=F64)[np.asarray(z)]
    return float(((k - c) ** 2).sum())


@dataclass
class KMeansResult:
    z: np.ndarray              # [N] last assignment
    centroids: np.ndarray      # [C][d] float64 holding float32 values
    counts: np.ndarray         # [C]
    offsets: np.ndarray        # [C+1] CSR offsets of each cluster in perm
    perm: np.ndarray           # [N] token ids grouped by cluster, ascending within
    history: List[np.ndarray] = field(default_factory=list)  # centroids after each update
    costs: List[float] = field(default_factory=list)         # cost of (z_it, C_it) per iteration


def kmeans(keys, init_idx, n_iters: int, bf16_operand: bool,
           keep_history: bool = False) -> KMeansResult:
    """Lloyd's k-means of one slice's prompt keys.

    Initial centroids are the keys at init_idx.  Each iteration assigns every
    key to its nearest centroid operand, then replaces each non-empty
    centroid by the mean of its keys.  With bf16_operand the distance is
    taken to the bfloat16 rounding of the float32 centroid: that is the
    operand a bf16 matrix-core contraction sees, and the decision is only
    exact against that operand.  The returned z is the last iteration's
    assignment and the centroids its update, so each centroid is the mean of
    the keys z assigns to it.
    """
    k = np.asarray(keys, dtype=F64)
    c = k[np.asarray(init_idx, dtype=np.int64)].copy()
    hist, costs = [], []
    z = np.zeros(k.shape[0], dtype=np.int64)
    for _ in range(n_iters):
        operand = round_to_bf16(c) if bf16_operand else c
        z = kmeans_assign(k, operand)
        c, _ = kmeans_update(k, z, c)
        if keep_history:
            hist.append(c.copy())
            costs.append(clustering_cost(k, z, c))
    return kmeans_finish(z, c, hist, costs)


def kmeans_finish(z, centroids, history=None, costs=None) -> KMeansResult:
    """The cluster layout of a final assignment: member counts, CSR offsets of
    each cluster and the token ids grouped by cluster (ascending inside a
    cluster), the order in which the pool stores the prompt rows."""
    z = np.asarray(z, dtype=np.int64)
    c = np.asarray(centroids, dtype=F64)
    counts = np.bincount(z, minlength=c.shape[0])
    offsets = np.zeros(c.shape[0] + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    perm = np.argsort(z, kind="stable")
    return KMeansResult(z=z, centroids=c, counts=counts, offsets=offsets,
                        perm=perm, history=list(history or []), costs=list(costs or []))


# ---------------------------------------------------------------------------
# decode-stage segments (Section 4.2 decode stage, Algorithm 1 store_cache)
# ---------------------------------------------------------------------------

def segment_mean(rows) -> np.ndarray:
    """Index vector of a temporal segment: the mean of its keys (float64 sum,
    one rounding to float32)."""
    r = np.asarray(rows, dtype=F64)
    return round_to_f32(r.sum(axis=0) / r.shape[0])


def page_units(keys, page_len: int):
    """Page-level index, the coarse-grained baseline of the management ablation
    (Appendix D.3): the tokens are cut into consecutive pages of page_len (the
    last one shorter when page_len does not divide the count), and each page
    is a unit whose index vector is its mean key, computed as a segment mean.
    Returns (reps [n_pages][d], starts [n_pages], sizes [n_pages])."""
    k = np.asarray(keys, dtype=F64)
    n = k.shape[0]
    if page_len < 1:
        raise ValueError("page_len must be >= 1")
    starts = np.arange(0, n, page_len, dtype=np.int64)
    sizes = np.minimum(page_len, n - starts)
    reps = np.stack([segment_mean(k[a:a + z]) for a, z in zip(starts, sizes)])
    return reps, starts, sizes


# ---------------------------------------------------------------------------
# semantic boundary test (Section 4.1 equation for r_t; Algorithm 1 decode loop)
# ---------------------------------------------------------------------------

def query_similarity(q, q_ref) -> float:
    """r = (1/H) * sum over heads of cos(q_ref^h, q^h).

    q, q_ref: [H][d].  The cosine's denominator is clamped at 1e-30, so a
    zero-norm query gives cosine 0 (the paper does not define that case).
    """
    a = np.asarray(q, dtype=F64)
    b = np.asarray(q_ref, dtype=F64)
    num = (a * b).sum(axis=-1)
    den = np.maximum(np.sqrt((a * a).sum(axis=-1)) * np.sqrt((b * b).sum(axis=-1)), 1e-30)
    return float((num / den).mean())


def boundary_fires(r: float, tau: float, first_step: bool) -> bool:
    """A new segment starts at the first step or when r drops strictly below tau."""
    return bool(first_step or r < tau)


def stride_fires(t: int, stride: int) -> bool:
    """The fixed-stride trigger of the retrieval ablation (Appendix D.3): a
    retrieval at the first decode step (t = 1) and then every `stride` steps."""
    return (t - 1) % stride == 0


# ---------------------------------------------------------------------------
# retrieval (Appendix B group-consistent score; Section 3.1 budget; Algorithm 1
# Retrieve)
# ---------------------------------------------------------------------------

def group_scores(q_group, reps, scale: float) -> np.ndarray:
    """A_u = (1/g) * sum_j softmax_u(q_j . rep_u * scale).

    q_group: [g][d] the query heads sharing one KV head; reps: [U][d] the
    index vectors (cluster centroids, then segment means).  The softmax runs
    over all U units, separately for each query head, then the g
    distributions are averaged.
    """
    q = np.asarray(q_group, dtype=F64)
    r = np.asarray(reps, dtype=F64)
    logits = (q @ r.T) * scale
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    p = e / e.sum(axis=1, keepdims=True)
    return p.mean(axis=0)


def select_budget(scores, unit_size, budget: int) -> Tuple[List[int], int]:
    """Top-scoring units whose total token count stays within the budget.

    Units are ranked by score, highest first, equal scores by lower unit id.
    Units are taken in that order until the next one would push the total
    above the budget (prefix stop), so the chosen set is always a prefix of
    the ranking.  Returns (unit ids in rank order, total tokens).
    """
    s = np.asarray(scores, dtype=F64)
    size = np.asarray(unit_size, dtype=np.int64)
    order = sorted(range(s.shape[0]), key=lambda u: (-s[u], u))
    chosen, total = [], 0
    for u in order:
        if total + int(size[u]) > budget:
            break
        chosen.append(u)
        total += int(size[u])
    return chosen, total


def gather_units(pool, unit_start, unit_size, units: Sequence[int]) -> np.ndarray:
    """Rows of the chosen units, in selection order, ascending inside a unit."""
    p = np.asarray(pool)
    idx = [r for u in units for r in range(int(unit_start[u]), int(unit_start[u]) + int(unit_size[u]))]
    if not idx:
        return np.zeros((0,) + p.shape[1:], dtype=F64)
    return np.asarray(p[np.asarray(idx)], dtype=F64)


# ---------------------------------------------------------------------------
# attention (Section 3.1)
# ---------------------------------------------------------------------------

def attention(q, k_rows, v_rows, scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """o_h = softmax(q_h K^T * scale) V for each query head h.

    q: [g][d]; k_rows, v_rows: [n][d].  Returns (o [g][d], lse [g]) where
    lse is the natural log of the softmax denominator including the max
    shift.  With no rows, o is zero and lse is -inf.
    """
    q = np.asarray(q, dtype=F64)
    k = np.asarray(k_rows, dtype=F64)
    v = np.asarray(v_rows, dtype=F64)
    if k.shape[0] == 0:
        return np.zeros((q.shape[0], v.shape[1] if v.ndim == 2 else q.shape[1])), np.full(q.shape[0], -np.inf)
    logits = (q @ k.T) * scale
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    denom = e.sum(axis=1, keepdims=True)
    o = (e / denom) @ v
    lse = (m + np.log(denom))[:, 0]
    return o, lse
