"""The decode loop of Algorithm 1 for one (sequence, layer) group, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per decode step t, in the order of Algorithm 1's decode phase:
  1. boundary test: r_t from the query heads of the layer (Section 4.1); a new
     segment starts at t = 1 or when r_t < tau.  The reference query is the
     previous step's query (mode "prev", the paper's equation) or the query
     of the last boundary (mode "anchor");
  2. on a boundary, Retrieve for every KV head of the group: group-consistent
     scores over the units evicted so far (Appendix B), budgeted selection,
     gather of the selected rows into KV_critical;
  3. store_cache for the decode stage: the new (k_t, v_t) enters the local
     window.  If the window already holds `window` tokens, its oldest
     segment leaves first: its mean key becomes a new unit's index vector and
     its rows are appended to the pool (Section 4.2 decode stage).  Segments
     are either fixed runs of `seg_len` tokens (segments="fixed") or
     delimited by the boundaries of step 1 (segments="boundary": Section 4.2
     partitions the generated KV at the semantic boundaries of Section 4.1;
     a segment also closes once it holds `seg_len` tokens, so that a full
     window always holds a closed segment, and seg_len < window is required);
  4. attention of each query head over [KV_critical : KV_local], the current
     token included.
KV_critical is kept unchanged between boundaries.

Ablation baselines (Appendix D.3, Appendix B): a fixed-stride trigger in place
of the boundary test, a page-level index in place of the prompt clusters
(prefill_state_from_pages), and per-head selection in place of the
group-consistent one.
"""
from __future__ import annotations

from collections import deque
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from .louiskv_oracle import (
    F64, attention, boundary_fires, gather_units, group_scores, page_units,
    query_similarity, segment_mean, select_budget, stride_fires, KMeansResult,
)


@dataclass
class PrefillState:
    """State after prefill for the KV heads of one group (lists indexed by KV head)."""
    reps: List[np.ndarray]         # [C][d] centroids (float64 holding float32 values)
    unit_start: List[np.ndarray]   # [C] first pool row of each cluster
    unit_size: List[np.ndarray]    # [C] member count of each cluster
    k_pool: List[np.ndarray]       # [P][d] prompt keys, cluster-contiguous
    v_pool: List[np.ndarray]       # [P][d] prompt values, same order


def prefill_state_from_kmeans(prompt_keys: Sequence, prompt_values: Sequence,
                              results: Sequence[KMeansResult]) -> PrefillState:
    """Pack each KV head's prompt rows cluster by cluster (the unified pool)."""
    reps, starts, sizes, kp, vp = [], [], [], [], []
    for k, v, res in zip(prompt_keys, prompt_values, results):
        k = np.asarray(k, dtype=F64)
        v = np.asarray(v, dtype=F64)
        reps.append(np.asarray(res.centroids, dtype=F64))
        starts.append(np.asarray(res.offsets[:-1], dtype=np.int64))
        sizes.append(np.asarray(res.counts, dtype=np.int64))
        kp.append(k[res.perm])
        vp.append(v[res.perm])
    return PrefillState(reps, starts, sizes, kp, vp)


def prefill_state_from_pages(prompt_keys: Sequence, prompt_values: Sequence, page_len: int) -> PrefillState:
    """The page-level baseline's prefill (Appendix D.3): no clustering; the
    pool holds the prompt in token order and each page of page_len tokens is
    a unit indexed by its mean key."""
    reps, starts, sizes, kp, vp = [], [], [], [], []
    for k, v in zip(prompt_keys, prompt_values):
        k = np.asarray(k, dtype=F64)
        r, a, z = page_units(k, page_len)
        reps.append(r)
        starts.append(a)
        sizes.append(z)
        kp.append(k)
        vp.append(np.asarray(v, dtype=F64))
    return PrefillState(reps, starts, sizes, kp, vp)


def head_scores(q_t, head: int, reps, scale: float) -> np.ndarray:
    """Per-head selection (the baseline that group-consistent selection
    replaces, Appendix B): query head `head` ranks the units of its KV head by
    its own softmax alone, i.e. the group score with a group of one."""
    return group_scores(np.asarray(q_t, dtype=F64)[head:head + 1], reps, scale)


def opens_segment(fire: bool, gen: int, open_first: Optional[int], seg_max: int) -> bool:
    """Boundary-delimited segments: token `gen` starts a new segment when there
    is no open one, when this step is a semantic boundary (Section 4.1, the
    is_new_segment of Algorithm 1), or when the open segment (first token
    open_first) already holds seg_max tokens."""
    return open_first is None or fire or gen - open_first >= seg_max


@dataclass
class StepRecord:
    t: int
    r: float                      # NaN at t = 1
    fire: bool
    scores: Optional[List[np.ndarray]]     # per selection list, when fired
    sel_units: Optional[List[List[int]]]   # per selection list, when fired
    n_sel: List[int]              # per selection list, current KV_critical size
    # (a selection list is a KV head; with selection="per_head" a query head)
    evicted_unit: Optional[int]   # unit id created at this step, if any
    out: np.ndarray               # [H_q][d]
    lse: np.ndarray               # [H_q]


class GroupDecoder:
    def __init__(self, prefill: PrefillState, n_q_heads: int, budget: int,
                 window: int, seg_len: int, tau: float, mode: str = "anchor",
                 scale: Optional[float] = None, segments: str = "fixed",
                 trigger: str = "boundary", stride: int = 16, selection: str = "group"):
        """trigger="stride" replaces the boundary test's decision by a
        retrieval every `stride` steps (r is still computed and the reference
        query still follows `mode`); selection="per_head" gives every query
        head its own selection and KV_critical (the ablation baselines of
        Appendix D.3 and Appendix B)."""
        if mode not in ("prev", "anchor"):
            raise ValueError(mode)
        if segments not in ("fixed", "boundary"):
            raise ValueError(segments)
        if trigger not in ("boundary", "stride") or stride < 1:
            raise ValueError((trigger, stride))
        if selection not in ("group", "per_head"):
            raise ValueError(selection)
        self.trigger, self.stride, self.selection = trigger, stride, selection
        if segments == "boundary" and not 1 <= seg_len < window:
            raise ValueError("boundary segments need 1 <= seg_len < window")
        self.segments = segments
        self.seg_first = deque()   # boundary mode: first generation index of each segment in the window
        self.h_kv = len(prefill.reps)
        self.g = n_q_heads // self.h_kv
        self.d = prefill.reps[0].shape[1]
        self.budget, self.window, self.seg_len = budget, window, seg_len
        self.tau, self.mode = tau, mode
        self.scale = 1.0 / np.sqrt(self.d) if scale is None else scale
        self.reps = [list(r) for r in prefill.reps]
        self.unit_start = [list(int(x) for x in s) for s in prefill.unit_start]
        self.unit_size = [list(int(x) for x in s) for s in prefill.unit_size]
        self.n_prompt = prefill.k_pool[0].shape[0]
        self.k_pool = [list(np.asarray(k, dtype=F64)) for k in prefill.k_pool]
        self.v_pool = [list(np.asarray(v, dtype=F64)) for v in prefill.v_pool]
        self.local = [deque() for _ in range(self.h_kv)]   # (gen index, k, v)
        # one KV_critical per selection list: per KV head, or per query head
        n_lists = self.h_kv * (self.g if selection == "per_head" else 1)
        self.crit_k = [np.zeros((0, self.d)) for _ in range(n_lists)]
        self.crit_v = [np.zeros((0, self.d)) for _ in range(n_lists)]
        self.crit_units: List[List[int]] = [[] for _ in range(n_lists)]
        self.q_ref = None
        self.t = 0
        self.n_evicted = 0

    def n_units(self) -> int:
        return len(self.reps[0])

    def step(self, q_t, k_t, v_t, fire_override: Optional[bool] = None,
             select_override: Optional[Sequence[Sequence[int]]] = None) -> StepRecord:
        """Advance one decode step.  q_t [H_q][d]; k_t, v_t [H_kv][d].

        fire_override / select_override let a checker adopt the other side's
        decision where the two differ only inside a near-tie.
        """
        q_t = np.asarray(q_t, dtype=F64)
        k_t = np.asarray(k_t, dtype=F64)
        v_t = np.asarray(v_t, dtype=F64)
        self.t += 1
        first = self.t == 1
        r = float("nan") if first else query_similarity(q_t, self.q_ref)
        if self.trigger == "stride":
            fire = stride_fires(self.t, self.stride)
        else:
            fire = boundary_fires(r, self.tau, first)
        if fire_override is not None:
            fire = bool(fire_override)
        if self.mode == "prev" or fire:
            self.q_ref = q_t.copy()

        scores = sels = None
        if fire:
            scores, sels = [], []
            per_head = self.selection == "per_head"
            for li in range(len(self.crit_k)):
                h = li // self.g if per_head else li
                reps = np.asarray(self.reps[h])
                if per_head:
                    a = head_scores(q_t, li, reps, self.scale)
                else:
                    a = group_scores(q_t[h * self.g:(h + 1) * self.g], reps, self.scale)
                if select_override is not None:
                    chosen = [int(u) for u in select_override[li]]
                else:
                    chosen, _ = select_budget(a, self.unit_size[h], self.budget)
                kp = np.asarray(self.k_pool[h])
                vp = np.asarray(self.v_pool[h])
                self.crit_k[li] = gather_units(kp, self.unit_start[h], self.unit_size[h], chosen)
                self.crit_v[li] = gather_units(vp, self.unit_start[h], self.unit_size[h], chosen)
                self.crit_units[li] = chosen
                scores.append(a)
                sels.append(chosen)

        evicted = None
        gen = self.t - 1                      # generation index of this step's token
        new_segment = False
        if self.segments == "boundary":
            new_segment = opens_segment(fire, gen, self.seg_first[-1] if self.seg_first else None, self.seg_len)
        if len(self.local[0]) >= self.window:
            evicted = self.n_units()
            if self.segments == "fixed":
                n_leave = self.seg_len
            else:
                first = self.seg_first.popleft()
                n_leave = (self.seg_first[0] if self.seg_first else gen) - first
            for h in range(self.h_kv):
                seg = [self.local[h].popleft() for _ in range(n_leave)]
                seg_k = np.stack([s[1] for s in seg])
                seg_v = np.stack([s[2] for s in seg])
                self.reps[h].append(segment_mean(seg_k))
                self.unit_start[h].append(self.n_prompt + seg[0][0])
                self.unit_size[h].append(n_leave)
                self.k_pool[h].extend(list(seg_k))
                self.v_pool[h].extend(list(seg_v))
            self.n_evicted += 1
        if new_segment:
            self.seg_first.append(gen)
        for h in range(self.h_kv):
            self.local[h].append((gen, k_t[h], v_t[h]))

        out = np.zeros((self.h_kv * self.g, self.d))
        lse = np.zeros(self.h_kv * self.g)
        per_head = self.selection == "per_head"
        for li in range(len(self.crit_k)):
            h = li // self.g if per_head else li
            heads = slice(li, li + 1) if per_head else slice(h * self.g, (h + 1) * self.g)
            lk = np.stack([x[1] for x in self.local[h]])
            lv = np.stack([x[2] for x in self.local[h]])
            kk = np.concatenate([self.crit_k[li], lk])
            vv = np.concatenate([self.crit_v[li], lv])
            o, l = attention(q_t[heads], kk, vv, self.scale)
            out[heads] = o
            lse[heads] = l
        return StepRecord(t=self.t, r=r, fire=fire, scores=scores, sel_units=sels,
                          n_sel=[int(x.shape[0]) for x in self.crit_k],
                          evicted_unit=evicted, out=out, lse=lse)
