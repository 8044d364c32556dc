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
"""
from __future__ import annotations

from collections import deque
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from .louiskv_oracle import (
    F64, attention, boundary_fires, gather_units, group_scores,
    query_similarity, segment_mean, select_budget, KMeansResult,
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
    scores: Optional[List[np.ndarray]]     # per KV head, when fired
    sel_units: Optional[List[List[int]]]   # per KV head, when fired
    n_sel: List[int]              # per KV head, current KV_critical size
    evicted_unit: Optional[int]   # unit id created at this step, if any
    out: np.ndarray               # [H_q][d]
    lse: np.ndarray               # [H_q]


class GroupDecoder:
    def __init__(self, prefill: PrefillState, n_q_heads: int, budget: int,
                 window: int, seg_len: int, tau: float, mode: str = "anchor",
                 scale: Optional[float] = None, segments: str = "fixed"):
        if mode not in ("prev", "anchor"):
            raise ValueError(mode)
        if segments not in ("fixed", "boundary"):
            raise ValueError(segments)
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
        self.crit_k = [np.zeros((0, self.d)) for _ in range(self.h_kv)]
        self.crit_v = [np.zeros((0, self.d)) for _ in range(self.h_kv)]
        self.crit_units: List[List[int]] = [[] for _ in range(self.h_kv)]
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
        fire = boundary_fires(r, self.tau, first)
        if fire_override is not None:
            fire = bool(fire_override)
        if self.mode == "prev" or fire:
            self.q_ref = q_t.copy()

        scores = sels = None
        if fire:
            scores, sels = [], []
            for h in range(self.h_kv):
                a = group_scores(q_t[h * self.g:(h + 1) * self.g], np.asarray(self.reps[h]), self.scale)
                if select_override is not None:
                    chosen = [int(u) for u in select_override[h]]
                else:
                    chosen, _ = select_budget(a, self.unit_size[h], self.budget)
                kp = np.asarray(self.k_pool[h])
                vp = np.asarray(self.v_pool[h])
                self.crit_k[h] = gather_units(kp, self.unit_start[h], self.unit_size[h], chosen)
                self.crit_v[h] = gather_units(vp, self.unit_start[h], self.unit_size[h], chosen)
                self.crit_units[h] = chosen
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
        for h in range(self.h_kv):
            lk = np.stack([x[1] for x in self.local[h]])
            lv = np.stack([x[2] for x in self.local[h]])
            kk = np.concatenate([self.crit_k[h], lk])
            vv = np.concatenate([self.crit_v[h], lv])
            o, l = attention(q_t[h * self.g:(h + 1) * self.g], kk, vv, self.scale)
            out[h * self.g:(h + 1) * self.g] = o
            lse[h * self.g:(h + 1) * self.g] = l
        return StepRecord(t=self.t, r=r, fire=fire, scores=scores, sel_units=sels,
                          n_sel=[int(x.shape[0]) for x in self.crit_k],
                          evicted_unit=evicted, out=out, lse=lse)
