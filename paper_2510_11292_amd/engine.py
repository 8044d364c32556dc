"""Buffers and call order of the LouisKV path for a batch of slices.

LouisKVEngine owns the device (or pinned-host) tensors of one batch of
(sequence, layer) groups and drives the library calls in the order of the
paper's Algorithm 1:

  prefill()  louiskv_cluster_prefill: k-means per slice, centroids as unit
             index vectors; louiskv_pack_pool: prompt K/V packed cluster by
             cluster into the pool.  With prefill_chunk set,
             louiskv_cluster_prefill_pipelined clusters the slices chunk by
             chunk and writes each chunk's pool rows on a second stream
             while the next chunk is clustered.
  step()     one decode step for every group: louiskv_boundary_check, then
             louiskv_retrieve for the groups that fired (scores see the units
             evicted before this step), louiskv_segment_output (window append,
             oldest-segment eviction), louiskv_sparse_decode_attn over
             [KV_critical : KV_local].  With fixed segments the boundary test
             and the store run as one launch (louiskv_decode_prologue) before
             the retrieval, which does not read what the store writes.  With segments="boundary" the output
             segments are delimited by the fired boundaries (the *_seg and
             louiskv_segment_output_boundary calls, per-slice window state
             on the device).

A call over few slices (a layer at a time, the group views below) runs the
whole step as louiskv_decode_step: the same stages in one launch (bf16; two
in float32) that spreads each slice over many blocks.

With the pool in device memory the engine runs zero-copy by default:
louiskv_retrieve_rows keeps KV_critical as a list of pool rows and
louiskv_sparse_decode_attn_rows reads them from the pool, so a fired step
copies nothing.  A pool in pinned host memory (or zero_copy=False) uses the
dense KV_critical buffers that louiskv_retrieve gathers; for a host pool the
default keeps them as a cache of pool rows (louiskv_retrieve_delta), so a
retrieval moves only the rows the previous selection did not hold.

EngineConfig also selects the ablation baselines of Appendix D.3 and
Appendix B: trigger="stride" (louiskv_fire_every in place of the boundary
test), index="pages" (louiskv_page_prefill in place of the clustering) and
selection="per_head" (louiskv_retrieve_rows_per_head and
louiskv_sparse_decode_attn_rows_per_head).

Python only allocates tensors and passes pointers; every step of the path
runs in the library's kernels.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Optional

import torch

from . import louiskv as L

MAX_UNITS = 8192   # units one slice's retrieval scores (the library's limit)
# a call over at most this many slices runs the decode step as louiskv_decode_step
# (one launch in bf16, each slice spread over many blocks); larger ones use the
# per-stage calls, whose kernels fill the chip with one block per slice
FUSED_STEP_MAX_SLICES = 64
# KV_critical over a host-resident pool: an LRU cache of this many budgets of
# pool rows per slice in HBM (the default; cache_rows overrides it)
HOST_CACHE_BUDGETS = 16


@dataclass(frozen=True)
class EngineConfig:
    n_slices: int
    n_kv_heads: int
    n_q_heads: int
    prompt_len: int
    n_clusters: int
    n_iters: int
    gen_len: int
    seg_len: int
    budget: int
    window: int
    tau: float
    mode: int = L.REF_ANCHOR
    head_dim: int = 128
    segments: str = "fixed"    # "fixed" seg_len-token runs, or "boundary" (seg_len is then the cap)
    # ablation baselines (Appendix D.3, Appendix B); the defaults are the method
    trigger: str = "boundary"  # "boundary" (the query-similarity test) or "stride" (every `stride` steps)
    stride: int = 16
    index: str = "clusters"    # "clusters" (k-means) or "pages" (n_clusters is then the page count)
    page_len: int = 16
    selection: str = "group"   # "group" (group-consistent) or "per_head"
    # boundary segments: a generation can evict up to one segment per step,
    # more units than a slice's retrieval can score (MAX_UNITS).  Such a
    # configuration is refused unless the caller accepts that segments past
    # the limit are dropped; segment_overflow() then reports whether any was.
    allow_unit_overflow: bool = False

    @property
    def n_groups(self) -> int:
        return self.n_slices // self.n_kv_heads

    @property
    def units_needed(self) -> int:
        """Units a slice can reach: clusters plus the segments the window can evict."""
        if self.segments == "boundary":
            return self.n_clusters + max(0, self.gen_len - self.window)   # one segment per step at most
        ev = 0 if self.gen_len <= self.window else (self.gen_len - self.window + self.seg_len - 1) // self.seg_len
        return self.n_clusters + ev

    @property
    def units_cap(self) -> int:
        if self.segments == "boundary":
            return min(self.units_needed, MAX_UNITS)
        ev = 0 if self.gen_len <= self.window else (self.gen_len - self.window + self.seg_len - 1) // self.seg_len
        return self.n_clusters + ev

    @property
    def pool_rows(self) -> int:
        return self.prompt_len + self.gen_len


def config_from_workload(wl, n_groups: Optional[int] = None, mode: int = L.REF_ANCHOR, **kw) -> EngineConfig:
    g = wl.n_groups if n_groups is None else n_groups
    base = dict(n_slices=g * wl.n_kv_heads, n_kv_heads=wl.n_kv_heads, n_q_heads=wl.n_q_heads,
                prompt_len=wl.prompt_len, n_clusters=wl.n_clusters, n_iters=wl.n_iters, gen_len=wl.gen_len,
                seg_len=wl.seg_len, budget=wl.budget, window=wl.window, tau=wl.tau, mode=mode,
                head_dim=wl.head_dim)
    base.update(kw)
    if base.get("index", "clusters") == "pages":
        # the prompt's units are its pages
        base["n_clusters"] = -(-base["prompt_len"] // base.get("page_len", 16))
    return EngineConfig(**base)


class LouisKVEngine:
    def __init__(self, cfg: EngineConfig, dtype: torch.dtype, device="cuda", pool_on_host: bool = False,
                 keep_scores: bool = False, out_dtype: Optional[torch.dtype] = None,
                 zero_copy: Optional[bool] = None, delta: Optional[bool] = None,
                 prefill_chunk: Optional[int] = None, copy_engine: bool = True, fuse_prologue: bool = True,
                 fused_step: Optional[bool] = None, cache_rows: Optional[int] = None):
        self.cfg = cfg
        self.dtype = dtype
        self.device = torch.device(device)
        self.pool_on_host = pool_on_host
        if zero_copy and pool_on_host:
            raise ValueError("zero-copy retrieval reads the pool from device memory; use zero_copy=False")
        self.zero_copy = (not pool_on_host) if zero_copy is None else bool(zero_copy)
        if delta and self.zero_copy:
            raise ValueError("delta transfers fill the KV_critical buffers; they need zero_copy=False")
        # KV_critical as a cache of pool rows: the default for a host-resident pool
        self.delta = (not self.zero_copy and pool_on_host) if delta is None else bool(delta)
        self.delta = self.delta and cfg.budget >= 1
        # cache_rows > budget keeps KV_critical as an LRU cache of that many
        # pool rows per slice (louiskv_retrieve_cached): rows selected again
        # after a few steps away are still resident and need no transfer
        if cache_rows is None and self.delta and pool_on_host:
            cache_rows = min(HOST_CACHE_BUDGETS * max(cfg.budget, 1), cfg.pool_rows, L.CACHE_MAX_ROWS)
        self.cached = cache_rows is not None and int(cache_rows) > max(cfg.budget, 1)
        if self.cached and not self.delta:
            raise ValueError("an LRU cache of pool rows needs delta transfers (zero_copy=False)")
        self.cache_rows = int(cache_rows) if self.cached else max(cfg.budget, 1)
        if cfg.trigger not in ("boundary", "stride") or cfg.stride < 1:
            raise ValueError((cfg.trigger, cfg.stride))
        if cfg.index not in ("clusters", "pages") or cfg.page_len < 1:
            raise ValueError((cfg.index, cfg.page_len))
        if cfg.selection not in ("group", "per_head"):
            raise ValueError(cfg.selection)
        self.per_head = cfg.selection == "per_head"
        # boundary test and fixed-segment store of a step in one launch
        # (louiskv_decode_prologue); with fuse_prologue=False as two calls
        self.fuse_prologue = bool(fuse_prologue)
        if self.per_head and not (self.zero_copy and cfg.segments == "fixed"):
            raise ValueError("per-head selection is built for zero-copy retrieval with fixed segments")
        S, d, cap, G = cfg.n_slices, cfg.head_dim, cfg.units_cap, cfg.n_groups
        # selection lists: one per KV-head slice, or one per query head
        nl = S * (cfg.n_q_heads // cfg.n_kv_heads if self.per_head else 1)
        dev = self.device
        i32 = dict(dtype=torch.int32, device=dev)
        self.reps = torch.zeros(S, cap, d, dtype=torch.float32, device=dev)
        self.unit_start = torch.zeros(S, cap, **i32)
        self.unit_size = torch.zeros(S, cap, **i32)
        self.assign = torch.zeros(S, cfg.prompt_len, **i32)
        self.perm = torch.zeros(S, cfg.prompt_len, **i32)
        if pool_on_host:
            self.k_pool = torch.empty(S, cfg.pool_rows, d, dtype=dtype, pin_memory=True)
            self.v_pool = torch.empty(S, cfg.pool_rows, d, dtype=dtype, pin_memory=True)
        else:
            self.k_pool = torch.empty(S, cfg.pool_rows, d, dtype=dtype, device=dev)
            self.v_pool = torch.empty(S, cfg.pool_rows, d, dtype=dtype, device=dev)
        self.k_local = torch.zeros(S, cfg.window, d, dtype=dtype, device=dev)
        self.v_local = torch.zeros(S, cfg.window, d, dtype=dtype, device=dev)
        if self.zero_copy:
            self.sel_rows = torch.zeros(nl, max(cfg.budget, 1), **i32)
            self.k_buf = self.v_buf = None
        else:
            self.sel_rows = None
            self.k_buf = torch.zeros(S, self.cache_rows, d, dtype=dtype, device=dev)
            self.v_buf = torch.zeros(S, self.cache_rows, d, dtype=dtype, device=dev)
        self.slot_step = torch.full((S, self.cache_rows), -1, **i32) if self.cached else None
        if self.delta:
            self.buf_row = torch.full((S, self.cache_rows), -1, **i32)
            self.slot_list = torch.zeros(S, max(cfg.budget, 1), **i32)
            self.n_fetched = torch.zeros(S, **i32)
        self.sel_units = torch.zeros(nl, cap, **i32)
        self.n_sel_units = torch.zeros(nl, **i32)
        self.n_sel = torch.zeros(nl, **i32)
        self.q_ref = torch.zeros(G, cfg.n_q_heads, d, dtype=dtype, device=dev)
        self.fire = torch.zeros(G, dtype=torch.uint8, device=dev)
        self.r = torch.zeros(G, dtype=torch.float64, device=dev)
        self.out = torch.zeros(G, cfg.n_q_heads, d, dtype=out_dtype or dtype, device=dev)
        self.lse = torch.zeros(G, cfg.n_q_heads, dtype=torch.float32, device=dev)
        self.scores = torch.zeros(nl, cap, dtype=torch.float64, device=dev) if keep_scores else None
        if cfg.segments not in ("fixed", "boundary"):
            raise ValueError(cfg.segments)
        if cfg.units_needed > MAX_UNITS and not cfg.allow_unit_overflow:
            raise ValueError(f"up to {cfg.units_needed} units per slice ({cfg.n_clusters} clusters and the segments "
                             f"of {cfg.gen_len} steps) exceed the {MAX_UNITS} a retrieval scores; segments past "
                             f"the limit would not be attended. Pass allow_unit_overflow=True to accept that and "
                             f"check segment_overflow().")
        self.seg_state = (torch.zeros(S, L.segment_state_ints(cfg.window), **i32)
                          if cfg.segments == "boundary" else None)
        dc = L.BF16 if dtype == torch.bfloat16 else L.F32
        u8 = dict(dtype=torch.uint8, device=dev)
        # prefill_chunk: cluster that many slices at a time and write each
        # chunk's pool rows on a second stream beside the next chunk's clustering
        self.prefill_chunk = None if prefill_chunk is None else max(1, min(int(prefill_chunk), S))
        self.copy_engine = bool(copy_engine)
        if cfg.index == "pages":
            self.ws_prefill = None
            self.prefill_chunk = None
        elif self.prefill_chunk is None:
            self.ws_prefill = torch.empty(L.cluster_prefill_workspace_size(S, cfg.prompt_len, cfg.n_clusters, dc),
                                          **u8)
        else:
            self.ws_prefill = torch.empty(L.cluster_prefill_pipelined_workspace_size(
                self.prefill_chunk, cfg.prompt_len, cfg.n_clusters, dc, pool_on_host, self.copy_engine), **u8)
            n_chunks = -(-S // self.prefill_chunk)
            self.chunk_events = [torch.cuda.Event() for _ in range(n_chunks + 1)]
            for e in self.chunk_events:
                e.record()
            self.copy_stream = torch.cuda.Stream(device=dev)
        g = cfg.n_q_heads // cfg.n_kv_heads
        rows = max(cfg.budget, 1)
        if self.per_head:
            self.ws_retrieve = torch.empty(L.retrieve_rows_workspace_size(nl, cap), **u8)
            self.ws_attn = torch.empty(max(L.sparse_decode_attn_rows_workspace_size(nl, 1, rows, cfg.window), 1),
                                       **u8)
        elif self.zero_copy:
            self.ws_retrieve = torch.empty(L.retrieve_rows_workspace_size(S, cap), **u8)
            self.ws_attn = torch.empty(max(L.sparse_decode_attn_rows_workspace_size(S, g, rows, cfg.window), 1), **u8)
        elif self.delta:
            self.ws_retrieve = torch.empty(L.retrieve_delta_workspace_size(S, cap, rows), **u8)
            self.ws_attn = torch.empty(max(L.sparse_decode_attn_rows_workspace_size(S, g, rows, cfg.window), 1), **u8)
        else:
            self.ws_retrieve = torch.empty(L.retrieve_workspace_size(S, cap, cfg.budget), **u8)
            self.ws_attn = torch.empty(max(L.sparse_decode_attn_workspace_size(S, g, rows, cfg.window), 1), **u8)
        # the whole decode step in one launch (louiskv_decode_step): built for
        # fixed segments over a device pool with the row-list KV_critical and
        # group-consistent selection; fused_step=None uses it for calls over
        # few slices (a layer at a time), True for every call, False never
        # (louiskv_decode_step_cached: the same with the LRU cache of pool
        # rows, in four launches, for device or host pools)
        step_shape_ok = (cfg.segments == "fixed" and cfg.trigger == "boundary" and not self.per_head
                         and cfg.n_q_heads // cfg.n_kv_heads in (1, 2, 4, 8))
        self._fused_cached = step_shape_ok and self.cached
        self._fused_ok = step_shape_ok and ((self.zero_copy and not pool_on_host) or self._fused_cached)
        if fused_step and not self._fused_ok:
            raise ValueError("the fused decode step needs fixed segments, group-consistent selection and either "
                             "zero-copy retrieval over a device pool or an LRU cache of pool rows")
        self.fused_step = fused_step
        self.ws_step = None
        if self._fused_ok and fused_step is not False:
            size = (L.decode_step_cached_workspace_size if self._fused_cached else L.decode_step_workspace_size)
            self.ws_step = torch.zeros(size(S, dc, g, cap, cfg.budget, cfg.window), **u8)
            if self._fused_cached:
                # the selected pool rows, the plan's input
                self.sel_rows_step = torch.zeros(S, cfg.budget, **i32)
        self.t = 0

    def segment_overflow(self) -> bool:
        """True if some evicted segment could not become a unit (the unit table
        was full), so its tokens are no longer attended (boundary segments;
        reads the state's overflow flag, a device-to-host copy)."""
        if self.seg_state is None:
            return False
        return bool((self.seg_state[:, 4] != 0).any())

    def _use_fused_step(self) -> bool:
        if not self._fused_ok or self.fused_step is False:
            return False
        return bool(self.fused_step) or self.cfg.n_slices <= FUSED_STEP_MAX_SLICES

    # ---------------------------------------------------------------- prefill
    def prefill(self, prompt_keys: torch.Tensor, prompt_values: torch.Tensor, init_idx: torch.Tensor,
                iter_events=None, pack_event=None) -> None:
        """k-means of the prompt keys (louiskv_cluster_prefill), then the pool
        write (louiskv_pack_pool).  pack_event, if given, is recorded between
        the two on the current stream."""
        c = self.cfg
        if c.index == "pages":
            L.page_prefill(prompt_keys, c.page_len, self.reps, self.unit_start, self.unit_size, prompt_values,
                           self.k_pool, self.v_pool, pool_on_host=self.pool_on_host)
            if pack_event is not None:
                pack_event.record()
        elif self.prefill_chunk is not None:
            if iter_events is not None or pack_event is not None:
                raise ValueError("the pipelined prefill takes no iteration or pack events")
            L.cluster_prefill_pipelined(prompt_keys, c.n_clusters, c.n_iters, init_idx, self.reps, self.unit_start,
                                        self.unit_size, self.assign, self.perm, prompt_values, self.k_pool,
                                        self.v_pool, self.prefill_chunk, self.chunk_events, self.copy_stream,
                                        pool_on_host=self.pool_on_host, copy_engine=self.copy_engine,
                                        workspace=self.ws_prefill)
        else:
            L.cluster_prefill(prompt_keys, c.n_clusters, c.n_iters, init_idx, self.reps, self.unit_start,
                              self.unit_size, self.assign, self.perm, iter_events=iter_events,
                              workspace=self.ws_prefill)
            if pack_event is not None:
                pack_event.record()
            L.pack_pool(prompt_keys, prompt_values, self.perm, self.k_pool, self.v_pool,
                        pool_on_host=self.pool_on_host)
        if self.seg_state is not None:
            L.segment_state_init(self.seg_state, c.window, c.n_clusters)
        if self.delta:
            self.buf_row.fill_(-1)
        if self.cached:
            self.slot_step.fill_(-1)
        self.t = 0

    # ------------------------------------------------------- layer by layer
    _PER_SLICE = ("reps", "unit_start", "unit_size", "assign", "perm", "k_pool", "v_pool", "k_local", "v_local",
                  "sel_rows", "sel_rows_step", "k_buf", "v_buf", "buf_row", "slot_step", "slot_list",
                  "n_fetched", "sel_units", "n_sel_units", "n_sel", "scores", "seg_state")
    _PER_GROUP = ("q_ref", "fire", "r", "out", "lse")

    def group_view(self, g: int, n: int = 1) -> "LouisKVEngine":
        """An engine over groups g .. g+n-1 alone (one layer of n sequences when
        the groups are ordered layer by layer) that shares this engine's
        storage: its calls read and write the same tensors, so a decode step
        can run layer by layer, as a model runs its layers."""
        import copy
        c = self.cfg
        if n < 1 or not 0 <= g or g + n > c.n_groups:
            raise IndexError((g, n))
        if self.per_head:
            raise ValueError("group views are built for group-consistent selection")
        h = c.n_kv_heads
        v = copy.copy(self)
        v.cfg = dataclasses.replace(c, n_slices=h * n)
        for name in self._PER_SLICE:
            t = getattr(self, name, None)
            if t is not None:
                setattr(v, name, t[g * h:(g + n) * h])
        for name in self._PER_GROUP:
            setattr(v, name, getattr(self, name)[g:g + n])
        # fewer slices per launch can take a larger workspace (split-KV
        # attention partials); the views run one after another and share it
        if not hasattr(self, "_view_ws_attn"):
            self._view_ws_attn = {}
        if n not in self._view_ws_attn:
            gs = c.n_q_heads // h
            rows = max(c.budget, 1)
            if self.zero_copy or self.delta:
                need = L.sparse_decode_attn_rows_workspace_size(h * n, gs, rows, c.window)
            else:
                need = L.sparse_decode_attn_workspace_size(h * n, gs, rows, c.window)
            self._view_ws_attn[n] = (self.ws_attn if need <= self.ws_attn.numel() else
                                     torch.empty(need, dtype=torch.uint8, device=self.device))
        v.ws_attn = self._view_ws_attn[n]
        # the fused step's workspace (counters zero between calls) sized for
        # the view, shared by the views of n groups, which run one at a time
        if self.ws_step is not None:
            if not hasattr(self, "_view_ws_step"):
                self._view_ws_step = {}
            if n not in self._view_ws_step:
                size = (L.decode_step_cached_workspace_size if self._fused_cached else L.decode_step_workspace_size)
                dc = L.BF16 if self.dtype == torch.bfloat16 else L.F32
                self._view_ws_step[n] = torch.zeros(size(h * n, dc, c.n_q_heads // h, c.units_cap, c.budget,
                                                         c.window), dtype=torch.uint8, device=self.device)
            v.ws_step = self._view_ws_step[n]
        return v

    def step_layer_by_layer(self, q_t: torch.Tensor, k_t: torch.Tensor, v_t: torch.Tensor,
                            groups_per_launch: int = 1) -> None:
        """One decode step run in launches of groups_per_launch consecutive
        groups (one layer at a time, the order in which a model produces its
        queries: with the groups ordered layer by layer, groups_per_launch =
        batch size gives one launch sequence per layer); results equal step()."""
        c = self.cfg
        h = c.n_kv_heads
        n = groups_per_launch
        if c.n_groups % n:
            raise ValueError(f"{c.n_groups} groups do not split into launches of {n}")
        if getattr(self, "_views_n", None) != n:
            self._views = [self.group_view(g, n) for g in range(0, c.n_groups, n)]
            self._views_n = n
        for i, v in enumerate(self._views):
            g = i * n
            v.t = self.t
            v.step(q_t[g:g + n], k_t[g * h:(g + n) * h], v_t[g * h:(g + n) * h])
        self.t += 1

    # ---------------------------------------------------------------- decode
    def n_units_before(self, t: int) -> int:
        """Units scorable at decode step t (0-based): clusters plus segments evicted before it."""
        if t == 0:
            return self.cfg.n_clusters
        return self.cfg.n_clusters + L.window_info(t - 1, self.cfg.window, self.cfg.seg_len)[1]

    def step(self, q_t: torch.Tensor, k_t: torch.Tensor, v_t: torch.Tensor) -> None:
        """One decode step: q_t [G][Hq][d], k_t and v_t [S][d]."""
        c = self.cfg
        t = self.t
        if self._use_fused_step():
            if self._fused_cached:
                L.decode_step_cached(q_t, self.q_ref, c.tau, c.mode, t, self.fire, self.r, k_t, v_t, self.k_local,
                                     self.v_local, c.seg_len, self.reps, self.unit_start, self.unit_size,
                                     c.n_clusters, self.k_pool, self.v_pool, c.prompt_len, c.budget, self.k_buf,
                                     self.v_buf, self.buf_row, self.slot_step, self.slot_list, self.sel_units,
                                     self.n_sel_units, self.n_sel, self.sel_rows_step, self.out, self.lse,
                                     n_fetched=self.n_fetched, scores_out=self.scores,
                                     pool_on_host=self.pool_on_host, workspace=self.ws_step)
            else:
                L.decode_step(q_t, self.q_ref, c.tau, c.mode, t, self.fire, self.r, k_t, v_t, self.k_local,
                              self.v_local, c.seg_len, self.reps, self.unit_start, self.unit_size, c.n_clusters,
                              self.k_pool, self.v_pool, c.prompt_len, c.budget, self.sel_units, self.n_sel_units,
                              self.n_sel, self.sel_rows, self.out, self.lse, scores_out=self.scores,
                              workspace=self.ws_step)
            self.t += 1
            return
        fused = self.fuse_prologue and c.trigger == "boundary" and self.seg_state is None
        if c.trigger == "stride":
            L.fire_every(self.fire, t, c.stride)
        elif fused:
            # the store writes only this step's new unit and pool rows, which
            # the retrieval below does not read, so it may come first
            L.decode_prologue(q_t, self.q_ref, c.tau, c.mode, t == 0, self.fire, self.r, k_t, v_t, self.k_local,
                              self.v_local, t, c.seg_len, self.reps, self.unit_start, self.unit_size, c.n_clusters,
                              self.k_pool, self.v_pool, c.prompt_len, pool_on_host=self.pool_on_host)
        else:
            L.boundary_check(q_t, self.q_ref, c.tau, c.mode, t == 0, self.fire, self.r)
        if self.seg_state is not None:
            self._step_boundary_segments(q_t, k_t, v_t)
            return
        if self.per_head:
            L.retrieve_rows_per_head(q_t, c.n_kv_heads, self.reps, self.unit_start, self.unit_size,
                                     self.n_units_before(t), c.budget, self.sel_units, self.n_sel_units, self.n_sel,
                                     self.sel_rows, fire=self.fire, scores_out=self.scores,
                                     workspace=self.ws_retrieve)
        elif self.zero_copy:
            L.retrieve_rows(q_t, c.n_kv_heads, self.reps, self.unit_start, self.unit_size, self.n_units_before(t),
                            c.budget, self.sel_units, self.n_sel_units, self.n_sel, self.sel_rows, fire=self.fire,
                            scores_out=self.scores, workspace=self.ws_retrieve)
        elif self.delta:
            self._retrieve_delta(q_t, self.n_units_before(t), None)
        else:
            L.retrieve(q_t, c.n_kv_heads, self.reps, self.unit_start, self.unit_size, self.n_units_before(t),
                       self.k_pool, self.v_pool, c.budget, self.sel_units, self.n_sel_units, self.n_sel,
                       self.k_buf, self.v_buf, fire=self.fire, pool_on_host=self.pool_on_host,
                       scores_out=self.scores, workspace=self.ws_retrieve)
        if not fused:
            L.segment_output(k_t, v_t, self.k_local, self.v_local, t, c.seg_len, self.reps, self.unit_start,
                             self.unit_size, c.n_clusters, self.k_pool, self.v_pool, c.prompt_len,
                             pool_on_host=self.pool_on_host)
        _, _, n_local, local_start = L.window_info(t, c.window, c.seg_len)
        if self.per_head:
            L.sparse_decode_attn_rows_per_head(q_t, c.n_kv_heads, self.k_pool, self.v_pool, self.sel_rows,
                                               self.n_sel, self.k_local, self.v_local, local_start, n_local,
                                               self.out, self.lse, workspace=self.ws_attn)
        elif self.zero_copy:
            L.sparse_decode_attn_rows(q_t, c.n_kv_heads, self.k_pool, self.v_pool, self.sel_rows, self.n_sel,
                                      self.k_local, self.v_local, local_start, n_local, self.out, self.lse,
                                      workspace=self.ws_attn)
        elif self.delta:
            L.sparse_decode_attn_rows(q_t, c.n_kv_heads, self.k_buf, self.v_buf, self.slot_list, self.n_sel,
                                      self.k_local, self.v_local, local_start, n_local, self.out, self.lse,
                                      workspace=self.ws_attn)
        else:
            L.sparse_decode_attn(q_t, c.n_kv_heads, self.k_buf, self.v_buf, self.n_sel, self.k_local,
                                 self.v_local, local_start, n_local, self.out, self.lse, workspace=self.ws_attn)
        self.t += 1

    def _step_boundary_segments(self, q_t, k_t, v_t) -> None:
        """The rest of step() with boundary-delimited segments: unit counts and
        windows are per slice, kept on the device in seg_state."""
        c = self.cfg
        t = self.t
        # units that can exist before this step: clusters plus one per step
        # since the window first filled
        bound = min(c.units_cap, c.n_clusters + max(0, t - c.window))
        if self.zero_copy:
            L.retrieve_rows_seg(q_t, c.n_kv_heads, self.reps, self.unit_start, self.unit_size, bound,
                                self.seg_state, c.window, c.budget, self.sel_units, self.n_sel_units, self.n_sel,
                                self.sel_rows, fire=self.fire, scores_out=self.scores, workspace=self.ws_retrieve)
        elif self.delta:
            self._retrieve_delta(q_t, bound, self.seg_state)
        else:
            L.retrieve_seg(q_t, c.n_kv_heads, self.reps, self.unit_start, self.unit_size, bound, self.seg_state,
                           c.window, self.k_pool, self.v_pool, c.budget, self.sel_units, self.n_sel_units,
                           self.n_sel, self.k_buf, self.v_buf, fire=self.fire, pool_on_host=self.pool_on_host,
                           scores_out=self.scores, workspace=self.ws_retrieve)
        L.segment_output_boundary(k_t, v_t, self.k_local, self.v_local, t, c.seg_len, self.fire, self.seg_state,
                                  self.reps, self.unit_start, self.unit_size, c.n_clusters, c.n_kv_heads,
                                  self.k_pool, self.v_pool, c.prompt_len, pool_on_host=self.pool_on_host)
        if self.zero_copy:
            L.sparse_decode_attn_rows_seg(q_t, c.n_kv_heads, self.k_pool, self.v_pool, self.sel_rows, self.n_sel,
                                          self.k_local, self.v_local, self.seg_state, t + 1, self.out, self.lse,
                                          workspace=self.ws_attn)
        elif self.delta:
            L.sparse_decode_attn_rows_seg(q_t, c.n_kv_heads, self.k_buf, self.v_buf, self.slot_list, self.n_sel,
                                          self.k_local, self.v_local, self.seg_state, t + 1, self.out, self.lse,
                                          workspace=self.ws_attn)
        else:
            L.sparse_decode_attn_seg(q_t, c.n_kv_heads, self.k_buf, self.v_buf, self.n_sel, self.k_local,
                                     self.v_local, self.seg_state, t + 1, self.out, self.lse, workspace=self.ws_attn)
        self.t += 1

    def _retrieve_delta(self, q_t, n_units: int, seg_state) -> None:
        """Retrieval into KV_critical kept as a cache of pool rows: only the
        selected rows the buffer lacks are copied (the buffer holds the last
        selection, or with cache_rows an LRU set of recently selected rows)."""
        c = self.cfg
        if self.cached:
            L.retrieve_cached(q_t, c.n_kv_heads, self.reps, self.unit_start, self.unit_size, n_units, self.k_pool,
                              self.v_pool, max(c.budget, 1), self.t, self.sel_units, self.n_sel_units, self.n_sel,
                              self.k_buf, self.v_buf, self.buf_row, self.slot_step, self.slot_list, fire=self.fire,
                              seg_state=seg_state, window=c.window, n_fetched=self.n_fetched,
                              pool_on_host=self.pool_on_host, scores_out=self.scores, workspace=self.ws_retrieve)
            return
        L.retrieve_delta(q_t, c.n_kv_heads, self.reps, self.unit_start, self.unit_size, n_units, self.k_pool,
                         self.v_pool, max(c.budget, 1), self.sel_units, self.n_sel_units, self.n_sel, self.k_buf,
                         self.v_buf, self.buf_row, self.slot_list, fire=self.fire, seg_state=seg_state,
                         window=c.window, n_fetched=self.n_fetched, pool_on_host=self.pool_on_host,
                         scores_out=self.scores, workspace=self.ws_retrieve)
