"""Seeded generators for keys, values, queries and k-means initial indices.

Recipe (per (sequence, layer, KV head) slice, each drawn from its own seeded
generator so any slice can be regenerated alone):

* keys: M = C true centres ~ N(0, I_d); a Markov chain over centres (start
  uniform; each token keeps the previous centre with probability 0.9, else
  draws a uniform one, possibly the same); key = centre[z] + 0.3 * N(0, I_d);
  channels 0-3 are then scaled by 8 (outlier channels).  The first P tokens
  are the prompt; the chain continues for the T generated tokens.
* values: N(0, 1) i.i.d.
* queries, per (sequence, layer), all query heads: q_1 ~ N(0, I); afterwards
  q_t = 0.97 q_{t-1} + 0.24 e_t, or q_t = e_t (a fresh draw) at a jump.  Jumps
  happen with probability p_jump per step and are shared by every layer and
  head of a sequence.
* storage: values are drawn in fp32 and rounded once to the workload's dtype
  (bf16 round-to-nearest-even via torch).
* k-means initial indices: the first C entries of a seeded permutation of the
  P prompt positions.

Values drawn on a CUDA device differ from values drawn on the CPU (different
generator engines); every comparison hands the same tensors to both sides.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Sequence

import torch

from .workloads import Workload

BASE_SEED = 251011292
_MASK = (1 << 64) - 1

# stream tags
_TAG_CENTRES, _TAG_CHAIN_STAY, _TAG_CHAIN_DRAW, _TAG_KEY_NOISE, _TAG_VALUES = 1, 2, 3, 4, 5
_TAG_QUERY_NOISE, _TAG_JUMPS, _TAG_INIT = 6, 7, 8


def _splitmix64(x: int) -> int:
    x = (x + 0x9E3779B97F4A7C15) & _MASK
    z = x
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def seed_for(*parts: int) -> int:
    """Deterministic 63-bit seed from a tuple of small integers."""
    h = BASE_SEED
    for p in parts:
        h = _splitmix64(h ^ (int(p) & _MASK))
    return h & ((1 << 63) - 1)


def _gen(device, *parts) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed_for(*parts))
    return g


def _wl_id(wl: Workload) -> int:
    return sum((i + 1) * ord(c) for i, c in enumerate(wl.name))


def storage_dtype(wl: Workload) -> torch.dtype:
    return torch.float32 if wl.dtype == "f32" else torch.bfloat16


def slice_keys_values(wl: Workload, seq: int, layer: int, kvh: int,
                      device="cpu", n_tokens: Optional[int] = None):
    """Keys and values of one slice, prompt first then generated tokens.

    Returns two tensors [n_tokens][d] in the workload's storage dtype, with
    n_tokens = P + T unless given.
    """
    n = wl.prompt_len + wl.gen_len if n_tokens is None else n_tokens
    d, m = wl.head_dim, wl.n_clusters
    wid = _wl_id(wl)
    centres = torch.randn(m, d, generator=_gen(device, wid, seq, layer, kvh, _TAG_CENTRES),
                          device=device, dtype=torch.float32)
    stay = torch.rand(n, generator=_gen(device, wid, seq, layer, kvh, _TAG_CHAIN_STAY),
                      device=device) < 0.9
    stay[0] = False
    draw = torch.randint(0, m, (n,), generator=_gen(device, wid, seq, layer, kvh, _TAG_CHAIN_DRAW),
                         device=device)
    pos = torch.arange(n, device=device)
    last_move = torch.where(stay, torch.zeros_like(pos), pos).cummax(0).values
    z = draw[last_move]
    keys = centres[z] + 0.3 * torch.randn(n, d, generator=_gen(device, wid, seq, layer, kvh, _TAG_KEY_NOISE),
                                          device=device, dtype=torch.float32)
    keys[:, :4] *= 8.0
    values = torch.randn(n, d, generator=_gen(device, wid, seq, layer, kvh, _TAG_VALUES),
                         device=device, dtype=torch.float32)
    dt = storage_dtype(wl)
    return keys.to(dt), values.to(dt)


def jump_steps(wl: Workload, seq: int, device="cpu", n_steps: Optional[int] = None) -> torch.Tensor:
    """Bool [T]: True where the query process restarts (shared by all layers/heads)."""
    t = wl.gen_len if n_steps is None else n_steps
    u = torch.rand(t, generator=_gen(device, _wl_id(wl), seq, _TAG_JUMPS), device=device)
    j = u < wl.p_jump
    if t > 0:
        j[0] = True  # q_1 is a fresh draw
    return j


def seq_queries(wl: Workload, seq: int, layers: Sequence[int], device="cpu",
                n_steps: Optional[int] = None) -> torch.Tensor:
    """Queries of several layers of one sequence: [T][len(layers)][H_q][d].

    Each layer's noise comes from its own (sequence, layer) generator, so the
    result does not depend on which layers are generated together.
    """
    t_len = wl.gen_len if n_steps is None else n_steps
    layers = list(layers)
    e = torch.empty(t_len, len(layers), wl.n_q_heads, wl.head_dim,
                    device=device, dtype=torch.float32)
    for i, layer in enumerate(layers):
        e[:, i] = torch.randn(t_len, wl.n_q_heads, wl.head_dim,
                              generator=_gen(device, _wl_id(wl), seq, layer, _TAG_QUERY_NOISE),
                              device=device, dtype=torch.float32)
    jumps = jump_steps(wl, seq, device, t_len)
    q = torch.empty_like(e)
    jl = jumps.tolist()
    for t in range(t_len):
        if jl[t]:
            q[t] = e[t]
        else:
            torch.add(0.97 * q[t - 1], e[t], alpha=0.24, out=q[t])
    return q.to(storage_dtype(wl))


def group_queries(wl: Workload, seq: int, layer: int, device="cpu",
                  n_steps: Optional[int] = None) -> torch.Tensor:
    """Queries of one (sequence, layer) for every decode step: [T][H_q][d]."""
    return seq_queries(wl, seq, [layer], device, n_steps)[:, 0]


def init_indices(wl: Workload, seq: int, layer: int, kvh: int) -> torch.Tensor:
    """First C positions of a seeded permutation of the prompt (int32, CPU)."""
    g = _gen("cpu", _wl_id(wl), seq, layer, kvh, _TAG_INIT)
    return torch.randperm(wl.prompt_len, generator=g)[: wl.n_clusters].to(torch.int32)


@dataclass
class SliceData:
    """Inputs for a set of (sequence, layer) groups, all their KV heads.

    Slice s of group index gi and KV head h is s = gi * H_kv + h.
    """
    wl: Workload
    groups: list                   # [(seq, layer)]
    prompt_keys: torch.Tensor      # [S][P][d]
    prompt_values: torch.Tensor    # [S][P][d]
    gen_keys: torch.Tensor         # [T][S][d]
    gen_values: torch.Tensor       # [T][S][d]
    queries: torch.Tensor          # [T][G][H_q][d]
    init_idx: torch.Tensor         # [S][C] int32 (same device)

    @property
    def n_slices(self) -> int:
        return self.prompt_keys.shape[0]


def make_slices(wl: Workload, device="cpu", groups: Optional[Sequence] = None,
                gen_len: Optional[int] = None) -> SliceData:
    """Generate every input for the given (sequence, layer) groups (default: all)."""
    if groups is None:
        groups = [(b, l) for b in range(wl.batch) for l in range(wl.n_layers)]
    groups = list(groups)
    t_len = wl.gen_len if gen_len is None else gen_len
    n_tok = wl.prompt_len + t_len
    dt = storage_dtype(wl)
    s_total = len(groups) * wl.n_kv_heads
    p = wl.prompt_len
    pk = torch.empty(s_total, p, wl.head_dim, dtype=dt, device=device)
    pv = torch.empty_like(pk)
    gk = torch.empty(t_len, s_total, wl.head_dim, dtype=dt, device=device)
    gv = torch.empty_like(gk)
    q = torch.empty(t_len, len(groups), wl.n_q_heads, wl.head_dim, dtype=dt, device=device)
    init = torch.empty(s_total, wl.n_clusters, dtype=torch.int32)
    for gi, (seq, layer) in enumerate(groups):
        for h in range(wl.n_kv_heads):
            s = gi * wl.n_kv_heads + h
            k, v = slice_keys_values(wl, seq, layer, h, device, n_tok)
            pk[s] = k[:p]
            pv[s] = v[:p]
            gk[:, s] = k[p:]
            gv[:, s] = v[p:]
            init[s] = init_indices(wl, seq, layer, h)
    by_seq = {}
    for gi, (seq, layer) in enumerate(groups):
        by_seq.setdefault(seq, []).append((gi, layer))
    for seq, items in by_seq.items():
        qs = seq_queries(wl, seq, [l for _, l in items], device, t_len)
        for i, (gi, _) in enumerate(items):
            q[:, gi] = qs[:, i]
    return SliceData(wl=wl, groups=groups, prompt_keys=pk, prompt_values=pv,
                     gen_keys=gk, gen_values=gv, queries=q, init_idx=init.to(device))
