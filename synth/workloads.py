"""The five synthetic workloads and their fixed parameters.

Shapes follow the paper's efficiency scenarios (Section 5.3: 32K-in/512-out,
500-in/16K-out, 32K-in/16K-out at batch 4) on a Llama-3.1-8B-like attention
geometry (32 layers, 8 KV heads, 32 query heads, head dim 128), plus a tiny
CPU-scale case and a 131K-token host-resident stress case.  Parameters the
paper leaves open are fixed here: local window W = 128 tokens (the paper's
short-input long-output setting, Section 5.2), no sink tokens, boundary
threshold 0.9, 32-token output segments.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    dtype: str            # "f32" or "bf16": storage type of keys, values, queries
    batch: int
    prompt_len: int       # P
    n_clusters: int       # C (also the number of true centres of the key process)
    n_iters: int          # Lloyd iterations
    gen_len: int          # T decode steps
    seg_len: int          # tokens per output segment
    budget: int           # B retrieved tokens per KV head
    window: int           # W local tokens kept on the GPU
    tau: float            # boundary threshold
    p_jump: float         # probability of a fresh query per step
    pool_on_host: bool    # the full KV pool lives in pinned host memory

    @property
    def group_size(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def n_groups(self) -> int:
        """(sequence, layer) pairs: the granularity of the boundary decision."""
        return self.batch * self.n_layers

    @property
    def n_slices(self) -> int:
        """(sequence, layer, KV head) triples: the granularity of clustering."""
        return self.n_groups * self.n_kv_heads

    @property
    def n_evicted_segments(self) -> int:
        if self.gen_len <= self.window:
            return 0
        return (self.gen_len - self.window + self.seg_len - 1) // self.seg_len

    @property
    def units_cap(self) -> int:
        return self.n_clusters + self.n_evicted_segments

    @property
    def pool_rows(self) -> int:
        return self.prompt_len + self.gen_len

    def replace(self, **kw) -> "Workload":
        return replace(self, **kw)


_COMMON = dict(n_kv_heads=8, n_q_heads=32, head_dim=128, n_iters=10,
               seg_len=32, window=128, tau=0.9)

WORKLOADS = {
    "tiny-4k": Workload(name="tiny-4k", n_layers=1, dtype="f32", batch=1,
                        prompt_len=4096, n_clusters=64, gen_len=256,
                        budget=512, p_jump=1 / 64, pool_on_host=False,
                        **_COMMON),
    "li-so-32k": Workload(name="li-so-32k", n_layers=32, dtype="bf16", batch=1,
                          prompt_len=32768, n_clusters=1024, gen_len=128,
                          budget=2048, p_jump=1 / 64, pool_on_host=False,
                          **_COMMON),
    "si-lo-16k": Workload(name="si-lo-16k", n_layers=32, dtype="bf16", batch=1,
                          prompt_len=1024, n_clusters=32, gen_len=16384,
                          budget=2048, p_jump=1 / 128, pool_on_host=False,
                          **_COMMON),
    "li-lo-32k-b4": Workload(name="li-lo-32k-b4", n_layers=32, dtype="bf16",
                             batch=4, prompt_len=32768, n_clusters=1024,
                             gen_len=16384, budget=4096, p_jump=1 / 64,
                             pool_on_host=False, **_COMMON),
    "host-131k": Workload(name="host-131k", n_layers=32, dtype="bf16", batch=1,
                          prompt_len=131072, n_clusters=4096, gen_len=8192,
                          budget=4096, p_jump=1 / 64, pool_on_host=True,
                          **_COMMON),
}

ORDER = ["tiny-4k", "li-so-32k", "si-lo-16k", "li-lo-32k-b4", "host-131k"]


def get_workload(name_or_index) -> Workload:
    if isinstance(name_or_index, int):
        return WORKLOADS[ORDER[name_or_index]]
    return WORKLOADS[name_or_index]


def tiny_workload(base: str = "tiny-4k", **kw) -> Workload:
    """A scaled-down variant of a workload, for CPU-seconds tests."""
    return WORKLOADS[base].replace(**kw)
