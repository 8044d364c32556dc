#!/usr/bin/env python
"""Synthetic ablations of the LouisKV decode path on one MI355X.

The paper's ablations (Section 5.4, Appendix D.3 and D.4, Appendix B) compare
the method with a fixed-stride trigger, a page-level index, per-head selection
and other thresholds, on models and datasets that are not available here.
This runs the same variants of the GPU path on the seeded synthetic workloads
and reports, per variant, what can be measured without a model:

  fire_rate         retrievals per (group, step)
  mass_recall       the share of each query head's dense attention probability
                    (over every token so far) that falls on the attended rows,
                    KV_critical plus the local window; mean and 10th percentile
                    over sampled slices, heads and steps
  topb_overlap      |selected pool rows  and  dense top-B pool rows| / B, with
                    the dense ranking averaged over the KV head's query group
                    (per query head for per-head selection)
  decode_steps_per_s  the decode loop of all layers as one HIP graph

Dense probabilities are computed in float32 with torch on sampled slices (an
evaluation of the selections, outside the path).  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# name -> EngineConfig overrides (tau, trigger, stride, index, page_len, seg_len, selection, mode); the
# page-level baseline uses 16-token pages on both sides (prompt pages and output segments)
VARIANTS = {
    "louiskv": {},
    "tau=0.5": {"tau": 0.5},
    "tau=0.7": {"tau": 0.7},
    "tau=0.8": {"tau": 0.8},
    "tau=0.95": {"tau": 0.95},
    "prev-query reference": {"mode": 0},
    "fixed stride 5": {"trigger": "stride", "stride": 5},
    "fixed stride 16": {"trigger": "stride", "stride": 16},
    "per-head selection": {"selection": "per_head"},
    "pages 16": {"index": "pages", "page_len": 16, "seg_len": 16},
    "every-step clusters": {"trigger": "stride", "stride": 1},
    "every-step pages 16": {"trigger": "stride", "stride": 1, "index": "pages", "page_len": 16, "seg_len": 16},
}


def log(msg: str) -> None:
    print(f"[ablations] {msg}", file=sys.stderr, flush=True)


def step_quality(eng, data, t, n_eval, topb):
    """(mass recall per evaluated head [n], top-B overlap per selection list [m])
    after decode step t for the first n_eval slices."""
    import torch
    from paper_2510_11292_amd import louiskv as L
    c = eng.cfg
    g = c.n_q_heads // c.n_kv_heads
    H = c.n_kv_heads
    d = c.head_dim
    _, n_ev, n_local, local_start = L.window_info(t, c.window, c.seg_len)
    n_pool = c.prompt_len + n_ev * c.seg_len           # pool rows holding a token so far
    S = n_eval
    kp = eng.k_pool[:S, :n_pool].float()
    ring = [(local_start + i) % c.window for i in range(n_local)]
    kl = eng.k_local[:S, ring].float()
    q = data.queries[t, :S // H].float().reshape(S, g, d)
    scale = 1.0 / d ** 0.5
    lp = torch.bmm(kp, q.transpose(1, 2).contiguous()) * scale        # [S][n_pool][g]
    ll = torch.bmm(kl, q.transpose(1, 2).contiguous()) * scale        # [S][n_local][g]
    lse = torch.logsumexp(torch.cat([lp, ll], dim=1), dim=1)          # [S][g]
    pp = torch.exp(lp - lse[:, None, :])                              # probabilities over pool rows
    p_local = torch.exp(ll - lse[:, None, :]).sum(1)                  # [S][g]
    per_head = eng.per_head
    nl = S * g if per_head else S
    rows = eng.sel_rows[:nl].long()
    n_sel = eng.n_sel[:nl]
    valid = torch.arange(rows.shape[1], device=rows.device)[None, :] < n_sel[:, None]
    rows = torch.where(valid, rows.clamp(0, n_pool - 1), 0)
    if per_head:
        # list s*g + j belongs to head j of slice s
        pj = pp.permute(0, 2, 1).reshape(S * g, n_pool)               # [S*g][n_pool]
        got = (torch.gather(pj, 1, rows) * valid).sum(1).reshape(S, g)
        rank_p = pj
    else:
        got = torch.stack([(torch.gather(pp[:, :, j], 1, rows) * valid).sum(1) for j in range(g)], dim=1)
        rank_p = pp.mean(2)                                            # group-averaged
    recall = (got + p_local).reshape(-1)
    k = min(topb, n_pool)
    top = torch.topk(rank_p, k, dim=1).indices
    hit = torch.zeros_like(rank_p, dtype=torch.bool)
    hit.scatter_(1, top, True)
    sel_hit = torch.gather(hit, 1, rows) & valid
    overlap = sel_hit.sum(1).float() / k
    return recall, overlap


def run_variant(name, over, wl, data, args):
    import torch
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    from paper_2510_11292_amd import louiskv as L
    kw = dict(over)
    mode = kw.pop("mode", L.REF_ANCHOR)
    cfg = config_from_workload(wl, mode=mode, **kw)
    dtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    eng = LouisKVEngine(cfg, dtype, "cuda", zero_copy=True)
    n_eval = min(args.eval_slices, cfg.n_slices) // cfg.n_kv_heads * cfg.n_kv_heads
    # quality pass: eager steps, evaluated every `metric_every` steps
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    fires = 0
    recalls, overlaps = [], []
    for t in range(wl.gen_len):
        eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        fires += int(eng.fire.sum())
        if t % args.metric_every == 0 or t == wl.gen_len - 1:
            r, o = step_quality(eng, data, t, n_eval, cfg.budget)
            recalls.append(r)
            overlaps.append(o)
    torch.cuda.synchronize()
    rec = torch.cat(recalls)
    ovl = torch.cat(overlaps)
    # speed pass: the whole decode loop as one graph after a fresh prefill
    def decode_all():
        for t in range(wl.gen_len):
            eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
    graph = torch.cuda.CUDAGraph()
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    torch.cuda.synchronize()
    eng.t = 0
    with torch.cuda.graph(graph):
        decode_all()
    ms = 0.0
    for _ in range(args.reps):
        eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        ms += e0.elapsed_time(e1)
    ms /= args.reps
    out = {
        "variant": name, "config": {k: v for k, v in over.items()},
        "fire_rate": fires / (wl.gen_len * cfg.n_groups),
        "mass_recall_mean": float(rec.mean()), "mass_recall_p10": float(torch.quantile(rec, 0.1)),
        "topb_overlap": float(ovl.mean()),
        "decode_steps_per_s": wl.gen_len / (ms / 1e3),
    }
    del graph, eng
    torch.cuda.empty_cache()
    log(f"{name:24s} fire {out['fire_rate']:.3f}  recall {out['mass_recall_mean']:.4f} "
        f"(p10 {out['mass_recall_p10']:.4f})  top-B overlap {out['topb_overlap']:.3f}  "
        f"{out['decode_steps_per_s']:.0f} steps/s")
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="li-so-32k")
    ap.add_argument("--gen-len", type=int, default=0, help="decode steps (default: the workload's)")
    ap.add_argument("--budget", type=int, default=0, help="retrieval budget B (default: the workload's)")
    ap.add_argument("--variants", default="", help="comma-separated subset of the variant names")
    ap.add_argument("--eval-slices", type=int, default=16, help="slices whose selections are evaluated")
    ap.add_argument("--metric-every", type=int, default=1, help="evaluate every this many steps")
    ap.add_argument("--reps", type=int, default=2)
    args = ap.parse_args()

    import torch
    import synth
    if not torch.cuda.is_available():
        print("ablations.py needs a GPU", file=sys.stderr)
        return 2
    wl = synth.get_workload(args.workload)
    if args.gen_len:
        wl = wl.replace(gen_len=args.gen_len)
    if args.budget:
        wl = wl.replace(budget=args.budget)
    if wl.pool_on_host:
        print("ablations.py evaluates device-resident pools (zero-copy selections)", file=sys.stderr)
        return 2
    names = [n.strip() for n in args.variants.split(",") if n.strip()] or list(VARIANTS)
    t0 = time.time()
    data = synth.make_slices(wl, "cuda")
    torch.cuda.synchronize()
    log(f"inputs for {data.n_slices} slices in {time.time() - t0:.1f}s")
    results = [run_variant(n, VARIANTS[n], wl, data, args) for n in names]
    print(json.dumps({
        "workload": wl.name, "decode_steps": wl.gen_len, "budget": wl.budget, "window": wl.window,
        "segment": wl.seg_len, "eval_slices": args.eval_slices, "metric_every": args.metric_every,
        "data": "synthetic", "variants": results,
    }), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
