"""The library called from plain C (tests/c_abi/abi_example.c, built by
__graft_entry__.build()): a k-means prefill and a decode loop through
include/louiskv.h alone give the same assignments, centroids and attention
outputs, bit for bit, as the same calls through the Python binding, and the
assignments agree with the oracle; a second C loop over
louiskv_decode_step equals the binding's one-launch step bit for bit."""
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
import synth  # noqa: E402
from parity_utils import check_kmeans_trajectory, gpu_kmeans_states, report, to64  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda"
EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "abi_example")


def test_c_caller_matches_python_binding(tmp_path):
    from paper_2510_11292_amd.engine import LouisKVEngine, config_from_workload
    if not os.path.exists(EXE):
        pytest.fail("tests/c_abi/abi_example is not built (run __graft_entry__.build())")
    wl = synth.get_workload("li-so-32k").replace(prompt_len=1024, n_clusters=32, gen_len=60, budget=256, window=32,
                                                 seg_len=8, n_iters=4)
    data = synth.make_slices(wl, DEV, groups=[(0, 3)])
    S, N, C, T = data.n_slices, wl.prompt_len, wl.n_clusters, wl.gen_len
    G, HQ = 1, wl.n_q_heads

    def raw(t):
        return t.detach().contiguous().cpu().view(torch.int16).numpy().tobytes() if t.dtype == torch.bfloat16 \
            else t.detach().contiguous().cpu().numpy().tobytes()
    (tmp_path / "meta.txt").write_text(f"{S} {N} {C} {wl.n_iters} {T} {wl.window} {wl.seg_len} {wl.budget} {G} "
                                       f"{HQ} {wl.n_kv_heads} {wl.tau!r}\n")
    for name, t in (("keys", data.prompt_keys), ("values", data.prompt_values), ("init", data.init_idx),
                    ("queries", data.queries), ("gen_keys", data.gen_keys), ("gen_values", data.gen_values)):
        (tmp_path / f"{name}.bin").write_bytes(raw(t))
    print(f"running {EXE}", flush=True)
    r = subprocess.run([EXE, str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    cfg = config_from_workload(wl, n_groups=1)
    # the C caller runs the per-stage calls, so the engine does too (not the
    # one-launch step it takes by default for a single group)
    eng = LouisKVEngine(cfg, torch.bfloat16, DEV, out_dtype=torch.float32, fuse_prologue=False, fused_step=False)
    eng.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    outs = []
    for t in range(T):
        eng.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        outs.append(eng.out.clone())
    torch.cuda.synchronize()
    cap = cfg.units_cap
    c_assign = np.frombuffer((tmp_path / "out_assign.bin").read_bytes(), dtype=np.int32).reshape(S, N)
    c_reps = np.frombuffer((tmp_path / "out_reps.bin").read_bytes(), dtype=np.float32).reshape(S, cap, 128)
    c_out = np.frombuffer((tmp_path / "out_attn.bin").read_bytes(), dtype=np.float32).reshape(T, G, HQ, 128)
    assert np.array_equal(c_assign, eng.assign.cpu().numpy())
    assert np.array_equal(c_reps, eng.reps.cpu().numpy())
    assert np.array_equal(c_out, torch.stack(outs).cpu().numpy())
    # the C loop over louiskv_decode_step: the binding's one-launch step bit
    # for bit, the per-stage calls up to the summation order of the attention
    c_step = np.frombuffer((tmp_path / "out_attn_step.bin").read_bytes(), dtype=np.float32).reshape(T, G, HQ, 128)
    eng2 = LouisKVEngine(cfg, torch.bfloat16, DEV, out_dtype=torch.float32, fused_step=True)
    eng2.prefill(data.prompt_keys, data.prompt_values, data.init_idx)
    outs2 = []
    for t in range(T):
        eng2.step(data.queries[t], data.gen_keys[t], data.gen_values[t])
        outs2.append(eng2.out.clone())
    torch.cuda.synchronize()
    assert np.array_equal(c_step, torch.stack(outs2).cpu().numpy())
    assert np.abs(c_step - c_out).max() <= 1e-5 * max(1.0, float(np.abs(c_out).max()))
    # and the clustering is the oracle's: equal, or a run whose every
    # iteration is an exact argmin and exact means up to excused near-ties
    from paper_2510_11292_amd import louiskv
    states = gpu_kmeans_states(louiskv, data.prompt_keys, data.init_idx, C)
    excused = 0
    for s in range(S):
        k64, init = to64(data.prompt_keys[s]), data.init_idx[s].cpu().numpy()
        res = oracle.kmeans(k64, init, wl.n_iters, True)
        if not np.array_equal(c_assign[s], res.z):
            excused += check_kmeans_trajectory(k64, init, wl.n_iters, True, lambda it: tuple(x[s] for x in states(it)))
    report("C caller k-means", dict(excused=excused), bound=max(2, S * N * wl.n_iters // 10000),
           of="assignment near-ties")
