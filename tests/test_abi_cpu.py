"""The C-ABI library without a GPU: it loads, exports every function the public
header declares, and its host-only logic (status strings, argument validation
that returns before any launch, the local-window rule) behaves as documented."""
import ctypes
import os
import re
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "louiskv.h")
LIB = os.path.join(ROOT, "paper_2510_11292_amd", "liblouiskv.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(louiskv_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("liblouiskv.so is not built; run `python -m paper_2510_11292_amd.build`")
    from paper_2510_11292_amd import louiskv
    return louiskv.load_library()


def test_exports_every_declared_function(lib):
    names = declared_functions()
    assert len(names) >= 13
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (louiskv_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    from paper_2510_11292_amd import louiskv
    assert sorted(louiskv.EXPORTED) == names


def test_version_and_status_strings(lib):
    assert lib.louiskv_abi_version() == 1
    for st in range(7):
        assert lib.louiskv_status_str(st)
    assert lib.louiskv_status_str(99) == b"unknown status"


def test_window_rule_matches_oracle_schedule(lib):
    """The library's window rule gives the eviction steps, live counts and ring
    positions that the oracle's decode loop produces."""
    import oracle
    from paper_2510_11292_amd import louiskv as L
    window, seg = 32, 8
    rng = np.random.default_rng(0)
    p, d, c = 40, 4, 4
    pk = rng.standard_normal((1, p, d))
    res = [oracle.kmeans(pk[0], np.arange(c), 1, False)]
    dec = oracle.GroupDecoder(oracle.prefill_state_from_kmeans(pk, pk, res), n_q_heads=1, budget=8,
                              window=window, seg_len=seg, tau=0.0)
    for t in range(150):
        rec = dec.step(rng.standard_normal((1, d)), rng.standard_normal((1, d)), rng.standard_normal((1, d)))
        ev, n_ev, n_local, start = L.window_info(t, window, seg)
        assert (ev >= 0) == (rec.evicted_unit is not None)
        if ev >= 0:
            assert rec.evicted_unit == c + ev
        assert n_ev == dec.n_evicted
        assert n_local == len(dec.local[0])
        assert start == dec.local[0][0][0] % window
    with pytest.raises(L.LouisKVError):
        L.window_info(0, 30, 8)


def test_validation_errors_return_before_launch(lib):
    """Bad arguments are rejected on the host with the documented status."""
    P = ctypes.c_void_p
    dummy = P(16)
    # NULL keys
    assert lib.louiskv_cluster_prefill(None, 1, 1, 64, 128, 8, 1, dummy, dummy, 8, dummy, dummy, dummy, dummy,
                                       None, None, None, 0, 0, None, dummy, 1 << 30, None) == 1
    # bad dtype
    assert lib.louiskv_cluster_prefill(dummy, 7, 1, 64, 128, 8, 1, dummy, dummy, 8, dummy, dummy, dummy, dummy,
                                       None, None, None, 0, 0, None, dummy, 1 << 30, None) == 3
    # head dim other than 128
    assert lib.louiskv_cluster_prefill(dummy, 1, 1, 64, 64, 8, 1, dummy, dummy, 8, dummy, dummy, dummy, dummy,
                                       None, None, None, 0, 0, None, dummy, 1 << 30, None) == 4
    # more clusters than tokens
    assert lib.louiskv_cluster_prefill(dummy, 1, 1, 64, 128, 65, 1, dummy, dummy, 80, dummy, dummy, dummy, dummy,
                                       None, None, None, 0, 0, None, dummy, 1 << 30, None) == 2
    # workspace too small
    assert lib.louiskv_cluster_prefill(dummy, 1, 1, 64, 128, 8, 1, dummy, dummy, 8, dummy, dummy, dummy, dummy,
                                       None, None, None, 0, 0, None, dummy, 16, None) == 5
    assert b"workspace" in lib.louiskv_last_error()
    # boundary: unknown mode, NULL output
    assert lib.louiskv_boundary_check(dummy, dummy, 1, 4, 32, 128, 0.9, 5, 0, None, dummy, None) == 2
    assert lib.louiskv_boundary_check(dummy, dummy, 1, 4, 32, 128, 0.9, 0, 0, None, None, None) == 1
    # retrieve: too many units, group size over the limit
    args = [dummy, 1, 8, 8, 4, 128, 0.088, dummy, dummy, dummy, 100, 200, dummy, dummy, 1000, 0, 64, None,
            dummy, dummy, dummy, dummy, dummy, None, dummy, 1 << 30, None]
    assert lib.louiskv_retrieve(*args) == 2
    args[10] = 50
    args[4] = 16
    assert lib.louiskv_retrieve(*args) == 4
    # attention: local window overflow
    assert lib.louiskv_sparse_decode_attn(dummy, 1, 8, 8, 4, 128, 0.088, dummy, dummy, dummy, 64, dummy, dummy,
                                          32, 0, 33, dummy, 1, None, dummy, 1 << 30, None) == 2
    # segment output: window not a multiple of the segment
    assert lib.louiskv_segment_output(dummy, dummy, 1, 8, 128, dummy, dummy, 30, 0, 8, dummy, dummy, dummy, 100, 10,
                                      None, None, 0, 0, 0, None) == 2


def test_boundary_segment_calls_validate_on_the_host(lib):
    """The boundary-delimited segment calls refuse a missing state, a cap not
    below the window and a state for a window too small, before any launch."""
    P = ctypes.c_void_p
    dummy = P(16)
    assert lib.louiskv_segment_state_ints(64) == 8 + 64
    assert lib.louiskv_segment_state_ints(1) == 0
    base = [dummy, dummy, 1, 8, 8, 128, dummy, dummy, 64, 0, 16, None, dummy, dummy, dummy, dummy, 200, 64,
            None, None, 0, 0, 0, None]
    # missing state
    a = list(base); a[12] = None
    assert lib.louiskv_segment_output_boundary(*a) == 1
    # cap not below the window
    a = list(base); a[10] = 64
    assert lib.louiskv_segment_output_boundary(*a) == 2
    a = list(base); a[10] = 0
    assert lib.louiskv_segment_output_boundary(*a) == 2
    # more clusters than unit slots
    a = list(base); a[17] = 201
    assert lib.louiskv_segment_output_boundary(*a) == 2
    # retrieval and attention need the state
    assert lib.louiskv_retrieve_rows_seg(dummy, 1, 8, 8, 4, 128, 0.088, dummy, dummy, dummy, 100, 50, None, 64, 64,
                                         None, dummy, dummy, dummy, dummy, None, dummy, 1 << 30, None) == 1
    assert lib.louiskv_sparse_decode_attn_rows_seg(dummy, 1, 8, 8, 4, 128, 0.088, dummy, dummy, 1000, dummy, dummy,
                                                   64, dummy, dummy, 64, dummy, 0, dummy, 1, None, dummy, 1 << 30,
                                                   None) == 2


def test_pipelined_prefill_validates_on_the_host(lib):
    """The pipelined prefill refuses a missing pool, a zero chunk and too few or
    NULL events before any launch; its workspace is one chunk's."""
    P = ctypes.c_void_p
    dummy = P(16)
    ev3 = (ctypes.c_void_p * 3)(16, 16, 16)
    ev3_null = (ctypes.c_void_p * 3)(16, None, 16)

    def call(k_pool=dummy, chunk=4, events=ev3, n_events=3, n_slices=8):
        return lib.louiskv_cluster_prefill_pipelined(
            dummy, 1, n_slices, 64, 128, 8, 1, dummy, dummy, 8, dummy, dummy, dummy, dummy,
            None, k_pool, None, 64, 0, chunk, 1, ctypes.cast(events, P) if events is not None else None, n_events,
            dummy, 1 << 30, None, None)

    assert call(k_pool=None) == 1
    assert call(chunk=0) == 2
    assert call(events=None) == 1
    assert call(n_events=2) == 1            # 8 slices in chunks of 4 need 3 events
    assert call(chunk=3, n_events=3) == 1   # chunks of 3 need 4
    assert call(events=ev3_null) == 1
    one = lib.louiskv_cluster_prefill_workspace_size(8, 32768, 128, 1024, 1)
    assert lib.louiskv_cluster_prefill_pipelined_workspace_size(8, 32768, 128, 1024, 1, 0, 1) == one
    assert lib.louiskv_cluster_prefill_pipelined_workspace_size(8, 32768, 128, 1024, 1, 1, 0) == one
    # host pool through the copy engines: plus one chunk of staged rows
    assert lib.louiskv_cluster_prefill_pipelined_workspace_size(8, 32768, 128, 1024, 1, 1, 1) == \
        one + 8 * 32768 * 256
    assert lib.louiskv_cluster_prefill_pipelined_workspace_size(0, 32768, 128, 1024, 1, 1, 1) == 0


def test_ablation_calls_validate_on_the_host(lib):
    """The ablation baselines' calls refuse bad arguments before any launch."""
    P = ctypes.c_void_p
    dummy = P(16)
    assert lib.louiskv_fire_every(None, 8, 0, 4, None) == 1
    assert lib.louiskv_fire_every(dummy, 8, 0, 0, None) == 2
    assert lib.louiskv_fire_every(dummy, 8, -1, 4, None) == 2
    # 1000 tokens in pages of 16 are 63 units: a table of 62 is too small
    assert lib.louiskv_page_prefill(dummy, None, 1, 2, 1000, 128, 16, dummy, 62, dummy, dummy, None, None, 0, 0,
                                    None) == 2
    assert lib.louiskv_page_prefill(dummy, None, 1, 2, 1000, 128, 0, dummy, 63, dummy, dummy, None, None, 0, 0,
                                    None) == 2
    assert lib.louiskv_page_prefill(dummy, None, 1, 2, 1000, 128, 16, dummy, 63, dummy, dummy, dummy, None, 999, 0,
                                    None) == 2
    assert lib.louiskv_page_prefill(dummy, None, 1, 2, 1000, 128, 16, dummy, 63, dummy, dummy, dummy, dummy, 1000, 0,
                                    None) == 1   # v_pool without values
    # per-head calls: a group of 9 query heads is past the limit
    assert lib.louiskv_retrieve_rows_per_head(dummy, 1, 8, 8, 9, 128, 0.1, dummy, dummy, dummy, 64, 64, 16, None,
                                              dummy, dummy, dummy, dummy, None, dummy, 1 << 30, None) == 4
    assert lib.louiskv_sparse_decode_attn_rows_per_head(dummy, 1, 8, 8, 9, 128, 0.1, dummy, dummy, 100, dummy,
                                                        dummy, 16, dummy, dummy, 8, 0, 1, dummy, 1, None, dummy,
                                                        1 << 30, None) == 4
    assert lib.louiskv_sparse_decode_attn_rows_per_head(dummy, 1, 8, 8, 4, 128, 0.1, dummy, dummy, 100, None,
                                                        dummy, 16, dummy, dummy, 8, 0, 1, dummy, 1, None, dummy,
                                                        1 << 30, None) == 1


def test_decode_prologue_validates_on_the_host(lib):
    """The fused boundary test and store refuse missing buffers, a bad mode
    and an eviction with no unit room before any launch."""
    P = ctypes.c_void_p
    d = P(16)

    def call(q=d, k_new=d, mode=1, step=0, units_cap=100, n_clusters=8):
        return lib.louiskv_decode_prologue(q, d, 1, 2, 32, 128, 0.9, mode, 1, None, d, k_new, d, 16, d, d, 64, step,
                                           16, d, d, d, units_cap, n_clusters, None, None, 0, 0, 0, None)
    assert call(q=None) == 1
    assert call(k_new=None) == 1
    assert call(mode=5) == 2
    # step 64 with a 64-token window and 16-token segments evicts segment 0
    # into unit n_clusters, which needs units_cap > n_clusters
    assert call(step=64, units_cap=8, n_clusters=8) == 2


def test_workspace_sizes_are_positive(lib):
    assert lib.louiskv_cluster_prefill_workspace_size(256, 32768, 128, 1024, 1) > 256 * 32768 * 4
    assert lib.louiskv_retrieve_workspace_size(256, 1024, 2048) > 0
    # one block per slice once there are enough slices: no split-KV partials
    assert lib.louiskv_sparse_decode_attn_workspace_size(256, 4, 128, 2048, 128) == 0
    assert lib.louiskv_sparse_decode_attn_workspace_size(8, 4, 128, 2048, 128) > 0
    assert lib.louiskv_cluster_prefill_workspace_size(0, 1, 128, 1, 1) == 0
    # the decode step's counters and flags (256 bytes apart, zero between
    # calls), then the selection's logits, part maxima and attention partials
    S, G, cap, budget, window = 8, 4, 1100, 2048, 128
    step = lib.louiskv_decode_step_workspace_size(S, 1, G, cap, budget, window)
    assert step >= 256 * (4 * S + 1) + S * cap * G * 8 + S * 32 * G * 8 + S * 32 * G * 130 * 4
    assert lib.louiskv_decode_step_workspace_size(S, 1, 9, cap, budget, window) == 0


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU; asked for more it exits with a message."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""
