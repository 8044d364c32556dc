"""ctypes binding of libLouisKV.

Each function marshals torch tensors into the C ABI of include/louiskv.h
(pointers, sizes, the current HIP stream) and raises LouisKVError on a
non-zero status.  All arithmetic happens in the library's HIP kernels; if the
library is not built this module fails loudly instead of computing anything.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblouiskv.so")

F32, BF16 = 0, 1
REF_PREV, REF_ANCHOR = 0, 1

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_F = ctypes.c_float
_D = ctypes.c_double

_SIGS = {
    "louiskv_abi_version": (ctypes.c_int, []),
    "louiskv_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "louiskv_last_error": (ctypes.c_char_p, []),
    "louiskv_window_info": (ctypes.c_int, [_I32, _I32, _I32, _P, _P, _P, _P]),
    "louiskv_cluster_prefill_workspace_size": (_SZ, [_I64, _I32, _I32, _I32, _I32]),
    "louiskv_cluster_prefill": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _I32, _P,
        _P, _I32, _P, _P, _P, _P,
        _P, _P, _P, _I64, _I32, _P, _P, _SZ, _P]),
    "louiskv_pack_pool": (ctypes.c_int, [_P, _P, _I32, _I64, _I32, _I32, _P, _P, _P, _I64, _I32, _P]),
    "louiskv_cluster_prefill_pipelined_workspace_size": (_SZ, [_I64, _I32, _I32, _I32, _I32, _I32, _I32]),
    "louiskv_cluster_prefill_pipelined": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _I32, _P,
        _P, _I32, _P, _P, _P, _P,
        _P, _P, _P, _I64, _I32, _I64, _I32, _P, _I64, _P, _SZ, _P, _P]),
    "louiskv_kmeans_assign": (ctypes.c_int, [_P, _I32, _I64, _I32, _I32, _I32, _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_kmeans_update": (ctypes.c_int, [_P, _I32, _I64, _I32, _I32, _I32, _P, _P, _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_segment_output": (ctypes.c_int, [
        _P, _P, _I32, _I64, _I32, _P, _P, _I32, _I32, _I32,
        _P, _P, _P, _I32, _I32, _P, _P, _I64, _I32, _I32, _P]),
    "louiskv_boundary_check": (ctypes.c_int, [_P, _P, _I32, _I64, _I32, _I32, _D, _I32, _I32, _P, _P, _P]),
    "louiskv_retrieve_workspace_size": (_SZ, [_I64, _I32, _I32]),
    "louiskv_retrieve": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _D,
        _P, _P, _P, _I32, _I32,
        _P, _P, _I64, _I32, _I32, _P,
        _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "louiskv_retrieve_rows_workspace_size": (_SZ, [_I64, _I32]),
    "louiskv_retrieve_rows": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _D,
        _P, _P, _P, _I32, _I32, _I32, _P,
        _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "louiskv_sparse_decode_attn_rows_workspace_size": (_SZ, [_I64, _I32, _I32, _I32, _I32]),
    "louiskv_sparse_decode_attn_rows": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _F,
        _P, _P, _I64, _P, _P, _I32, _P, _P, _I32, _I32, _I32,
        _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_decode_step_workspace_size": (_SZ, [_I64, _I32, _I32, _I32, _I32, _I32]),
    "louiskv_decode_step_cached_workspace_size": (_SZ, [_I64, _I32, _I32, _I32, _I32, _I32]),
    "louiskv_decode_step": (ctypes.c_int, [
        _P, _P, _I32, _I64, _I32, _I32, _I32, _D, _I32, _I32, _P, _P,
        _P, _P, _P, _P, _I32, _I32, _P, _P, _P, _I32, _I32,
        _P, _P, _I64, _I32, _I32, _P, _P, _P, _P, _P, _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_decode_step_cached": (ctypes.c_int, [
        _P, _P, _I32, _I64, _I32, _I32, _I32, _D, _I32, _I32, _P, _P,
        _P, _P, _P, _P, _I32, _I32, _P, _P, _P, _I32, _I32,
        _P, _P, _I64, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P,
        _P, _P, _P, _P, _P, _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_sparse_decode_attn_rows_noalloc": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _F,
        _P, _P, _I64, _P, _P, _I32, _P, _P, _I32, _I32, _I32,
        _P, _I32, _P, _P]),
    "louiskv_fire_every": (ctypes.c_int, [_P, _I64, _I32, _I32, _P]),
    "louiskv_decode_prologue": (ctypes.c_int, [
        _P, _P, _I32, _I64, _I32, _I32, _D, _I32, _I32, _P, _P,
        _P, _P, _I64, _P, _P, _I32, _I32, _I32, _P, _P, _P, _I32, _I32, _P, _P, _I64, _I32, _I32, _P]),
    "louiskv_page_prefill": (ctypes.c_int, [
        _P, _P, _I32, _I64, _I32, _I32, _I32, _P, _I32, _P, _P, _P, _P, _I64, _I32, _P]),
    "louiskv_retrieve_rows_per_head": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _D,
        _P, _P, _P, _I32, _I32, _I32, _P,
        _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "louiskv_sparse_decode_attn_rows_per_head": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _F,
        _P, _P, _I64, _P, _P, _I32, _P, _P, _I32, _I32, _I32,
        _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_sparse_decode_attn_workspace_size": (_SZ, [_I64, _I32, _I32, _I32, _I32]),
    "louiskv_sparse_decode_attn": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _F,
        _P, _P, _P, _I32, _P, _P, _I32, _I32, _I32,
        _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_segment_state_ints": (_SZ, [_I32]),
    "louiskv_segment_state_init": (ctypes.c_int, [_P, _I64, _I32, _I32, _P]),
    "louiskv_segment_output_boundary": (ctypes.c_int, [
        _P, _P, _I32, _I64, _I32, _I32, _P, _P, _I32, _I32, _I32, _P, _P,
        _P, _P, _P, _I32, _I32, _P, _P, _I64, _I32, _I32, _P]),
    "louiskv_retrieve_seg": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _D,
        _P, _P, _P, _I32, _I32, _P, _I32,
        _P, _P, _I64, _I32, _I32, _P,
        _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "louiskv_retrieve_rows_seg": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _D,
        _P, _P, _P, _I32, _I32, _P, _I32, _I32, _P,
        _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "louiskv_sparse_decode_attn_seg": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _F,
        _P, _P, _P, _I32, _P, _P, _I32, _P, _I32,
        _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_sparse_decode_attn_rows_seg": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _F,
        _P, _P, _I64, _P, _P, _I32, _P, _P, _I32, _P, _I32,
        _P, _I32, _P, _P, _SZ, _P]),
    "louiskv_retrieve_delta_workspace_size": (_SZ, [_I64, _I32, _I32]),
    "louiskv_retrieve_delta": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _D,
        _P, _P, _P, _I32, _I32, _P, _I32,
        _P, _P, _I64, _I32, _I32, _P,
        _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "louiskv_retrieve_cached": (ctypes.c_int, [
        _P, _I32, _I64, _I32, _I32, _I32, _D,
        _P, _P, _P, _I32, _I32, _P, _I32,
        _P, _P, _I64, _I32, _I32, _I32, _I32, _P,
        _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
}

EXPORTED = sorted(_SIGS)

_lib = None


class LouisKVError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libLouisKV status {status}: {message}")
        self.status = status


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load (once) and return the library; raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"libLouisKV is not built ({p} missing); run `python -m paper_2510_11292_amd.build`")
    lib = ctypes.CDLL(p)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


def _check(status: int) -> None:
    if status != 0:
        lib = load_library()
        raise LouisKVError(status, lib.louiskv_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("libLouisKV needs contiguous tensors")
    return ctypes.c_void_p(t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _ws(nbytes: int, device, workspace: Optional[torch.Tensor]):
    if workspace is None:
        workspace = torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)
    return workspace, workspace.numel() * workspace.element_size()


def abi_version() -> int:
    return load_library().louiskv_abi_version()


def window_info(step: int, window: int, seg_len: int):
    """(evicted_segment or -1, n_evicted, n_local, local_start) after storing token `step`."""
    out = [ctypes.c_int32() for _ in range(4)]
    _check(load_library().louiskv_window_info(step, window, seg_len, *[ctypes.byref(o) for o in out]))
    return tuple(o.value for o in out)


def cluster_prefill_workspace_size(n_slices, n_tokens, n_clusters, dtype_code, d=128) -> int:
    return load_library().louiskv_cluster_prefill_workspace_size(n_slices, n_tokens, d, n_clusters, dtype_code)


def cluster_prefill(keys, n_clusters: int, n_iters: int, init_idx, reps, unit_start, unit_size, assign, perm,
                    values=None, k_pool=None, v_pool=None, pool_on_host: bool = False,
                    iter_events: Optional[Sequence] = None, workspace=None, stream=None):
    s, n, d = keys.shape
    dt = _dtype_code(keys)
    ws, wsb = _ws(cluster_prefill_workspace_size(s, n, n_clusters, dt, d), keys.device, workspace)
    pool_rows = k_pool.shape[1] if k_pool is not None else (v_pool.shape[1] if v_pool is not None else 0)
    ev = None
    if iter_events is not None:
        arr = (ctypes.c_void_p * len(iter_events))(*[e.cuda_event for e in iter_events])
        ev = ctypes.cast(arr, ctypes.c_void_p)
    _check(load_library().louiskv_cluster_prefill(
        _ptr(keys), dt, s, n, d, n_clusters, n_iters, _ptr(init_idx),
        _ptr(reps), reps.shape[1], _ptr(unit_start), _ptr(unit_size), _ptr(assign), _ptr(perm),
        _ptr(values), _ptr(k_pool), _ptr(v_pool), pool_rows, int(pool_on_host), ev,
        _ptr(ws), wsb, _stream(stream)))


def cluster_prefill_pipelined_workspace_size(slices_per_chunk, n_tokens, n_clusters, dtype_code, pool_on_host,
                                             copy_engine, d=128) -> int:
    return load_library().louiskv_cluster_prefill_pipelined_workspace_size(
        slices_per_chunk, n_tokens, d, n_clusters, dtype_code, int(pool_on_host), int(copy_engine))


def cluster_prefill_pipelined(keys, n_clusters: int, n_iters: int, init_idx, reps, unit_start, unit_size, assign,
                              perm, values, k_pool, v_pool, slices_per_chunk: int, chunk_events: Sequence,
                              copy_stream, pool_on_host: bool = False, copy_engine: bool = True, workspace=None,
                              stream=None):
    """louiskv_cluster_prefill_pipelined: chunk_events holds ceil(S / chunk) + 1
    torch.cuda.Event objects (recorded once already, so that they exist)."""
    s, n, d = keys.shape
    dt = _dtype_code(keys)
    ws, wsb = _ws(cluster_prefill_pipelined_workspace_size(min(slices_per_chunk, s), n, n_clusters, dt,
                                                           pool_on_host, copy_engine, d), keys.device, workspace)
    arr = (ctypes.c_void_p * len(chunk_events))(*[e.cuda_event for e in chunk_events])
    _check(load_library().louiskv_cluster_prefill_pipelined(
        _ptr(keys), dt, s, n, d, n_clusters, n_iters, _ptr(init_idx),
        _ptr(reps), reps.shape[1], _ptr(unit_start), _ptr(unit_size), _ptr(assign), _ptr(perm),
        _ptr(values), _ptr(k_pool), _ptr(v_pool), k_pool.shape[1], int(pool_on_host), slices_per_chunk,
        int(copy_engine), ctypes.cast(arr, ctypes.c_void_p), len(chunk_events), _ptr(ws), wsb, _stream(stream),
        _stream(copy_stream)))


def kmeans_assign(keys, n_clusters: int, centroids, assign, workspace=None, stream=None):
    s, n, d = keys.shape
    dt = _dtype_code(keys)
    ws, wsb = _ws(cluster_prefill_workspace_size(s, n, n_clusters, dt, d), keys.device, workspace)
    _check(load_library().louiskv_kmeans_assign(
        _ptr(keys), dt, s, n, d, n_clusters, _ptr(centroids), centroids.shape[1], _ptr(assign),
        _ptr(ws), wsb, _stream(stream)))


def kmeans_update(keys, n_clusters: int, assign, centroids_in, centroids_out, counts=None, workspace=None,
                  stream=None):
    s, n, d = keys.shape
    dt = _dtype_code(keys)
    ws, wsb = _ws(cluster_prefill_workspace_size(s, n, n_clusters, dt, d), keys.device, workspace)
    _check(load_library().louiskv_kmeans_update(
        _ptr(keys), dt, s, n, d, n_clusters, _ptr(assign), _ptr(centroids_in), _ptr(centroids_out),
        centroids_out.shape[1], _ptr(counts), _ptr(ws), wsb, _stream(stream)))


def segment_output(k_new, v_new, k_local, v_local, step: int, seg_len: int, reps, unit_start, unit_size,
                   n_clusters: int, k_pool=None, v_pool=None, prompt_len: int = 0, pool_on_host: bool = False,
                   stream=None):
    s, d = k_new.shape
    pool_rows = k_pool.shape[1] if k_pool is not None else 0
    _check(load_library().louiskv_segment_output(
        _ptr(k_new), _ptr(v_new), _dtype_code(k_new), s, d, _ptr(k_local), _ptr(v_local), k_local.shape[1],
        step, seg_len, _ptr(reps), _ptr(unit_start), _ptr(unit_size), reps.shape[1], n_clusters,
        _ptr(k_pool), _ptr(v_pool), pool_rows, prompt_len, int(pool_on_host), _stream(stream)))


def boundary_check(q, q_ref, tau: float, mode: int, first_step: bool, fire_out, r_out=None, stream=None):
    g, h, d = q.shape
    _check(load_library().louiskv_boundary_check(
        _ptr(q), _ptr(q_ref), _dtype_code(q), g, h, d, float(tau), int(mode), int(first_step),
        _ptr(r_out), _ptr(fire_out), _stream(stream)))


def retrieve_workspace_size(n_slices, units_cap, budget) -> int:
    return load_library().louiskv_retrieve_workspace_size(n_slices, units_cap, budget)


def retrieve(q, n_kv_heads: int, reps, unit_start, unit_size, n_units: int, k_pool, v_pool, budget: int,
             sel_units, n_sel_units, n_sel, k_buf, v_buf, fire=None, scale: Optional[float] = None,
             pool_on_host: bool = False, scores_out=None, workspace=None, stream=None):
    g, hq, d = q.shape
    s = reps.shape[0]
    cap = reps.shape[1]
    ws, wsb = _ws(retrieve_workspace_size(s, cap, budget), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_retrieve(
        _ptr(q), _dtype_code(q), s, n_kv_heads, hq // n_kv_heads, d, float(sc),
        _ptr(reps), _ptr(unit_start), _ptr(unit_size), cap, n_units,
        _ptr(k_pool), _ptr(v_pool), k_pool.shape[1], int(pool_on_host), budget, _ptr(fire),
        _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(k_buf), _ptr(v_buf), _ptr(scores_out),
        _ptr(ws), wsb, _stream(stream)))


def sparse_decode_attn_workspace_size(n_slices, group_size, buf_rows, window, d=128) -> int:
    return load_library().louiskv_sparse_decode_attn_workspace_size(n_slices, group_size, d, buf_rows, window)


def sparse_decode_attn(q, n_kv_heads: int, k_buf, v_buf, n_sel, k_local, v_local, local_start: int, n_local: int,
                       out, lse_out=None, scale: Optional[float] = None, workspace=None, stream=None):
    g, hq, d = q.shape
    s = n_sel.shape[0]
    gs = hq // n_kv_heads
    buf_rows = k_buf.shape[1] if k_buf is not None else 0
    window = k_local.shape[1] if k_local is not None else 0
    ws, wsb = _ws(sparse_decode_attn_workspace_size(s, gs, buf_rows, window, d), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_sparse_decode_attn(
        _ptr(q), _dtype_code(q), s, n_kv_heads, gs, d, float(sc), _ptr(k_buf), _ptr(v_buf), _ptr(n_sel), buf_rows,
        _ptr(k_local), _ptr(v_local), window, local_start, n_local, _ptr(out), _dtype_code(out), _ptr(lse_out),
        _ptr(ws), wsb, _stream(stream)))


def retrieve_rows_workspace_size(n_slices, units_cap) -> int:
    return load_library().louiskv_retrieve_rows_workspace_size(n_slices, units_cap)


def retrieve_rows(q, n_kv_heads: int, reps, unit_start, unit_size, n_units: int, budget: int, sel_units,
                  n_sel_units, n_sel, sel_rows, fire=None, scale: Optional[float] = None, scores_out=None,
                  workspace=None, stream=None):
    """Selection as a list of pool rows (no copy); sel_rows is [S][budget] int32."""
    g, hq, d = q.shape
    s = reps.shape[0]
    cap = reps.shape[1]
    ws, wsb = _ws(retrieve_rows_workspace_size(s, cap), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_retrieve_rows(
        _ptr(q), _dtype_code(q), s, n_kv_heads, hq // n_kv_heads, d, float(sc),
        _ptr(reps), _ptr(unit_start), _ptr(unit_size), cap, n_units, budget, _ptr(fire),
        _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(sel_rows), _ptr(scores_out),
        _ptr(ws), wsb, _stream(stream)))


def sparse_decode_attn_rows_workspace_size(n_slices, group_size, budget, window, d=128) -> int:
    return load_library().louiskv_sparse_decode_attn_rows_workspace_size(n_slices, group_size, d, budget, window)


def sparse_decode_attn_rows(q, n_kv_heads: int, k_pool, v_pool, sel_rows, n_sel, k_local, v_local,
                            local_start: int, n_local: int, out, lse_out=None, scale: Optional[float] = None,
                            workspace=None, stream=None):
    """Attention over the listed pool rows followed by the local window."""
    g, hq, d = q.shape
    s = n_sel.shape[0]
    gs = hq // n_kv_heads
    budget = sel_rows.shape[1]
    window = k_local.shape[1] if k_local is not None else 0
    ws, wsb = _ws(sparse_decode_attn_rows_workspace_size(s, gs, budget, window, d), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_sparse_decode_attn_rows(
        _ptr(q), _dtype_code(q), s, n_kv_heads, gs, d, float(sc), _ptr(k_pool), _ptr(v_pool), k_pool.shape[1],
        _ptr(sel_rows), _ptr(n_sel), budget, _ptr(k_local), _ptr(v_local), window, local_start, n_local,
        _ptr(out), _dtype_code(out), _ptr(lse_out), _ptr(ws), wsb, _stream(stream)))


def decode_step_workspace_size(n_slices: int, dtype_code: int, group_size: int, units_cap: int, budget: int,
                               window: int) -> int:
    return int(load_library().louiskv_decode_step_workspace_size(n_slices, dtype_code, group_size, units_cap,
                                                                 budget, window))


def decode_step(q, q_ref, tau: float, mode: int, step: int, fire, r_out, k_new, v_new, k_local, v_local,
                seg_len: int, reps, unit_start, unit_size, n_clusters: int, k_pool, v_pool, prompt_len: int,
                budget: int, sel_units, n_sel_units, n_sel, sel_rows, out, lse_out=None, scores_out=None,
                workspace=None, stream=None):
    """One decode step (boundary, store, retrieval of the fired groups, attention)
    in one launch (bf16; two in float32).  workspace: zero-filled before its
    first use."""
    g, hq, d = q.shape
    s = k_new.shape[0]
    h = s // g
    window = k_local.shape[1]
    dt = _dtype_code(q)
    if workspace is None:
        workspace = torch.zeros(decode_step_workspace_size(s, dt, hq // h, reps.shape[1], budget, window),
                                dtype=torch.uint8, device=q.device)
    _check(load_library().louiskv_decode_step(
        _ptr(q), _ptr(q_ref), dt, g, hq, h, d, float(tau), mode, step, _ptr(r_out), _ptr(fire),
        _ptr(k_new), _ptr(v_new), _ptr(k_local), _ptr(v_local), window, seg_len, _ptr(reps), _ptr(unit_start),
        _ptr(unit_size), reps.shape[1], n_clusters, _ptr(k_pool), _ptr(v_pool), k_pool.shape[1], prompt_len,
        budget, _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(sel_rows), _ptr(scores_out), _ptr(out),
        _dtype_code(out), _ptr(lse_out), _ptr(workspace), workspace.numel(), _stream(stream)))


def decode_step_cached_workspace_size(n_slices: int, dtype_code: int, group_size: int, units_cap: int, budget: int,
                                      window: int) -> int:
    return int(load_library().louiskv_decode_step_cached_workspace_size(n_slices, dtype_code, group_size, units_cap,
                                                                        budget, window))


def decode_step_cached(q, q_ref, tau: float, mode: int, step: int, fire, r_out, k_new, v_new, k_local, v_local,
                       seg_len: int, reps, unit_start, unit_size, n_clusters: int, k_pool, v_pool, prompt_len: int,
                       budget: int, k_buf, v_buf, buf_row, slot_step, slot_list, sel_units, n_sel_units, n_sel,
                       sel_rows, out, lse_out=None, n_fetched=None, scores_out=None, pool_on_host: bool = False,
                       workspace=None, stream=None):
    """One decode step with KV_critical kept as an LRU cache of k_buf.shape[1]
    pool rows, in four launches.  workspace: zero-filled before its first use."""
    g, hq, d = q.shape
    s = k_new.shape[0]
    h = s // g
    window = k_local.shape[1]
    dt = _dtype_code(q)
    if workspace is None:
        workspace = torch.zeros(decode_step_cached_workspace_size(s, dt, hq // h, reps.shape[1], budget, window),
                                dtype=torch.uint8, device=q.device)
    _check(load_library().louiskv_decode_step_cached(
        _ptr(q), _ptr(q_ref), dt, g, hq, h, d, float(tau), mode, step, _ptr(r_out), _ptr(fire),
        _ptr(k_new), _ptr(v_new), _ptr(k_local), _ptr(v_local), window, seg_len, _ptr(reps), _ptr(unit_start),
        _ptr(unit_size), reps.shape[1], n_clusters, _ptr(k_pool), _ptr(v_pool), k_pool.shape[1], int(pool_on_host),
        prompt_len, budget, k_buf.shape[1], _ptr(k_buf), _ptr(v_buf), _ptr(buf_row), _ptr(slot_step),
        _ptr(slot_list), _ptr(n_fetched), _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(sel_rows),
        _ptr(scores_out), _ptr(out), _dtype_code(out), _ptr(lse_out), _ptr(workspace), workspace.numel(),
        _stream(stream)))


NOALLOC_SCRATCH_BYTES = 8 << 20   # LOUISKV_NOALLOC_SCRATCH_BYTES


def sparse_decode_attn_rows_noalloc(q, n_kv_heads: int, k_pool, v_pool, sel_rows, n_sel, k_local, v_local,
                                    local_start: int, n_local: int, out, lse_out=None,
                                    scale: Optional[float] = None, stream=None):
    """sparse_decode_attn_rows without a workspace: the split-KV partials use
    the library's static device array (at most NOALLOC_SCRATCH_BYTES)."""
    g, hq, d = q.shape
    s = n_sel.shape[0]
    gs = hq // n_kv_heads
    budget = sel_rows.shape[1]
    window = k_local.shape[1] if k_local is not None else 0
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_sparse_decode_attn_rows_noalloc(
        _ptr(q), _dtype_code(q), s, n_kv_heads, gs, d, float(sc), _ptr(k_pool), _ptr(v_pool), k_pool.shape[1],
        _ptr(sel_rows), _ptr(n_sel), budget, _ptr(k_local), _ptr(v_local), window, local_start, n_local,
        _ptr(out), _dtype_code(out), _ptr(lse_out), _stream(stream)))


def decode_prologue(q, q_ref, tau: float, mode: int, first_step: bool, fire, r_out, k_new, v_new, k_local, v_local,
                    step: int, seg_len: int, reps, unit_start, unit_size, n_clusters: int, k_pool=None, v_pool=None,
                    prompt_len: int = 0, pool_on_host: bool = False, stream=None):
    """boundary_check and segment_output (fixed segments) in one launch."""
    g, hq, d = q.shape
    s = k_new.shape[0]
    window = k_local.shape[1]
    pool_rows = k_pool.shape[1] if k_pool is not None else 0
    _check(load_library().louiskv_decode_prologue(
        _ptr(q), _ptr(q_ref), _dtype_code(q), g, hq, d, float(tau), mode, int(first_step), _ptr(r_out), _ptr(fire),
        _ptr(k_new), _ptr(v_new), s, _ptr(k_local), _ptr(v_local), window, step, seg_len, _ptr(reps),
        _ptr(unit_start), _ptr(unit_size), reps.shape[1], n_clusters, _ptr(k_pool), _ptr(v_pool), pool_rows,
        prompt_len, int(pool_on_host), _stream(stream)))


# ------------------------------------------------------ ablation baselines

def fire_every(fire, step: int, stride: int, stream=None):
    """Fixed-stride trigger: fire[g] = (step % stride == 0) for every group."""
    _check(load_library().louiskv_fire_every(_ptr(fire), fire.shape[0], step, stride, _stream(stream)))


def page_prefill(keys, page_len: int, reps, unit_start, unit_size, values=None, k_pool=None, v_pool=None,
                 pool_on_host: bool = False, stream=None):
    """Page-level index of the prompt (mean key per page), pool in token order."""
    s, n, d = keys.shape
    pool_rows = k_pool.shape[1] if k_pool is not None else 0
    _check(load_library().louiskv_page_prefill(
        _ptr(keys), _ptr(values), _dtype_code(keys), s, n, d, page_len, _ptr(reps), reps.shape[1],
        _ptr(unit_start), _ptr(unit_size), _ptr(k_pool), _ptr(v_pool), pool_rows, int(pool_on_host),
        _stream(stream)))


def retrieve_rows_per_head(q, n_kv_heads: int, reps, unit_start, unit_size, n_units: int, budget: int, sel_units,
                           n_sel_units, n_sel, sel_rows, fire=None, scale: Optional[float] = None, scores_out=None,
                           workspace=None, stream=None):
    """One selection per query head; outputs have n_slices * group_size lists."""
    g, hq, d = q.shape
    s = reps.shape[0]
    cap = reps.shape[1]
    gs = hq // n_kv_heads
    ws, wsb = _ws(retrieve_rows_workspace_size(s * gs, cap), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_retrieve_rows_per_head(
        _ptr(q), _dtype_code(q), s, n_kv_heads, gs, d, float(sc),
        _ptr(reps), _ptr(unit_start), _ptr(unit_size), cap, n_units, budget, _ptr(fire),
        _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(sel_rows), _ptr(scores_out),
        _ptr(ws), wsb, _stream(stream)))


def sparse_decode_attn_rows_per_head(q, n_kv_heads: int, k_pool, v_pool, sel_rows, n_sel, k_local, v_local,
                                     local_start: int, n_local: int, out, lse_out=None, scale: Optional[float] = None,
                                     workspace=None, stream=None):
    """Attention of every query head over its own listed pool rows and its KV
    head's local window."""
    g, hq, d = q.shape
    s = k_pool.shape[0]
    gs = hq // n_kv_heads
    budget = sel_rows.shape[1]
    window = k_local.shape[1] if k_local is not None else 0
    ws, wsb = _ws(sparse_decode_attn_rows_workspace_size(s * gs, 1, budget, window, d), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_sparse_decode_attn_rows_per_head(
        _ptr(q), _dtype_code(q), s, n_kv_heads, gs, d, float(sc), _ptr(k_pool), _ptr(v_pool), k_pool.shape[1],
        _ptr(sel_rows), _ptr(n_sel), budget, _ptr(k_local), _ptr(v_local), window, local_start, n_local,
        _ptr(out), _dtype_code(out), _ptr(lse_out), _ptr(ws), wsb, _stream(stream)))


# ------------------------------------------------ boundary-delimited segments

def segment_state_ints(window: int) -> int:
    """int32 entries per slice of the segment state (louiskv_segment_state_ints)."""
    return load_library().louiskv_segment_state_ints(window)


def segment_state_init(seg_state, window: int, n_clusters: int, stream=None):
    """Segment state before decode step 0 (clusters only, empty window)."""
    _check(load_library().louiskv_segment_state_init(_ptr(seg_state), seg_state.shape[0], window, n_clusters,
                                                     _stream(stream)))


def segment_output_boundary(k_new, v_new, k_local, v_local, step: int, seg_max: int, fire, seg_state, reps,
                            unit_start, unit_size, n_clusters: int, n_kv_heads: int, k_pool=None, v_pool=None,
                            prompt_len: int = 0, pool_on_host: bool = False, stream=None):
    s, d = k_new.shape
    pool_rows = k_pool.shape[1] if k_pool is not None else 0
    _check(load_library().louiskv_segment_output_boundary(
        _ptr(k_new), _ptr(v_new), _dtype_code(k_new), s, n_kv_heads, d, _ptr(k_local), _ptr(v_local),
        k_local.shape[1], step, seg_max, _ptr(fire), _ptr(seg_state), _ptr(reps), _ptr(unit_start),
        _ptr(unit_size), reps.shape[1], n_clusters, _ptr(k_pool), _ptr(v_pool), pool_rows, prompt_len,
        int(pool_on_host), _stream(stream)))


def retrieve_seg(q, n_kv_heads: int, reps, unit_start, unit_size, max_units: int, seg_state, window: int, k_pool,
                 v_pool, budget: int, sel_units, n_sel_units, n_sel, k_buf, v_buf, fire=None,
                 scale: Optional[float] = None, pool_on_host: bool = False, scores_out=None, workspace=None,
                 stream=None):
    g, hq, d = q.shape
    s = reps.shape[0]
    cap = reps.shape[1]
    ws, wsb = _ws(retrieve_workspace_size(s, cap, budget), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_retrieve_seg(
        _ptr(q), _dtype_code(q), s, n_kv_heads, hq // n_kv_heads, d, float(sc),
        _ptr(reps), _ptr(unit_start), _ptr(unit_size), cap, max_units, _ptr(seg_state), window,
        _ptr(k_pool), _ptr(v_pool), k_pool.shape[1], int(pool_on_host), budget, _ptr(fire),
        _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(k_buf), _ptr(v_buf), _ptr(scores_out),
        _ptr(ws), wsb, _stream(stream)))


def retrieve_rows_seg(q, n_kv_heads: int, reps, unit_start, unit_size, max_units: int, seg_state, window: int,
                      budget: int, sel_units, n_sel_units, n_sel, sel_rows, fire=None, scale: Optional[float] = None,
                      scores_out=None, workspace=None, stream=None):
    g, hq, d = q.shape
    s = reps.shape[0]
    cap = reps.shape[1]
    ws, wsb = _ws(retrieve_rows_workspace_size(s, cap), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_retrieve_rows_seg(
        _ptr(q), _dtype_code(q), s, n_kv_heads, hq // n_kv_heads, d, float(sc),
        _ptr(reps), _ptr(unit_start), _ptr(unit_size), cap, max_units, _ptr(seg_state), window, budget,
        _ptr(fire), _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(sel_rows), _ptr(scores_out),
        _ptr(ws), wsb, _stream(stream)))


def sparse_decode_attn_seg(q, n_kv_heads: int, k_buf, v_buf, n_sel, k_local, v_local, seg_state, n_tokens: int,
                           out, lse_out=None, scale: Optional[float] = None, workspace=None, stream=None):
    g, hq, d = q.shape
    s = n_sel.shape[0]
    gs = hq // n_kv_heads
    buf_rows = k_buf.shape[1] if k_buf is not None else 0
    window = k_local.shape[1]
    ws, wsb = _ws(sparse_decode_attn_workspace_size(s, gs, buf_rows, window, d), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_sparse_decode_attn_seg(
        _ptr(q), _dtype_code(q), s, n_kv_heads, gs, d, float(sc), _ptr(k_buf), _ptr(v_buf), _ptr(n_sel), buf_rows,
        _ptr(k_local), _ptr(v_local), window, _ptr(seg_state), n_tokens, _ptr(out), _dtype_code(out),
        _ptr(lse_out), _ptr(ws), wsb, _stream(stream)))


def sparse_decode_attn_rows_seg(q, n_kv_heads: int, k_pool, v_pool, sel_rows, n_sel, k_local, v_local, seg_state,
                                n_tokens: int, out, lse_out=None, scale: Optional[float] = None, workspace=None,
                                stream=None):
    g, hq, d = q.shape
    s = n_sel.shape[0]
    gs = hq // n_kv_heads
    budget = sel_rows.shape[1]
    window = k_local.shape[1]
    ws, wsb = _ws(sparse_decode_attn_rows_workspace_size(s, gs, budget, window, d), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_sparse_decode_attn_rows_seg(
        _ptr(q), _dtype_code(q), s, n_kv_heads, gs, d, float(sc), _ptr(k_pool), _ptr(v_pool), k_pool.shape[1],
        _ptr(sel_rows), _ptr(n_sel), budget, _ptr(k_local), _ptr(v_local), window, _ptr(seg_state), n_tokens,
        _ptr(out), _dtype_code(out), _ptr(lse_out), _ptr(ws), wsb, _stream(stream)))


def retrieve_delta_workspace_size(n_slices, units_cap, budget) -> int:
    return load_library().louiskv_retrieve_delta_workspace_size(n_slices, units_cap, budget)


def retrieve_delta(q, n_kv_heads: int, reps, unit_start, unit_size, n_units: int, k_pool, v_pool, budget: int,
                   sel_units, n_sel_units, n_sel, k_buf, v_buf, buf_row, slot_list, fire=None, seg_state=None,
                   window: int = 0, n_fetched=None, scale: Optional[float] = None, pool_on_host: bool = False,
                   scores_out=None, workspace=None, stream=None):
    """Retrieval into KV_critical as a cache of pool rows (only new rows are copied)."""
    g, hq, d = q.shape
    s = reps.shape[0]
    cap = reps.shape[1]
    ws, wsb = _ws(retrieve_delta_workspace_size(s, cap, budget), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_retrieve_delta(
        _ptr(q), _dtype_code(q), s, n_kv_heads, hq // n_kv_heads, d, float(sc),
        _ptr(reps), _ptr(unit_start), _ptr(unit_size), cap, n_units, _ptr(seg_state), window,
        _ptr(k_pool), _ptr(v_pool), k_pool.shape[1], int(pool_on_host), budget, _ptr(fire),
        _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(k_buf), _ptr(v_buf), _ptr(buf_row),
        _ptr(slot_list), _ptr(n_fetched), _ptr(scores_out), _ptr(ws), wsb, _stream(stream)))


CACHE_MAX_ROWS = 65536   # louiskv_retrieve_cached: slots per slice at most


def retrieve_cached(q, n_kv_heads: int, reps, unit_start, unit_size, n_units: int, k_pool, v_pool, budget: int,
                    step: int, sel_units, n_sel_units, n_sel, k_buf, v_buf, buf_row, slot_step, slot_list, fire=None,
                    seg_state=None, window: int = 0, n_fetched=None, scale: Optional[float] = None,
                    pool_on_host: bool = False, scores_out=None, workspace=None, stream=None):
    """Retrieval into KV_critical kept as an LRU cache of k_buf.shape[1] pool rows."""
    g, hq, d = q.shape
    s = reps.shape[0]
    cap = reps.shape[1]
    ws, wsb = _ws(retrieve_delta_workspace_size(s, cap, budget), q.device, workspace)
    sc = (1.0 / d ** 0.5) if scale is None else scale
    _check(load_library().louiskv_retrieve_cached(
        _ptr(q), _dtype_code(q), s, n_kv_heads, hq // n_kv_heads, d, float(sc),
        _ptr(reps), _ptr(unit_start), _ptr(unit_size), cap, n_units, _ptr(seg_state), window,
        _ptr(k_pool), _ptr(v_pool), k_pool.shape[1], int(pool_on_host), budget, k_buf.shape[1], step, _ptr(fire),
        _ptr(sel_units), _ptr(n_sel_units), _ptr(n_sel), _ptr(k_buf), _ptr(v_buf), _ptr(buf_row), _ptr(slot_step),
        _ptr(slot_list), _ptr(n_fetched), _ptr(scores_out), _ptr(ws), wsb, _stream(stream)))


def pack_pool(keys, values, perm, k_pool, v_pool=None, pool_on_host: bool = False, stream=None):
    """Prompt K/V rows into the pools in perm order (each cluster contiguous)."""
    s, n, d = keys.shape
    _check(load_library().louiskv_pack_pool(
        _ptr(keys), _ptr(values), _dtype_code(keys), s, n, d, _ptr(perm), _ptr(k_pool), _ptr(v_pool),
        k_pool.shape[1], int(pool_on_host), _stream(stream)))
