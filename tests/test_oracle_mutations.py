"""Plant plausible mistakes in the oracle (on the CPU) and check that at least
one pin fails for each: the pins are strong enough to notice a dropped term,
a flipped sign, a wrong axis, a wrong tie-break or a wrong budget rule."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
import oracle  # noqa: E402
import oracle.louiskv_oracle as L  # noqa: E402
import oracle.decode_driver as DD  # noqa: E402
from oracle_pins import ALL_PINS  # noqa: E402

F64 = np.float64
ORIG = {n: getattr(L, n) for n in ("kmeans_update", "group_scores", "attention")}
ORIG_PREFILL = DD.prefill_state_from_kmeans


def _sqdist_plus(keys, centroids):
    k = np.asarray(keys, F64); c = np.asarray(centroids, F64)
    return (k * k).sum(1)[:, None] + 2.0 * (k @ c.T) + (c * c).sum(1)[None, :]


def _sqdist_no_cnorm(keys, centroids):
    k = np.asarray(keys, F64); c = np.asarray(centroids, F64)
    return (k * k).sum(1)[:, None] - 2.0 * (k @ c.T)


def _assign_ties_high(keys, centroids, chunk=8192):
    d = L.squared_distances(keys, centroids)
    return d.shape[1] - 1 - np.argmin(d[:, ::-1], axis=1)


def _update_off_by_one(keys, z, prev):
    k = np.asarray(keys, F64); prev = np.asarray(prev, F64)
    counts = np.bincount(z, minlength=prev.shape[0])
    sums = np.zeros_like(prev); np.add.at(sums, z, k)
    out = prev.copy(); nz = counts > 0
    out[nz] = L.round_to_f32(sums[nz] / (counts[nz][:, None] + 1))
    return out, counts


def _update_empty_zero(keys, z, prev):
    out, counts = ORIG["kmeans_update"](keys, z, prev)
    out[counts == 0] = 0.0
    return out, counts


def _no_bf16(x):
    return np.asarray(x, F64)


def _similarity_sum(q, q_ref):
    a = np.asarray(q, F64); b = np.asarray(q_ref, F64)
    den = np.maximum(np.linalg.norm(a, axis=-1) * np.linalg.norm(b, axis=-1), 1e-30)
    return float(((a * b).sum(-1) / den).sum())


def _fires_le(r, tau, first):
    return bool(first or r <= tau)


def _scores_wrong_axis(q_group, reps, scale):
    lg = (np.asarray(q_group, F64) @ np.asarray(reps, F64).T) * scale
    e = np.exp(lg - lg.max(0, keepdims=True))
    return (e / e.sum(0, keepdims=True)).mean(0)


def _scores_no_scale(q_group, reps, scale):
    return ORIG["group_scores"](q_group, reps, 1.0)


def _select_skip(scores, unit_size, budget):
    s = np.asarray(scores, F64)
    order = sorted(range(len(s)), key=lambda u: (-s[u], u))
    chosen, tot = [], 0
    for u in order:
        if tot + int(unit_size[u]) <= budget:
            chosen.append(u); tot += int(unit_size[u])
    return chosen, tot


def _select_ties_high(scores, unit_size, budget):
    s = np.asarray(scores, F64)
    order = sorted(range(len(s)), key=lambda u: (-s[u], -u))
    chosen, tot = [], 0
    for u in order:
        if tot + int(unit_size[u]) > budget:
            break
        chosen.append(u); tot += int(unit_size[u])
    return chosen, tot


def _attention_k_as_v(q, k_rows, v_rows, scale):
    return ORIG["attention"](q, k_rows, k_rows, scale)


def _attention_no_scale(q, k_rows, v_rows, scale):
    return ORIG["attention"](q, k_rows, v_rows, 1.0)


def _segment_mean_f64(rows):
    r = np.asarray(rows, F64)
    return r.sum(0) / (r.shape[0] - 1)


def _opens_no_cap(fire, gen, open_first, seg_max):
    return open_first is None or fire


def _opens_cap_late(fire, gen, open_first, seg_max):
    return open_first is None or fire or gen - open_first > seg_max


def _opens_ignores_fire(fire, gen, open_first, seg_max):
    return open_first is None or gen - open_first >= seg_max


def _stride_late(t, stride):
    return t % stride == 0


def _pages_drop_tail(keys, page_len):
    k = np.asarray(keys, F64)
    n = k.shape[0] // page_len * page_len
    starts = np.arange(0, n, page_len, dtype=np.int64)
    sizes = np.full(len(starts), page_len, dtype=np.int64)
    reps = np.stack([L.segment_mean(k[a:a + page_len]) for a in starts])
    return reps, starts, sizes


def _head_scores_first_head(q_t, head, reps, scale):
    return L.group_scores(np.asarray(q_t, F64)[0:1], reps, scale)


def _head_scores_group(q_t, head, reps, scale):
    base = head - head % 2
    return L.group_scores(np.asarray(q_t, F64)[base:base + 2], reps, scale)


def _prefill_token_order(prompt_keys, prompt_values, results):
    st = ORIG_PREFILL(prompt_keys, prompt_values, results)
    st.k_pool = [np.asarray(k, F64) for k in prompt_keys]
    st.v_pool = [np.asarray(v, F64) for v in prompt_values]
    return st


MUTATIONS = {
    "distance_cross_term_sign": ("squared_distances", _sqdist_plus),
    "distance_dropped_centroid_norm": ("squared_distances", _sqdist_no_cnorm),
    "assign_ties_to_highest": ("kmeans_assign", _assign_ties_high),
    "update_divides_by_n_plus_1": ("kmeans_update", _update_off_by_one),
    "update_zeroes_empty_cluster": ("kmeans_update", _update_empty_zero),
    "operand_not_rounded_to_bf16": ("round_to_bf16", _no_bf16),
    "similarity_sum_not_mean": ("query_similarity", _similarity_sum),
    "boundary_fires_on_equal": ("boundary_fires", _fires_le),
    "softmax_over_heads": ("group_scores", _scores_wrong_axis),
    "score_scale_dropped": ("group_scores", _scores_no_scale),
    "budget_skip_and_continue": ("select_budget", _select_skip),
    "select_ties_to_highest": ("select_budget", _select_ties_high),
    "attention_keys_as_values": ("attention", _attention_k_as_v),
    "attention_scale_dropped": ("attention", _attention_no_scale),
    "segment_mean_wrong_count": ("segment_mean", _segment_mean_f64),
    "segment_without_length_cap": ("opens_segment", _opens_no_cap),
    "segment_cap_one_late": ("opens_segment", _opens_cap_late),
    "segment_ignores_boundary": ("opens_segment", _opens_ignores_fire),
    "stride_first_fire_late": ("stride_fires", _stride_late),
    "pages_drop_ragged_tail": ("page_units", _pages_drop_tail),
    "per_head_uses_first_head": ("head_scores", _head_scores_first_head),
    "per_head_uses_group_average": ("head_scores", _head_scores_group),
    "pool_left_in_token_order": ("prefill_state_from_kmeans", _prefill_token_order),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    for mod in (L, oracle, DD):
        if hasattr(mod, attr):
            monkeypatch.setattr(mod, attr, fn)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(oracle)
        except AssertionError:
            failed.append(pin.__name__)
            break
        except Exception:
            failed.append(pin.__name__ + " (error)")
            break
    assert failed, f"no pin catches mutation {name}"
