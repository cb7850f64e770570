"""Planted mistakes in the oracle must be caught by its pins.

Each case swaps one oracle function for a plausibly wrong variant (on the CPU)
and checks that at least one pin test then fails.
"""

import math

import numpy as np
import pytest

import oracle as O
import oracle.prhs_oracle as M
from tests import test_oracle_pins as P


def _wrong_scale_dense(q, K, V, scale=None):
    return _orig["dense_attention"](q, K, V, 1.0)


def _tie_high_index(sigma, n0, k, sink, window):
    sink_end, win_start = M.region_bounds(n0, sink, window)
    pos = np.arange(sink_end, win_start)
    if pos.size == 0 or k <= 0:
        return np.zeros(0, dtype=np.int64)
    order = np.lexsort((-pos, -np.asarray(sigma, float)[pos]))
    return pos[order][:k]


def _reuse_without_new_tokens(s_star, m, r, n0, n, sink, window):
    return _orig["reuse_set"](s_star, m, r, n0, n0, sink, window)


def _reuse_no_clip(s_star, m, r, n0, n, sink, window):
    s_star = np.asarray(s_star, dtype=np.int64)
    sink_end, win_start = M.region_bounds(n0, sink, window)
    neigh = (s_star[:m, None] + np.arange(-r, r + 1)[None, :]).ravel()
    parts = [np.arange(0, sink_end), s_star, neigh, np.arange(win_start, n)]
    return np.unique(np.concatenate(parts))


def _min_over_group(Qg, K):
    Qg = np.atleast_2d(np.asarray(Qg, float))
    K = np.asarray(K, float)
    return (K @ Qg.T).min(axis=1) if K.shape[0] else np.zeros(0)


def _window_off_by_one(n0, sink, window):
    sink_end = min(sink, n0)
    return sink_end, max(sink_end, n0 - window - 1)


def _m_is_k_over_2(k_b, topk_len, dilate_m=-1):
    m = k_b // 2 if dilate_m < 0 else dilate_m
    return max(0, min(m, topk_len))


def _lse_missing_max(q, K, V, scale=None):
    y, lse = _orig["dense_attention"](q, K, V, scale)
    z = M.attention_logits(q, K, scale)
    return y, (lse - z.max()) if z.size else lse


def _schedule_layer_only(step, layer, s, G):
    return layer % G == 0


def _similar_ignoring_sign(q_now, q_ref, tau):
    a, b = np.ravel(q_now).astype(float), np.ravel(q_ref).astype(float)
    dot = float(a @ b)
    return dot * dot > tau * tau * float(a @ a) * float(b @ b)


def _gate_oldest_first(Qg_now, anchors, tau):
    for step, Qg_ref in list(anchors):
        if M.group_similar(Qg_now, Qg_ref, tau):
            return step
    return None


def _group_any_head(Qg_now, Qg_ref, tau):
    Qn, Qr = np.atleast_2d(Qg_now), np.atleast_2d(Qg_ref)
    return any(M.query_similar(Qn[h], Qr[h], tau) for h in range(Qn.shape[0]))


def _psaw_start_p_not_p_minus_1(layer0, n_layers, n, sink, l_s, phi, alpha):
    P = M.psaw_boundary(layer0 + 1, n_layers, n, l_s, phi, alpha)
    return max(min(sink, n), P)


def _psaw_zero_based_layer(layer, n_layers, t, l_s, phi, alpha):
    if layer - 1 < l_s:
        return 0
    e = alpha * (layer - 1 - l_s) / (n_layers - l_s)
    return int(math.floor((1.0 - phi ** e) * t))


def _mi_without_factor_2(delta, L):
    return M.binary_entropy(delta) + delta * math.log(L)


def _mi_in_bits(delta, L):
    h = 0.0 if delta <= 0.0 or delta >= 1.0 else (
        -delta * math.log2(delta) - (1 - delta) * math.log2(1 - delta))
    return 2.0 * (h + delta * math.log2(L))


def _binary_entropy_one_term(x):
    return 0.0 if x <= 0.0 or x >= 1.0 else -x * math.log(x)


def _budget_ceil(n0, k=None, k_num=0, k_den=0):
    if k_den and k_den > 0:
        return (k_num * n0 + k_den - 1) // k_den
    return int(k)


_orig = {name: getattr(M, name) for name in
         ["dense_attention", "topk_middle", "reuse_set", "ranking_scores",
          "region_bounds", "dilation_m", "is_refresh"]}

PINS = [getattr(P, n) for n in dir(P) if n.startswith("test_")]

def _prefill_vis_at_i(layer0, n_layers, T, sink, l_s, phi, alpha):
    return np.array([M.psaw_visible_start(layer0, n_layers, max(i, 1), sink, l_s, phi, alpha)
                     for i in range(T)], dtype=np.int64)


def _prefill_set_inclusive_mask(i, sink, vis=None):
    S = np.arange(i + 1, dtype=np.int64)
    return S if vis is None else S[(S < sink) | (S > vis)]


MUTANTS = [
    ("dense_attention", _wrong_scale_dense),
    ("dense_attention", _lse_missing_max),
    ("topk_middle", _tie_high_index),
    ("reuse_set", _reuse_without_new_tokens),
    ("reuse_set", _reuse_no_clip),
    ("ranking_scores", _min_over_group),
    ("region_bounds", _window_off_by_one),
    ("dilation_m", _m_is_k_over_2),
    ("is_refresh", _schedule_layer_only),
    ("query_similar", _similar_ignoring_sign),
    ("gate_choice", _gate_oldest_first),
    ("group_similar", _group_any_head),
    ("psaw_visible_start", _psaw_start_p_not_p_minus_1),
    ("psaw_boundary", _psaw_zero_based_layer),
    ("psaw_prefill_visible", _prefill_vis_at_i),
    ("prefill_visible_set", _prefill_set_inclusive_mask),
    ("mi_loss_bound", _mi_without_factor_2),
    ("mi_loss_bound", _mi_in_bits),
    ("binary_entropy", _binary_entropy_one_term),
    ("budget_k", _budget_ceil),
]


@pytest.mark.parametrize("name,fn", MUTANTS, ids=[f"{n}:{f.__name__}" for n, f in MUTANTS])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    monkeypatch.setattr(M, name, fn)
    monkeypatch.setattr(O, name, fn)
    failed = []
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"no pin caught the mutant {fn.__name__} of {name}"
