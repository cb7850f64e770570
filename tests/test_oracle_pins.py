"""Pins of the CPU oracle to facts the paper and the mathematics fix.

Each test checks the oracle against something other than itself: closed forms,
brute-force enumeration, an independent library routine, identities proved in
the paper's appendices, and budgets the paper prints (tests/golden).
"""

import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle as O
from tests.compare import topk_layout

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_budgets.json")


def grid(rng, *shape, scale=1.0):
    """Values on the j/16 grid (|j| <= 255)."""
    x = rng.standard_normal(shape) * scale
    return np.clip(np.round(x * 16), -255, 255) / 16


# ---------------------------------------------------------------- dense attention

def test_dense_equal_keys_gives_mean_value():
    # all logits equal => uniform weights => y = mean(V)  (Eq. attn_eq)
    rng = np.random.default_rng(0)
    k = rng.standard_normal(16)
    K = np.tile(k, (9, 1))
    V = rng.standard_normal((9, 16))
    q = rng.standard_normal(16)
    y, lse = O.dense_attention(q, K, V)
    np.testing.assert_allclose(y, V.mean(0), rtol=0, atol=1e-14)
    assert lse == pytest.approx(q @ k / 4.0 + math.log(9), abs=1e-12)


def test_dense_single_key_returns_its_value():
    rng = np.random.default_rng(1)
    q, k, v = rng.standard_normal((3, 8))
    y, lse = O.dense_attention(q, k[None], v[None])
    np.testing.assert_array_equal(y, v)
    assert lse == pytest.approx(q @ k / math.sqrt(8), abs=1e-14)


def test_dense_dominant_key():
    # one logit exceeds every other by 60: its weight is 1 - O(n e^-60)
    rng = np.random.default_rng(2)
    d = 4
    K = np.zeros((7, d))
    K[3, 0] = 60.0 * math.sqrt(d)
    q = np.array([1.0, 0, 0, 0])
    V = rng.standard_normal((7, d))
    y, _ = O.dense_attention(q, K, V)
    np.testing.assert_allclose(y, V[3], atol=1e-20 + 7 * math.exp(-60) * np.abs(V).max())


def test_dense_matches_torch_sdpa_fp64():
    rng = np.random.default_rng(3)
    for n, d in [(1, 8), (5, 64), (300, 128)]:
        q = rng.standard_normal(d)
        K = rng.standard_normal((n, d)) * 2
        V = rng.standard_normal((n, d))
        y, _ = O.dense_attention(q, K, V)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.tensor(q)[None, None, None], torch.tensor(K)[None, None],
            torch.tensor(V)[None, None]).numpy()[0, 0, 0]
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-13)


def test_dense_matches_scalar_loop_and_lse():
    # independent plain-Python evaluation of Eq. attn_eq
    rng = np.random.default_rng(4)
    n, d = 11, 6
    q = rng.standard_normal(d)
    K = rng.standard_normal((n, d))
    V = rng.standard_normal((n, d))
    logits = [sum(q[t] * K[i][t] for t in range(d)) / math.sqrt(d) for i in range(n)]
    Z = sum(math.exp(z) for z in logits)
    yref = [sum(math.exp(logits[i]) / Z * V[i][t] for i in range(n)) for t in range(d)]
    y, lse = O.dense_attention(q, K, V)
    np.testing.assert_allclose(y, yref, rtol=1e-13, atol=1e-14)
    assert lse == pytest.approx(math.log(Z), rel=1e-14)
    A = O.attention_weights(q, K)
    np.testing.assert_allclose(A, [math.exp(z) / Z for z in logits], rtol=1e-13)


def test_empty_set_attention():
    y, lse = O.sparse_attention(np.ones(4), np.ones((3, 4)), np.ones((3, 4)), [])
    np.testing.assert_array_equal(y, np.zeros(4))
    assert lse == -math.inf


# ---------------------------------------------------------------- scores and Z1 exactness

def test_ranking_score_is_group_max_of_raw_dot():
    rng = np.random.default_rng(5)
    Qg = rng.standard_normal((4, 8))
    K = rng.standard_normal((10, 8))
    s = O.ranking_scores(Qg, K)
    for i in range(10):
        ref = max(sum(Qg[h][t] * K[i][t] for t in range(8)) for h in range(4))
        assert s[i] == pytest.approx(ref, abs=1e-12)


def test_grid_scores_exact_in_float32_any_order():
    # The generator's grid makes fp32 dot products exact in every order, so the
    # GPU's fp32 scores equal the oracle's fp64 scores bit for bit.
    rng = np.random.default_rng(6)
    for d in (64, 128):
        q = grid(rng, d, scale=4.0)
        K = grid(rng, 200, d, scale=4.0)
        ref = O.ranking_scores(q, K)
        seq = np.zeros(200, dtype=np.float32)
        for t in range(d):
            seq = (seq + (q[t].astype(np.float32) * K[:, t].astype(np.float32))).astype(np.float32)
        rev = np.zeros(200, dtype=np.float32)
        for t in reversed(range(d)):
            rev = (rev + (q[t].astype(np.float32) * K[:, t].astype(np.float32))).astype(np.float32)
        pair = (K.astype(np.float32) * q.astype(np.float32)).sum(axis=1, dtype=np.float32)
        for v in (seq, rev, pair):
            assert np.array_equal(v.astype(np.float64), ref)
        # extreme grid values: the worst-case magnitude is still exact
        qx = np.full(d, 255 / 16)
        Kx = np.full((1, d), -255 / 16)
        assert O.ranking_scores(qx, Kx)[0] == np.float32(d * (255 / 16) ** 2) * -1


# ---------------------------------------------------------------- top-k oracle

def test_topk_brute_force_max_mass():
    # the top-k set maximises retained mass over every k-subset of the middle
    # range (Thm. oracle); checked by enumeration on tiny inputs
    rng = np.random.default_rng(7)
    for trial in range(40):
        n0 = int(rng.integers(1, 13))
        sink, window = int(rng.integers(0, 3)), int(rng.integers(0, 4))
        k = int(rng.integers(0, 6))
        d = 4
        q = grid(rng, d, scale=2)
        K = grid(rng, n0, d, scale=2)
        A = O.attention_weights(q, K)
        sigma = O.ranking_scores(q, K)
        S = O.topk_middle(sigma, n0, k, sink, window)
        best = O.brute_force_topk_mass(A, n0, k, sink, window)
        sink_end, win_start = O.region_bounds(n0, sink, window)
        assert len(S) == min(k, max(0, win_start - sink_end))
        assert O.retained_mass(A, S) == pytest.approx(best, abs=1e-14)


def test_topk_order_and_tie_break_lowest_index():
    # ties on the score resolve to the lower position; output order is
    # (score desc, position asc); checked against Python's sort of tuples
    rng = np.random.default_rng(8)
    for trial in range(50):
        n0 = int(rng.integers(5, 60))
        sigma = rng.integers(-3, 4, size=n0).astype(np.float64)  # many ties
        sink, window = 2, 3
        k = int(rng.integers(1, n0))
        S = O.topk_middle(sigma, n0, k, sink, window)
        mid = [i for i in range(n0) if sink <= i < n0 - window]
        ref = sorted(mid, key=lambda i: (-sigma[i], i))[:k]
        assert list(S) == ref


def test_topk_negative_zero_ties_positive_zero():
    sigma = np.array([0.0, -0.0, 0.0, -0.0, -1.0])
    S = O.topk_middle(sigma, 5, 3, 0, 0)
    assert list(S) == [0, 1, 2]


def test_topk_degenerate_ranges():
    sigma = np.arange(10, dtype=np.float64)
    assert list(O.topk_middle(sigma, 10, 0, 2, 2)) == []
    assert list(O.topk_middle(sigma, 10, 99, 2, 2)) == [7, 6, 5, 4, 3, 2]
    assert list(O.topk_middle(sigma, 4, 3, 2, 2)) == []   # n0 <= sink + window
    assert list(O.topk_middle(sigma, 3, 3, 4, 0)) == []   # n0 < sink


# ---------------------------------------------------------------- set algebra

def _anchor_by_definition(s_star, n0, sink, window):
    return sorted({i for i in range(n0) if i < sink} | set(int(x) for x in s_star)
                  | {i for i in range(n0) if i >= n0 - window})


def _reuse_by_definition(s_star, m, r, n0, n, sink, window):
    out = {i for i in range(n) if i < sink}
    out |= set(int(x) for x in s_star)
    for p in list(s_star)[:m]:
        for j in range(-r, r + 1):
            if 0 <= p + j < n:
                out.add(int(p + j))
    out |= {i for i in range(n) if i >= max(min(sink, n0), n0 - window)}
    return sorted(out)


def test_sets_brute_force_random():
    rng = np.random.default_rng(9)
    for trial in range(400):
        n0 = int(rng.integers(0, 40))
        n = n0 + int(rng.integers(0, 6))
        sink = int(rng.integers(0, 6))
        window = int(rng.integers(0, 8))
        k = int(rng.integers(0, 12))
        r = int(rng.integers(0, 3))
        sigma = rng.integers(-4, 5, size=max(n, 1)).astype(np.float64)
        S = O.topk_middle(sigma, n0, k, sink, window)
        m = O.dilation_m(k, len(S), -1 if trial % 2 else int(rng.integers(0, 5)))
        assert list(O.anchor_set(S, n0, sink, window)) == _anchor_by_definition(S, n0, sink, window)
        assert list(O.reuse_set(S, m, r, n0, n, sink, window)) == \
            _reuse_by_definition(S, m, r, n0, n, sink, window)


def test_reuse_set_grows_by_the_decoded_tail():
    # R(n) = R(n0) followed by [n0, n) for every n >= n0: dilated neighbours of
    # middle positions stay below n0 and [n0, n) lies in the window.  Checked
    # against the set-by-definition, including window 0 and wide radii.
    rng = np.random.default_rng(12)
    for trial in range(400):
        n0 = int(rng.integers(0, 40))
        sink = int(rng.integers(0, 6))
        window = int(rng.integers(0, 8))
        k = int(rng.integers(0, 12))
        r = int(rng.integers(0, 4))
        sigma = rng.integers(-4, 5, size=max(n0, 1)).astype(np.float64)
        S = O.topk_middle(sigma, n0, k, sink, window)
        m = O.dilation_m(k, len(S))
        base = _reuse_by_definition(S, m, r, n0, n0, sink, window)
        assert all(i < n0 for i in base)
        for n in range(n0, n0 + 6):
            assert list(O.reuse_set(S, m, r, n0, n, sink, window)) == base + list(range(n0, n))


def test_reuse_at_range_edges_and_overlaps():
    # top-m at the first and last middle positions; neighbours land in the
    # sink and window (no duplicates) or are clipped
    sink, window, n0, n = 3, 4, 20, 22
    S = np.array([3, 15, 9])
    R = O.reuse_set(S, 2, 1, n0, n, sink, window)
    assert list(R) == [0, 1, 2, 3, 4, 9, 14, 15, 16, 17, 18, 19, 20, 21]
    R0 = O.reuse_set(np.array([0]), 1, 2, 1, 1, 0, 0)
    assert list(R0) == [0]


def test_reuse_radius_zero_and_m_zero_equal_plain_sharing():
    rng = np.random.default_rng(10)
    sigma = rng.standard_normal(100)
    S = O.topk_middle(sigma, 90, 20, 4, 8)
    base = O.reuse_set(S, 0, 1, 90, 95, 4, 8)
    assert list(base) == list(O.reuse_set(S, 7, 0, 90, 95, 4, 8))
    expect = sorted(set(range(4)) | set(S.tolist()) | set(range(82, 95)))
    assert list(base) == expect


def test_isolated_dilation_size_closed_form():
    # isolated top-m winners each add exactly 2r neighbours: |S_hat| = C + 2rm
    sink, window, n0 = 4, 32, 1000
    k, r = 30, 1
    sigma = np.zeros(n0)
    winners = np.arange(10, 10 + 10 * k, 10)[:k]
    sigma[winners] = np.linspace(100, 50, k)
    S = O.topk_middle(sigma, n0, k, sink, window)
    assert sorted(S.tolist()) == winners.tolist()
    m = O.dilation_m(k, len(S))
    assert m == 10
    C = O.anchor_set(S, n0, sink, window)
    R = O.reuse_set(S, m, r, n0, n0, sink, window)
    assert len(C) == sink + k + window
    assert len(R) == sink + k + window + 2 * r * m


# ---------------------------------------------------------------- golden budgets

def test_golden_paper_budgets():
    g = json.load(open(GOLDEN))
    gs = g["gsm8k_coqa"]
    sink = gs["C_t"] - gs["C_local"] - gs["k"]
    assert sink == 8
    n0 = 2000
    sigma = np.zeros(n0)
    sigma[np.arange(100, 100 + 3 * gs["k"], 3)] = 1.0  # k spread winners
    S = O.topk_middle(sigma, n0, gs["k"], sink, gs["C_local"])
    C = O.anchor_set(S, n0, sink, gs["C_local"])
    assert len(C) == gs["C_t"]                        # C = C_sink + k + C_local
    m = O.dilation_m(gs["k"], len(S))
    assert m == 29 and g["defaults"]["r"] == 1
    R = O.reuse_set(S, m, 1, n0, n0, sink, gs["C_local"])
    assert gs["C_t"] <= len(R) <= gs["C_t"] + 2 * m
    lb = g["longbench"]
    C_lb = lb["C_sink"] + lb["k"] + lb["C_local"]
    assert C_lb == lb["budget"]
    m_lb = lb["k"] // 3
    # the paper's average dilated shared set lies within [C, C + 2 r m]
    assert C_lb <= lb["avg_shared_set"] <= C_lb + 2 * m_lb
    C_star = lb["C_sink"] + lb["k_cis_star"] + lb["C_local"]
    assert C_star <= lb["cis_star_avg_budget"] <= C_star + 2 * (lb["k_cis_star"] // 3)


# ---------------------------------------------------------------- invariant: a full budget is dense attention

def test_full_budget_reproduces_dense():
    # k >= |middle| (or window >= n) gives R = [0, n): sparse == dense
    rng = np.random.default_rng(11)
    for (n0, extra, sink, window, k) in [(50, 3, 4, 8, 1000), (50, 0, 4, 64, 10), (7, 2, 0, 0, 7)]:
        n = n0 + extra
        d = 16
        q = rng.standard_normal(d)
        K = rng.standard_normal((n, d))
        V = rng.standard_normal((n, d))
        sigma = O.ranking_scores(q, K)
        S = O.topk_middle(sigma, n0, k, sink, window)
        R = O.reuse_set(S, O.dilation_m(k, len(S)), 1, n0, n, sink, window)
        assert list(R) == list(range(n))
        y_s, l_s = O.sparse_attention(q, K, V, R)
        y_d, l_d = O.dense_attention(q, K, V)
        np.testing.assert_allclose(y_s, y_d, rtol=0, atol=1e-15)
        assert l_s == pytest.approx(l_d, abs=1e-15)
        if extra == 0:
            C = O.anchor_set(S, n0, sink, window)
            assert list(C) == list(range(n0))


# ---------------------------------------------------------------- mass relations (appendices)

def _random_case(rng, n=200, d=32):
    q = rng.standard_normal(d)
    K = rng.standard_normal((n, d)) * 1.5
    V = rng.standard_normal((n, d))
    return q, K, V


def test_tv_identity_and_kl_identity():
    # ||A - A~_S||_TV = delta_S (Lemma tv); KL(A~_S || A) = log 1/tau_S (U2)
    rng = np.random.default_rng(12)
    for _ in range(20):
        q, K, V = _random_case(rng)
        A = O.attention_weights(q, K)
        S = np.sort(rng.choice(200, size=int(rng.integers(1, 200)), replace=False))
        At = O.renormalised(A, S)
        assert O.tv_distance(A, At) == pytest.approx(O.dropped_mass(A, S), abs=1e-14)
        assert O.kl_divergence(At, A) == pytest.approx(-math.log(O.retained_mass(A, S)), abs=1e-12)


def test_output_error_bounded_by_dropped_mass():
    # |y - y_S|_inf <= 2 delta_S max|v| (from the TV identity)
    rng = np.random.default_rng(13)
    for _ in range(30):
        q, K, V = _random_case(rng)
        S = np.sort(rng.choice(200, size=int(rng.integers(1, 200)), replace=False))
        A = O.attention_weights(q, K)
        y, _ = O.dense_attention(q, K, V)
        ys, _ = O.sparse_attention(q, K, V, S)
        assert np.abs(y - ys).max() <= 2 * O.dropped_mass(A, S) * np.abs(V).max() + 1e-13


def test_family_best_is_minimal_dropped_mass():
    # the per-head top-k member of the family beats every random member
    rng = np.random.default_rng(14)
    sink, window, k = 4, 16, 20
    for _ in range(20):
        q, K, V = _random_case(rng)
        n = K.shape[0]
        A = O.attention_weights(q, K)
        best = O.family_best_dropped(A, n, sink, window, k)
        S = O.anchor_set(O.topk_middle(O.ranking_scores(q, K), n, k, sink, window), n, sink, window)
        assert O.dropped_mass(A, S) == pytest.approx(best, abs=1e-14)
        mid = np.arange(sink, n - window)
        for _ in range(20):
            Sr = O.anchor_set(rng.choice(mid, size=k, replace=False), n, sink, window)
            assert best <= O.dropped_mass(A, Sr) + 1e-15


def test_cis_retained_mass_gap():
    # Prop. cis-beta: on fixed keys, a later query reusing the dilated set of
    # the reference query keeps tau_pre(q') >= tau*(q') - 2 ||A(q') - A(q)||_1
    rng = np.random.default_rng(15)
    sink, window, k, n, d = 4, 16, 24, 300, 32
    for _ in range(30):
        K = rng.standard_normal((n, d)) * 1.5
        q = rng.standard_normal(d)
        Sq = O.topk_middle(O.ranking_scores(q, K), n, k, sink, window)
        R = O.reuse_set(Sq, O.dilation_m(k, len(Sq)), 1, n, n, sink, window)
        qp = q
        for _ in range(8):
            qp = 0.9 * qp + math.sqrt(0.19) * rng.standard_normal(d)
            A_q = O.attention_weights(q, K)
            A_p = O.attention_weights(qp, K)
            d_att = np.abs(A_p - A_q).sum()
            tau_star = 1.0 - O.family_best_dropped(A_p, n, sink, window, k)
            tau_pre = O.retained_mass(A_p, R)
            assert tau_pre >= tau_star - 2 * d_att - 1e-13


def test_attention_variation_lipschitz_bound():
    # ||A(q') - A(q)||_1 <= 2 K_max / sqrt(d) * ||q' - q|| (CIS appendix lemmas)
    rng = np.random.default_rng(16)
    for _ in range(50):
        n, d = 100, 16
        K = rng.standard_normal((n, d))
        q = rng.standard_normal(d)
        qp = q + rng.standard_normal(d) * rng.uniform(0.01, 1.0)
        lhs = np.abs(O.attention_weights(qp, K) - O.attention_weights(q, K)).sum()
        kmax = np.linalg.norm(K, axis=1).max()
        assert lhs <= 2 * kmax / math.sqrt(d) * np.linalg.norm(qp - q) + 1e-14


def test_mi_bound_monotone_on_restricted_domain():
    # g is increasing on (0, L/(1+L)] (footnote to Eq. pohs bound)
    for L in (2, 10, 1000, 131072):
        xs = np.linspace(1e-9, L / (1 + L), 2000)
        gs = [O.mi_loss_bound(x, L) for x in xs]
        assert all(b >= a - 1e-12 for a, b in zip(gs, gs[1:]))
    assert O.mi_loss_bound(0.0, 100) == 0.0


def test_binary_entropy_closed_forms_and_library():
    # h_b in nats: h_b(1/2) = ln 2, h_b(1/4) = 2 ln 2 - (3/4) ln 3, symmetric
    # about 1/2, and equal to scipy's Shannon entropy of the pmf (x, 1 - x)
    from scipy.stats import entropy
    assert O.binary_entropy(0.5) == pytest.approx(math.log(2), abs=1e-15)
    assert O.binary_entropy(0.25) == pytest.approx(2 * math.log(2) - 0.75 * math.log(3), abs=1e-15)
    for x in (1e-6, 0.01, 0.3, 0.77, 0.999):
        assert O.binary_entropy(x) == pytest.approx(O.binary_entropy(1 - x), abs=1e-15)
        assert O.binary_entropy(x) == pytest.approx(float(entropy([x, 1 - x])), rel=1e-13)
    assert O.binary_entropy(0.0) == 0.0 and O.binary_entropy(1.0) == 0.0


def test_mi_bound_closed_forms():
    # Eq. mi_bound, g(d) = 2 [h_b(d) + d ln L], with entropy and log in the
    # same base (nats).  Hand values: d = 1/2, L = 2 gives 2 (ln 2 + ln 2 / 2)
    # = 3 ln 2; d = 1/4, L = 8 gives 2 (2 ln 2 - 3/4 ln 3 + 3/4 ln 2).
    assert O.mi_loss_bound(0.5, 2) == pytest.approx(3 * math.log(2), abs=1e-14)
    assert O.mi_loss_bound(0.25, 8) == pytest.approx(
        2 * (2.75 * math.log(2) - 0.75 * math.log(3)), abs=1e-14)
    # h_b(d) + d ln L is maximised where its derivative ln((1 - d) / d) + ln L
    # vanishes, at d = L / (1 + L) (the end of the footnote's domain), and the
    # maximum is ln(1 + L): so g peaks at 2 ln(1 + L) there and nowhere higher
    for L in (2, 7, 100, 4096, 131072):
        d_star = L / (1 + L)
        assert O.mi_loss_bound(d_star, L) == pytest.approx(2 * math.log1p(L), rel=1e-13)
        xs = np.linspace(1e-6, 1 - 1e-6, 997)
        assert max(O.mi_loss_bound(x, L) for x in xs) <= 2 * math.log1p(L) + 1e-12


def test_mi_bound_dominates_entropy_continuity():
    # the bound's building block (entropy continuity, MI-bound appendix,
    # Step 2): |H(P) - H(Q)| <= h_b(eps) + eps ln m for pmfs on m <= L
    # symbols with TV distance eps; so g(eps) / 2 bounds it for random pairs
    from scipy.stats import entropy
    rng = np.random.default_rng(40)
    for _ in range(300):
        m = int(rng.integers(2, 40))
        P = rng.dirichlet(np.ones(m))
        Q = rng.dirichlet(np.ones(m) * rng.uniform(0.2, 5))
        eps = O.tv_distance(P, Q)
        if eps >= m / (1 + m):
            continue
        gap = abs(float(entropy(P)) - float(entropy(Q)))
        assert gap <= O.mi_loss_bound(eps, m) / 2 + 1e-12


def test_proportional_budget_closed_forms():
    # reading of the throughput sweep's "top-k 5% of each sequence's length":
    # k_b = floor(n0 / 20), integer arithmetic, recomputed per refresh
    cases = {1000: 50, 1019: 50, 1020: 51, 8192: 409, 16368: 818, 19: 0, 20: 1, 0: 0}
    for n0, kb in cases.items():
        assert O.budget_k(n0, k_num=1, k_den=20) == kb
    # 3/64 of n0 and a fixed budget
    assert O.budget_k(4096, k_num=3, k_den=64) == 192
    assert O.budget_k(4095, k_num=3, k_den=64) == 191
    assert O.budget_k(4096, k=256) == 256 and O.budget_k(10, k=256) == 256


# ---------------------------------------------------------------- schedule

def test_retrieval_ratio_closed_form():
    # rho_hat = 1 / (s G) when T is a multiple of s and N of G (Sec. 5.1)
    for s, G, T, N in [(4, 1, 16, 1), (4, 4, 16, 32), (8, 4, 16, 32), (8, 1, 16, 32)]:
        assert O.retrieval_ratio(T, N, s, G) == pytest.approx(1.0 / (s * G))


def test_decode_oracle_schedule_and_anchor_state():
    rng = np.random.default_rng(17)
    L, T, g, d, n_ctx = 4, 8, 2, 16, 60
    sink, window, k, s, G = 2, 4, 6, 4, 2
    K = [rng.standard_normal((n_ctx + T, d)) for _ in range(L)]
    Q = [[rng.standard_normal((g, d)) for _ in range(T)] for _ in range(L)]
    dec = O.DecodeOracle(sink, window, s, G, r=1, k=k)
    for j in range(T):
        n = n_ctx + j + 1
        for l in range(L):
            S = dec.step_set(l, j, Q[l][j], K[l], n)
            a = (l // G) * G
            j0 = (j // s) * s
            n0 = n_ctx + j0 + 1
            s_star = O.topk_middle(O.ranking_scores(Q[a][j0], K[a][:n0]), n0, k, sink, window)
            if l == a and j == j0:
                expect = O.anchor_set(s_star, n0, sink, window)
            else:
                expect = O.reuse_set(s_star, k // 3, 1, n0, n, sink, window)
            assert list(S) == list(expect)


def test_topk_layout_partitions_by_rank_then_position():
    # the library's layout of S*: its m top-ranked members, then the rest, each
    # part ascending; the set and the top-m set are those of the ranked S*
    rng = np.random.default_rng(18)
    sigma = rng.integers(-5, 6, size=300).astype(float)
    S = O.topk_middle(sigma, 300, 40, 4, 16)
    for m in (0, 1, 13, 40):
        lay = topk_layout(S, m)
        assert sorted(lay.tolist()) == sorted(S.tolist())
        assert set(lay[:m].tolist()) == set(S[:m].tolist())
        assert list(lay[:m]) == sorted(lay[:m]) and list(lay[m:]) == sorted(lay[m:])


# ---------------------------------------------------------------- similarity gate

def test_query_similarity_closed_forms():
    # Eq. cos_sim on vectors of known angle
    e = np.zeros(8)
    e[0] = 1.0
    assert O.query_similar(e, 3 * e, 0.99)                  # same direction, any length
    assert not O.query_similar(e, e, 1.0)                   # cos = 1 is not > 1
    f = np.zeros(8)
    f[1] = 2.0
    assert not O.query_similar(e, f, 0.0)                   # orthogonal
    assert not O.query_similar(e, -e, 0.0)                  # opposite
    assert not O.query_similar(np.zeros(8), e, 0.0)         # zero query
    for deg, tau, want in ((30, 0.8, True), (30, 0.9, False), (40, 0.76, True), (40, 0.77, False)):
        th = math.radians(deg)
        v = np.zeros(8)
        v[0], v[1] = math.cos(th), math.sin(th)
        assert O.query_similar(e, 5 * v, tau) == want, (deg, tau)


def test_group_similarity_needs_every_head():
    rng = np.random.default_rng(21)
    Q = rng.standard_normal((4, 16))
    R = Q + 0.01 * rng.standard_normal((4, 16))
    assert O.group_similar(Q, R, 0.9)
    R[2] = -R[2]
    assert not O.group_similar(Q, R, 0.9)


def test_gate_chooses_most_recent_similar_anchor():
    e0, e1 = np.eye(2)
    q = np.array([[1.0, 0.2]])
    anchors = [(0, np.array([[1.0, 0.0]])), (1, np.array([[0.0, 1.0]])), (2, np.array([[1.0, 0.1]]))]
    assert O.gate_choice(q, anchors, 0.8) == 2
    assert O.gate_choice(q, anchors[:2], 0.8) == 0
    assert O.gate_choice(q, anchors[1:2], 0.8) is None
    assert O.gate_choice(q, [], 0.0) is None


def _on_grid(x):
    return np.clip(np.round(x * 16), -255, 255) / 16


def _run_schedule(dec, Qs, K, n_ctx, L, T):
    sets = {}
    for j in range(T):
        for l in range(L):
            sets[(l, j)] = dec.step_set(l, j, Qs[l][j], K[l], n_ctx + j + 1)
    return sets


def _gate_inputs(seed, L=4, T=8, g=2, d=16, n=220):
    rng = np.random.default_rng(seed)
    K = [grid(rng, n + T, d) for _ in range(L)]
    base = rng.standard_normal((L, g, d))
    Qs = [[_on_grid(base[l] + 0.3 * rng.standard_normal((g, d))) for _ in range(T)] for l in range(L)]
    return K, Qs, n


def test_gate_tau_one_retrieves_every_step():
    # cos > 1 never holds: every anchor-layer step retrieves, which is the
    # fixed schedule with a refresh at every step
    K, Qs, n = _gate_inputs(3)
    kw = dict(sink=4, window=16, G=2, r=1, k=24)
    gated = O.GatedDecodeOracle(s=4, tau=1.0, **kw)
    fixed = O.DecodeOracle(s=1, **kw)
    a = _run_schedule(gated, Qs, K, n, 4, 8)
    b = _run_schedule(fixed, Qs, K, n, 4, 8)
    assert all(np.array_equal(a[x], b[x]) for x in a)
    assert gated.retrievals == gated.decisions


def test_gate_tau_zero_positive_queries_is_the_block_schedule():
    # queries with positive dot products share from the block's first step:
    # the fixed schedule with refresh every s steps, retrieval ratio 1/s
    K, Qs, n = _gate_inputs(4)
    Qs = [[np.abs(q) for q in row] for row in Qs]
    kw = dict(sink=4, window=16, G=2, r=1, k=24)
    gated = O.GatedDecodeOracle(s=4, tau=0.0, **kw)
    fixed = O.DecodeOracle(s=4, **kw)
    a = _run_schedule(gated, Qs, K, n, 4, 8)
    b = _run_schedule(fixed, Qs, K, n, 4, 8)
    assert all(np.array_equal(a[x], b[x]) for x in a)
    assert gated.retrievals * 4 == gated.decisions


def test_gate_mixed_decisions_follow_the_rule():
    # step 2 is unlike step 0 and retrieves; step 3 resembles both and uses
    # the more recent step 2; non-anchor layers follow their anchor's choice
    d, n = 16, 200
    rng = np.random.default_rng(5)
    K = [grid(rng, n + 4, d) for _ in range(2)]
    u = np.zeros(d)
    u[:4] = 1.0
    w = np.zeros(d)
    w[4:8] = 1.0                 # orthogonal to u
    q = {0: u, 1: u, 2: w, 3: u + w}
    Qs = [[q[j][None, :] for j in range(4)] for _ in range(2)]
    dec = O.GatedDecodeOracle(sink=2, window=8, s=4, G=2, tau=0.5, k=10)
    sets = _run_schedule(dec, Qs, K, n, 2, 4)
    assert [dec.decision[(0, j)] for j in range(4)] == [0, 0, 2, 2]
    assert dec.retrievals == 2
    S0 = O.topk_middle(O.ranking_scores(q[0][None, :], K[0][: n + 1]), n + 1, 10, 2, 8)
    S2 = O.topk_middle(O.ranking_scores(q[2][None, :], K[0][: n + 3]), n + 3, 10, 2, 8)
    m = O.dilation_m(10, 10)
    assert np.array_equal(sets[(0, 1)], O.reuse_set(S0, m, 1, n + 1, n + 2, 2, 8))
    assert np.array_equal(sets[(0, 2)], O.anchor_set(S2, n + 3, 2, 8))
    assert np.array_equal(sets[(1, 2)], O.reuse_set(S2, m, 1, n + 3, n + 3, 2, 8))
    assert np.array_equal(sets[(0, 3)], O.reuse_set(S2, m, 1, n + 3, n + 4, 2, 8))


# ---------------------------------------------------------------- PSAW

def test_psaw_boundary_closed_forms():
    # Eq. psaw: nothing below l_s and at l_s itself (phi^0 = 1); at the top
    # layer l = N the boundary is floor((1 - phi^alpha) t)
    N, l_s, phi, alpha = 32, 24, 0.7, 1.0
    assert all(O.psaw_boundary(l, N, 1000, l_s, phi, alpha) == 0 for l in range(1, l_s + 1))
    assert O.psaw_boundary(N, N, 1000, l_s, phi, alpha) == 300
    assert O.psaw_boundary(N, N, 10, l_s, 0.5, 2.0) == 7            # 1 - 0.25 = 0.75
    b = [O.psaw_boundary(l, N, 4096, l_s, phi, alpha) for l in range(l_s, N + 1)]
    assert b == sorted(b) and b[-1] < 4096 * 0.31                   # monotone in depth
    assert O.psaw_boundary(N, N, 4096, l_s, phi, 0.0) == 0          # alpha = 0: no pruning


def test_psaw_visible_set_by_definition():
    # 1-based masked range (C_sink, P) against the 0-based restriction
    N, l_s, phi, alpha, sink = 8, 6, 0.6, 1.0, 3
    for layer0 in range(N):
        for n in (1, 2, 3, 5, 40, 97):
            P = O.psaw_boundary(layer0 + 1, N, n, l_s, phi, alpha)
            visible1 = [p for p in range(1, n + 1) if p <= sink or p >= P]
            start = O.psaw_visible_start(layer0, N, n, sink, l_s, phi, alpha)
            S = np.arange(n)
            assert list(O.psaw_restrict(S, start, sink, n) + 1) == visible1, (layer0, n)


def test_psaw_schedule_is_the_cis_set_under_the_mask():
    # CPE: the schedule with PSAW attends exactly the CIS set restricted to
    # the visible positions; without pruning layers it is the CIS schedule
    K, Qs, n = _gate_inputs(8, L=4, T=6)
    kw = dict(sink=4, window=16, s=3, G=2, r=1, k=24)
    for psaw in ((4, 2, 0.5, 1.0), (4, 5, 0.5, 1.0)):
        plain = _run_schedule(O.DecodeOracle(**kw), Qs, K, n, 4, 6)
        cpe = _run_schedule(O.DecodeOracle(psaw=psaw, **kw), Qs, K, n, 4, 6)
        for (l, j), S in plain.items():
            start = O.psaw_visible_start(l, 4, n + j + 1, 4, *psaw[1:])
            assert np.array_equal(cpe[(l, j)], O.psaw_restrict(S, start, 4, n + j + 1))
            if psaw[1] == 5:
                assert np.array_equal(cpe[(l, j)], S)
        top = cpe[(3, 5)]
        if psaw[1] == 2:
            start = O.psaw_visible_start(3, 4, n + 6, 4, 2, 0.5, 1.0)
            assert start > 4 and not np.any((top >= 4) & (top < start))


# ---------------------------------------------------------------- PSAW at prefill

def _causal_matrix_form(Q, K, V, scale):
    # the whole prompt at once: masked logit matrix, row softmax, one product
    T = Q.shape[0]
    Z = (Q @ K[:T].T) * scale
    Z[np.triu_indices(T, 1)] = -np.inf
    mx = Z.max(axis=1, keepdims=True)
    E = np.exp(Z - mx)
    den = E.sum(axis=1, keepdims=True)
    return (E / den) @ V[:T], (mx + np.log(den)).ravel()


def test_prefill_causal_matches_matrix_form():
    rng = np.random.default_rng(71)
    T, d = 37, 16
    Q, K, V = (rng.standard_normal((T, d)) for _ in range(3))
    y, lse = O.prefill_attention(Q, K, V, T)
    y2, lse2 = _causal_matrix_form(Q, K, V, 1 / math.sqrt(d))
    assert np.allclose(y, y2, atol=1e-12) and np.allclose(lse, lse2, atol=1e-12)
    # below the pruning depth PSAW leaves the prompt causal
    vis = O.psaw_prefill_visible(2, 8, T, 4, 6, 0.7, 1.0)
    assert list(vis) == [min(4, i + 1) for i in range(T)]
    y3, _ = O.prefill_attention(Q, K, V, T, sink=4, vis_start=vis)
    assert np.allclose(y3, y2, atol=1e-12)


def test_prefill_psaw_top_layer_and_monotone():
    N, l_s, phi, alpha, sink = 32, 24, 0.7, 1.0, 4
    vis = O.psaw_prefill_visible(N - 1, N, 500, sink, l_s, phi, alpha)
    assert list(vis) == [max(min(sink, i + 1), math.floor(0.3 * (i + 1)) - 1) for i in range(500)]
    for layer0 in range(l_s - 1, N):
        v = O.psaw_prefill_visible(layer0, N, 300, sink, l_s, phi, alpha)
        assert np.all(np.diff(v) >= 0)        # the window's start only moves forward


def test_prefill_row_is_the_decode_set_at_its_length():
    # query i of a prefill sees what a decode step at length i + 1 sees
    N, l_s, phi, alpha, sink = 8, 5, 0.5, 1.5, 3
    for layer0 in (4, 6, 7):
        vis = O.psaw_prefill_visible(layer0, N, 60, sink, l_s, phi, alpha)
        for i in range(60):
            n = i + 1
            start = O.psaw_visible_start(layer0, N, n, sink, l_s, phi, alpha)
            assert np.array_equal(O.prefill_visible_set(i, sink, int(vis[i])),
                                  O.psaw_restrict(np.arange(n), start, sink, n))
            P = O.psaw_boundary(layer0 + 1, N, n, l_s, phi, alpha)
            visible1 = [p for p in range(1, n + 1) if p <= sink or p >= P]
            assert list(O.prefill_visible_set(i, sink, int(vis[i])) + 1) == visible1


def test_prefill_psaw_rows_match_masked_matrix_form():
    # the top layer of a small prompt: each row against the matrix form with
    # the masked columns removed by hand
    rng = np.random.default_rng(72)
    T, d, sink = 50, 8, 2
    Q, K, V = (rng.standard_normal((T, d)) for _ in range(3))
    vis = O.psaw_prefill_visible(3, 4, T, sink, 2, 0.3, 1.0)
    assert vis[-1] > sink
    y, lse = O.prefill_attention(Q, K, V, T, sink=sink, vis_start=vis)
    for i in range(T):
        cols = [j for j in range(i + 1) if j < sink or j >= vis[i]]
        z = (K[cols] @ Q[i]) / math.sqrt(d)
        w = np.exp(z - z.max())
        assert np.allclose(y[i], (w / w.sum()) @ V[cols], atol=1e-12)
        assert abs(lse[i] - (z.max() + math.log(w.sum()))) < 1e-12
    # rows past the prompt are empty
    y4, lse4 = O.prefill_attention(Q, K, V, 20)
    assert np.all(y4[20:] == 0) and np.all(np.isneginf(lse4[20:]))
