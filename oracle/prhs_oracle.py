"""CPU oracle for the Pre-hoc Sparsity (PrHS) decode hot path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
CPU-baseline leg of the benchmark may import or call this module.  The product
path (the HIP library and its Python binding) never routes through it, and this
module imports nothing from the product package.

Everything is plain NumPy in float64, one (batch, kv-head) unit at a time, with
explicit ordering wherever order matters.  Token positions are 0-based; the
paper counts from 1.  Each function names the passage of the paper it follows
("Near-Oracle KV Selection via Pre-hoc Sparsity for Long-Context Inference").

Readings of passages that the paper leaves open:

* Positions are 0-based and ranges half-open.  The current decode token is
  already in the cache, so a query at context length ``n`` attends ``[0, n)``
  (the sum in Eq. attn_eq runs up to and including step t).
* The sink is ``[0, C_sink)``, the recency window at anchor length ``n0`` is
  ``[n0 - C_local, n0)`` and the middle range searched by top-k is what lies
  between them (Sec. 4.1, Selection Criteria).
* Ranking uses the raw dot product ``q . k`` (no 1/sqrt(d)); softmax is
  monotone, so the ranking equals the ranking by attention weight.  For a
  grouped-query head group the key's score is the max over the group's query
  heads.  Equal scores are ordered by ascending position.
* The dilated shared set keeps the sink, the anchor's top-k, the +-r
  neighbourhood of its top-m and every position from the anchor's window start
  up to the current length (Eq. neighboring, with the neighbourhood clipped to
  the valid positions as in the CIS parameterisation appendix).
* PSAW at prefill: the query at position i has the i + 1 tokens [0, i] in
  view, so Eq. psaw is taken at t = i + 1; it attends the causal range [0, i]
  restricted to the sink and [max(C_sink, P - 1), i] (the same set a decode
  step at length i + 1 attends).
* Cross-layer sharing: groups of G consecutive layers; the first layer of a
  group is the anchor that scores; the others reuse its selection over their
  own K/V.  Refresh happens at decode steps j with j mod s == 0.
"""

from __future__ import annotations

import itertools
import math

import numpy as np

__all__ = [
    "attention_logits",
    "attention_weights",
    "dense_attention",
    "sparse_attention",
    "ranking_scores",
    "region_bounds",
    "budget_k",
    "dilation_m",
    "topk_middle",
    "anchor_set",
    "reuse_set",
    "is_refresh",
    "anchor_layer",
    "retrieval_ratio",
    "retained_mass",
    "dropped_mass",
    "family_best_dropped",
    "binary_entropy",
    "mi_loss_bound",
    "tv_distance",
    "kl_divergence",
    "renormalised",
    "DecodeOracle",
    "query_similar",
    "group_similar",
    "gate_choice",
    "GatedDecodeOracle",
    "psaw_boundary",
    "psaw_visible_start",
    "psaw_restrict",
    "psaw_prefill_visible",
    "prefill_visible_set",
    "prefill_attention",
]


# ---------------------------------------------------------------------------
# Attention (Sec. 2.1, Eq. attn_eq)
# ---------------------------------------------------------------------------

def _f64(x):
    return np.asarray(x, dtype=np.float64)


def attention_logits(q, K, scale=None):
    """Scaled logits q.k_i / sqrt(d) for every cached key (Eq. attn_eq)."""
    q = _f64(q)
    K = _f64(K)
    d = q.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    return (K @ q) * scale


def attention_weights(q, K, scale=None):
    """Softmax attention weights A_i(q) over all cached keys (Eq. attn_eq).

    Computed with a max shift; the shift cancels in the ratio.
    """
    z = attention_logits(q, K, scale)
    if z.size == 0:
        return z
    e = np.exp(z - z.max())
    return e / e.sum()


def dense_attention(q, K, V, scale=None):
    """Full decode attention over keys [0, n): returns (y, lse).

    y = sum_i A_i v_i and lse = log sum_i exp(q.k_i * scale) (Eq. attn_eq).
    An empty cache gives y = 0 and lse = -inf.
    """
    V = _f64(V)
    z = attention_logits(q, K, scale)
    if z.size == 0:
        return np.zeros(V.shape[-1]), -math.inf
    zmax = z.max()
    e = np.exp(z - zmax)
    s = e.sum()
    y = (e @ V) / s
    return y, float(zmax + math.log(s))


def sparse_attention(q, K, V, S, scale=None):
    """Token-sparse attention restricted to the index set S (Def. 3.1, Sec. 2.2).

    The weights are the softmax over S only, i.e. the renormalised distribution
    A_i / tau_S of the unified-bounds appendix.  Returns (y, lse); an empty S
    gives y = 0 and lse = -inf.
    """
    S = np.asarray(S, dtype=np.int64)
    K = _f64(K)
    V = _f64(V)
    return dense_attention(q, K[S], V[S], scale)


# ---------------------------------------------------------------------------
# Selection (Sec. 4.1, Selection Criteria; top-k oracle of Sec. 2.3)
# ---------------------------------------------------------------------------

def ranking_scores(Qg, K):
    """Key ranking score sigma_i = max over the query heads of a KV-head group
    of the raw dot product q_h . k_i.

    Qg has shape [g, d] (g = 1 for multi-head attention), K has shape [n, d].
    """
    Qg = np.atleast_2d(_f64(Qg))
    K = _f64(K)
    if K.shape[0] == 0:
        return np.zeros(0)
    return (K @ Qg.T).max(axis=1)


def region_bounds(n0, sink, window):
    """(sink_end, win_start) for anchor length n0.

    sink = [0, sink_end), window = [win_start, n0), middle = [sink_end, win_start).
    When sink and window overlap the middle is empty.
    """
    sink_end = min(sink, n0)
    win_start = max(sink_end, n0 - window)
    return sink_end, win_start


def budget_k(n0, k=None, k_num=0, k_den=0):
    """Middle budget for a sequence: a fixed k, or floor(k_num * n0 / k_den)
    when a proportional budget is given (integer arithmetic)."""
    if k_den and k_den > 0:
        return (k_num * n0) // k_den
    return int(k)


def dilation_m(k_b, topk_len, dilate_m=-1):
    """Number of top-ranked indices that are dilated: floor(k/3) by default
    (Sec. 5.1 defaults), clamped to the number actually selected."""
    m = k_b // 3 if dilate_m < 0 else dilate_m
    return max(0, min(m, topk_len))


def topk_middle(sigma, n0, k, sink, window):
    """Top-k oracle over the middle range (Sec. 4.1 Selection Criteria).

    sigma holds the score of every position [0, len(sigma)); only positions in
    the middle range of anchor length n0 compete.  Returns the selected
    positions ordered by (score descending, position ascending), so its first m
    entries are the top-m winners.  min(k, |middle|) entries are returned.
    """
    sink_end, win_start = region_bounds(n0, sink, window)
    pos = np.arange(sink_end, win_start, dtype=np.int64)
    if pos.size == 0 or k <= 0:
        return np.zeros(0, dtype=np.int64)
    sc = _f64(sigma)[pos]
    order = np.lexsort((pos, -sc))  # primary: -score, secondary: position
    return pos[order][: min(k, pos.size)]


def anchor_set(s_star, n0, sink, window):
    """Critical set C_t = sink U S* U window at the anchor (Sec. 4.1),
    ascending and without duplicates."""
    sink_end, win_start = region_bounds(n0, sink, window)
    parts = [np.arange(0, sink_end), np.asarray(s_star, dtype=np.int64),
             np.arange(win_start, n0)]
    return np.unique(np.concatenate(parts).astype(np.int64))


def reuse_set(s_star, m, r, n0, n, sink, window):
    """Dilated shared set used by a later step or another layer of the group.

    S_hat = S* U {p + j : p in top-m of S*, |j| <= r} (Eq. neighboring), the
    neighbourhood clipped to [0, n); plus the sink and every position from the
    anchor's window start up to the current length n.  Ascending, unique.
    """
    s_star = np.asarray(s_star, dtype=np.int64)
    sink_end, win_start = region_bounds(n0, sink, window)
    top_m = s_star[:m]
    neigh = (top_m[:, None] + np.arange(-r, r + 1)[None, :]).ravel()
    neigh = neigh[(neigh >= 0) & (neigh < n)]
    parts = [np.arange(0, min(sink_end, n)), s_star, neigh, np.arange(win_start, n)]
    return np.unique(np.concatenate(parts).astype(np.int64))


# ---------------------------------------------------------------------------
# Schedule (Sec. 4.1 blocks; retrieval ratio of Sec. 5.1)
# ---------------------------------------------------------------------------

def is_refresh(step, layer, s, G):
    """A (layer, step) pair scores and selects itself iff the step opens a
    block of s decode steps and the layer opens a group of G layers."""
    return step % s == 0 and layer % G == 0


def anchor_layer(layer, G):
    return (layer // G) * G


def retrieval_ratio(T, num_layers, s, G):
    """Average per-step retrieval ratio rho_hat = mean_t R_t / (H * N)
    (Sec. 5.1) for the pure step/layer schedule.  Heads retrieve together, so
    the head count cancels."""
    per_step = []
    for t in range(T):
        r_t = sum(1 for l in range(num_layers) if is_refresh(t, l, s, G))
        per_step.append(r_t / num_layers)
    return float(np.mean(per_step))


# ---------------------------------------------------------------------------
# Mass accounting (Sec. 2.3 and the unified-bounds appendix)
# ---------------------------------------------------------------------------

def retained_mass(A, S):
    """tau_S = sum over S of A_i."""
    return float(_f64(A)[np.asarray(S, dtype=np.int64)].sum())


def dropped_mass(A, S):
    """delta_S = 1 - tau_S."""
    return 1.0 - retained_mass(A, S)


def renormalised(A, S):
    """Truncated and renormalised distribution A_i / tau_S on S, 0 elsewhere."""
    A = _f64(A)
    out = np.zeros_like(A)
    S = np.asarray(S, dtype=np.int64)
    out[S] = A[S] / A[S].sum()
    return out


def tv_distance(P, Q):
    return 0.5 * float(np.abs(_f64(P) - _f64(Q)).sum())


def kl_divergence(P, Q):
    """KL(P || Q) over the support of P."""
    P = _f64(P)
    Q = _f64(Q)
    m = P > 0
    return float((P[m] * np.log(P[m] / Q[m])).sum())


def family_best_dropped(A, n, sink, window, k):
    """Smallest dropped mass over the family sink U window U (any k middle
    positions): the per-head top-k oracle of Sec. 2.3 restricted to the
    middle range, with the current length as anchor length."""
    A = _f64(A)
    sink_end, win_start = region_bounds(n, sink, window)
    mid = A[sink_end:win_start]
    kk = min(k, mid.size)
    best_mid = np.sort(mid)[::-1][:kk].sum() if kk > 0 else 0.0
    kept = A[:sink_end].sum() + A[win_start:n].sum() + best_mid
    return 1.0 - float(kept)


def binary_entropy(x):
    if x <= 0.0 or x >= 1.0:
        return 0.0
    return -x * math.log(x) - (1.0 - x) * math.log(1.0 - x)


def mi_loss_bound(delta, L):
    """g(delta) = 2 [h_b(delta) + delta log L] (Eq. mi_bound)."""
    return 2.0 * (binary_entropy(delta) + delta * math.log(L))


# ---------------------------------------------------------------------------
# Whole decode schedule over layers and steps
# ---------------------------------------------------------------------------

class DecodeOracle:
    """Runs the selection schedule of the hot path for one (batch, kv-head)
    unit across layers and decode steps, on explicit arrays.

    q[l][j]  : [g, d] query heads of the group at layer l, decode step j
    K[l], V[l]: [n_max, d] the unit's cache at layer l
    n_ctx    : cached context before step 0; step j attends n = n_ctx + j + 1.

    The anchor layer of a group at a refresh step attends its undilated
    critical set C(n0); every other (layer, step) attends the dilated shared
    set built from the group's latest anchor top-k (Sec. 4.1 and Def. 3.2, Sec. 2.2).
    With psaw = (n_layers, l_s, phi, alpha) every attended set is further
    restricted to the layer's PSAW-visible positions (CPE, Sec. 4.2 and 4.4);
    the selection itself is unchanged.
    """

    def __init__(self, sink, window, s, G, r=1, k=None, k_num=0, k_den=0,
                 dilate_m=-1, scale=None, psaw=None):
        self.sink = sink
        self.window = window
        self.s = s
        self.G = G
        self.r = r
        self.k = k
        self.k_num = k_num
        self.k_den = k_den
        self.dilate_m = dilate_m
        self.scale = scale
        self.psaw = psaw
        self.state = {}  # anchor layer -> (s_star, n0, k_b)

    def refresh(self, layer, Qg, K, n0):
        k_b = budget_k(n0, self.k, self.k_num, self.k_den)
        sigma = ranking_scores(Qg, _f64(K)[:n0])
        s_star = topk_middle(sigma, n0, k_b, self.sink, self.window)
        self.state[anchor_layer(layer, self.G)] = (s_star, n0, k_b)
        return s_star, anchor_set(s_star, n0, self.sink, self.window)

    def shared(self, layer, n):
        s_star, n0, k_b = self.state[anchor_layer(layer, self.G)]
        m = dilation_m(k_b, len(s_star), self.dilate_m)
        return reuse_set(s_star, m, self.r, n0, n, self.sink, self.window)

    def step_set(self, layer, step, Qg, K, n):
        """Index set that (layer, step) attends at current length n."""
        if is_refresh(step, layer, self.s, self.G):
            _, S = self.refresh(layer, Qg, K, n)
        else:
            S = self.shared(layer, n)
        return _psaw_apply(self.psaw, S, layer, n, self.sink)

    def attend(self, Qg, K, V, S):
        """Sparse attention of every query head of the group over S."""
        Qg = np.atleast_2d(_f64(Qg))
        outs = [sparse_attention(Qg[h], K, V, S, self.scale) for h in range(Qg.shape[0])]
        return np.stack([o[0] for o in outs]), np.array([o[1] for o in outs])


# ---------------------------------------------------------------------------
# Progressive sliding attention window (Sec. 4.2, Eq. psaw)
# ---------------------------------------------------------------------------

def psaw_boundary(layer, n_layers, t, l_s, phi, alpha):
    """P_l(t) of Eq. psaw for 1-based layer `layer` of `n_layers` at 1-based
    step t: 0 below the pruning depth l_s, else floor((1 - phi^(alpha (l -
    l_s) / (N - l_s))) t)."""
    if layer < l_s:
        return 0
    e = alpha * (layer - l_s) / (n_layers - l_s)
    return int(math.floor((1.0 - phi ** e) * t))


def psaw_visible_start(layer0, n_layers, n, sink, l_s, phi, alpha):
    """First visible non-sink 0-based position for 0-based layer `layer0` at
    current length n.  Eq. psaw masks the 1-based positions strictly between
    C_sink and P_l(t) (layer l = layer0 + 1, t = n); in 0-based terms the
    masked range is [C_sink, P - 1), so the visible set is [0, C_sink) U
    [max(C_sink, P - 1), n)."""
    P = psaw_boundary(layer0 + 1, n_layers, n, l_s, phi, alpha)
    sink_end = min(sink, n)
    return max(sink_end, P - 1)


def psaw_restrict(S, start, sink, n):
    """Index set S intersected with the PSAW-visible positions [0, C_sink) U
    [start, n) (CPE: the CIS set under the PSAW mask, Sec. 4.4)."""
    S = np.asarray(S, dtype=np.int64)
    sink_end = min(sink, n)
    return S[(S < sink_end) | ((S >= start) & (S < n))]


# ---------------------------------------------------------------------------
# PSAW at prefill (Sec. 4.2: the window narrows during prefill as well as
# decoding; the prefill panel of the PSAW/ETF figure)
# ---------------------------------------------------------------------------

def psaw_prefill_visible(layer0, n_layers, T, sink, l_s, phi, alpha):
    """First visible non-sink position of every query of a prefill of T
    tokens at 0-based layer `layer0`.  The query at 0-based position i has
    the i + 1 tokens [0, i] in view, so Eq. psaw is taken at t = i + 1: its
    first visible position is psaw_visible_start(layer0, ..., n = i + 1).
    Returns int64 [T]."""
    return np.array([psaw_visible_start(layer0, n_layers, i + 1, sink, l_s, phi, alpha)
                     for i in range(T)], dtype=np.int64)


def prefill_visible_set(i, sink, vis=None):
    """Keys the query at position i attends at prefill: the causal range
    [0, i] (Eq. attn_eq over the tokens in view), restricted under PSAW to
    [0, C_sink) U [vis, i]."""
    S = np.arange(i + 1, dtype=np.int64)
    return S if vis is None else psaw_restrict(S, vis, sink, i + 1)


def prefill_attention(Q, K, V, n, sink=0, vis_start=None, scale=None):
    """Prefill attention of one query head over a prompt of n tokens: row i
    of Q (position i) attends prefill_visible_set(i, sink, vis_start[i]) of
    its kv head's K, V; rows at positions >= n (past the prompt) give y = 0
    and lse = -inf.  Returns (y [T][d], lse [T])."""
    Q = _f64(Q)
    T, d = Q.shape
    y = np.zeros((T, d))
    lse = np.full(T, -np.inf)
    for i in range(min(T, n)):
        S = prefill_visible_set(i, sink, None if vis_start is None else int(vis_start[i]))
        y[i], lse[i] = sparse_attention(Q[i], K[: i + 1], V[: i + 1], S, scale)
    return y, lse


# ---------------------------------------------------------------------------
# Similarity gate (Sec. 4.1, Similarity Criteria; Eq. cos_sim)
# ---------------------------------------------------------------------------

def query_similar(q_now, q_ref, tau):
    """Whether sim(q_now, q_ref) = q_now . q_ref / (|q_now| |q_ref|) exceeds
    tau, for 0 <= tau <= 1 (Eq. cos_sim).

    Decided without a square root or a division: sim > tau holds exactly when
    the dot product is positive and dot^2 > tau^2 |q_now|^2 |q_ref|^2.  The
    three sums are formed in float64 and the comparison is evaluated as
    dot * dot > (tau * tau) * n_now * n_ref in that order, so that any
    implementation computing the same exact sums takes the same decision.
    A zero query is similar to nothing."""
    a = _f64(q_now).ravel()
    b = _f64(q_ref).ravel()
    dot = float(np.dot(a, b))
    n_now = float(np.dot(a, a))
    n_ref = float(np.dot(b, b))
    t = float(tau)
    return dot > 0.0 and dot * dot > (t * t) * n_now * n_ref


def group_similar(Qg_now, Qg_ref, tau):
    """A kv head's group shares only when every one of its query heads is
    similar to the same head of the reference step (the paper gates each
    head; a grouped-query kv head serves all of its query heads)."""
    Qn = np.atleast_2d(_f64(Qg_now))
    Qr = np.atleast_2d(_f64(Qg_ref))
    return all(query_similar(Qn[h], Qr[h], tau) for h in range(Qn.shape[0]))


def gate_choice(Qg_now, anchors, tau):
    """Sec. 4.1: a later query shares when an earlier query of its block is
    similar, choosing the most recent such query.  `anchors` lists the
    block's earlier retrieving steps as (step, Qg) in step order; returns the
    chosen step, or None when the query must retrieve."""
    for step, Qg_ref in reversed(list(anchors)):
        if group_similar(Qg_now, Qg_ref, tau):
            return step
    return None


class GatedDecodeOracle:
    """The schedule with the similarity gate, for one (batch, kv-head) unit.

    Blocks of s decode steps restrict sharing to adjacent queries.  At the
    anchor layer of each group of G layers, the block's first step retrieves;
    a later step shares the selection of the most recent earlier retrieving
    step of the block whose queries are similar (gate_choice), else it
    retrieves and becomes a reference itself.  A retrieving step attends its
    undilated critical set C(n); every other (layer, step) attends the
    dilated shared set of the selection it uses, grown by the tokens decoded
    since that selection (Sec. 4.1; Def. 3.2, Sec. 2.2).  The retrieval ratio
    is the fraction of (anchor layer, step) pairs that retrieve.  psaw as in
    DecodeOracle."""

    def __init__(self, sink, window, s, G, tau, r=1, k=None, k_num=0, k_den=0,
                 dilate_m=-1, scale=None, psaw=None):
        self.sink = sink
        self.window = window
        self.s = s
        self.G = G
        self.tau = tau
        self.r = r
        self.k = k
        self.k_num = k_num
        self.k_den = k_den
        self.dilate_m = dilate_m
        self.scale = scale
        self.psaw = psaw
        self.anchors = {}    # anchor layer -> [(step, Qg, s_star, n0, k_b)] of the block
        self.decision = {}   # (anchor layer, step) -> step whose selection is used
        self.retrievals = 0
        self.decisions = 0

    def _retrieve(self, layer, step, Qg, K, n):
        k_b = budget_k(n, self.k, self.k_num, self.k_den)
        sigma = ranking_scores(Qg, _f64(K)[:n])
        s_star = topk_middle(sigma, n, k_b, self.sink, self.window)
        self.anchors[layer].append((step, np.atleast_2d(_f64(Qg)).copy(), s_star, n, k_b))
        return s_star

    def _shared_of(self, layer, src, n):
        for step, _, s_star, n0, k_b in self.anchors[layer]:
            if step == src:
                m = dilation_m(k_b, len(s_star), self.dilate_m)
                return reuse_set(s_star, m, self.r, n0, n, self.sink, self.window)
        raise KeyError(src)

    def step_set(self, layer, step, Qg, K, n):
        """Index set that (layer, step) attends at current length n.  K is
        read only where the anchor layer retrieves."""
        return _psaw_apply(self.psaw, self._step_set(layer, step, Qg, K, n), layer, n, self.sink)

    def _step_set(self, layer, step, Qg, K, n):
        a = anchor_layer(layer, self.G)
        if layer == a:
            if step % self.s == 0:
                self.anchors[a] = []
            src = gate_choice(Qg, [(st, q) for st, q, *_ in self.anchors[a]], self.tau)
            self.decisions += 1
            if src is None:
                self.retrievals += 1
                s_star = self._retrieve(a, step, Qg, K, n)
                self.decision[(a, step)] = step
                return anchor_set(s_star, n, self.sink, self.window)
            self.decision[(a, step)] = src
            return self._shared_of(a, src, n)
        return self._shared_of(a, self.decision[(a, step)], n)

    def attend(self, Qg, K, V, S):
        """Sparse attention of every query head of the group over S."""
        Qg = np.atleast_2d(_f64(Qg))
        outs = [sparse_attention(Qg[h], K, V, S, self.scale) for h in range(Qg.shape[0])]
        return np.stack([o[0] for o in outs]), np.array([o[1] for o in outs])


def _psaw_apply(psaw, S, layer, n, sink):
    if psaw is None:
        return S
    n_layers, l_s, phi, alpha = psaw
    start = psaw_visible_start(layer, n_layers, n, sink, l_s, phi, alpha)
    return psaw_restrict(S, start, sink, n)


def brute_force_topk_mass(A, n0, k, sink, window):
    """Largest retained mass over every k-subset of the middle range, by
    enumeration (tiny inputs only); used to pin the top-k oracle."""
    sink_end, win_start = region_bounds(n0, sink, window)
    mid = list(range(sink_end, win_start))
    kk = min(k, len(mid))
    best = -1.0
    A = _f64(A)
    for comb in itertools.combinations(mid, kk):
        best = max(best, float(A[list(comb)].sum()))
    return best
