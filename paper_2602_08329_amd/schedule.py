"""Host-side decode schedule over layers and steps (Sec. 4.1 blocks, Def. 3.2
sharing, layer groups).

For decode step j and layer l:
  * (l, j) with prhs_schedule == REFRESH (j % s == 0 and l % G == 0) runs
    prhs_select on its own q and K, then attends its critical set C(n0);
  * every other layer of the group attends the dilated shared set R(n) over
    its own K/V.
R(n) is R(n0) followed by the positions decoded since the anchor, [n0, n)
(dilated neighbours of the middle range stay below n0 and [n0, n) lies in the
recency window).  By default the refresh therefore writes R(n0) in the same
launch (prhs_select_shared), and later steps attend R(n0) plus that tail
through prhs_reuse_decode_attn.  With per_step_sets=True, prhs_dilate_reuse
instead builds R(n) at every step and prhs_sparse_decode_attn attends it.
The carried state is the per-group top-k buffer, the shared set and the anchor
lengths n0, which are simply the sequence lengths of the refresh step.
"""

from __future__ import annotations

import math

import torch

from . import binding as B


def psaw_defaults(n_layers):
    """Sec. 5.1: pruning from l_s = floor(3 N / 4), phi = 0.7, alpha = 1."""
    return (3 * n_layers) // 4, 0.7, 1.0


def psaw_layers(n_layers, sink, psaw):
    """Window descriptors (binding.psaw) of the layers that can mask keys
    under psaw = (l_s, phi, alpha): the 1-based layer l = layer + 1 masks
    only when l > l_s (at l = l_s the factor is 1 - phi^0 = 0).  Returns
    {layer: descriptor}; the library evaluates Eq. psaw from them."""
    if psaw is None:
        return {}
    l_s, phi, alpha = psaw
    return {l: B.psaw(l, n_layers, l_s, phi, alpha, sink) for l in range(n_layers) if l + 1 > l_s}


def capture_steps(fn, steps):
    """Captures the launches of fn(j) for j in steps (for example a runner's
    step, selection_step or dense_step) into a HIP graph and returns it
    (torch.cuda.CUDAGraph); replay() reruns the same launches on the same
    buffers, back to back on the current stream and without host launch
    overhead.  Every launch of the path takes the current stream and none
    records a memset, so a replay computes what the eager calls compute.  The
    runner's host-side schedule checks run at capture time."""
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for j in steps:
            fn(j)
    return graph


class DecodeRunner:
    """Runs the hot path of a synthetic workload (paper_2602_08329_amd.synth)
    whose inputs already live on the GPU."""

    def __init__(self, inp, device="cuda", per_step_sets=False, psaw=None):
        w = inp.w
        self.per_step_sets = per_step_sets
        self.reuses = w.G > 1 or w.s > 1   # some layer-step attends a shared set
        self.w = w
        self.inp = inp
        self.device = torch.device(device)
        self.L = len(inp.K)
        self.groups = (self.L + w.G - 1) // w.G
        self.scale = 1.0 / math.sqrt(w.d)
        T, Bsz = w.steps, w.batch
        lens = torch.tensor([[n + j + 1 for n in w.n_ctx] for j in range(T)], dtype=torch.int32)
        self.seq_lens = lens.to(self.device)
        self.max_seq_len = w.capacity
        self.params = B.params(k=w.k, k_num=w.k_num, k_den=w.k_den, sink=w.sink,
                               window=w.window, dilate_m=w.dilate_m, dilate_r=w.r,
                               refresh_every=w.s, layer_group=w.G)
        table = inp.block_table.to(self.device) if inp.block_table is not None else None
        # one descriptor per (layer, step): only the lengths pointer differs
        self.kv = [[B.KV(inp.K[l], inp.V[l], self.seq_lens[j], self.max_seq_len, w.hq, table)
                    for j in range(T)] for l in range(self.L)]
        self.k_cap = max(1, B.prhs_max_topk(self.params, self.max_seq_len))
        self.set_cap = max(1, B.prhs_set_capacity(self.params, self.max_seq_len),
                           min(self.max_seq_len, w.sink + self.k_cap + w.window))
        dev = self.device
        i32 = torch.int32
        G_ = self.groups
        self.topk_idx = torch.zeros(G_, Bsz, w.hkv, self.k_cap, dtype=i32, device=dev)
        self.topk_len = torch.zeros(G_, Bsz, w.hkv, dtype=i32, device=dev)
        self.anchor_set = torch.zeros(G_, Bsz, w.hkv, self.set_cap, dtype=i32, device=dev)
        self.anchor_len = torch.zeros(G_, Bsz, w.hkv, dtype=i32, device=dev)
        self.shared_set = torch.zeros(G_, Bsz, w.hkv, self.set_cap, dtype=i32, device=dev)
        self.shared_len = torch.zeros(G_, Bsz, w.hkv, dtype=i32, device=dev)
        self.anchor_step = [None] * G_
        kv0 = self.kv[0][0]
        self.ws_select = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SELECT, kv0, self.params), dev)
        self.ws_attn = B.workspace(
            B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv0, self.params, self.set_cap), dev)
        self.ws_dense = B.workspace(B.prhs_workspace_size(B.PRHS_OP_DENSE_ATTN, kv0, self.params), dev)
        self.out = torch.zeros(Bsz, w.hq, w.d, dtype=torch.float32, device=dev)
        self.lse = torch.zeros(Bsz, w.hq, dtype=torch.float32, device=dev)
        # PSAW (Sec. 4.2): psaw = (l_s, phi, alpha); the layers that can mask
        # attend the schedule's sets through the pool form (identity rows and
        # per-unit anchor lengths) with their window descriptor
        self.psaw = psaw
        self.psaw_desc = psaw_layers(self.L, w.sink, psaw)
        if self.psaw_desc:
            self.unit_ids = torch.arange(Bsz * w.hkv, dtype=i32, device=dev)
            self.unit_lens = self.seq_lens.repeat_interleave(w.hkv, dim=1).contiguous()

    def psaw_start(self, l, j):
        """First visible non-sink position of every sequence at layer l, step
        j (host list, from the library's Eq. psaw), or None when the layer
        does not mask."""
        ps = self.psaw_desc.get(l)
        if ps is None:
            return None
        return [B.prhs_psaw_first_visible(ps, n + j + 1) for n in self.w.n_ctx]

    # -- pieces -------------------------------------------------------------
    def refresh(self, gi, j):
        l = gi * self.w.G
        if self.per_step_sets or not self.reuses:
            B.prhs_select(self.kv[l][j], self.inp.q[l, j], self.params, self.topk_idx[gi],
                          self.topk_len[gi], self.anchor_set[gi], self.anchor_len[gi],
                          self.ws_select)
        else:
            B.prhs_select_shared(self.kv[l][j], self.inp.q[l, j], self.params, self.topk_idx[gi],
                                 self.topk_len[gi], self.anchor_set[gi], self.anchor_len[gi],
                                 self.shared_set[gi], self.shared_len[gi], self.ws_select)
        self.anchor_step[gi] = j

    def _anchor(self, gi, j):
        j0 = self.anchor_step[gi]
        if j0 is None or j - j0 >= self.w.s or j < j0:
            raise RuntimeError(f"group {gi} has no anchor for step {j}")
        return j0

    def share(self, gi, j):
        j0 = self._anchor(gi, j)
        n = self.seq_lens[j] if self.per_step_sets else self.seq_lens[j0]
        B.prhs_dilate_reuse(self.params, self.topk_idx[gi], self.topk_len[gi], self.seq_lens[j0],
                            n, self.shared_set[gi], self.shared_len[gi])

    def shares_at(self, j):
        """Groups whose shared set prhs_dilate_reuse (re)builds at step j (in
        the default mode the refresh writes it)."""
        w = self.w
        if self.per_step_sets:
            return list(range(self.groups)) if (w.G > 1 or j % w.s != 0) else []
        return []

    def set_for(self, l, j):
        """(set, len, tail_start) that layer l attends at step j: the rows are
        set[:len], then [tail_start[b], n_b) when tail_start is not None."""
        gi = l // self.w.G
        if B.prhs_schedule(j, l, self.params) == B.PRHS_REFRESH:
            return self.anchor_set[gi], self.anchor_len[gi], None
        j0 = self._anchor(gi, j)
        tail = None if self.per_step_sets else self.seq_lens[j0]
        return self.shared_set[gi], self.shared_len[gi], tail

    def attend(self, l, j, out=None, lse=None):
        s, n, tail = self.set_for(l, j)
        out = self.out if out is None else out
        lse = self.lse if lse is None else lse
        ps = self.psaw_desc.get(l)
        if ps is not None:
            # the same set through the pool form, under the layer's PSAW mask
            if tail is None:
                utail = self.unit_lens[j]
            else:
                utail = tail.repeat_interleave(self.w.hkv).contiguous()
            B.prhs_pool_decode_attn(self.kv[l][j], self.inp.q[l, j], s, n, self.unit_ids, utail,
                                    self.scale, out, lse, self.ws_attn, psaw=ps)
        elif tail is None:
            B.prhs_sparse_decode_attn(self.kv[l][j], self.inp.q[l, j], s, n, self.scale, out, lse,
                                      self.ws_attn)
        else:
            B.prhs_reuse_decode_attn(self.kv[l][j], self.inp.q[l, j], s, n, tail, self.scale, out,
                                     lse, self.ws_attn)

    def dense(self, l, j, out=None, lse=None):
        B.prhs_dense_decode_attn(self.kv[l][j], self.inp.q[l, j], self.scale,
                                 self.out if out is None else out,
                                 self.lse if lse is None else lse, self.ws_dense)

    # -- whole decode steps -------------------------------------------------
    def selection_step(self, j):
        """Refresh and reuse-set construction of step j for every group."""
        w = self.w
        shares = set(self.shares_at(j))
        for gi in range(self.groups):
            if B.prhs_schedule(j, gi * w.G, self.params) == B.PRHS_REFRESH:
                self.refresh(gi, j)
            if gi in shares:
                self.share(gi, j)

    def step(self, j, outs=None):
        """One sparse decode step j over every layer; outs[l] receives layer
        l's (out, lse) when given."""
        self.selection_step(j)
        for l in range(self.L):
            o = None if outs is None else outs[l]
            self.attend(l, j, *(o if o is not None else (None, None)))

    def dense_step(self, j, outs=None):
        for l in range(self.L):
            o = None if outs is None else outs[l]
            self.dense(l, j, *(o if o is not None else (None, None)))


class GatedDecodeRunner(DecodeRunner):
    """The decode schedule with the similarity gate (Sec. 4.1, Similarity
    Criteria): blocks of s steps; at every step each group's anchor layer
    takes the gate and refreshes its retrieving units (prhs_gate_select: the
    gate inside the refresh launch where that is one fused kernel), and every
    layer attends its pool row plus the decoded tail through
    prhs_pool_decode_attn.  Per group the state is the block's reference
    queries, retrieval flags and lengths per slot, and the set pool
    [2][s][B][Hkv][set_cap] (kind 0 critical sets, kind 1 shared sets).

    With concurrent=True, step() runs the two kinds of unit concurrently
    (Sec. 4.4: shared heads need no retrieval, so their attention does not
    wait for it): the current stream takes the gate, the refresh and then
    the retrieving units' attention; a second stream of the same priority
    takes the same gate decisions without recording them (prhs_gate, record
    off, into arrays of its own) and attends the sharing units.  The two
    launches of a layer write disjoint units and use separate workspaces.
    Otherwise step() is selection_step() and every layer's attend(), one
    launch after another (the faster order on this GPU: a launch restricted
    to half the units keeps half the workgroups busy for about as long as a
    full launch takes)."""

    def __init__(self, inp, device="cuda", tau=0.8, psaw=None, concurrent=False):
        super().__init__(inp, device, psaw=psaw)
        w = self.w
        self.tau = float(tau)
        self.concurrent = concurrent
        dev, i32 = self.device, torch.int32
        G_, S, U = self.groups, w.s, w.batch * w.hkv
        q = inp.q
        self.ref_q = torch.zeros((G_, S) + tuple(q.shape[2:]), dtype=q.dtype, device=dev)
        self.ref_valid = torch.zeros(G_, S, U, dtype=i32, device=dev)
        self.slot_lens = torch.zeros(G_, S, w.batch, dtype=i32, device=dev)
        self.pool = torch.zeros(G_, 2, S, w.batch, w.hkv, self.set_cap, dtype=i32, device=dev)
        self.pool_len = torch.zeros(G_, 2, S, w.batch, w.hkv, dtype=i32, device=dev)
        self.choice = torch.zeros(G_, U, dtype=i32, device=dev)
        self.row_anchor = torch.zeros(G_, U, dtype=i32, device=dev)
        self.row_other = torch.zeros(G_, U, dtype=i32, device=dev)
        self.tail = torch.zeros(G_, U, dtype=i32, device=dev)
        # the sharing branch's own copy of the decisions and its workspace
        self.side_choice = torch.zeros(G_, U, dtype=i32, device=dev)
        self.side_row_anchor = torch.zeros(G_, U, dtype=i32, device=dev)
        self.side_row_other = torch.zeros(G_, U, dtype=i32, device=dev)
        self.side_tail = torch.zeros(G_, U, dtype=i32, device=dev)
        self.ws_attn_side = torch.zeros_like(self.ws_attn)
        self.side_stream = None
        self.gated_step = [None] * G_

    def _gate_order(self, gi, j):
        if j % self.w.s != 0 and self.gated_step[gi] != j - 1:
            raise RuntimeError(f"group {gi}: the gate runs at every step of a block in order")

    def selection_step(self, j):
        w = self.w
        slot = j % w.s
        for gi in range(self.groups):
            self._gate_order(gi, j)
            l = gi * w.G
            B.prhs_gate_select(self.kv[l][j], self.inp.q[l, j], self.params, self.tau, slot,
                               self.ref_q[gi], self.ref_valid[gi], self.slot_lens[gi],
                               self.choice[gi], self.row_anchor[gi], self.row_other[gi],
                               self.tail[gi], self.topk_idx[gi], self.topk_len[gi],
                               self.pool[gi, 0, slot], self.pool_len[gi, 0, slot],
                               self.pool[gi, 1, slot], self.pool_len[gi, 1, slot], self.ws_select)
            self.gated_step[gi] = j

    def set_for(self, l, j):
        """(pool, pool_len, unit_row, unit_tail) that layer l attends at step j."""
        gi = l // self.w.G
        if self.gated_step[gi] != j:
            raise RuntimeError(f"group {gi} has not been gated at step {j}")
        rows = self.row_anchor[gi] if l % self.w.G == 0 else self.row_other[gi]
        return self.pool[gi], self.pool_len[gi], rows, self.tail[gi]

    def attend(self, l, j, out=None, lse=None):
        pool, plen, rows, tail = self.set_for(l, j)
        B.prhs_pool_decode_attn(self.kv[l][j], self.inp.q[l, j], pool, plen, rows, tail,
                                self.scale, self.out if out is None else out,
                                self.lse if lse is None else lse, self.ws_attn,
                                psaw=self.psaw_desc.get(l))

    def step(self, j, outs=None):
        """One gated decode step over every layer; outs[l] receives layer
        l's (out, lse) when given."""
        if not self.concurrent:
            return DecodeRunner.step(self, j, outs)
        w = self.w
        slot = j % w.s
        main = torch.cuda.current_stream(self.device)
        if self.side_stream is None:
            self.side_stream = torch.cuda.Stream(self.device)   # default priority
        side = self.side_stream

        def dest(l):
            o = None if outs is None else outs[l]
            return (self.out, self.lse) if o is None else o

        side.wait_stream(main)
        with torch.cuda.stream(side):
            for gi in range(self.groups):
                self._gate_order(gi, j)
                l0 = gi * w.G
                B.prhs_gate(self.inp.q[l0, j], self.seq_lens[j], self.tau, slot, self.ref_q[gi],
                            self.ref_valid[gi], self.slot_lens[gi], self.side_choice[gi],
                            self.side_row_anchor[gi], self.side_row_other[gi],
                            self.side_tail[gi], w.hkv, stream=side, record=False)
                for l in range(l0, min(l0 + w.G, self.L)):
                    rows = self.side_row_anchor[gi] if l == l0 else self.side_row_other[gi]
                    out, lse = dest(l)
                    B.prhs_pool_decode_attn(self.kv[l][j], self.inp.q[l, j], self.pool[gi],
                                            self.pool_len[gi], rows, self.side_tail[gi],
                                            self.scale, out, lse, self.ws_attn_side,
                                            stream=side, psaw=self.psaw_desc.get(l),
                                            unit_gate=self.side_choice[gi],
                                            units_side=B.PRHS_UNITS_SHARING)
        self.selection_step(j)
        for gi in range(self.groups):
            l0 = gi * w.G
            for l in range(l0, min(l0 + w.G, self.L)):
                rows = self.row_anchor[gi] if l == l0 else self.row_other[gi]
                out, lse = dest(l)
                B.prhs_pool_decode_attn(self.kv[l][j], self.inp.q[l, j], self.pool[gi],
                                        self.pool_len[gi], rows, self.tail[gi], self.scale, out,
                                        lse, self.ws_attn, psaw=self.psaw_desc.get(l),
                                        unit_gate=self.choice[gi],
                                        units_side=B.PRHS_UNITS_RETRIEVING)
        main.wait_stream(side)

    def retrieving_units(self):
        """Units of every group that retrieved at the last gated step."""
        return int((self.choice < 0).sum().item())
