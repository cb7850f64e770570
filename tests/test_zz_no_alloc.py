"""The no-allocation sparse attention entry point: its outputs equal those of
prhs_sparse_decode_attn (same kernels, its own workspace) bit for bit, on two
calls in a row whose second input is smaller, and both are within the
tolerance of the oracle on sampled heads."""

import math

import numpy as np
import pytest
import torch

import oracle as O
from paper_2602_08329_amd import binding as B
from paper_2602_08329_amd import synth

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


def _case(batch, hq, hkv, lens, cap, seed):
    inp = synth.random_inputs(batch, hq, hkv, 128, lens, seed=seed, device=DEV)
    seq = torch.tensor(lens, dtype=torch.int32, device=DEV)
    kv = B.KV(inp.K[0], inp.V[0], seq, inp.w.capacity, hq)
    rng = np.random.default_rng(seed)
    idx = torch.zeros(batch, hkv, cap, dtype=torch.int32)
    ln = torch.zeros(batch, hkv, dtype=torch.int32)
    sets = {}
    for b in range(batch):
        for g in range(hkv):
            size = int(rng.integers(1, min(cap, lens[b]) + 1))
            S = np.sort(rng.choice(lens[b], size=size, replace=False))
            sets[(b, g)] = S
            idx[b, g, :size] = torch.tensor(S, dtype=torch.int32)
            ln[b, g] = size
    return inp, kv, idx.to(DEV), ln.to(DEV), sets


def _run(inp, kv, idx, ln, static):
    B_, Hq = kv.c.batch, kv.c.num_q_heads
    out = torch.full((B_, Hq, 128), float("nan"), device=DEV)
    lse = torch.full((B_, Hq), float("nan"), device=DEV)
    scale = 1 / math.sqrt(128)
    if static:
        B.prhs_sparse_decode_attn_static(kv, inp.q[0, 0], idx, ln, scale, out, lse)
    else:
        ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv, None, idx.shape[-1]),
                         DEV)
        B.prhs_sparse_decode_attn(kv, inp.q[0, 0], idx, ln, scale, out, lse, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def test_static_scratch_matches_workspace_entry_point():
    # first call: many split units (the scratch holds their partials); second
    # call: a smaller batch, fewer heads and shorter sets over a fresh cache,
    # so the scratch still holds the first call's larger contents
    for case in [dict(batch=3, hq=32, hkv=8, lens=(9000, 5000, 3000), cap=4000, seed=81),
                 dict(batch=1, hq=8, hkv=2, lens=(2000,), cap=900, seed=82)]:
        print(f"case {case}", flush=True)
        inp, kv, idx, ln, sets = _case(**case)
        ys, ls = _run(inp, kv, idx, ln, static=True)
        yw, lw = _run(inp, kv, idx, ln, static=False)
        assert not np.isnan(ys).any()
        assert np.array_equal(ys, yw) and np.array_equal(ls, lw)
        G = case["hq"] // case["hkv"]
        for (b, g) in list(sets)[:: max(1, len(sets) // 5)]:
            K, V = synth.gather_unit(inp, 0, b, g, case["lens"][b])
            Qg = synth.query_group(inp, 0, 0, b, g)
            for i in range(G):
                yr, lr = O.sparse_attention(Qg[i], K, V, sets[(b, g)])
                h = g * G + i
                assert np.abs(ys[b, h] - yr).max() <= 2e-3 * np.abs(yr).max()
                assert abs(ls[b, h] - lr) <= 1e-4 * max(1.0, abs(lr))
