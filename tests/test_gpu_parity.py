"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Index sets are compared bit for bit (inputs on the j/16 grid make GPU fp32
scores exact, see the synth module); attention outputs per (batch, query head)
must satisfy |y_gpu - y_ref|_inf / |y_ref|_inf <= 2e-3 for bf16 inputs and
1e-5 for fp32 inputs, with y_ref the fp64 oracle over the same set.
"""

import math

import numpy as np
import pytest
import torch

import oracle as O
from tests.compare import topk_layout
from paper_2602_08329_amd import binding as B
from paper_2602_08329_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
TOL = {"bf16": 2e-3, "f32": 1e-5}
LSE_TOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def lens_tensor(lens):
    return torch.tensor(list(lens), dtype=torch.int32, device=DEV)


def kv_for(inp, lens, layer=0):
    t = lens_tensor(lens)
    table = inp.block_table
    return B.KV(inp.K[layer], inp.V[layer], t, inp.w.capacity, inp.w.hq, table), t


def assert_close(y, lse, y_ref, lse_ref, tol, label):
    y = np.asarray(y, dtype=np.float64)
    if not np.isfinite(lse_ref):
        assert np.all(y == 0.0), f"{label}: empty set must give zeros"
        assert lse == -math.inf, f"{label}: empty set must give lse=-inf"
        return
    den = np.abs(y_ref).max()
    err = np.abs(y - y_ref).max() / (den if den > 0 else 1.0)
    assert err <= tol, f"{label}: rel err {err:.3e} > {tol}"
    assert abs(lse - lse_ref) <= LSE_TOL * max(1.0, abs(lse_ref)), \
        f"{label}: lse {lse} vs {lse_ref}"


def run_dense(inp, lens, layer=0, step=0):
    kv, _ = kv_for(inp, lens, layer)
    w = inp.w
    out = torch.full((w.batch, w.hq, w.d), float("nan"), device=DEV)
    lse = torch.full((w.batch, w.hq), float("nan"), device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_DENSE_ATTN, kv), DEV)
    B.prhs_dense_decode_attn(kv, inp.q[layer, step], 1 / math.sqrt(w.d), out, lse, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def run_sparse(inp, lens, sets, set_cap, layer=0, step=0):
    w = inp.w
    kv, _ = kv_for(inp, lens, layer)
    idx = torch.zeros(w.batch, w.hkv, set_cap, dtype=torch.int32)
    ln = torch.zeros(w.batch, w.hkv, dtype=torch.int32)
    for (b, g), S in sets.items():
        idx[b, g, : len(S)] = torch.tensor(S, dtype=torch.int32)
        ln[b, g] = len(S)
    idx, ln = idx.to(DEV), ln.to(DEV)
    out = torch.full((w.batch, w.hq, w.d), float("nan"), device=DEV)
    lse = torch.full((w.batch, w.hq), float("nan"), device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv, None, set_cap), DEV)
    B.prhs_sparse_decode_attn(kv, inp.q[layer, step], idx, ln, 1 / math.sqrt(w.d), out, lse, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


DENSE_CASES = [
    # dtype, d, paged, Hq, Hkv, lens
    ("bf16", 128, False, 8, 2, (1, 37, 300, 1025)),
    ("bf16", 64, True, 4, 4, (700, 5, 64)),
    ("bf16", 128, True, 32, 8, (4100, 129)),
    ("bf16", 128, False, 16, 1, (2000,)),
    ("f32", 64, False, 4, 4, (129, 3000)),
    ("f32", 128, True, 4, 2, (17, 450, 33)),
]


@pytest.mark.parametrize("dtype,d,paged,hq,hkv,lens", DENSE_CASES)
def test_dense_attention(dtype, d, paged, hq, hkv, lens):
    inp = synth.random_inputs(len(lens), hq, hkv, d, lens, dtype=dtype, paged=paged,
                              seed=11 + d + len(lens), grid=False, key_scale=1.5, device=DEV)
    y, lse = run_dense(inp, lens)
    g = hq // hkv
    for b, n in enumerate(lens):
        for hk in range(hkv):
            K, V = synth.gather_unit(inp, 0, b, hk, n)
            Qg = synth.query_group(inp, 0, 0, b, hk)
            for j in range(g):
                h = hk * g + j
                yr, lr = O.dense_attention(Qg[j], K, V)
                assert_close(y[b, h], lse[b, h], yr, lr, TOL[dtype], f"b{b} h{h} n{n}")


def test_dense_zero_length_gives_empty():
    inp = synth.random_inputs(2, 4, 2, 128, (50, 70), seed=5, device=DEV)
    y, lse = run_dense(inp, (0, 70))
    assert np.all(y[0] == 0) and np.all(lse[0] == -np.inf)
    assert np.isfinite(y[1]).all()


SPARSE_CASES = [
    ("bf16", 128, False, 8, 2, (900, 77, 2500)),
    ("bf16", 128, True, 32, 8, (3000, 1200)),
    ("bf16", 64, False, 4, 4, (500, 640)),
    ("f32", 64, True, 4, 4, (1000, 40)),
]


@pytest.mark.parametrize("dtype,d,paged,hq,hkv,lens", SPARSE_CASES)
def test_sparse_attention_oracle_sets(dtype, d, paged, hq, hkv, lens):
    inp = synth.random_inputs(len(lens), hq, hkv, d, lens, dtype=dtype, paged=paged,
                              seed=23 + d, grid=False, key_scale=1.5, device=DEV)
    rng = np.random.default_rng(7)
    sets = {}
    for b, n in enumerate(lens):
        for g in range(hkv):
            kind = (b * hkv + g) % 4
            if kind == 0:
                S = []                                    # empty set
            elif kind == 1:
                S = list(range(n))                        # everything
            else:
                size = int(rng.integers(1, n + 1))
                S = sorted(rng.choice(n, size=size, replace=False).tolist())
            sets[(b, g)] = S
    set_cap = max(len(s) for s in sets.values()) + 5
    y, lse = run_sparse(inp, lens, sets, set_cap)
    gq = hq // hkv
    for (b, g), S in sets.items():
        K, V = synth.gather_unit(inp, 0, b, g, lens[b])
        Qg = synth.query_group(inp, 0, 0, b, g)
        for j in range(gq):
            yr, lr = O.sparse_attention(Qg[j], K, V, S)
            assert_close(y[b, g * gq + j], lse[b, g * gq + j], yr, lr, TOL[dtype],
                         f"b{b} g{g} |S|={len(S)}")


@pytest.mark.parametrize("paged", [False, True])
def test_sparse_attention_more_units_than_cus(paged):
    """More unsplit units than CUs (several workgroups per CU), with varied
    lengths and set sizes: every unit's output lands in its own place."""
    lens = tuple(100 + (i * 379) % 1100 for i in range(150))
    hq, hkv = 8, 2
    inp = synth.random_inputs(len(lens), hq, hkv, 128, lens, paged=paged, seed=91,
                              grid=False, key_scale=1.5, device=DEV)
    rng = np.random.default_rng(11)
    sets = {}
    for b, n in enumerate(lens):
        for g in range(hkv):
            size = int(rng.integers(1, min(n, 400) + 1))
            sets[(b, g)] = sorted(rng.choice(n, size=size, replace=False).tolist())
    y, lse = run_sparse(inp, lens, sets, 400)
    gq = hq // hkv
    for (b, g), S in sets.items():
        K, V = synth.gather_unit(inp, 0, b, g, lens[b])
        Qg = synth.query_group(inp, 0, 0, b, g)
        for j in range(gq):
            yr, lr = O.sparse_attention(Qg[j], K, V, S)
            assert_close(y[b, g * gq + j], lse[b, g * gq + j], yr, lr, TOL["bf16"],
                         f"b{b} g{g} |S|={len(S)}")


@pytest.mark.parametrize("dtype,set_cap", [("bf16", 512), ("bf16", 513), ("f32", 512), ("f32", 513)])
def test_sparse_attention_unsplit_boundary(dtype, set_cap):
    """Sets of at most 512 rows per unit run in one launch without a merge,
    longer ones split across workgroups: both sides of that boundary, with
    sets filling the capacity and shorter ones."""
    lens = (700, 512, 90)
    d, hq, hkv = (128, 8, 2) if dtype == "bf16" else (64, 4, 4)
    inp = synth.random_inputs(len(lens), hq, hkv, d, lens, dtype=dtype, paged=False,
                              seed=41, grid=False, key_scale=1.5, device=DEV)
    rng = np.random.default_rng(11)
    sets = {}
    for b, n in enumerate(lens):
        for g in range(hkv):
            top = min(n, set_cap)
            size = top if g == 0 else int(rng.integers(1, top + 1))
            sets[(b, g)] = sorted(rng.choice(n, size=size, replace=False).tolist())
    y, lse = run_sparse(inp, lens, sets, set_cap)
    gq = hq // hkv
    for (b, g), S in sets.items():
        K, V = synth.gather_unit(inp, 0, b, g, lens[b])
        Qg = synth.query_group(inp, 0, 0, b, g)
        for j in range(gq):
            yr, lr = O.sparse_attention(Qg[j], K, V, S)
            assert_close(y[b, g * gq + j], lse[b, g * gq + j], yr, lr, TOL[dtype],
                         f"b{b} g{g} |S|={len(S)}")


def test_attention_skips_entries_and_pages_outside_the_cache():
    """Device arrays the host cannot check: set entries outside [0, n) (negative,
    at or past n, huge), block-table entries outside the page pool (-1, past
    the last page) and a sequence length beyond max_seq_len.  The kernels skip
    such entries and pages and clamp the length, so the outputs are attention
    over the remaining valid positions."""
    lens = (300, 200)
    inp = synth.random_inputs(2, 8, 2, 128, lens, paged=True, seed=61, grid=False,
                              key_scale=1.5, device=DEV)
    w = inp.w
    ps = w.page_size
    table = inp.block_table.clone()
    P = inp.K[0].shape[0]
    bad = {(0, 1): -1, (1, 0): P + 7, (0, 3): 1 << 30}
    for (b, pg), v in bad.items():
        table[b, pg] = v
    kv = B.KV(inp.K[0], inp.V[0], lens_tensor(lens), w.capacity, w.hq, table)
    rng = np.random.default_rng(17)
    set_cap = 160
    idx = torch.zeros(2, 2, set_cap, dtype=torch.int32)
    ln = torch.zeros(2, 2, dtype=torch.int32)
    sets = {}
    for b, n in enumerate(lens):
        for g in range(2):
            S = sorted(rng.choice(n, size=120, replace=False).tolist())
            S = [-5, -1] + S + [n, n + 100, w.capacity + 5, 1 << 30]
            idx[b, g, : len(S)] = torch.tensor(S, dtype=torch.int32)
            ln[b, g] = len(S)
            sets[(b, g)] = [i for i in S if 0 <= i < n and (b, i // ps) not in bad]
    out = torch.full((2, 8, 128), float("nan"), device=DEV)
    lse = torch.full((2, 8), float("nan"), device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv, None, set_cap), DEV)
    B.prhs_sparse_decode_attn(kv, inp.q[0, 0], idx.to(DEV), ln.to(DEV), 1 / math.sqrt(128), out,
                              lse, ws)
    torch.cuda.synchronize()
    y, ls = out.cpu().numpy(), lse.cpu().numpy()
    for (b, g), S in sets.items():
        K, V = synth.gather_unit(inp, 0, b, g, lens[b])
        Qg = synth.query_group(inp, 0, 0, b, g)
        for j in range(4):
            yr, lr = O.sparse_attention(Qg[j], K, V, S)
            assert_close(y[b, g * 4 + j], ls[b, g * 4 + j], yr, lr, TOL["bf16"], f"b{b} g{g}")
    # a length beyond max_seq_len is clamped to it: dense attention over the
    # whole cache of the longest sequence (every row of it is valid)
    big = torch.tensor([w.capacity + 1000, lens[1]], dtype=torch.int32, device=DEV)
    kvc = B.KV(inp.K[0], inp.V[0], big, w.capacity, w.hq, inp.block_table)
    out.fill_(float("nan"))
    wsd = B.workspace(B.prhs_workspace_size(B.PRHS_OP_DENSE_ATTN, kvc), DEV)
    B.prhs_dense_decode_attn(kvc, inp.q[0, 0], 1 / math.sqrt(128), out, lse, wsd)
    torch.cuda.synchronize()
    y, ls = out.cpu().numpy(), lse.cpu().numpy()
    for g in range(2):
        K, V = synth.gather_unit(inp, 0, 0, g, w.capacity)
        Qg = synth.query_group(inp, 0, 0, 0, g)
        for j in range(4):
            yr, lr = O.dense_attention(Qg[j], K, V)
            assert_close(y[0, g * 4 + j], ls[0, g * 4 + j], yr, lr, TOL["bf16"], f"clamped g{g}")


def test_sparse_full_set_matches_dense_kernel():
    lens = (1500, 333)
    inp = synth.random_inputs(2, 8, 2, 128, lens, seed=31, grid=False, device=DEV)
    sets = {(b, g): list(range(lens[b])) for b in range(2) for g in range(2)}
    ys, ls = run_sparse(inp, lens, sets, 1600)
    yd, ld = run_dense(inp, lens)
    for b in range(2):
        for h in range(8):
            den = np.abs(yd[b, h]).max()
            assert np.abs(ys[b, h] - yd[b, h]).max() / den <= 2e-3
            assert abs(ls[b, h] - ld[b, h]) <= 1e-4 * max(1, abs(ld[b, h]))


# ---------------------------------------------------------------- selection

def run_select(inp, lens, p, layer=0, step=0):
    w = inp.w
    kv, _ = kv_for(inp, lens, layer)
    k_cap = max(1, B.prhs_max_topk(p, w.capacity))
    set_cap = max(1, min(w.capacity, p.sink + k_cap + p.window))
    topk = torch.full((w.batch, w.hkv, k_cap), -7, dtype=torch.int32, device=DEV)
    tlen = torch.full((w.batch, w.hkv), -7, dtype=torch.int32, device=DEV)
    sidx = torch.full((w.batch, w.hkv, set_cap), -7, dtype=torch.int32, device=DEV)
    slen = torch.full((w.batch, w.hkv), -7, dtype=torch.int32, device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SELECT, kv, p), DEV)
    zb = B.select_zero_bytes(kv)
    ws.fill_(0xAB)   # beyond the histogram region the workspace needs no initialisation
    ws[:zb].zero_()
    B.prhs_select(kv, inp.q[layer, step], p, topk, tlen, sidx, slen, ws)
    torch.cuda.synchronize()
    assert not ws[:zb].any(), "the histogram region is not left zero"
    return topk.cpu().numpy(), tlen.cpu().numpy(), sidx.cpu().numpy(), slen.cpu().numpy()


def oracle_select(inp, lens, p, layer=0, step=0):
    res = {}
    for b, n0 in enumerate(lens):
        for g in range(inp.w.hkv):
            K, _ = synth.gather_unit(inp, layer, b, g, n0)
            Qg = synth.query_group(inp, layer, step, b, g)
            kb = O.budget_k(n0, p.k, p.k_num, p.k_den)
            S = O.topk_middle(O.ranking_scores(Qg, K), n0, kb, p.sink, p.window)
            res[(b, g)] = (S, O.anchor_set(S, n0, p.sink, p.window))
    return res


def check_select(inp, lens, p, layer=0, step=0):
    topk, tlen, sidx, slen = run_select(inp, lens, p, layer, step)
    ref = oracle_select(inp, lens, p, layer, step)
    for (b, g), (S, C) in ref.items():
        assert tlen[b, g] == len(S), f"b{b} g{g}: topk_len {tlen[b, g]} != {len(S)}"
        kb = O.budget_k(lens[b], p.k, p.k_num, p.k_den)
        expect = topk_layout(S, O.dilation_m(kb, len(S), p.dilate_m))
        assert np.array_equal(topk[b, g, : len(S)], expect), f"b{b} g{g}: top-k differs"
        assert slen[b, g] == len(C), f"b{b} g{g}: set_len {slen[b, g]} != {len(C)}"
        assert np.array_equal(sidx[b, g, : len(C)], C), f"b{b} g{g}: anchor set differs"
    return topk, tlen


SELECT_CASES = [
    # name, dtype, d, paged, hq, hkv, lens, params
    # few rows, middle range within LDS: the keyed path (multi-workgroup
    # scoring, then one selection workgroup per row)
    ("ragged-gqa", "bf16", 128, False, 8, 2, (5000, 2100, 70), dict(k=300, sink=4, window=64)),
    ("mha-d64-paged", "bf16", 64, True, 4, 4, (3000, 1500), dict(k=100, sink=4, window=32)),
    ("g8", "bf16", 128, False, 16, 2, (4500,), dict(k=64, sink=0, window=0)),
    ("k-ge-middle", "bf16", 128, False, 4, 2, (400, 900), dict(k=2000, sink=4, window=16)),
    ("k-zero", "bf16", 128, False, 4, 2, (400, 900), dict(k=0, sink=4, window=16)),
    ("short-seqs", "bf16", 128, False, 4, 2, (3, 20, 21, 22), dict(k=5, sink=4, window=16)),
    ("ratio", "bf16", 128, True, 8, 2, (9000, 4100), dict(k_num=1, k_den=20, sink=4, window=128)),
    ("f32", "f32", 64, False, 4, 4, (1025, 300), dict(k=64, sink=4, window=32)),
    ("f32-paged-gqa", "f32", 128, True, 8, 2, (2000,), dict(k=50, sink=2, window=8)),
    ("big-k", "bf16", 128, False, 4, 1, (20000,), dict(k=9000, sink=4, window=64)),
    ("keyed-128-rows", "bf16", 128, False, 32, 8, tuple(300 + (i * 997) % 5000 for i in range(16)),
     dict(k=150, sink=4, window=32)),
    # middle ranges beyond LDS: the radix path (score, filter, finish),
    # including a k whose level-1 ties overflow the LDS buffer
    ("radix-ragged-gqa", "bf16", 128, False, 8, 2, (30000, 26000, 70), dict(k=300, sink=4, window=64)),
    ("radix-paged-d64", "bf16", 64, True, 4, 4, (27000,), dict(k=100, sink=4, window=32)),
    ("radix-big-k", "bf16", 128, False, 4, 1, (30000,), dict(k=12000, sink=4, window=64)),
    ("radix-f32-paged", "f32", 128, True, 8, 2, (26000,), dict(k=50, sink=2, window=8)),
    ("radix-ratio", "bf16", 128, True, 8, 2, (40000, 25000), dict(k_num=1, k_den=20, sink=4, window=128)),
    ("radix-g16", "bf16", 128, True, 32, 2, (30000,), dict(k=200, sink=4, window=64)),
    # odd budget (an odd sort buffer: the finish kernel's bitmaps start one
    # entry further to stay 16-byte aligned) and a cache capacity that is not
    # a whole number of 128-position groups
    ("radix-odd-k", "bf16", 128, False, 8, 2, (30007, 26001), dict(k=301, sink=3, window=61)),
    # 17 sequences x 8 kv heads = 136 rows, more than half the CUs: the
    # single-launch refresh path
    ("fused-ragged", "bf16", 128, False, 32, 8,
     (3000, 2100, 70, 1500, 999, 2048, 300, 2999, 1200, 640, 77, 2500, 1800, 33, 2222, 1024, 1700),
     dict(k=150, sink=4, window=32)),
    ("fused-mha-d64", "bf16", 64, False, 8, 8, (900, 1300) * 8 + (1100,), dict(k=60, sink=2, window=16)),
    ("fused-k-ge-middle", "bf16", 128, False, 16, 8, (400, 150) * 8 + (300,), dict(k=5000, sink=4, window=16)),
    ("fused-k-zero", "bf16", 128, False, 16, 8, (400, 900) * 8 + (600,), dict(k=0, sink=4, window=16)),
    ("fused-short", "bf16", 128, False, 8, 8, (3, 20, 21, 22, 40, 60, 5, 1) * 2 + (9,),
     dict(k=5, sink=4, window=16)),
    ("fused-ratio", "bf16", 128, False, 32, 8, (9000, 4100) * 8 + (6000,),
     dict(k_num=1, k_den=20, sink=4, window=128)),
    # 40 x 8 = 320 rows, more than the CUs: workgroups take rows by length rank
    ("fused-balanced", "bf16", 128, False, 16, 8,
     tuple(300 + (i * 389) % 2700 for i in range(38)) + (1500, 1500),
     dict(k=100, sink=4, window=32)),
    ("fused-balanced-d64", "bf16", 64, False, 8, 8,
     tuple(40 + (i * 577) % 3000 for i in range(40)), dict(k=70, sink=2, window=16)),
    # long middle ranges on 136 rows: up to ~21k keys the key array fits LDS
    # beside the 1024-thread workgroup's staging; beyond, 512 threads
    ("fused-wide-21k", "bf16", 128, False, 32, 8, (21000, 16000) * 8 + (12000,),
     dict(k=1000, sink=4, window=128)),
    ("fused-narrow-24k", "bf16", 128, False, 32, 8, (24000, 23000) * 8 + (20000,),
     dict(k_num=1, k_den=20, sink=4, window=128)),
    # more rows than CUs with long middle ranges: two 512-thread workgroups
    # would not share a CU's LDS, so 1024-thread ones take the rows by length
    ("fused-wide-many-rows", "bf16", 128, False, 32, 8, tuple(15000 + 31 * i for i in range(33)),
     dict(k_num=1, k_den=20, sink=4, window=128)),
    # more than 256 sequences: no length ranking, one row per workgroup in order
    ("fused-many-seqs", "bf16", 128, False, 4, 1, tuple(100 + (i * 131) % 1200 for i in range(260)),
     dict(k=40, sink=4, window=16)),
    # short rows, two workgroups side by side per CU, more than two rounds of
    # rows over the CUs (serpentine length order)
    ("fused-three-rounds", "bf16", 128, False, 8, 4, tuple(50 + (i * 97) % 700 for i in range(150)),
     dict(k=30, sink=4, window=16)),
    # the largest query group (16 heads per kv head) on each path
    ("g16-keyed", "bf16", 128, True, 32, 2, (6000, 2500), dict(k=200, sink=4, window=64)),
    ("g16-fused", "bf16", 128, False, 16, 1, tuple(900 + 37 * i for i in range(136)),
     dict(k=50, sink=4, window=16)),
]


@pytest.mark.parametrize("name,dtype,d,paged,hq,hkv,lens,pk", SELECT_CASES,
                         ids=[c[0] for c in SELECT_CASES])
def test_select_bit_exact(name, dtype, d, paged, hq, hkv, lens, pk):
    inp = synth.random_inputs(len(lens), hq, hkv, d, lens, dtype=dtype, paged=paged,
                              seed=41 + len(name), grid=True, device=DEV)
    check_select(inp, lens, B.params(**pk))


def check_select_shared(inp, lens, p):
    """prhs_select_shared: top-k and anchor set as prhs_select, plus the
    dilated shared set at the anchor length equal to the oracle's R(n0)."""
    w = inp.w
    kv, _ = kv_for(inp, lens)
    k_cap = max(1, B.prhs_max_topk(p, w.capacity))
    set_cap = max(1, B.prhs_set_capacity(p, w.capacity))
    shape = (w.batch, w.hkv)
    topk = torch.full(shape + (k_cap,), -7, dtype=torch.int32, device=DEV)
    tlen = torch.full(shape, -7, dtype=torch.int32, device=DEV)
    sidx = torch.full(shape + (set_cap,), -7, dtype=torch.int32, device=DEV)
    slen = torch.full(shape, -7, dtype=torch.int32, device=DEV)
    hidx = torch.full(shape + (set_cap,), -7, dtype=torch.int32, device=DEV)
    hlen = torch.full(shape, -7, dtype=torch.int32, device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SELECT, kv, p), DEV)
    zb = B.select_zero_bytes(kv)
    ws.fill_(0xCD)
    ws[:zb].zero_()
    B.prhs_select_shared(kv, inp.q[0, 0], p, topk, tlen, sidx, slen, hidx, hlen, ws)
    torch.cuda.synchronize()
    assert not ws[:zb].any(), "the histogram region is not left zero"
    topk, tlen, sidx, slen = (t.cpu().numpy() for t in (topk, tlen, sidx, slen))
    hidx, hlen = hidx.cpu().numpy(), hlen.cpu().numpy()
    for (b, g), (S, C) in oracle_select(inp, lens, p).items():
        kb = O.budget_k(lens[b], p.k, p.k_num, p.k_den)
        m = O.dilation_m(kb, len(S), p.dilate_m)
        assert tlen[b, g] == len(S) and np.array_equal(topk[b, g, : len(S)], topk_layout(S, m))
        assert slen[b, g] == len(C) and np.array_equal(sidx[b, g, : len(C)], C)
        R = O.reuse_set(S, m, p.dilate_r, lens[b], lens[b], p.sink, p.window)
        assert hlen[b, g] == len(R), f"b{b} g{g}: shared_len {hlen[b, g]} != {len(R)}"
        assert np.array_equal(hidx[b, g, : len(R)], R), f"b{b} g{g}: shared set differs"


SHARED_VARIANTS = [dict(dilate_r=1), dict(dilate_r=2, dilate_m=7), dict(dilate_r=0)]


@pytest.mark.parametrize("name,dtype,d,paged,hq,hkv,lens,pk", SELECT_CASES,
                         ids=[c[0] for c in SELECT_CASES])
def test_select_shared_bit_exact(name, dtype, d, paged, hq, hkv, lens, pk):
    inp = synth.random_inputs(len(lens), hq, hkv, d, lens, dtype=dtype, paged=paged,
                              seed=43 + len(name), grid=True, device=DEV)
    for var in SHARED_VARIANTS:
        check_select_shared(inp, lens, B.params(refresh_every=4, **pk, **var))


WIDE_DILATION_CASES = [c for c in SELECT_CASES
                       if c[0] in ("ragged-gqa", "fused-ragged", "fused-mha-d64", "keyed-128-rows",
                                   "radix-ragged-gqa")]


@pytest.mark.parametrize("r", [31, 32, 40, 63, 64, 70])
@pytest.mark.parametrize("name,dtype,d,paged,hq,hkv,lens,pk", WIDE_DILATION_CASES,
                         ids=[c[0] for c in WIDE_DILATION_CASES])
def test_select_shared_wide_dilation(name, dtype, d, paged, hq, hkv, lens, pk, r):
    """Dilation radii around one and two bitmap words (neighbours that reach
    past the next 32 and 64 middle positions)."""
    inp = synth.random_inputs(len(lens), hq, hkv, d, lens, dtype=dtype, paged=paged,
                              seed=7 + r, grid=True, device=DEV)
    check_select_shared(inp, lens, B.params(refresh_every=4, **pk, dilate_r=r, dilate_m=25))


@pytest.mark.parametrize("r", [33, 64])
def test_select_shared_two_bitmap_segments(r):
    """A radius of a word or more keeps the radix finish in its segmented
    form (a marked neighbour bitmap); a middle range of about 70k positions
    then spans two segments, with top-m winners placed on both sides of the
    boundary whose neighbours cross it."""
    lens = (70100, 20000)
    hq, hkv = 4, 1
    inp = synth.random_inputs(2, hq, hkv, 128, lens, seed=31 + r, grid=True, device=DEV)
    K = inp.K[0]
    for b, n in enumerate(lens):
        # bands around the segment boundaries a 65,408-position segment
        # would have (4 + 65408 from the sink), and at the middle
        for c in (4 + 65408, n // 2):
            if c + 200 >= n - 64:
                continue
            pos = torch.arange(c - 150, c + 150, 7, device=DEV)
            K[b, 0, pos] = (4 * inp.q[0, 0, b, 0]).to(K.dtype)
    check_select_shared(inp, lens, B.params(refresh_every=4, k=400, sink=4, window=64,
                                            dilate_r=r))


def test_select_shared_clustered_top_m_long_middle():
    """Top-m winners packed in bands (stride 5) at 1/4, 1/3, 1/2, 2/3 and 3/4
    of middle ranges beyond LDS (the radix path): neighbours of winners on
    either side of any split of the range into equal parts must all land in
    the shared set."""
    lens = (30000, 40000)
    hq, hkv = 4, 2
    G = hq // hkv
    inp = synth.random_inputs(2, hq, hkv, 128, lens, seed=21, grid=True, device=DEV)
    K = inp.K[0]
    for b, n in enumerate(lens):
        lo, hi = 4, n - 64
        for f in (1 / 4, 1 / 3, 1 / 2, 2 / 3, 3 / 4):
            c = lo + int((hi - lo) * f)
            pos = torch.arange(c - 80, c + 80, 5, device=DEV)
            for g in range(hkv):
                # 4 q of the group's first head: far above every random score
                K[b, g, pos] = (4 * inp.q[0, 0, b, g * G]).to(K.dtype)
    for r in (1, 5, 31):
        check_select_shared(inp, lens, B.params(refresh_every=4, k=600, sink=4, window=64,
                                                dilate_r=r))


def test_select_shared_window_zero_edges():
    # no window: a top-m winner at the last middle position has its right
    # neighbour at n0, outside [0, n0); a winner at the first has its left
    # neighbour in the sink; coarse grid, many ties
    for lens in ((600, 1500, 9), (700,) * 16):
        hkv = 8 if len(lens) == 16 else 2
        inp = synth.random_inputs(len(lens), 2 * hkv, hkv, 128, lens, seed=59, grid=True,
                                  device=DEV)
        for K in inp.K:
            K.copy_(torch.where(torch.isnan(K), K, torch.clamp(torch.round(K.float()), -1, 1).to(K.dtype) / 16))
        check_select_shared(inp, lens, B.params(k=40, sink=3, window=0, dilate_r=3))


def test_select_all_ties_lowest_positions():
    # every key equal: each score ties, so the top-k are the lowest middle positions
    lens = (3000, 1800)
    inp = synth.random_inputs(2, 8, 2, 128, lens, seed=3, grid=True, device=DEV)
    for K in inp.K:
        K.copy_(torch.where(torch.isnan(K), K, torch.full_like(K, 0.25)))
    p = B.params(k=200, sink=4, window=64)
    topk, tlen = check_select(inp, lens, p)
    assert list(topk[0, 0, :5]) == [4, 5, 6, 7, 8]   # the top m = the lowest positions


def test_select_fused_all_ties():
    # all scores equal on the single-launch path (136 rows): ties go to the
    # lower positions
    lens = (2500, 1700) * 8 + (2100,)
    inp = synth.random_inputs(17, 8, 8, 128, lens, seed=14, grid=True, device=DEV)
    for K in inp.K:
        K.copy_(torch.where(torch.isnan(K), K, torch.full_like(K, 0.75)))
    topk, tlen = check_select(inp, lens, B.params(k=120, sink=4, window=32))
    assert list(topk[0, 0, :3]) == [4, 5, 6]


def test_select_all_ties_beyond_lds_budget():
    # every score equal on a row longer than LDS (radix path) and than the
    # finish kernel's LDS tie buffer: the tie-break runs through the global
    # radix levels over positions
    lens = (30000,)
    inp = synth.random_inputs(1, 4, 1, 128, lens, seed=12, grid=True, device=DEV)
    for K in inp.K:
        K.copy_(torch.where(torch.isnan(K), K, torch.full_like(K, -0.5)))
    topk, tlen = check_select(inp, lens, B.params(k=300, sink=4, window=64))
    assert list(topk[0, 0, :3]) == [4, 5, 6]


def test_select_largest_supported_topk():
    # k = PRHS_MAX_TOPK on middle ranges beyond LDS (the radix path, whose
    # finish kernel keeps every winner in LDS), one row clamped to its middle
    lens = (40000, 16050)
    inp = synth.random_inputs(2, 4, 1, 128, lens, seed=14, grid=True, device=DEV)
    check_select(inp, lens, B.params(k=B.PRHS_MAX_TOPK, sink=4, window=64))


@pytest.mark.parametrize("lens", [(6000, 2500), (30000, 26000)], ids=["keyed", "radix"])
def test_select_coarse_grid_many_ties(lens):
    # values in {-1/16, 0, 1/16}: very many exact ties at the threshold
    inp = synth.random_inputs(2, 8, 2, 128, lens, seed=4, grid=True, device=DEV)
    for t in inp.K + [inp.q]:
        t.copy_(torch.where(torch.isnan(t), t, torch.clamp(torch.round(t.float()), -1, 1).to(t.dtype) / 16))
    check_select(inp, lens, B.params(k=500, sink=4, window=64))


def test_select_negative_zero_scores():
    # scores of exactly +0 and -0 rank equal; ties break to the lower position
    lens = (600,)
    inp = synth.random_inputs(1, 2, 1, 64, lens, dtype="f32", seed=6, grid=True, device=DEV)
    q = inp.q
    q.zero_()
    q[0, 0, 0, 0, 0] = 1.0
    q[0, 0, 0, 1, 0] = -1.0      # second head of the group: scores are -k
    K = inp.K[0]
    K[0, 0, :600, 0] = 0.0       # every key scores +0 on head 0 and -0 on head 1
    K[0, 0, 100, 0] = -0.0
    check_select(inp, lens, B.params(k=10, sink=4, window=8))


def test_select_reuses_workspace_across_calls():
    lens = (3000, 1000)
    inp = synth.random_inputs(2, 8, 2, 128, lens, seed=8, grid=True, layers=2, device=DEV)
    p = B.params(k=120, sink=4, window=32)
    for layer in (0, 1, 0):
        check_select(inp, lens, p, layer=layer)


# ---------------------------------------------------------------- dilation / reuse

def test_dilate_reuse_bit_exact():
    lens0 = (5000, 2000, 30)
    steps = 6
    inp = synth.random_inputs(3, 8, 2, 128, lens0, seed=9, grid=True, steps=steps, device=DEV)
    for pk in (dict(k=300, sink=4, window=64, dilate_r=1),
               dict(k=90, sink=0, window=0, dilate_r=2, dilate_m=40),
               dict(k=300, sink=4, window=64, dilate_r=0),
               dict(k_num=1, k_den=20, sink=4, window=16, dilate_r=1),
               dict(k=9000, sink=4, window=64, dilate_r=1)):
        p = B.params(refresh_every=steps, **pk)
        topk, tlen, _, _ = run_select(inp, lens0, p)
        ref = oracle_select(inp, lens0, p)
        topk_d = torch.tensor(topk, device=DEV)
        tlen_d = torch.tensor(tlen, device=DEV)
        set_cap = B.prhs_set_capacity(p, inp.w.capacity)
        anchor = lens_tensor(lens0)
        for j in range(steps):
            lens = tuple(n + j for n in lens0)
            sidx = torch.full((3, 2, set_cap), -7, dtype=torch.int32, device=DEV)
            slen = torch.full((3, 2), -7, dtype=torch.int32, device=DEV)
            B.prhs_dilate_reuse(p, topk_d, tlen_d, anchor, lens_tensor(lens), sidx, slen)
            torch.cuda.synchronize()
            sidx, slen = sidx.cpu().numpy(), slen.cpu().numpy()
            for (b, g), (S, _) in ref.items():
                kb = O.budget_k(lens0[b], p.k, p.k_num, p.k_den)
                m = O.dilation_m(kb, len(S), p.dilate_m)
                R = O.reuse_set(S, m, p.dilate_r, lens0[b], lens[b], p.sink, p.window)
                assert slen[b, g] == len(R), f"step {j} b{b} g{g}"
                assert np.array_equal(sidx[b, g, : len(R)], R), f"step {j} b{b} g{g}"


def run_reuse(inp, lens, idx, ln, anchor, layer=0, step=0):
    w = inp.w
    kv, _ = kv_for(inp, lens, layer)
    out = torch.full((w.batch, w.hq, w.d), float("nan"), device=DEV)
    lse = torch.full((w.batch, w.hq), float("nan"), device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv, None, idx.shape[-1]), DEV)
    B.prhs_reuse_decode_attn(kv, inp.q[layer, step], idx, ln, lens_tensor(anchor),
                             1 / math.sqrt(w.d), out, lse, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


@pytest.mark.parametrize("dtype,d,paged,hq,hkv", [("bf16", 128, False, 8, 2),
                                                  ("bf16", 128, True, 32, 8),
                                                  ("f32", 64, False, 4, 4)])
def test_reuse_attention_equals_per_step_set(dtype, d, paged, hq, hkv):
    # set built once at the anchor length, attended at later lengths with the
    # tail [n0, n): same rows, same outputs as the oracle over R(n)
    lens0 = (3000, 700, 40)
    steps = 8
    inp = synth.random_inputs(3, hq, hkv, d, lens0, dtype=dtype, paged=paged, seed=41 + d,
                              grid=True, steps=steps, device=DEV)
    p = B.params(k=150, sink=4, window=32, dilate_r=1, refresh_every=steps)
    topk, tlen, _, _ = run_select(inp, lens0, p)
    ref = oracle_select(inp, lens0, p)
    set_cap = B.prhs_set_capacity(p, inp.w.capacity)
    sidx = torch.zeros(3, hkv, set_cap, dtype=torch.int32, device=DEV)
    slen = torch.zeros(3, hkv, dtype=torch.int32, device=DEV)
    anchor = lens_tensor(lens0)
    B.prhs_dilate_reuse(p, torch.tensor(topk, device=DEV), torch.tensor(tlen, device=DEV),
                        anchor, anchor, sidx, slen)
    gq = hq // hkv
    for j in (0, 1, steps - 1):
        lens = tuple(n + j for n in lens0)
        y, lse = run_reuse(inp, lens, sidx, slen, lens0, step=j)
        for (b, g), (S, _) in ref.items():
            kb = O.budget_k(lens0[b], p.k, p.k_num, p.k_den)
            R = O.reuse_set(S, O.dilation_m(kb, len(S)), 1, lens0[b], lens[b], 4, 32)
            K, V = synth.gather_unit(inp, 0, b, g, lens[b])
            Qg = synth.query_group(inp, 0, j, b, g)
            for i in range(gq):
                yr, lr = O.sparse_attention(Qg[i], K, V, R)
                assert_close(y[b, g * gq + i], lse[b, g * gq + i], yr, lr, TOL[dtype],
                             f"step {j} b{b} g{g}")


def test_reuse_attention_skips_set_entries_past_anchor():
    # set entries at or beyond n0 are covered by the tail and not attended
    # twice; an anchor length of 0 leaves only the tail [0, n): dense attention;
    # an anchor length past n is clamped to n (no tail)
    lens = (900, 260, 50)
    inp = synth.random_inputs(3, 8, 2, 128, lens, seed=43, grid=False, device=DEV)
    cap = 1000
    sets = {(0, 0): list(range(0, 900, 3)), (0, 1): list(range(850, 900)),
            (1, 0): list(range(260)), (1, 1): [5, 100, 259],
            (2, 0): [0, 1, 2], (2, 1): []}
    anchor = (600, 0, 70)
    idx = torch.zeros(3, 2, cap, dtype=torch.int32)
    ln = torch.zeros(3, 2, dtype=torch.int32)
    for (b, g), S in sets.items():
        idx[b, g, : len(S)] = torch.tensor(S, dtype=torch.int32)
        ln[b, g] = len(S)
    y, lse = run_reuse(inp, lens, idx.to(DEV), ln.to(DEV), anchor)
    for (b, g), S in sets.items():
        n0 = min(max(anchor[b], 0), lens[b])
        R = sorted(set(i for i in S if i < n0) | set(range(n0, lens[b])))
        K, V = synth.gather_unit(inp, 0, b, g, lens[b])
        Qg = synth.query_group(inp, 0, 0, b, g)
        for i in range(4):
            yr, lr = O.sparse_attention(Qg[i], K, V, R)
            assert_close(y[b, g * 4 + i], lse[b, g * 4 + i], yr, lr, TOL["bf16"], f"b{b} g{g}")
    yd, ld = run_dense(inp, lens)
    assert np.abs(y[1] - yd[1]).max() <= 2e-3 * np.abs(yd[1]).max()


def test_reuse_attention_many_splits_ragged():
    # several splits per unit and a tail crossing split boundaries
    lens0 = (20000, 9000)
    inp = synth.random_inputs(2, 32, 8, 128, lens0, seed=47, grid=True, steps=8, device=DEV)
    p = B.params(k=1500, sink=4, window=128, dilate_r=1, refresh_every=8)
    topk, tlen, _, _ = run_select(inp, lens0, p)
    ref = oracle_select(inp, lens0, p)
    set_cap = B.prhs_set_capacity(p, inp.w.capacity)
    sidx = torch.zeros(2, 8, set_cap, dtype=torch.int32, device=DEV)
    slen = torch.zeros(2, 8, dtype=torch.int32, device=DEV)
    anchor = lens_tensor(lens0)
    B.prhs_dilate_reuse(p, torch.tensor(topk, device=DEV), torch.tensor(tlen, device=DEV),
                        anchor, anchor, sidx, slen)
    j = 7
    lens = tuple(n + j for n in lens0)
    y, lse = run_reuse(inp, lens, sidx, slen, lens0, step=j)
    for (b, g) in [(0, 0), (0, 7), (1, 3)]:
        S = ref[(b, g)][0]
        R = O.reuse_set(S, O.dilation_m(1500, len(S)), 1, lens0[b], lens[b], 4, 128)
        K, V = synth.gather_unit(inp, 0, b, g, lens[b])
        Qg = synth.query_group(inp, 0, j, b, g)
        for i in range(4):
            yr, lr = O.sparse_attention(Qg[i], K, V, R)
            assert_close(y[b, g * 4 + i], lse[b, g * 4 + i], yr, lr, TOL["bf16"], f"b{b} g{g}")


def test_split_merge_workspace_reused_across_calls():
    # one attention workspace for consecutive calls whose units split a
    # different number of ways (including one split and empty units): the
    # merge of every call is complete and the workspace is left reusable.
    # The workspace starts as NaN bytes, so a merge that let a split slot
    # no call wrote into its arithmetic would give NaN.
    inp = synth.random_inputs(2, 32, 8, 128, (9000, 3000), seed=53, grid=False, device=DEV)
    rng = np.random.default_rng(53)
    cap = 8200
    kv, _ = kv_for(inp, (9000, 3000))
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv, None, cap), DEV)
    ws.fill_(0xFF)
    for call in range(4):
        lens = (9000 - 1000 * call, 3000 - 700 * call)
        sets = {}
        for b in range(2):
            for g in range(8):
                size = 0 if (b + g + call) % 7 == 0 else int(rng.integers(1, min(cap, lens[b]) + 1))
                sets[(b, g)] = sorted(rng.choice(lens[b], size=size, replace=False).tolist())
        kv, _ = kv_for(inp, lens)
        idx = torch.zeros(2, 8, cap, dtype=torch.int32)
        ln = torch.zeros(2, 8, dtype=torch.int32)
        for (b, g), S in sets.items():
            idx[b, g, : len(S)] = torch.tensor(S, dtype=torch.int32)
            ln[b, g] = len(S)
        out = torch.full((2, 32, 128), float("nan"), device=DEV)
        lse = torch.full((2, 32), float("nan"), device=DEV)
        B.prhs_sparse_decode_attn(kv, inp.q[0, 0], idx.to(DEV), ln.to(DEV), 1 / math.sqrt(128),
                                  out, lse, ws)
        torch.cuda.synchronize()
        y, ls = out.cpu().numpy(), lse.cpu().numpy()
        assert not np.isnan(y).any(), f"call {call}: unmerged heads"
        for (b, g) in [(0, 0), (0, 5), (1, 2), (1, 7), ((call + 1) % 2, (call * 3) % 8)]:
            K, V = synth.gather_unit(inp, 0, b, g, lens[b])
            Qg = synth.query_group(inp, 0, 0, b, g)
            for i in range(4):
                yr, lr = O.sparse_attention(Qg[i], K, V, sets[(b, g)])
                assert_close(y[b, g * 4 + i], ls[b, g * 4 + i], yr, lr, TOL["bf16"],
                             f"call {call} b{b} g{g}")


def test_empty_batch_is_a_no_op_on_every_entry_point():
    # batch 0: every call returns OK without touching the device buffers
    inp = synth.random_inputs(1, 8, 2, 128, (100,), seed=71, device=DEV)
    kv0 = B.KV(inp.K[0][:0], inp.V[0][:0], torch.zeros(0, dtype=torch.int32, device=DEV),
               inp.w.capacity, 8)
    p = B.params(k=8, sink=4, window=8, refresh_every=2)
    q0 = inp.q[0, 0][:0]
    z3 = torch.zeros(0, 2, 64, dtype=torch.int32, device=DEV)
    z2 = torch.zeros(0, 2, dtype=torch.int32, device=DEV)
    out = torch.zeros(0, 8, 128, device=DEV)
    lse = torch.zeros(0, 8, device=DEV)
    ws = B.workspace(1, DEV)
    B.prhs_select(kv0, q0, p, z3, z2, z3, z2, ws)
    B.prhs_select_shared(kv0, q0, p, z3, z2, z3, z2, z3.clone(), z2.clone(), ws)
    B.prhs_sparse_decode_attn(kv0, q0, z3, z2, 0.1, out, lse, ws)
    B.prhs_reuse_decode_attn(kv0, q0, z3, z2, torch.zeros(0, dtype=torch.int32, device=DEV),
                             0.1, out, lse, ws)
    B.prhs_dense_decode_attn(kv0, q0, 0.1, out, lse, ws)
    torch.cuda.synchronize()


# ---------------------------------------------------------------- off-grid inputs

OFFGRID = ["g8", "ratio", "f32", "f32-paged-gqa", "keyed-128-rows", "radix-ragged-gqa",
           "radix-paged-d64", "radix-f32-paged", "radix-ratio", "fused-ragged",
           "fused-mha-d64", "fused-narrow-24k", "g16-keyed", "g16-fused"]


def _near_threshold(sym, sigma, tau, tol, what):
    for x in sym:
        assert abs(sigma[x] - tau) <= tol, \
            f"{what}: position {x} differs with score {sigma[x]!r} vs threshold {tau!r} (tol {tol:.2e})"


@pytest.mark.parametrize("name", OFFGRID)
def test_select_off_grid_within_rounding_of_threshold(name):
    # N(0, 1) inputs that are not on the grid: the library's fp32 scores may
    # differ from the exact ones by the dot-product rounding bound
    # gamma_d * sum_d |q_d k_d| (gamma_d = d u / (1 - d u), u = 2^-24), so a
    # position may swap in or out of the top k (or the top m) only when its
    # exact score lies within twice the row's largest bound of the k-th
    # (m-th) largest exact score; everything else must agree, and the anchor
    # and shared sets must be exactly those the library's own top-k defines.
    case = next(c for c in SELECT_CASES if c[0] == name)
    _, dtype, d, paged, hq, hkv, lens, pk = case
    inp = synth.random_inputs(len(lens), hq, hkv, d, lens, dtype=dtype, paged=paged,
                              seed=97 + len(name), grid=False, device=DEV)
    p = B.params(refresh_every=4, dilate_r=1, **pk)
    w = inp.w
    kv, _ = kv_for(inp, lens)
    k_cap = max(1, B.prhs_max_topk(p, w.capacity))
    set_cap = max(1, B.prhs_set_capacity(p, w.capacity))
    shape = (w.batch, w.hkv)
    topk = torch.full(shape + (k_cap,), -7, dtype=torch.int32, device=DEV)
    tlen = torch.full(shape, -7, dtype=torch.int32, device=DEV)
    sidx = torch.full(shape + (set_cap,), -7, dtype=torch.int32, device=DEV)
    slen = torch.full(shape, -7, dtype=torch.int32, device=DEV)
    hidx = torch.full(shape + (set_cap,), -7, dtype=torch.int32, device=DEV)
    hlen = torch.full(shape, -7, dtype=torch.int32, device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SELECT, kv, p), DEV)
    B.prhs_select_shared(kv, inp.q[0, 0], p, topk, tlen, sidx, slen, hidx, hlen, ws)
    torch.cuda.synchronize()
    topk, tlen, sidx, slen = (t.cpu().numpy() for t in (topk, tlen, sidx, slen))
    hidx, hlen = hidx.cpu().numpy(), hlen.cpu().numpy()
    swaps = 0
    for b, n0 in enumerate(lens):
        for g in range(w.hkv):
            K = synth.gather_unit(inp, 0, b, g, n0)[0]
            Qg = synth.query_group(inp, 0, 0, b, g)
            sigma = O.ranking_scores(Qg, K)
            gam = d * 2.0 ** -24 / (1 - d * 2.0 ** -24)
            bound = gam * (np.abs(K) @ np.abs(Qg).T).max(axis=1)
            kb = O.budget_k(n0, p.k, p.k_num, p.k_den)
            S = O.topk_middle(sigma, n0, kb, p.sink, p.window)
            m = O.dilation_m(kb, len(S), p.dilate_m)
            got = topk[b, g, : tlen[b, g]]
            assert tlen[b, g] == len(S), f"b{b} g{g}: topk_len"
            top, rest = got[:m], got[m:]
            assert list(top) == sorted(top) and list(rest) == sorted(rest)
            assert len(set(got.tolist())) == len(got)
            se, wst = O.region_bounds(n0, p.sink, p.window)
            assert np.all((got >= se) & (got < wst))
            if len(S):
                tol = 2 * bound[se:wst].max()
                sym = set(got.tolist()) ^ set(S.tolist())
                _near_threshold(sym, sigma, sigma[S[-1]], tol, f"{name} b{b} g{g} top-k")
                if m:
                    symm = set(top.tolist()) ^ set(S[:m].tolist())
                    _near_threshold(symm, sigma, sigma[S[m - 1]], tol, f"{name} b{b} g{g} top-m")
                    swaps += len(symm)
                swaps += len(sym)
            own = np.concatenate([top, rest])
            C = O.anchor_set(own, n0, p.sink, p.window)
            assert slen[b, g] == len(C) and np.array_equal(sidx[b, g, : len(C)], C)
            R = O.reuse_set(own, m, p.dilate_r, n0, n0, p.sink, p.window)
            assert hlen[b, g] == len(R) and np.array_equal(hidx[b, g, : len(R)], R)
    print(f"{name}: {swaps} positions swapped at a threshold")
