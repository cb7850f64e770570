"""The C-ABI library on the host: it loads, exports every symbol the header
declares, its pure host logic matches the oracle's definitions, and every
validation error returns its status before any device work (so these tests
need no GPU; no call here reaches a kernel launch)."""

import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle as O
from paper_2602_08329_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "prhs.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        from paper_2602_08329_amd import build
        build.build()
    return B.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(prhs_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def test_abi_version(L):
    assert L.prhs_abi_version() == 2


def test_schedule_matches_oracle(L):
    for s in (1, 2, 4, 8):
        for G in (1, 2, 4):
            p = B.params(k=8, refresh_every=s, layer_group=G)
            for j in range(20):
                for l in range(9):
                    got = B.prhs_schedule(j, l, p)
                    assert got == (B.PRHS_REFRESH if O.is_refresh(j, l, s, G) else B.PRHS_REUSE)
    assert B.prhs_schedule(-1, 0, B.params()) == -1
    assert B.prhs_schedule(0, 0, B.params(refresh_every=0)) == -1


def test_max_topk_matches_oracle_budget(L):
    rng = np.random.default_rng(0)
    for _ in range(300):
        n = int(rng.integers(0, 5000))
        sink, window = int(rng.integers(0, 20)), int(rng.integers(0, 300))
        if rng.random() < 0.5:
            p = B.params(k=int(rng.integers(0, 3000)), sink=sink, window=window)
            kb = p.k
        else:
            num, den = int(rng.integers(0, 5)), int(rng.integers(1, 40))
            p = B.params(k_num=num, k_den=den, sink=sink, window=window)
            kb = O.budget_k(n, k_num=num, k_den=den)
        se, ws = O.region_bounds(n, sink, window)
        assert B.prhs_max_topk(p, n) == min(kb, ws - se)


def test_set_capacity_bounds_every_schedule_set(L):
    # the capacity covers the largest anchor or shared set the oracle builds
    rng = np.random.default_rng(1)
    for _ in range(200):
        n_ctx = int(rng.integers(1, 300))
        s = int(rng.integers(1, 9))
        sink, window, k = int(rng.integers(0, 8)), int(rng.integers(0, 40)), int(rng.integers(0, 80))
        r = int(rng.integers(0, 3))
        p = B.params(k=k, sink=sink, window=window, dilate_r=r, refresh_every=s)
        cap = B.prhs_set_capacity(p, n_ctx + s)
        sigma = rng.integers(-5, 5, size=n_ctx + s).astype(float)
        for j0 in range(s):
            n0 = n_ctx + 1
            S = O.topk_middle(sigma, n0, k, sink, window)
            m = O.dilation_m(k, len(S))
            assert len(O.anchor_set(S, n0, sink, window)) <= cap
            for j in range(s):
                assert len(O.reuse_set(S, m, r, n0, n0 + j, sink, window)) <= cap


def _kv(**over):
    f = dict(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=128, dtype=B.PRHS_BF16,
             layout=B.PRHS_KV_CONTIGUOUS, capacity=1024, page_size=16, max_pages=64,
             num_pages=128, k=0x1000, v=0x2000, block_table=None, seq_lens=0x3000,
             max_seq_len=1000)
    f.update(over)
    return B.PrhsKv(**f)


def _select(L, kv, p, k_cap=64, set_cap=200, ws_bytes=None, q=0x4000):
    n = ctypes.c_size_t(0)
    L.prhs_workspace_size(B.PRHS_OP_SELECT, ctypes.byref(kv), ctypes.byref(p), 0, ctypes.byref(n))
    wsb = n.value if ws_bytes is None else ws_bytes
    return L.prhs_select(ctypes.byref(kv), q, ctypes.byref(p), 0x5000, 0x6000, k_cap, 0x7000,
                         0x8000, set_cap, 0x9000, wsb, None)


@pytest.mark.parametrize("over,status,msg", [
    (dict(num_q_heads=6, num_kv_heads=4), B.PRHS_E_INVALID, "multiple"),
    (dict(num_q_heads=34, num_kv_heads=2), B.PRHS_E_UNSUPPORTED, "<= 16"),
    (dict(head_dim=96), B.PRHS_E_UNSUPPORTED, "head_dim"),
    (dict(dtype=7), B.PRHS_E_UNSUPPORTED, "dtype"),
    (dict(capacity=10), B.PRHS_E_INVALID, "capacity"),
    (dict(layout=B.PRHS_KV_PAGED, block_table=None), B.PRHS_E_INVALID, "block_table"),
    (dict(layout=B.PRHS_KV_PAGED, block_table=0xA000, max_pages=2), B.PRHS_E_INVALID, "max_pages"),
    (dict(layout=5), B.PRHS_E_UNSUPPORTED, "layout"),
    (dict(max_seq_len=1 << 22, capacity=1 << 22), B.PRHS_E_UNSUPPORTED, "max_seq_len"),
    (dict(k=None), B.PRHS_E_INVALID, "NULL"),
    (dict(seq_lens=None), B.PRHS_E_INVALID, "seq_lens"),
    (dict(batch=-1), B.PRHS_E_INVALID, "batch"),
])
def test_select_shape_validation(L, over, status, msg):
    st = _select(L, _kv(**over), B.params(k=32, sink=4, window=64))
    assert st == status
    assert msg in L.prhs_last_error().decode()


@pytest.mark.parametrize("over,status", [
    (dict(k=-1), B.PRHS_E_INVALID),
    (dict(refresh_every=0), B.PRHS_E_INVALID),
    (dict(layer_group=0), B.PRHS_E_INVALID),
    (dict(sink=-2), B.PRHS_E_INVALID),
    (dict(window=-1), B.PRHS_E_INVALID),
    (dict(dilate_r=-1), B.PRHS_E_INVALID),
    (dict(k_num=-1, k_den=20), B.PRHS_E_INVALID),
])
def test_select_param_validation(L, over, status):
    base = dict(k=32, sink=4, window=64)
    base.update(over)
    assert _select(L, _kv(), B.params(**base)) == status


def test_select_capacity_and_workspace_errors(L):
    p = B.params(k=32, sink=4, window=64)
    assert _select(L, _kv(), p, k_cap=31) == B.PRHS_E_CAPACITY
    assert "k_cap" in L.prhs_last_error().decode()
    assert _select(L, _kv(), p, set_cap=99) == B.PRHS_E_CAPACITY
    assert _select(L, _kv(), p, ws_bytes=100) == B.PRHS_E_WORKSPACE
    assert _select(L, _kv(), p, q=None) == B.PRHS_E_INVALID
    big = B.params(k=20000, sink=0, window=0)
    kv = _kv(capacity=30000, max_seq_len=30000)
    assert _select(L, kv, big, k_cap=20000, set_cap=30000) == B.PRHS_E_UNSUPPORTED
    # the largest budget the selection supports, and one past it, on a middle
    # range beyond LDS (the radix path, whose winners stay in LDS)
    kv = _kv(capacity=40000, max_seq_len=40000)
    at = B.params(k=B.PRHS_MAX_TOPK, sink=4, window=64)
    past = B.params(k=B.PRHS_MAX_TOPK + 1, sink=4, window=64)
    assert _select(L, kv, past, k_cap=B.PRHS_MAX_TOPK + 1, set_cap=40000) == B.PRHS_E_UNSUPPORTED
    assert "sort limit" in L.prhs_last_error().decode()
    assert _select(L, kv, at, k_cap=B.PRHS_MAX_TOPK, set_cap=40000, ws_bytes=0) == B.PRHS_E_WORKSPACE


def test_attention_validation(L):
    kv = _kv()
    n = ctypes.c_size_t(0)
    assert L.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, ctypes.byref(kv), None, 300,
                                 ctypes.byref(n)) == 0
    assert n.value > 0
    st = L.prhs_sparse_decode_attn(ctypes.byref(kv), 0x1, 0x2, 0x3, 300, 0.1, 0x4, None, 0x5,
                                   n.value - 1, None)
    assert st == B.PRHS_E_WORKSPACE
    st = L.prhs_sparse_decode_attn(ctypes.byref(kv), 0x1, None, 0x3, 300, 0.1, 0x4, None, 0x5,
                                   n.value, None)
    assert st == B.PRHS_E_INVALID
    st = L.prhs_sparse_decode_attn(ctypes.byref(kv), 0x1, 0x2, 0x3, 300, float("nan"), 0x4, None,
                                   0x5, n.value, None)
    assert st == B.PRHS_E_INVALID
    # the reuse variant: same checks plus its anchor lengths
    st = L.prhs_reuse_decode_attn(ctypes.byref(kv), 0x1, 0x2, 0x3, 300, None, 0.1, 0x4, None, 0x5,
                                  n.value, None)
    assert st == B.PRHS_E_INVALID
    assert b"anchor_lens" in L.prhs_last_error()
    st = L.prhs_reuse_decode_attn(ctypes.byref(kv), 0x1, 0x2, 0x3, 300, 0x6, 0.1, 0x4, None, 0x5,
                                  n.value - 1, None)
    assert st == B.PRHS_E_WORKSPACE
    st = L.prhs_reuse_decode_attn(ctypes.byref(kv), 0x1, 0x2, 0x3, -1, 0x6, 0.1, 0x4, None, 0x5,
                                  n.value, None)
    assert st == B.PRHS_E_INVALID
    kv0 = _kv(batch=0, k=None, v=None, seq_lens=None)
    assert L.prhs_reuse_decode_attn(ctypes.byref(kv0), None, None, None, 8, None, 0.1, None, None,
                                    None, 0, None) == B.PRHS_OK
    st = L.prhs_dense_decode_attn(ctypes.byref(_kv(head_dim=80)), 0x1, 0.1, 0x4, None, 0x5, 1 << 30,
                                  None)
    assert st == B.PRHS_E_UNSUPPORTED
    st = L.prhs_dense_decode_attn(ctypes.byref(kv), None, 0.1, 0x4, None, 0x5, 1 << 30, None)
    assert st == B.PRHS_E_INVALID


def test_select_shared_validation(L):
    kv = _kv()
    p = B.params(k=8, window=4, refresh_every=4)
    cap = L.prhs_set_capacity(ctypes.byref(p), kv.max_seq_len)
    n = ctypes.c_size_t(0)
    assert L.prhs_workspace_size(B.PRHS_OP_SELECT, ctypes.byref(kv), ctypes.byref(p), 0,
                                 ctypes.byref(n)) == 0
    args = lambda shared, set_cap: (ctypes.byref(kv), 0x1, ctypes.byref(p), 0x2, 0x3, 64, 0x4, 0x5,
                                    set_cap, shared, 0x7, 0x8, n.value, None)
    assert L.prhs_select_shared(*args(None, cap)) == B.PRHS_E_INVALID
    # the shared set needs room for the dilation as well (prhs_set_capacity)
    assert L.prhs_select_shared(*args(0x6, cap - 1)) == B.PRHS_E_CAPACITY
    assert b"shared set" in L.prhs_last_error()
    kv0 = _kv(batch=0, k=None, v=None, seq_lens=None)
    assert L.prhs_select_shared(ctypes.byref(kv0), None, ctypes.byref(p), None, None, 8, None, None,
                                cap, None, None, None, 0, None) == B.PRHS_OK


def test_gate_validation(L):
    def gate(batch=2, hq=8, hkv=2, d=128, dtype=B.PRHS_BF16, tau=0.8, S=4, slot=1, ptr=0x10):
        return L.prhs_gate(batch, hq, hkv, d, dtype, ptr, ptr, tau, S, slot, ptr, ptr, ptr, ptr, ptr,
                           ptr, ptr, 1, None)
    assert gate(tau=1.5) == B.PRHS_E_INVALID
    assert gate(tau=-0.1) == B.PRHS_E_INVALID
    assert gate(tau=float("nan")) == B.PRHS_E_INVALID
    assert gate(slot=4) == B.PRHS_E_INVALID and b"slot" in L.prhs_last_error()
    assert gate(slot=-1) == B.PRHS_E_INVALID
    assert gate(hq=6, hkv=4) == B.PRHS_E_INVALID
    assert gate(dtype=7) == B.PRHS_E_UNSUPPORTED
    assert gate(ptr=None) == B.PRHS_E_INVALID
    assert gate(batch=0, ptr=None) == B.PRHS_OK      # nothing to do, no device work


def test_select_gated_and_pool_attention_validation(L):
    kv = _kv()
    p = B.params(k=8, window=4, refresh_every=4)
    cap = L.prhs_set_capacity(ctypes.byref(p), kv.max_seq_len)
    n = ctypes.c_size_t(0)
    L.prhs_workspace_size(B.PRHS_OP_SELECT, ctypes.byref(kv), ctypes.byref(p), 0, ctypes.byref(n))
    st = L.prhs_select_gated(ctypes.byref(kv), 0x1, ctypes.byref(p), None, 0x2, 0x3, 64, 0x4, 0x5,
                             cap, 0x6, 0x7, 0x8, n.value, None)
    assert st == B.PRHS_E_INVALID and b"choice" in L.prhs_last_error()
    st = L.prhs_select_gated(ctypes.byref(kv), 0x1, ctypes.byref(p), 0x9, 0x2, 0x3, 64, 0x4, 0x5,
                             cap - 1, 0x6, 0x7, 0x8, n.value, None)
    assert st == B.PRHS_E_CAPACITY
    L.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, ctypes.byref(kv), None, 300, ctypes.byref(n))
    good = B.psaw(7, 8, 6, 0.7, 1.0, 4)
    pool = lambda rows, urow, ps, wsb, gate=None, side=0: L.prhs_pool_decode_attn(  # noqa: E731
        ctypes.byref(kv), 0x1, 0x2, 0x3, rows, 300, urow, 0x5, gate, side,
        None if ps is None else ctypes.byref(ps), 0.1, 0x6, None, 0x7, wsb, None)
    assert pool(-1, 0x4, None, n.value) == B.PRHS_E_INVALID
    assert pool(8, None, None, n.value) == B.PRHS_E_INVALID
    assert pool(8, 0x4, B.psaw(7, 8, 6, 0.7, 1.0, -2), n.value) == B.PRHS_E_INVALID
    assert pool(8, 0x4, B.psaw(8, 8, 6, 0.7, 1.0, 4), n.value) == B.PRHS_E_INVALID
    assert pool(8, 0x4, good, n.value - 1) == B.PRHS_E_WORKSPACE
    # the unit filter: a known side, and the gate's choice with a filter
    assert pool(8, 0x4, None, n.value, gate=0x9, side=3) == B.PRHS_E_INVALID
    assert pool(8, 0x4, None, n.value, gate=None, side=B.PRHS_UNITS_SHARING) == B.PRHS_E_INVALID
    assert b"unit_gate" in L.prhs_last_error()
    assert pool(8, 0x4, None, n.value - 1, gate=0x9,
                side=B.PRHS_UNITS_RETRIEVING) == B.PRHS_E_WORKSPACE


def test_gate_select_validation(L):
    kv = _kv()
    p = B.params(k=8, window=4, refresh_every=4)
    cap = L.prhs_set_capacity(ctypes.byref(p), kv.max_seq_len)
    n = ctypes.c_size_t(0)
    L.prhs_workspace_size(B.PRHS_OP_SELECT, ctypes.byref(kv), ctypes.byref(p), 0, ctypes.byref(n))

    def gs(kv=kv, tau=0.8, S=4, slot=1, ptr=0x10, set_cap=cap, wsb=n.value):
        return L.prhs_gate_select(ctypes.byref(kv), 0x1, ctypes.byref(p), tau, S, slot, ptr, ptr,
                                  ptr, ptr, ptr, ptr, ptr, 0x2, 0x3, 64, 0x4, 0x5, set_cap, 0x6,
                                  0x7, 0x8, wsb, None)
    assert gs(tau=1.2) == B.PRHS_E_INVALID and b"tau" in L.prhs_last_error()
    assert gs(slot=4) == B.PRHS_E_INVALID
    assert gs(ptr=None) == B.PRHS_E_INVALID
    assert gs(set_cap=cap - 1) == B.PRHS_E_CAPACITY
    assert gs(wsb=0) == B.PRHS_E_WORKSPACE
    assert gs(kv=_kv(head_dim=96)) == B.PRHS_E_UNSUPPORTED
    kv0 = _kv(batch=0, k=None, v=None, seq_lens=None)
    assert L.prhs_gate_select(ctypes.byref(kv0), None, ctypes.byref(p), 0.8, 4, 0, None, None,
                              None, None, None, None, None, None, None, 8, None, None, cap, None,
                              None, None, 0, None) == B.PRHS_OK


def test_dilate_validation_and_empty_batch(L):
    p = B.params(k=8)
    assert L.prhs_dilate_reuse(ctypes.byref(p), 2, 0, 1, 1, 8, 1, 1, 1, 1, 8, None) == B.PRHS_E_INVALID
    assert L.prhs_dilate_reuse(ctypes.byref(p), 2, 2, None, 1, 8, 1, 1, 1, 1, 8, None) == B.PRHS_E_INVALID
    # an empty batch is a no-op that never touches the device
    assert L.prhs_dilate_reuse(ctypes.byref(p), 0, 2, None, None, 8, None, None, None, None, 8,
                               None) == B.PRHS_OK
    kv0 = _kv(batch=0, k=None, v=None, seq_lens=None)
    assert _select(L, kv0, B.params(k=8, window=4), q=None) == B.PRHS_OK


def test_prefill_validation(L):
    kv = _kv()
    pre = lambda kv=kv, q=0x4000, T=300, sink=4, scale=0.1, out=0x5000: L.prhs_prefill_attn(  # noqa: E731
        ctypes.byref(kv), q, T, ctypes.byref(B.psaw(7, 8, 6, 0.7, 1.0, sink)), scale, out, None,
        None)
    for bad in (0.0, -0.1, float("nan"), float("inf")):
        assert pre(scale=bad) == B.PRHS_E_INVALID
    assert b"scale" in L.prhs_last_error()
    assert pre(T=-1) == B.PRHS_E_INVALID
    assert pre(sink=-1) == B.PRHS_E_INVALID
    assert pre(q=None) == B.PRHS_E_INVALID
    assert pre(out=None) == B.PRHS_E_INVALID
    assert pre(kv=_kv(dtype=B.PRHS_F32)) == B.PRHS_E_UNSUPPORTED
    assert pre(kv=_kv(layout=B.PRHS_KV_PAGED, block_table=None)) == B.PRHS_E_INVALID
    assert pre(T=0, q=None, out=None) == B.PRHS_OK     # nothing to do, no device work
    kv0 = _kv(batch=0, k=None, v=None, seq_lens=None)
    assert pre(kv=kv0, q=None, out=None) == B.PRHS_OK


def test_workspace_size_errors(L):
    n = ctypes.c_size_t(7)
    assert L.prhs_workspace_size(99, None, None, 0, ctypes.byref(n)) == B.PRHS_E_INVALID
    assert L.prhs_workspace_size(B.PRHS_OP_SELECT, None, None, 0, ctypes.byref(n)) == B.PRHS_E_INVALID
    assert L.prhs_workspace_size(B.PRHS_OP_DILATE_REUSE, None, None, 0, ctypes.byref(n)) == B.PRHS_OK
    assert n.value == 0


def test_binding_marshalling_checks():
    # shape and dtype checks of the Python layer run before the C call
    K = torch.zeros(1, 2, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        B.KV(K, K.float(), torch.zeros(1, dtype=torch.int32), 8, 2)
    with pytest.raises(ValueError):
        B.KV(K, K, torch.zeros(2, dtype=torch.int32), 8, 2)
    kv = B.KV(K, K, torch.zeros(1, dtype=torch.int32), 8, 2)
    with pytest.raises(ValueError):
        B.prhs_sparse_decode_attn(kv, torch.zeros(1, 2, 64, dtype=torch.float32),
                                  torch.zeros(1, 2, 8, dtype=torch.int32),
                                  torch.zeros(1, 2, dtype=torch.int32), 0.1,
                                  torch.zeros(1, 2, 64), None, torch.zeros(8, dtype=torch.uint8))


@pytest.mark.parametrize("N,l_s,phi,alpha,sink", [(32, 24, 0.7, 1.0, 4), (8, 6, 0.3, 1.0, 16),
                                                  (8, 4, 0.5, 1.5, 2), (4, 2, 0.01, 3.0, 0),
                                                  (1, 0, 0.7, 1.0, 4), (12, 1, 0.95, 0.2, 70)])
def test_psaw_first_visible_matches_oracle(L, N, l_s, phi, alpha, sink):
    # Eq. psaw lives in the library: its first visible position equals the
    # oracle's at every layer and at lengths across the whole range (decode
    # lengths and every prefill row of a short prompt)
    lens = list(range(0, 301)) + [1023, 4096, 4097, 32769, 131073, 131088, (1 << 22) - 1]
    for layer in range(N):
        ps = B.psaw(layer, N, l_s, phi, alpha, sink)
        got = [B.prhs_psaw_first_visible(ps, n) for n in lens]
        ref = [O.psaw_visible_start(layer, N, n, sink, l_s, phi, alpha) for n in lens]
        assert got == ref, (layer, [(n, a, b) for n, a, b in zip(lens, got, ref) if a != b][:5])
        pre = O.psaw_prefill_visible(layer, N, 300, sink, l_s, phi, alpha)
        assert got[1:301] == pre.tolist()


def test_psaw_descriptor_validation(L):
    bad = [B.psaw(-1, 8, 6, 0.7, 1.0, 4), B.psaw(8, 8, 6, 0.7, 1.0, 4), B.psaw(0, 0, 0, 0.7, 1.0, 4),
           B.psaw(7, 8, 8, 0.7, 1.0, 4), B.psaw(7, 8, -1, 0.7, 1.0, 4), B.psaw(7, 8, 6, 0.0, 1.0, 4),
           B.psaw(7, 8, 6, 1.5, 1.0, 4), B.psaw(7, 8, 6, 0.7, -1.0, 4),
           B.psaw(7, 8, 6, 0.7, float("inf"), 4), B.psaw(7, 8, 6, float("nan"), 1.0, 4),
           B.psaw(7, 8, 6, 0.7, 1.0, -1)]
    for ps in bad:
        assert L.prhs_psaw_first_visible(ctypes.byref(ps), 100) == -1
        assert L.prhs_last_error()
        with pytest.raises(B.PrhsError):
            B.prhs_psaw_first_visible(ps, 100)
    assert L.prhs_psaw_first_visible(None, 100) == -1
    assert L.prhs_psaw_first_visible(ctypes.byref(B.psaw(7, 8, 6, 0.7, 1.0, 4)), -1) == -1
    # phi = 1 masks nothing at any depth
    assert B.prhs_psaw_first_visible(B.psaw(7, 8, 6, 1.0, 1.0, 4), 1000) == 4


def _host_kv(B_=2, hq=8, hkv=2, cap=64, d=64):
    K = torch.zeros(B_, hkv, cap, d, dtype=torch.bfloat16)
    return B.KV(K, K.clone(), torch.full((B_,), cap, dtype=torch.int32), cap, hq)


def _i32(*shape):
    return torch.zeros(*shape, dtype=torch.int32)


def test_binding_rejects_wrong_shapes_before_any_launch():
    # every tensor's shape is checked against the cache descriptor: a wrong
    # one raises ValueError in the binding, before the library is called
    kv = _host_kv()
    q, ws = torch.zeros(2, 8, 64, dtype=torch.bfloat16), torch.zeros(16, dtype=torch.uint8)
    out, lse = torch.zeros(2, 8, 64), torch.zeros(2, 8)
    sets, lens = _i32(2, 2, 40), _i32(2, 2)
    cases = [
        lambda: B.prhs_sparse_decode_attn(kv, q, sets, lens, 0.1, torch.zeros(2, 2, 64), lse, ws),
        lambda: B.prhs_sparse_decode_attn(kv, q, sets, lens, 0.1, out, torch.zeros(2, 2), ws),
        lambda: B.prhs_sparse_decode_attn(kv, q, _i32(2, 8, 40), _i32(2, 8), 0.1, out, lse, ws),
        lambda: B.prhs_sparse_decode_attn(kv, q, sets, _i32(2, 3), 0.1, out, lse, ws),
        lambda: B.prhs_sparse_decode_attn(kv, q[:1], sets, lens, 0.1, out, lse, ws),
        lambda: B.prhs_reuse_decode_attn(kv, q, sets, lens, _i32(3), 0.1, out, lse, ws),
        lambda: B.prhs_dense_decode_attn(kv, q, 0.1, torch.zeros(2, 8, 32), lse, ws),
        lambda: B.prhs_select(kv, q, B.params(k=4), _i32(2, 8, 4), _i32(2, 2), sets, lens, ws),
        lambda: B.prhs_select(kv, q, B.params(k=4), _i32(2, 2, 4), _i32(2), sets, lens, ws),
        lambda: B.prhs_select_shared(kv, q, B.params(k=4), _i32(2, 2, 4), _i32(2, 2), sets, lens,
                                     _i32(2, 2, 39), lens, ws),
        lambda: B.prhs_select_gated(kv, q, B.params(k=4), _i32(2), _i32(2, 2, 4), _i32(2, 2), sets,
                                    lens, sets.clone(), lens.clone(), ws),
        lambda: B.prhs_pool_decode_attn(kv, q, _i32(6, 40), _i32(5), _i32(4), _i32(4), 0.1, out,
                                        lse, ws),
        lambda: B.prhs_pool_decode_attn(kv, q, _i32(6, 40), _i32(6), _i32(3), _i32(4), 0.1, out,
                                        lse, ws),
        lambda: B.prhs_pool_decode_attn(kv, q, _i32(6, 40), _i32(6), _i32(4), _i32(5), 0.1, out,
                                        lse, ws),
        lambda: B.prhs_dilate_reuse(B.params(k=4), _i32(2, 2, 4), _i32(2, 2), _i32(3), _i32(2),
                                    sets, lens),
        lambda: B.prhs_dilate_reuse(B.params(k=4), _i32(2, 2, 4), _i32(2, 2), _i32(2), _i32(2),
                                    _i32(2, 3, 40), lens),
        lambda: B.prhs_gate(q, _i32(2), 0.8, 0, torch.zeros(4, 2, 8, 64, dtype=torch.bfloat16),
                            _i32(4, 4), _i32(4, 2), _i32(3), _i32(4), _i32(4), _i32(4), 2),
        lambda: B.prhs_prefill_attn(kv, torch.zeros(2, 8, 10, 64, dtype=torch.bfloat16), 0.1,
                                    torch.zeros(2, 8, 9, 64)),
        lambda: B.prhs_prefill_attn(kv, torch.zeros(2, 8, 10, 64, dtype=torch.bfloat16), 0.1,
                                    torch.zeros(2, 8, 10, 64), torch.zeros(2, 8, 11)),
    ]
    for i, call in enumerate(cases):
        with pytest.raises(ValueError):
            call()
            pytest.fail(f"case {i} was not rejected")


def test_binding_rejects_host_tensors():
    # correctly shaped tensors that are not on the GPU never reach the library
    kv = _host_kv()
    q, ws = torch.zeros(2, 8, 64, dtype=torch.bfloat16), torch.zeros(16, dtype=torch.uint8)
    out, lse = torch.zeros(2, 8, 64), torch.zeros(2, 8)
    with pytest.raises(ValueError, match="GPU"):
        B.prhs_sparse_decode_attn(kv, q, _i32(2, 2, 40), _i32(2, 2), 0.1, out, lse, ws)
    with pytest.raises(ValueError, match="GPU"):
        B.prhs_dense_decode_attn(kv, q, 0.1, out, None, ws)
    with pytest.raises(ValueError, match="GPU"):
        B.prhs_dilate_reuse(B.params(k=4), _i32(2, 2, 4), _i32(2, 2), _i32(2), _i32(2),
                            _i32(2, 2, 40), _i32(2, 2))
    with pytest.raises(ValueError, match="GPU"):
        B.prhs_gate(q, _i32(2), 0.8, 0, torch.zeros(4, 2, 8, 64, dtype=torch.bfloat16),
                    _i32(4, 4), _i32(4, 2), _i32(4), _i32(4), _i32(4), _i32(4), 2)


def test_static_attention_rejects_partials_beyond_its_scratch(L):
    # partials of 64 x 64 heads x many splits exceed the 16 MiB static array:
    # rejected on the host, before any device work
    kv = _kv(batch=64, num_q_heads=64, num_kv_heads=8, capacity=100000, max_seq_len=100000)
    st = L.prhs_sparse_decode_attn_static(ctypes.byref(kv), 0x1, 0x2, 0x3, 100000, 0.1, 0x4, None,
                                          None)
    assert st == B.PRHS_E_UNSUPPORTED and b"static scratch" in L.prhs_last_error()
    n = ctypes.c_size_t(0)
    L.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, ctypes.byref(kv), None, 100000, ctypes.byref(n))
    assert n.value > 16 << 20
    # an empty batch is a no-op
    kv0 = _kv(batch=0, k=None, v=None, seq_lens=None)
    assert L.prhs_sparse_decode_attn_static(ctypes.byref(kv0), None, None, None, 64, 0.1, None,
                                            None, None) == B.PRHS_OK
