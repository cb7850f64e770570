"""ctypes binding of libprhs (include/prhs.h).

Argument marshalling only: tensors are checked for device, dtype, shape and
contiguity, then their data pointers and the current HIP stream are handed to
the C ABI.  Every step of the hot path runs in the library's HIP kernels; there
is no fallback.  ``lib()`` raises when the library has not been built.
"""

from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libprhs.so")

PRHS_OK = 0
PRHS_E_INVALID = -1
PRHS_E_UNSUPPORTED = -2
PRHS_E_CAPACITY = -3
PRHS_E_WORKSPACE = -4
PRHS_E_DEVICE = -5

PRHS_F32 = 0
PRHS_BF16 = 1
PRHS_KV_CONTIGUOUS = 0
PRHS_KV_PAGED = 1

PRHS_OP_SELECT = 0
PRHS_OP_DILATE_REUSE = 1
PRHS_OP_SPARSE_ATTN = 2
PRHS_OP_DENSE_ATTN = 3

PRHS_REUSE = 0
PRHS_REFRESH = 1
PRHS_MAX_TOPK = 16384

EXPORTS = [
    "prhs_abi_version", "prhs_max_topk", "prhs_set_capacity", "prhs_workspace_size",
    "prhs_schedule", "prhs_select", "prhs_select_shared", "prhs_dilate_reuse", "prhs_sparse_decode_attn",
    "prhs_reuse_decode_attn", "prhs_dense_decode_attn", "prhs_gate", "prhs_select_gated",
    "prhs_pool_decode_attn", "prhs_prefill_attn", "prhs_last_error",
]


class PrhsKv(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("layout", ctypes.c_int32),
        ("capacity", ctypes.c_int32), ("page_size", ctypes.c_int32),
        ("max_pages", ctypes.c_int32), ("num_pages", ctypes.c_int32),
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p), ("seq_lens", ctypes.c_void_p),
        ("max_seq_len", ctypes.c_int32),
    ]


class PrhsParams(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_int32), ("k_num", ctypes.c_int32), ("k_den", ctypes.c_int32),
        ("sink", ctypes.c_int32), ("window", ctypes.c_int32),
        ("dilate_m", ctypes.c_int32), ("dilate_r", ctypes.c_int32),
        ("refresh_every", ctypes.c_int32), ("layer_group", ctypes.c_int32),
    ]


class PrhsError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"prhs status {status}: {message}")
        self.status = status


_lib = None


def lib():
    """The loaded libprhs; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2602_08329_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        i32, vp, sz = ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
        P = ctypes.POINTER
        L.prhs_abi_version.restype = i32
        L.prhs_abi_version.argtypes = []
        L.prhs_max_topk.restype = i32
        L.prhs_max_topk.argtypes = [P(PrhsParams), i32]
        L.prhs_set_capacity.restype = i32
        L.prhs_set_capacity.argtypes = [P(PrhsParams), i32]
        L.prhs_workspace_size.restype = i32
        L.prhs_workspace_size.argtypes = [i32, P(PrhsKv), P(PrhsParams), i32, P(sz)]
        L.prhs_schedule.restype = i32
        L.prhs_schedule.argtypes = [i32, i32, P(PrhsParams)]
        L.prhs_select.restype = i32
        L.prhs_select.argtypes = [P(PrhsKv), vp, P(PrhsParams), vp, vp, i32, vp, vp, i32, vp, sz, vp]
        L.prhs_select_shared.restype = i32
        L.prhs_select_shared.argtypes = [P(PrhsKv), vp, P(PrhsParams), vp, vp, i32, vp, vp, i32,
                                         vp, vp, vp, sz, vp]
        L.prhs_dilate_reuse.restype = i32
        L.prhs_dilate_reuse.argtypes = [P(PrhsParams), i32, i32, vp, vp, i32, vp, vp, vp, vp, i32, vp]
        L.prhs_sparse_decode_attn.restype = i32
        L.prhs_sparse_decode_attn.argtypes = [P(PrhsKv), vp, vp, vp, i32, ctypes.c_float, vp, vp,
                                              vp, sz, vp]
        L.prhs_reuse_decode_attn.restype = i32
        L.prhs_reuse_decode_attn.argtypes = [P(PrhsKv), vp, vp, vp, i32, vp, ctypes.c_float, vp,
                                             vp, vp, sz, vp]
        L.prhs_dense_decode_attn.restype = i32
        L.prhs_dense_decode_attn.argtypes = [P(PrhsKv), vp, ctypes.c_float, vp, vp, vp, sz, vp]
        L.prhs_gate.restype = i32
        L.prhs_gate.argtypes = [i32, i32, i32, i32, i32, vp, vp, ctypes.c_double, i32, i32, vp, vp,
                                vp, vp, vp, vp, vp, vp]
        L.prhs_select_gated.restype = i32
        L.prhs_select_gated.argtypes = [P(PrhsKv), vp, P(PrhsParams), vp, vp, vp, i32, vp, vp, i32,
                                        vp, vp, vp, sz, vp]
        L.prhs_pool_decode_attn.restype = i32
        L.prhs_pool_decode_attn.argtypes = [P(PrhsKv), vp, vp, vp, i32, i32, vp, vp, vp, i32,
                                            ctypes.c_float, vp, vp, vp, sz, vp]
        L.prhs_prefill_attn.restype = i32
        L.prhs_prefill_attn.argtypes = [P(PrhsKv), vp, i32, vp, i32, ctypes.c_float, vp, vp, vp]
        L.prhs_last_error.restype = ctypes.c_char_p
        L.prhs_last_error.argtypes = []
        _lib = L
    return _lib


def check(status):
    if status != PRHS_OK:
        raise PrhsError(status, lib().prhs_last_error().decode())


def params(k=0, sink=4, window=0, dilate_m=-1, dilate_r=1, refresh_every=1, layer_group=1,
           k_num=0, k_den=0):
    return PrhsParams(k, k_num, k_den, sink, window, dilate_m, dilate_r, refresh_every, layer_group)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t, dtype, name, dims=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dims is not None and t.dim() != dims:
        raise ValueError(f"{name} must have {dims} dims, got {t.dim()}")


class KV:
    """A layer's KV cache descriptor; holds references to the tensors it
    points to.  Contiguous K, V: [B][Hkv][capacity][d]; paged: [P][Hkv][ps][d]
    with block_table [B][max_pages] int32."""

    def __init__(self, K, V, seq_lens, max_seq_len, num_q_heads, block_table=None):
        if K.dtype not in (torch.float32, torch.bfloat16) or V.dtype != K.dtype:
            raise ValueError("K and V must both be float32 or bfloat16")
        _need(K, K.dtype, "K", 4)
        _need(V, K.dtype, "V", 4)
        if V.shape != K.shape:
            raise ValueError("K and V shapes differ")
        _need(seq_lens, torch.int32, "seq_lens", 1)
        self._keep = (K, V, seq_lens, block_table)
        d = K.shape[3]
        dt = PRHS_F32 if K.dtype == torch.float32 else PRHS_BF16
        if block_table is None:
            B, Hkv, cap, _ = K.shape
            self.c = PrhsKv(B, num_q_heads, Hkv, d, dt, PRHS_KV_CONTIGUOUS, cap, 0, 0, 0,
                            K.data_ptr(), V.data_ptr(), None, seq_lens.data_ptr(), max_seq_len)
        else:
            _need(block_table, torch.int32, "block_table", 2)
            P, Hkv, ps, _ = K.shape
            B, max_pages = block_table.shape
            self.c = PrhsKv(B, num_q_heads, Hkv, d, dt, PRHS_KV_PAGED, 0, ps, max_pages, P,
                            K.data_ptr(), V.data_ptr(), block_table.data_ptr(),
                            seq_lens.data_ptr(), max_seq_len)
        if seq_lens.numel() != self.c.batch:
            raise ValueError("seq_lens must have one entry per sequence")
        self.dtype = K.dtype

    def with_seq_lens(self, seq_lens, max_seq_len=None):
        """Same cache, other lengths (a new descriptor)."""
        K, V, _, table = self._keep
        return KV(K, V, seq_lens, self.c.max_seq_len if max_seq_len is None else max_seq_len,
                  self.c.num_q_heads, table)


def prhs_max_topk(p, max_seq_len):
    return lib().prhs_max_topk(ctypes.byref(p), max_seq_len)


def prhs_set_capacity(p, max_seq_len):
    return lib().prhs_set_capacity(ctypes.byref(p), max_seq_len)


def prhs_schedule(step, layer, p):
    return lib().prhs_schedule(step, layer, ctypes.byref(p))


def prhs_workspace_size(op, kv=None, p=None, set_cap=0):
    n = ctypes.c_size_t(0)
    check(lib().prhs_workspace_size(op, None if kv is None else ctypes.byref(kv.c),
                                    None if p is None else ctypes.byref(p), set_cap,
                                    ctypes.byref(n)))
    return n.value


def workspace(nbytes, device):
    """A zero-filled device workspace.  No entry point needs its workspace
    initialised; zeros keep runs reproducible."""
    return torch.zeros(max(1, nbytes), dtype=torch.uint8, device=device)


def _q_dtype(kv, q):
    _need(q, kv.dtype, "q", 3)
    if q.shape != (kv.c.batch, kv.c.num_q_heads, kv.c.head_dim):
        raise ValueError(f"q must be [B][Hq][d], got {tuple(q.shape)}")


def prhs_select(kv, q, p, topk_idx, topk_len, set_idx, set_len, ws, stream=None):
    _q_dtype(kv, q)
    for t, n, dims in ((topk_idx, "topk_idx", 3), (topk_len, "topk_len", 2),
                       (set_idx, "set_idx", 3), (set_len, "set_len", 2)):
        _need(t, torch.int32, n, dims)
    _need(ws, torch.uint8, "ws")
    check(lib().prhs_select(ctypes.byref(kv.c), _ptr(q), ctypes.byref(p), _ptr(topk_idx),
                            _ptr(topk_len), topk_idx.shape[-1], _ptr(set_idx), _ptr(set_len),
                            set_idx.shape[-1], _ptr(ws), ws.numel(), _stream(stream)))


def prhs_select_shared(kv, q, p, topk_idx, topk_len, set_idx, set_len, shared_idx, shared_len, ws,
                       stream=None):
    """prhs_select that also writes the dilated shared set at the anchor
    length (shared_idx has the same capacity as set_idx)."""
    _q_dtype(kv, q)
    for t, n, dims in ((topk_idx, "topk_idx", 3), (topk_len, "topk_len", 2),
                       (set_idx, "set_idx", 3), (set_len, "set_len", 2),
                       (shared_idx, "shared_idx", 3), (shared_len, "shared_len", 2)):
        _need(t, torch.int32, n, dims)
    if shared_idx.shape != set_idx.shape:
        raise ValueError("shared_idx must have the shape of set_idx")
    _need(ws, torch.uint8, "ws")
    check(lib().prhs_select_shared(ctypes.byref(kv.c), _ptr(q), ctypes.byref(p), _ptr(topk_idx),
                                   _ptr(topk_len), topk_idx.shape[-1], _ptr(set_idx),
                                   _ptr(set_len), set_idx.shape[-1], _ptr(shared_idx),
                                   _ptr(shared_len), _ptr(ws), ws.numel(), _stream(stream)))


def prhs_dilate_reuse(p, topk_idx, topk_len, anchor_lens, seq_lens, set_idx, set_len, stream=None):
    for t, n, dims in ((topk_idx, "topk_idx", 3), (topk_len, "topk_len", 2),
                       (anchor_lens, "anchor_lens", 1), (seq_lens, "seq_lens", 1),
                       (set_idx, "set_idx", 3), (set_len, "set_len", 2)):
        _need(t, torch.int32, n, dims)
    B, Hkv, k_cap = topk_idx.shape
    check(lib().prhs_dilate_reuse(ctypes.byref(p), B, Hkv, _ptr(topk_idx), _ptr(topk_len), k_cap,
                                  _ptr(anchor_lens), _ptr(seq_lens), _ptr(set_idx), _ptr(set_len),
                                  set_idx.shape[-1], _stream(stream)))


def prhs_sparse_decode_attn(kv, q, set_idx, set_len, scale, out, lse, ws, stream=None):
    _q_dtype(kv, q)
    _need(set_idx, torch.int32, "set_idx", 3)
    _need(set_len, torch.int32, "set_len", 2)
    _need(out, torch.float32, "out", 3)
    if lse is not None:
        _need(lse, torch.float32, "lse", 2)
    _need(ws, torch.uint8, "ws")
    check(lib().prhs_sparse_decode_attn(ctypes.byref(kv.c), _ptr(q), _ptr(set_idx), _ptr(set_len),
                                        set_idx.shape[-1], float(scale), _ptr(out), _ptr(lse),
                                        _ptr(ws), ws.numel(), _stream(stream)))


def prhs_reuse_decode_attn(kv, q, set_idx, set_len, anchor_lens, scale, out, lse, ws,
                           stream=None):
    """Attention over set U [anchor_lens[b], n_b): the reused set of a later
    step, with the set built once at the anchor length."""
    _q_dtype(kv, q)
    _need(set_idx, torch.int32, "set_idx", 3)
    _need(set_len, torch.int32, "set_len", 2)
    _need(anchor_lens, torch.int32, "anchor_lens", 1)
    _need(out, torch.float32, "out", 3)
    if lse is not None:
        _need(lse, torch.float32, "lse", 2)
    _need(ws, torch.uint8, "ws")
    check(lib().prhs_reuse_decode_attn(ctypes.byref(kv.c), _ptr(q), _ptr(set_idx), _ptr(set_len),
                                       set_idx.shape[-1], _ptr(anchor_lens), float(scale),
                                       _ptr(out), _ptr(lse), _ptr(ws), ws.numel(),
                                       _stream(stream)))


def prhs_gate(q, seq_lens, tau, slot, ref_q, ref_valid, slot_lens, choice, row_anchor, row_other,
              tail, num_kv_heads, stream=None):
    """Similarity gate for block step `slot`: q [B][Hq][d]; ref_q
    [S][B][Hq][d] (dtype of q); ref_valid [S][B*Hkv]; slot_lens [S][B];
    choice, row_anchor, row_other, tail [B*Hkv] int32 outputs."""
    if q.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("q must be bf16 or fp32")
    _need(q, q.dtype, "q", 3)
    _need(ref_q, q.dtype, "ref_q", 4)
    B, Hq, d = q.shape
    S = ref_q.shape[0]
    if tuple(ref_q.shape[1:]) != (B, Hq, d):
        raise ValueError("ref_q must be [S][B][Hq][d]")
    for t, n, shape in ((seq_lens, "seq_lens", (B,)), (ref_valid, "ref_valid", (S, B * num_kv_heads)),
                        (slot_lens, "slot_lens", (S, B)), (choice, "choice", (B * num_kv_heads,)),
                        (row_anchor, "row_anchor", (B * num_kv_heads,)),
                        (row_other, "row_other", (B * num_kv_heads,)),
                        (tail, "tail", (B * num_kv_heads,))):
        _need(t, torch.int32, n)
        if tuple(t.shape) != shape:
            raise ValueError(f"{n} must have shape {shape}, got {tuple(t.shape)}")
    dt = PRHS_BF16 if q.dtype == torch.bfloat16 else PRHS_F32
    check(lib().prhs_gate(B, Hq, num_kv_heads, d, dt, _ptr(q), _ptr(seq_lens), float(tau), S,
                          int(slot), _ptr(ref_q), _ptr(ref_valid), _ptr(slot_lens), _ptr(choice),
                          _ptr(row_anchor), _ptr(row_other), _ptr(tail), _stream(stream)))


def prhs_select_gated(kv, q, p, choice, topk_idx, topk_len, set_idx, set_len, shared_idx, shared_len,
                      ws, stream=None):
    """prhs_select_shared for the units with choice < 0 only."""
    _q_dtype(kv, q)
    _need(choice, torch.int32, "choice")
    for t, n, dims in ((topk_idx, "topk_idx", 3), (topk_len, "topk_len", 2),
                       (set_idx, "set_idx", 3), (set_len, "set_len", 2),
                       (shared_idx, "shared_idx", 3), (shared_len, "shared_len", 2)):
        _need(t, torch.int32, n, dims)
    if shared_idx.shape != set_idx.shape:
        raise ValueError("shared_idx must have the shape of set_idx")
    _need(ws, torch.uint8, "ws")
    check(lib().prhs_select_gated(ctypes.byref(kv.c), _ptr(q), ctypes.byref(p), _ptr(choice),
                                  _ptr(topk_idx), _ptr(topk_len), topk_idx.shape[-1],
                                  _ptr(set_idx), _ptr(set_len), set_idx.shape[-1],
                                  _ptr(shared_idx), _ptr(shared_len), _ptr(ws), ws.numel(),
                                  _stream(stream)))


def prhs_pool_decode_attn(kv, q, pool_idx, pool_len, unit_row, unit_tail, scale, out, lse, ws,
                          stream=None, psaw_start=None, psaw_sink=0):
    """Attention where unit u attends pool row unit_row[u] plus the tail
    [unit_tail[u], n_b), without the positions [psaw_sink, psaw_start[b])
    when psaw_start [B] is given.  pool_idx [..][set_cap] (any leading dims,
    flattened to rows), pool_len with the same leading dims."""
    if psaw_start is not None:
        _need(psaw_start, torch.int32, "psaw_start", 1)
    _q_dtype(kv, q)
    _need(pool_idx, torch.int32, "pool_idx")
    _need(pool_len, torch.int32, "pool_len")
    cap = pool_idx.shape[-1]
    rows = pool_idx.numel() // max(cap, 1)
    if pool_len.numel() != rows:
        raise ValueError("pool_len must have one entry per pool row")
    _need(unit_row, torch.int32, "unit_row")
    _need(unit_tail, torch.int32, "unit_tail")
    _need(out, torch.float32, "out", 3)
    if lse is not None:
        _need(lse, torch.float32, "lse", 2)
    _need(ws, torch.uint8, "ws")
    check(lib().prhs_pool_decode_attn(ctypes.byref(kv.c), _ptr(q), _ptr(pool_idx), _ptr(pool_len),
                                      rows, cap, _ptr(unit_row), _ptr(unit_tail),
                                      _ptr(psaw_start), int(psaw_sink), float(scale), _ptr(out),
                                      _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)))


def prhs_prefill_attn(kv, q, scale, out, lse=None, vis_start=None, sink=0, stream=None):
    """Causal prefill attention of the prompts (kv holds them; seq_lens are
    their lengths) for the queries q [B][Hq][T][d] at positions 0 .. T - 1,
    under the PSAW mask when vis_start [T] int32 is given."""
    _need(q, kv.dtype, "q", 4)
    B_, H_, T, d = q.shape
    if (B_, H_, d) != (kv.c.batch, kv.c.num_q_heads, kv.c.head_dim):
        raise ValueError(f"q must be [B][Hq][T][d], got {tuple(q.shape)}")
    _need(out, torch.float32, "out", 4)
    if tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must have q's shape")
    if lse is not None:
        _need(lse, torch.float32, "lse", 3)
        if tuple(lse.shape) != (B_, H_, T):
            raise ValueError("lse must be [B][Hq][T]")
    if vis_start is not None:
        _need(vis_start, torch.int32, "vis_start", 1)
        if vis_start.numel() != T:
            raise ValueError("vis_start must have T entries")
    check(lib().prhs_prefill_attn(ctypes.byref(kv.c), _ptr(q), int(T), _ptr(vis_start), int(sink),
                                  float(scale), _ptr(out), _ptr(lse), _stream(stream)))


def prhs_dense_decode_attn(kv, q, scale, out, lse, ws, stream=None):
    _q_dtype(kv, q)
    _need(out, torch.float32, "out", 3)
    if lse is not None:
        _need(lse, torch.float32, "lse", 2)
    _need(ws, torch.uint8, "ws")
    check(lib().prhs_dense_decode_attn(ctypes.byref(kv.c), _ptr(q), float(scale), _ptr(out),
                                       _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)))
