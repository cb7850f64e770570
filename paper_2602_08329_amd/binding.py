"""ctypes binding of libprhs (include/prhs.h).

Argument marshalling only: every tensor is checked for dtype, contiguity and
its exact shape against the cache descriptor, and for living on the cache's
GPU, before its data pointer and the current HIP stream are handed to the C
ABI (so a wrongly shaped or host tensor raises ValueError instead of reaching
a kernel).  Every step of the hot path runs in the library's HIP kernels; there
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
PRHS_UNITS_ALL = 0
PRHS_UNITS_RETRIEVING = 1
PRHS_UNITS_SHARING = 2
PRHS_MAX_TOPK = 16000

EXPORTS = [
    "prhs_abi_version", "prhs_max_topk", "prhs_set_capacity", "prhs_workspace_size",
    "prhs_schedule", "prhs_select", "prhs_select_shared", "prhs_dilate_reuse", "prhs_sparse_decode_attn",
    "prhs_sparse_decode_attn_static",
    "prhs_reuse_decode_attn", "prhs_dense_decode_attn", "prhs_gate", "prhs_gate_select",
    "prhs_select_gated",
    "prhs_pool_decode_attn", "prhs_prefill_attn", "prhs_psaw_first_visible", "prhs_last_error",
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


class PrhsPsaw(ctypes.Structure):
    _fields_ = [
        ("layer", ctypes.c_int32), ("num_layers", ctypes.c_int32), ("l_s", ctypes.c_int32),
        ("sink", ctypes.c_int32), ("phi", ctypes.c_double), ("alpha", ctypes.c_double),
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
        L.prhs_sparse_decode_attn_static.restype = i32
        L.prhs_sparse_decode_attn_static.argtypes = [P(PrhsKv), vp, vp, vp, i32, ctypes.c_float, vp,
                                                     vp, vp]
        L.prhs_reuse_decode_attn.restype = i32
        L.prhs_reuse_decode_attn.argtypes = [P(PrhsKv), vp, vp, vp, i32, vp, ctypes.c_float, vp,
                                             vp, vp, sz, vp]
        L.prhs_dense_decode_attn.restype = i32
        L.prhs_dense_decode_attn.argtypes = [P(PrhsKv), vp, ctypes.c_float, vp, vp, vp, sz, vp]
        L.prhs_gate.restype = i32
        L.prhs_gate.argtypes = [i32, i32, i32, i32, i32, vp, vp, ctypes.c_double, i32, i32, vp, vp,
                                vp, vp, vp, vp, vp, i32, vp]
        L.prhs_gate_select.restype = i32
        L.prhs_gate_select.argtypes = [P(PrhsKv), vp, P(PrhsParams), ctypes.c_double, i32, i32, vp,
                                       vp, vp, vp, vp, vp, vp, vp, vp, i32, vp, vp, i32, vp, vp,
                                       vp, sz, vp]
        L.prhs_select_gated.restype = i32
        L.prhs_select_gated.argtypes = [P(PrhsKv), vp, P(PrhsParams), vp, vp, vp, i32, vp, vp, i32,
                                        vp, vp, vp, sz, vp]
        L.prhs_pool_decode_attn.restype = i32
        L.prhs_pool_decode_attn.argtypes = [P(PrhsKv), vp, vp, vp, i32, i32, vp, vp, vp, i32,
                                            P(PrhsPsaw), ctypes.c_float, vp, vp, vp, sz, vp]
        L.prhs_prefill_attn.restype = i32
        L.prhs_prefill_attn.argtypes = [P(PrhsKv), vp, i32, P(PrhsPsaw), ctypes.c_float, vp, vp, vp]
        L.prhs_psaw_first_visible.restype = i32
        L.prhs_psaw_first_visible.argtypes = [P(PrhsPsaw), i32]
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


def psaw(layer, num_layers, l_s, phi, alpha, sink):
    """Descriptor of one layer's progressive sliding attention window (Eq. psaw)."""
    return PrhsPsaw(int(layer), int(num_layers), int(l_s), int(sink), float(phi), float(alpha))


def prhs_psaw_first_visible(ps, n):
    """First visible non-sink position of the window `ps` with n tokens in view."""
    v = lib().prhs_psaw_first_visible(ctypes.byref(ps), int(n))
    if v < 0:
        raise PrhsError(PRHS_E_INVALID, lib().prhs_last_error().decode())
    return v


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _ref(x):
    return None if x is None else ctypes.byref(x)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t, dtype, name, shape=None, dims=None):
    """Type, dtype, contiguity and shape (exact `shape`, or `dims` dimensions)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dims is not None and t.dim() != dims:
        raise ValueError(f"{name} must have {dims} dims, got {t.dim()}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _on_device(device, **tensors):
    """Every given tensor lives on `device`, a GPU (checked after the shapes,
    just before the launch)."""
    if device.type != "cuda":
        raise ValueError(f"the cache lives on {device}; the library runs on the GPU")
    for name, t in tensors.items():
        if t is not None and t.device != device:
            raise ValueError(f"{name} is on {t.device}, the cache on {device}")


class KV:
    """A layer's KV cache descriptor; holds references to the tensors it
    points to.  Contiguous K, V: [B][Hkv][capacity][d]; paged: [P][Hkv][ps][d]
    with block_table [B][max_pages] int32."""

    def __init__(self, K, V, seq_lens, max_seq_len, num_q_heads, block_table=None):
        if K.dtype not in (torch.float32, torch.bfloat16) or V.dtype != K.dtype:
            raise ValueError("K and V must both be float32 or bfloat16")
        _need(K, K.dtype, "K", dims=4)
        _need(V, K.dtype, "V", shape=K.shape)
        _need(seq_lens, torch.int32, "seq_lens", dims=1)
        self._keep = (K, V, seq_lens, block_table)
        d = K.shape[3]
        dt = PRHS_F32 if K.dtype == torch.float32 else PRHS_BF16
        if block_table is None:
            B, Hkv, cap, _ = K.shape
            self.c = PrhsKv(B, num_q_heads, Hkv, d, dt, PRHS_KV_CONTIGUOUS, cap, 0, 0, 0,
                            K.data_ptr(), V.data_ptr(), None, seq_lens.data_ptr(), max_seq_len)
        else:
            _need(block_table, torch.int32, "block_table", dims=2)
            P, Hkv, ps, _ = K.shape
            B, max_pages = block_table.shape
            self.c = PrhsKv(B, num_q_heads, Hkv, d, dt, PRHS_KV_PAGED, 0, ps, max_pages, P,
                            K.data_ptr(), V.data_ptr(), block_table.data_ptr(),
                            seq_lens.data_ptr(), max_seq_len)
        if seq_lens.numel() != self.c.batch:
            raise ValueError("seq_lens must have one entry per sequence")
        self.dtype = K.dtype
        self.device = K.device

    # shapes the entry points expect, from the descriptor
    @property
    def units(self):
        return self.c.batch * self.c.num_kv_heads

    def q_shape(self):
        return (self.c.batch, self.c.num_q_heads, self.c.head_dim)

    def per_unit(self, last=None):
        base = (self.c.batch, self.c.num_kv_heads)
        return base if last is None else base + (last,)

    def check_device(self, **tensors):
        K, V, seq_lens, table = self._keep
        _on_device(self.device, K=K, V=V, seq_lens=seq_lens, block_table=table, **tensors)

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
    """A zero-filled device workspace: a selection workspace needs its
    leading histogram region (select_zero_bytes) zero before its first use;
    the other workspaces need no initialisation."""
    return torch.zeros(max(1, nbytes), dtype=torch.uint8, device=device)


def select_zero_bytes(kv):
    """Bytes at the front of a selection workspace that must be zero when a
    call starts and that every call leaves zero (per-row histograms and
    counters of batch x num_kv_heads rows)."""
    rows = kv.c.batch * kv.c.num_kv_heads

    def a256(x):
        return (x + 255) // 256 * 256
    return 2 * a256(rows * 8192) + a256(rows * 16)


def _q(kv, q):
    _need(q, kv.dtype, "q", shape=kv.q_shape())


def _outputs(kv, out, lse):
    _need(out, torch.float32, "out", shape=kv.q_shape())
    if lse is not None:
        _need(lse, torch.float32, "lse", shape=kv.q_shape()[:2])


def _ws(ws):
    _need(ws, torch.uint8, "ws", dims=1)


def _selection_outputs(kv, topk_idx, topk_len, set_idx, set_len, shared_idx=None,
                       shared_len=None):
    _need(topk_idx, torch.int32, "topk_idx", dims=3)
    _need(topk_idx, torch.int32, "topk_idx", shape=kv.per_unit(topk_idx.shape[-1]))
    _need(topk_len, torch.int32, "topk_len", shape=kv.per_unit())
    _need(set_idx, torch.int32, "set_idx", dims=3)
    _need(set_idx, torch.int32, "set_idx", shape=kv.per_unit(set_idx.shape[-1]))
    _need(set_len, torch.int32, "set_len", shape=kv.per_unit())
    if shared_idx is not None or shared_len is not None:
        _need(shared_idx, torch.int32, "shared_idx", shape=set_idx.shape)
        _need(shared_len, torch.int32, "shared_len", shape=kv.per_unit())


def prhs_select(kv, q, p, topk_idx, topk_len, set_idx, set_len, ws, stream=None):
    _q(kv, q)
    _selection_outputs(kv, topk_idx, topk_len, set_idx, set_len)
    _ws(ws)
    kv.check_device(q=q, topk_idx=topk_idx, topk_len=topk_len, set_idx=set_idx, set_len=set_len,
                    ws=ws)
    check(lib().prhs_select(ctypes.byref(kv.c), _ptr(q), ctypes.byref(p), _ptr(topk_idx),
                            _ptr(topk_len), topk_idx.shape[-1], _ptr(set_idx), _ptr(set_len),
                            set_idx.shape[-1], _ptr(ws), ws.numel(), _stream(stream)))


def prhs_select_shared(kv, q, p, topk_idx, topk_len, set_idx, set_len, shared_idx, shared_len, ws,
                       stream=None):
    """prhs_select that also writes the dilated shared set at the anchor
    length (shared_idx has the same capacity as set_idx)."""
    _q(kv, q)
    _selection_outputs(kv, topk_idx, topk_len, set_idx, set_len, shared_idx, shared_len)
    _ws(ws)
    kv.check_device(q=q, topk_idx=topk_idx, topk_len=topk_len, set_idx=set_idx, set_len=set_len,
                    shared_idx=shared_idx, shared_len=shared_len, ws=ws)
    check(lib().prhs_select_shared(ctypes.byref(kv.c), _ptr(q), ctypes.byref(p), _ptr(topk_idx),
                                   _ptr(topk_len), topk_idx.shape[-1], _ptr(set_idx),
                                   _ptr(set_len), set_idx.shape[-1], _ptr(shared_idx),
                                   _ptr(shared_len), _ptr(ws), ws.numel(), _stream(stream)))


def prhs_dilate_reuse(p, topk_idx, topk_len, anchor_lens, seq_lens, set_idx, set_len, stream=None):
    _need(topk_idx, torch.int32, "topk_idx", dims=3)
    B, Hkv, k_cap = topk_idx.shape
    _need(topk_len, torch.int32, "topk_len", shape=(B, Hkv))
    _need(anchor_lens, torch.int32, "anchor_lens", shape=(B,))
    _need(seq_lens, torch.int32, "seq_lens", shape=(B,))
    _need(set_idx, torch.int32, "set_idx", dims=3)
    _need(set_idx, torch.int32, "set_idx", shape=(B, Hkv, set_idx.shape[-1]))
    _need(set_len, torch.int32, "set_len", shape=(B, Hkv))
    _on_device(topk_idx.device, topk_len=topk_len, anchor_lens=anchor_lens, seq_lens=seq_lens,
               set_idx=set_idx, set_len=set_len)
    check(lib().prhs_dilate_reuse(ctypes.byref(p), B, Hkv, _ptr(topk_idx), _ptr(topk_len), k_cap,
                                  _ptr(anchor_lens), _ptr(seq_lens), _ptr(set_idx), _ptr(set_len),
                                  set_idx.shape[-1], _stream(stream)))


def _sets(kv, set_idx, set_len):
    _need(set_idx, torch.int32, "set_idx", dims=3)
    _need(set_idx, torch.int32, "set_idx", shape=kv.per_unit(set_idx.shape[-1]))
    _need(set_len, torch.int32, "set_len", shape=kv.per_unit())


def prhs_sparse_decode_attn(kv, q, set_idx, set_len, scale, out, lse, ws, stream=None):
    _q(kv, q)
    _sets(kv, set_idx, set_len)
    _outputs(kv, out, lse)
    _ws(ws)
    kv.check_device(q=q, set_idx=set_idx, set_len=set_len, out=out, lse=lse, ws=ws)
    check(lib().prhs_sparse_decode_attn(ctypes.byref(kv.c), _ptr(q), _ptr(set_idx), _ptr(set_len),
                                        set_idx.shape[-1], float(scale), _ptr(out), _ptr(lse),
                                        _ptr(ws), ws.numel(), _stream(stream)))


def prhs_sparse_decode_attn_static(kv, q, set_idx, set_len, scale, out, lse, stream=None):
    """prhs_sparse_decode_attn with its split-K partials in the library's
    static device array instead of a workspace: no allocation anywhere.
    Calls that overlap on one GPU race."""
    _q(kv, q)
    _sets(kv, set_idx, set_len)
    _outputs(kv, out, lse)
    kv.check_device(q=q, set_idx=set_idx, set_len=set_len, out=out, lse=lse)
    check(lib().prhs_sparse_decode_attn_static(ctypes.byref(kv.c), _ptr(q), _ptr(set_idx),
                                               _ptr(set_len), set_idx.shape[-1], float(scale),
                                               _ptr(out), _ptr(lse), _stream(stream)))


def prhs_reuse_decode_attn(kv, q, set_idx, set_len, anchor_lens, scale, out, lse, ws,
                           stream=None):
    """Attention over set U [anchor_lens[b], n_b): the reused set of a later
    step, with the set built once at the anchor length."""
    _q(kv, q)
    _sets(kv, set_idx, set_len)
    _need(anchor_lens, torch.int32, "anchor_lens", shape=(kv.c.batch,))
    _outputs(kv, out, lse)
    _ws(ws)
    kv.check_device(q=q, set_idx=set_idx, set_len=set_len, anchor_lens=anchor_lens, out=out,
                    lse=lse, ws=ws)
    check(lib().prhs_reuse_decode_attn(ctypes.byref(kv.c), _ptr(q), _ptr(set_idx), _ptr(set_len),
                                       set_idx.shape[-1], _ptr(anchor_lens), float(scale),
                                       _ptr(out), _ptr(lse), _ptr(ws), ws.numel(),
                                       _stream(stream)))


def _gate_arrays(q, seq_lens, ref_q, ref_valid, slot_lens, choice, row_anchor, row_other, tail,
                 num_kv_heads):
    if not isinstance(q, torch.Tensor) or q.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("q must be a bf16 or fp32 tensor")
    _need(q, q.dtype, "q", dims=3)
    B_, Hq, d = q.shape
    _need(ref_q, q.dtype, "ref_q", dims=4)
    S = ref_q.shape[0]
    _need(ref_q, q.dtype, "ref_q", shape=(S, B_, Hq, d))
    U = B_ * num_kv_heads
    for t, n, shape in ((seq_lens, "seq_lens", (B_,)), (ref_valid, "ref_valid", (S, U)),
                        (slot_lens, "slot_lens", (S, B_)), (choice, "choice", (U,)),
                        (row_anchor, "row_anchor", (U,)), (row_other, "row_other", (U,)),
                        (tail, "tail", (U,))):
        _need(t, torch.int32, n, shape=shape)
    return S


def prhs_gate(q, seq_lens, tau, slot, ref_q, ref_valid, slot_lens, choice, row_anchor, row_other,
              tail, num_kv_heads, stream=None, record=True):
    """Similarity gate for block step `slot`: q [B][Hq][d]; ref_q
    [S][B][Hq][d] (dtype of q); ref_valid [S][B*Hkv]; slot_lens [S][B];
    choice, row_anchor, row_other, tail [B*Hkv] int32 outputs.  With
    record=False the step is decided but not recorded (ref_q, ref_valid and
    slot_lens are only read)."""
    S = _gate_arrays(q, seq_lens, ref_q, ref_valid, slot_lens, choice, row_anchor, row_other, tail,
                     num_kv_heads)
    _on_device(q.device, seq_lens=seq_lens, ref_q=ref_q, ref_valid=ref_valid,
               slot_lens=slot_lens, choice=choice, row_anchor=row_anchor, row_other=row_other,
               tail=tail)
    B_, Hq, d = q.shape
    dt = PRHS_BF16 if q.dtype == torch.bfloat16 else PRHS_F32
    check(lib().prhs_gate(B_, Hq, num_kv_heads, d, dt, _ptr(q), _ptr(seq_lens), float(tau), S,
                          int(slot), _ptr(ref_q), _ptr(ref_valid), _ptr(slot_lens), _ptr(choice),
                          _ptr(row_anchor), _ptr(row_other), _ptr(tail), 1 if record else 0,
                          _stream(stream)))


def prhs_gate_select(kv, q, p, tau, slot, ref_q, ref_valid, slot_lens, choice, row_anchor,
                     row_other, tail, topk_idx, topk_len, set_idx, set_len, shared_idx,
                     shared_len, ws, stream=None):
    """prhs_gate (recording the step) and the refresh of the retrieving units
    in one call; the gate runs inside the refresh launch where that is one
    fused kernel."""
    _q(kv, q)
    seq_lens = kv._keep[2]
    S = _gate_arrays(q, seq_lens, ref_q, ref_valid, slot_lens, choice, row_anchor, row_other, tail,
                     kv.c.num_kv_heads)
    _selection_outputs(kv, topk_idx, topk_len, set_idx, set_len, shared_idx, shared_len)
    _ws(ws)
    kv.check_device(q=q, ref_q=ref_q, ref_valid=ref_valid, slot_lens=slot_lens, choice=choice,
                    row_anchor=row_anchor, row_other=row_other, tail=tail, topk_idx=topk_idx,
                    topk_len=topk_len, set_idx=set_idx, set_len=set_len, shared_idx=shared_idx,
                    shared_len=shared_len, ws=ws)
    check(lib().prhs_gate_select(ctypes.byref(kv.c), _ptr(q), ctypes.byref(p), float(tau), S,
                                 int(slot), _ptr(ref_q), _ptr(ref_valid), _ptr(slot_lens),
                                 _ptr(choice), _ptr(row_anchor), _ptr(row_other), _ptr(tail),
                                 _ptr(topk_idx), _ptr(topk_len), topk_idx.shape[-1], _ptr(set_idx),
                                 _ptr(set_len), set_idx.shape[-1], _ptr(shared_idx),
                                 _ptr(shared_len), _ptr(ws), ws.numel(), _stream(stream)))


def prhs_select_gated(kv, q, p, choice, topk_idx, topk_len, set_idx, set_len, shared_idx, shared_len,
                      ws, stream=None):
    """prhs_select_shared for the units with choice < 0 only."""
    _q(kv, q)
    _need(choice, torch.int32, "choice", shape=(kv.units,))
    _selection_outputs(kv, topk_idx, topk_len, set_idx, set_len, shared_idx, shared_len)
    _ws(ws)
    kv.check_device(q=q, choice=choice, topk_idx=topk_idx, topk_len=topk_len, set_idx=set_idx,
                    set_len=set_len, shared_idx=shared_idx, shared_len=shared_len, ws=ws)
    check(lib().prhs_select_gated(ctypes.byref(kv.c), _ptr(q), ctypes.byref(p), _ptr(choice),
                                  _ptr(topk_idx), _ptr(topk_len), topk_idx.shape[-1],
                                  _ptr(set_idx), _ptr(set_len), set_idx.shape[-1],
                                  _ptr(shared_idx), _ptr(shared_len), _ptr(ws), ws.numel(),
                                  _stream(stream)))


def prhs_pool_decode_attn(kv, q, pool_idx, pool_len, unit_row, unit_tail, scale, out, lse, ws,
                          stream=None, psaw=None, unit_gate=None, units_side=PRHS_UNITS_ALL):
    """Attention where unit u attends pool row unit_row[u] plus the tail
    [unit_tail[u], n_b), under the layer's PSAW mask (Eq. psaw) when psaw (a
    PrhsPsaw) is given.  pool_idx [..][set_cap] (any leading dims, flattened
    to rows), pool_len with the same leading dims.  units_side (with the
    gate's choice as unit_gate) restricts the launch to the retrieving or
    the sharing units; the others' outputs are left as they are."""
    if units_side != PRHS_UNITS_ALL:
        _need(unit_gate, torch.int32, "unit_gate", shape=(kv.units,))
    _q(kv, q)
    _need(pool_idx, torch.int32, "pool_idx")
    if pool_idx.dim() < 1:
        raise ValueError("pool_idx must have at least one dimension")
    cap = pool_idx.shape[-1]
    rows = pool_idx.numel() // max(cap, 1)
    _need(pool_len, torch.int32, "pool_len", shape=pool_idx.shape[:-1])
    _need(unit_row, torch.int32, "unit_row", shape=(kv.units,))
    _need(unit_tail, torch.int32, "unit_tail", shape=(kv.units,))
    _outputs(kv, out, lse)
    _ws(ws)
    if psaw is not None and not isinstance(psaw, PrhsPsaw):
        raise TypeError("psaw must be a PrhsPsaw (binding.psaw(...))")
    kv.check_device(q=q, pool_idx=pool_idx, pool_len=pool_len, unit_row=unit_row,
                    unit_tail=unit_tail, unit_gate=unit_gate, out=out, lse=lse, ws=ws)
    check(lib().prhs_pool_decode_attn(ctypes.byref(kv.c), _ptr(q), _ptr(pool_idx), _ptr(pool_len),
                                      rows, cap, _ptr(unit_row), _ptr(unit_tail),
                                      _ptr(unit_gate) if units_side != PRHS_UNITS_ALL else None,
                                      int(units_side), _ref(psaw), float(scale), _ptr(out),
                                      _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)))


def prhs_prefill_attn(kv, q, scale, out, lse=None, psaw=None, stream=None):
    """Causal prefill attention of the prompts (kv holds them; seq_lens are
    their lengths) for the queries q [B][Hq][T][d] at positions 0 .. T - 1,
    under the layer's PSAW mask (Eq. psaw) when psaw (a PrhsPsaw) is given."""
    _need(q, kv.dtype, "q", dims=4)
    B_, H_, T, d = q.shape
    _need(q, kv.dtype, "q", shape=(kv.c.batch, kv.c.num_q_heads, T, kv.c.head_dim))
    _need(out, torch.float32, "out", shape=q.shape)
    if lse is not None:
        _need(lse, torch.float32, "lse", shape=(B_, H_, T))
    if psaw is not None and not isinstance(psaw, PrhsPsaw):
        raise TypeError("psaw must be a PrhsPsaw (binding.psaw(...))")
    kv.check_device(q=q, out=out, lse=lse)
    check(lib().prhs_prefill_attn(ctypes.byref(kv.c), _ptr(q), int(T), _ref(psaw), float(scale),
                                  _ptr(out), _ptr(lse), _stream(stream)))


def prhs_dense_decode_attn(kv, q, scale, out, lse, ws, stream=None):
    _q(kv, q)
    _outputs(kv, out, lse)
    _ws(ws)
    kv.check_device(q=q, out=out, lse=lse, ws=ws)
    check(lib().prhs_dense_decode_attn(ctypes.byref(kv.c), _ptr(q), float(scale), _ptr(out),
                                       _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)))
