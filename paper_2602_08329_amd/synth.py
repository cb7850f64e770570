"""Seeded synthetic decode workloads shaped like the paper's experiments.

This module only draws inputs: queries, a K/V cache per layer and the paged
block table.  It holds none of the selection or attention arithmetic; both the
HIP path and the CPU oracle consume what it produces.

Recipe (the paper's datasets and model weights are not available, so these
inputs stand in for them):

* Q, K, V are N(0, 1).  Decode queries of one head follow an AR(1) process
  across steps, q_{j+1} = 0.9 q_j + sqrt(0.19) e_j.
* Per (batch, kv-head) let qbar be the mean query over the group's heads and
  the decode steps, u = qbar / |qbar|.  "Heavy" keys get c * u added with
  c = boost * sqrt(d) / |qbar|, which raises their logit under the mean query
  by ``boost`` (3, plus an Exp(1) tail for the long-context workload).
* A distance bias adds b_i * u to key i so that its mean-query logit rises by
  2 i / (n_tot - 1): attention scores fall roughly linearly with distance
  from the current token (exponential-recency appendix of the paper).
* Adjacent layers can be correlated: X^l = c X^{l-1} + sqrt(1 - c^2) Z, for
  keys and for the queries of step 0; heavy positions are shared by layers.
* Every element is finally rounded to the grid j/16 with |j| <= 255.  Such
  values are exact in bf16 and fp32 and every partial sum of a dot product of
  length <= 128 is an integer multiple of 2^-8 below 2^16, so it is exact in
  fp32 in any summation order: GPU and CPU scores agree bit for bit.
"""

from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import numpy as np
import torch

GRID = 16.0
GRID_MAX = 255


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str               # "f32" or "bf16"
    layers: int
    batch: int
    hq: int
    hkv: int
    d: int
    n_ctx: tuple             # cached context per sequence before decode step 0
    steps: int               # decode steps T; step j attends n_ctx + j + 1 keys
    k: int                   # fixed middle budget (unused when k_den > 0)
    window: int
    sink: int
    s: int                   # refresh period in steps
    G: int                   # layer-group size
    r: int = 1
    dilate_m: int = -1       # -1: floor(k / 3)
    k_num: int = 0           # proportional budget k_b = floor(k_num * n0 / k_den)
    k_den: int = 0
    paged: bool = False
    page_size: int = 16
    heavy: int = 8           # heavy positions per (batch, kv-head)
    heavy_tail: bool = False  # add an Exp(1) boost tail
    layer_corr: float = 0.0
    seed: int = 1234

    @property
    def g(self):
        return self.hq // self.hkv

    @property
    def capacity(self):
        """Tokens per (batch, kv-head) the cache must hold."""
        return max(self.n_ctx) + self.steps

    def replace(self, **kw):
        return dataclasses.replace(self, **kw)


def _seq_lengths(seed, batch, nmax):
    rng = np.random.default_rng(np.random.SeedSequence(seed + 7))
    lo = (nmax + 1) // 2
    return tuple(int(x) for x in rng.integers(lo, nmax - 16 + 1, size=batch))


def workload(index, batch=None, nmax=None, block=None):
    """The paper-shaped workloads.

    0 tiny fp32 MHA; 1 LLaMA-2-7B-shaped MHA at 4k; 2 Mistral-7B-shaped GQA at
    32k; 3 LLaMA-3-8B-shaped GQA at 128k on a paged cache; 4 GQA throughput
    sweep with mixed sequence lengths (batch in {16, 64}, nmax in {8k, 16k});
    5 the operator benchmark of the efficiency evaluation (Sec. 5.4):
    LLaMA-2-7B-shaped MHA, batch in {8, 16}, context in {1k, 2k, 4k}, token
    budget 1/8 of the context with C_sink 16 and C_local 64 (the budget split
    of Sec. 5.3), CIS blocks of `block` in {8, 16} steps, no layer sharing.
    """
    if index == 0:
        return Workload("tiny-mha-f32-1k", "f32", 1, 1, 4, 4, 64, (1024,), 16,
                        k=64, window=32, sink=4, s=4, G=1, heavy=8, seed=1234)
    if index == 1:
        return Workload("llama2-7b-mha-4k", "bf16", 32, 8, 32, 32, 128, (4096,) * 8, 16,
                        k=256, window=64, sink=4, s=4, G=4, heavy=8, layer_corr=0.8,
                        seed=1235)
    if index == 2:
        return Workload("mistral-7b-gqa-32k", "bf16", 32, 4, 32, 8, 128, (32768,) * 4, 16,
                        k=1024, window=128, sink=4, s=8, G=4, heavy=8, layer_corr=0.8,
                        seed=1236)
    if index == 3:
        return Workload("llama3-8b-gqa-128k-paged", "bf16", 32, 1, 32, 8, 128, (131072,), 16,
                        k=2048, window=256, sink=4, s=8, G=1, paged=True, page_size=16,
                        heavy=round(0.005 * 131072), heavy_tail=True, seed=1237)
    if index == 4:
        batch = 16 if batch is None else batch
        nmax = 16384 if nmax is None else nmax
        return Workload(f"gqa-sweep-b{batch}-n{nmax}", "bf16", 32, batch, 32, 8, 128,
                        _seq_lengths(1238 + batch + nmax, batch, nmax), 16,
                        k=0, k_num=1, k_den=20, window=128, sink=4, s=4, G=1, heavy=8,
                        seed=1238)
    if index == 5:
        batch = 16 if batch is None else batch
        nmax = 2048 if nmax is None else nmax
        block = 16 if block is None else block
        return Workload(f"paper-op-b{batch}-n{nmax}-s{block}", "bf16", 32, batch, 32, 32, 128,
                        (nmax,) * batch, 16, k=max(0, nmax // 8 - 80), window=64, sink=16,
                        s=block, G=1, heavy=8, layer_corr=0.8, seed=1239 + batch + nmax + block)
    raise ValueError(f"no workload {index}")


def _round_grid(x):
    return torch.clamp(torch.round(x * GRID), -GRID_MAX, GRID_MAX) / GRID


@dataclass
class Inputs:
    """Generated inputs.  Tensors live on the requested device.

    q      [layers][steps][B][Hq][d]
    K, V   per layer: contiguous [B][Hkv][cap][d] or paged [P][Hkv][ps][d]
    block_table [B][max_pages] int32 (paged only)
    n_ctx  [B] int
    """
    w: Workload
    q: torch.Tensor
    K: list
    V: list
    block_table: torch.Tensor = None
    n_ctx: tuple = ()
    num_pages: int = 0
    heavy_pos: torch.Tensor = None
    meta: dict = field(default_factory=dict)

    def seq_lens(self, step):
        return [n + step + 1 for n in self.n_ctx]


def generate(w: Workload, device="cpu", layers=None, torch_dtype=None):
    """Draw a workload's inputs on ``device`` (seeded; deterministic per
    device type).  ``layers`` limits how many layers are materialised."""
    L = w.layers if layers is None else layers
    dt = torch_dtype or (torch.float32 if w.dtype == "f32" else torch.bfloat16)
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    B, Hq, Hkv, d, T, g = w.batch, w.hq, w.hkv, w.d, w.steps, w.g
    cap = w.capacity
    n_tot = [n + T for n in w.n_ctx]

    def randn(*shape):
        return torch.randn(*shape, generator=gen, device=dev, dtype=torch.float32)

    c_l = w.layer_corr
    s_l = math.sqrt(max(0.0, 1.0 - c_l * c_l))

    # queries: layer-correlated start, AR(1) across steps
    q = torch.empty(L, T, B, Hq, d, device=dev, dtype=torch.float32)
    q0 = randn(B, Hq, d)
    for l in range(L):
        if l > 0:
            q0 = c_l * q0 + s_l * randn(B, Hq, d) if c_l > 0 else randn(B, Hq, d)
        qj = q0
        for j in range(T):
            if j > 0:
                qj = 0.9 * qj + math.sqrt(0.19) * randn(B, Hq, d)
            q[l, j] = qj

    # heavy positions per (b, kv-head), shared by every layer, in the middle range
    H = max(1, w.heavy)
    heavy_pos = torch.zeros(B, Hkv, H, dtype=torch.int64, device=dev)
    heavy_boost = torch.full((B, Hkv, H), 3.0, device=dev)
    for b in range(B):
        lo = w.sink
        hi = max(lo + 1, w.n_ctx[b] - w.window)
        heavy_pos[b] = torch.randint(lo, hi, (Hkv, H), generator=gen, device=dev)
    if w.heavy_tail:
        u = torch.rand(B, Hkv, H, generator=gen, device=dev)
        heavy_boost = heavy_boost - torch.log1p(-u.clamp(max=1 - 1e-7))

    # distance bias per position (mean-query logit rises by 2 i / (n_tot - 1))
    pos = torch.arange(cap, device=dev, dtype=torch.float32)
    dist = torch.zeros(B, cap, device=dev)
    valid = torch.zeros(B, cap, device=dev)
    for b in range(B):
        dist[b, : n_tot[b]] = 2.0 * pos[: n_tot[b]] / max(1, n_tot[b] - 1)
        valid[b, : n_tot[b]] = 1.0

    Ks, Vs = [], []
    kbase = None
    for l in range(L):
        z = randn(B, Hkv, cap, d)
        if kbase is None or c_l == 0:
            kbase = z
        else:
            kbase = c_l * kbase + s_l * z
        qbar = q[l].reshape(T, B, Hkv, g, d).mean(dim=(0, 3))          # [B][Hkv][d]
        qn = qbar.norm(dim=-1, keepdim=True).clamp_min(1e-6)
        u = qbar / qn
        unit = math.sqrt(d) / qn                                        # [B][Hkv][1]
        Kl = kbase + (dist[:, None, :, None] * unit[:, :, None, :]) * u[:, :, None, :]
        add = torch.zeros(B, Hkv, cap, device=dev)
        add.scatter_add_(2, heavy_pos, heavy_boost)
        Kl = Kl + (add[..., None] * unit[:, :, None, :]) * u[:, :, None, :]
        Vl = randn(B, Hkv, cap, d)
        mask = valid[:, None, :, None]
        Ks.append((_round_grid(Kl) * mask).to(dt))
        Vs.append((_round_grid(Vl) * mask).to(dt))
    qg = _round_grid(q).to(dt)

    inp = Inputs(w, qg, Ks, Vs, n_ctx=tuple(w.n_ctx), heavy_pos=heavy_pos)
    if w.paged:
        _to_paged(inp, gen, dev)
    return inp


def _to_paged(inp, gen, dev):
    """Scatter the contiguous caches into fixed-size pages whose physical
    order is a seeded random permutation; fills the block table."""
    w = inp.w
    ps = w.page_size
    B, Hkv, d = w.batch, w.hkv, w.d
    cap = w.capacity
    max_pages = (cap + ps - 1) // ps
    P = B * max_pages
    perm = torch.randperm(P, generator=gen, device=dev)
    table = perm.reshape(B, max_pages).to(torch.int32)
    pad = max_pages * ps - cap
    newK, newV = [], []
    for Kc, Vc in zip(inp.K, inp.V):
        out = []
        for X in (Kc, Vc):
            Xp = torch.nn.functional.pad(X, (0, 0, 0, pad)) if pad else X
            Xp = Xp.reshape(B, Hkv, max_pages, ps, d).permute(0, 2, 1, 3, 4)
            Xp = Xp.reshape(P, Hkv, ps, d)
            phys = torch.empty((P, Hkv, ps, d), dtype=Xp.dtype, device=Xp.device)
            phys[table.reshape(-1).long()] = Xp
            out.append(phys)
        newK.append(out[0])
        newV.append(out[1])
    inp.K, inp.V = newK, newV
    inp.block_table = table
    inp.num_pages = P


def gather_unit(inp, layer, b, h_kv, n):
    """The first n cached (K, V) rows of one (batch, kv-head) unit as float64
    NumPy arrays, resolved through the block table for paged caches."""
    w = inp.w
    if w.paged:
        ps = w.page_size
        pages = (n + ps - 1) // ps
        tab = inp.block_table[b, :pages].long()
        K = inp.K[layer][tab, h_kv].reshape(-1, w.d)[:n]
        V = inp.V[layer][tab, h_kv].reshape(-1, w.d)[:n]
    else:
        K = inp.K[layer][b, h_kv, :n]
        V = inp.V[layer][b, h_kv, :n]
    return (K.float().cpu().numpy().astype(np.float64),
            V.float().cpu().numpy().astype(np.float64))


def query_group(inp, layer, step, b, h_kv):
    """The g query heads of kv-head h_kv as a float64 [g, d] array."""
    g = inp.w.g
    qg = inp.q[layer, step, b, h_kv * g:(h_kv + 1) * g]
    return qg.float().cpu().numpy().astype(np.float64)


def random_inputs(batch, hq, hkv, d, lens, dtype="bf16", paged=False, page_size=16, seed=0,
                  grid=True, layers=1, steps=1, key_scale=1.0, device="cpu", spare_pages=3):
    """Unstructured seeded cache for parity tests: N(0, key_scale^2) keys,
    N(0, 1) values and queries, optionally rounded to the j/16 grid.  Sequence
    b holds lens[b] valid tokens at step 0 (step j holds lens[b] + j); every
    cache row beyond the valid tokens, and every unused page, is NaN so that a
    read past the end shows up in the results."""
    lens = tuple(int(x) for x in lens)
    w = Workload(f"random-{seed}", dtype, layers, batch, hq, hkv, d,
                 tuple(n - 1 for n in lens), steps, k=0, window=0, sink=0, s=1, G=1,
                 paged=paged, page_size=page_size, seed=seed)
    dt = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    cap = max(max(lens) + steps - 1, 1)

    def draw(*shape, scale=1.0):
        x = torch.randn(*shape, generator=gen) * scale
        return _round_grid(x) if grid else x

    q = draw(layers, steps, batch, hq, d).to(dt)
    valid = torch.zeros(batch, 1, cap, 1, dtype=torch.bool)
    for b, n in enumerate(lens):
        valid[b, :, : n + steps - 1] = True
    Ks, Vs = [], []
    for _ in range(layers):
        K = draw(batch, hkv, cap, d, scale=key_scale)
        V = draw(batch, hkv, cap, d)
        nan = torch.tensor(float("nan"))
        Ks.append(torch.where(valid, K, nan).to(dt))
        Vs.append(torch.where(valid, V, nan).to(dt))
    inp = Inputs(w.replace(n_ctx=tuple(n - 1 for n in lens)), q, Ks, Vs, n_ctx=tuple(n - 1 for n in lens))
    if paged:
        ps = page_size
        max_pages = (cap + ps - 1) // ps
        P = batch * max_pages + spare_pages
        perm = torch.randperm(P, generator=gen)
        table = perm[: batch * max_pages].reshape(batch, max_pages).to(torch.int32)
        pad = max_pages * ps - cap
        newK, newV = [], []
        for Kc, Vc in zip(inp.K, inp.V):
            out = []
            for X in (Kc, Vc):
                Xp = torch.nn.functional.pad(X.float(), (0, 0, 0, pad), value=float("nan")) if pad else X.float()
                Xp = Xp.reshape(batch, hkv, max_pages, ps, d).permute(0, 2, 1, 3, 4).reshape(-1, hkv, ps, d)
                phys = torch.full((P, hkv, ps, d), float("nan"))
                phys[table.reshape(-1).long()] = Xp
                out.append(phys.to(dt))
            newK.append(out[0])
            newV.append(out[1])
        inp.K, inp.V = newK, newV
        inp.block_table = table
        inp.num_pages = P
    if device != "cpu":
        inp.q = inp.q.to(device)
        inp.K = [x.to(device) for x in inp.K]
        inp.V = [x.to(device) for x in inp.V]
        if inp.block_table is not None:
            inp.block_table = inp.block_table.to(device)
    return inp
