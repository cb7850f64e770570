#!/usr/bin/env python3
"""Decode-step benchmark of the PrHS hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1]

A step is one decode step of the whole hot path over every layer of the
workload: refresh selection (score, top-k, anchor set) where the schedule asks
for it, the dilated shared set of every layer group (built once per refresh;
later steps attend it plus the tokens decoded since), and sparse decode
attention of every layer.  Inputs are seeded synthetic tensors already
resident in HBM.  The same steps are timed with dense decode attention for the
speedup.  Prints one JSON line on stdout; progress goes to stderr.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

METRIC = ("sparse decode-attn µs/layer-step + effective HBM GB/s (% peak); "
          "speedup vs dense")
HBM_PEAK_GBPS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def attention_bytes(w, rows):
    """Algorithmic bytes of one sparse attention launch over `rows` gathered
    (batch, kv-head) rows in total: K and V rows plus their indices, the
    queries, and the outputs y and lse."""
    e = 4 if w.dtype == "f32" else 2
    return rows * (2 * w.d * e + 4) + w.batch * w.hq * w.d * e + w.batch * w.hq * (w.d + 1) * 4


def dense_bytes(w, lens):
    """Algorithmic bytes of one dense attention launch over sequences of the
    given lengths: every cached K and V row once, the queries, y and lse."""
    e = 4 if w.dtype == "f32" else 2
    return (2 * w.hkv * w.d * e * int(sum(lens)) + w.batch * w.hq * w.d * e
            + w.batch * w.hq * (w.d + 1) * 4)


def torch_sum_gbps():
    """A library read stream for reference: torch's sum over a 4 GiB fp32
    tensor, 5 timed passes after one warm-up.  (The dense attention kernel,
    which reads every cached K and V row once, is the faster stream; its rate
    is reported as dense_gbps.)"""
    import torch
    x = torch.ones(1 << 30, dtype=torch.float32, device="cuda")
    x.sum()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        x.sum()
    e1.record()
    torch.cuda.synchronize()
    gbps = 5 * x.numel() * 4 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del x
    return round(gbps, 1)


def middle_len(w, n0):
    se = min(w.sink, n0)
    return max(se, n0 - w.window) - se


def record_step(run, j, gated):
    """Runs the selection of decode step j (untimed) and returns the set rows
    each layer attends and the step's algorithmic selection bytes: middle
    keys read by the refreshing rows (d e each), their queries, the top-k,
    critical-set and shared-set entries written; for the gate, the queries it
    reads and records; for a separate shared-set build, top-k read and set
    written."""
    import torch
    w = run.w
    e = 4 if w.dtype == "f32" else 2
    qbytes = w.batch * w.hq * w.d * e
    run.selection_step(j)
    torch.cuda.synchronize()
    sel = 0
    lens_j = [w.n_ctx[b] + j + 1 for b in range(w.batch)]
    if gated:
        slot = j % w.s
        choice = run.choice.view(run.groups, w.batch, w.hkv).cpu()
        retr = choice < 0
        mid = sum(middle_len(w, lens_j[b]) * int(retr[:, b].sum()) for b in range(w.batch))
        written = 0
        for gi in range(run.groups):
            r = retr[gi].to(run.topk_len.device)
            written += int(run.topk_len[gi][r].sum() + run.pool_len[gi, 0, slot][r].sum()
                           + run.pool_len[gi, 1, slot][r].sum())
        sel += run.groups * qbytes * (2 + slot) + mid * w.d * e + written * 4
        if bool(retr.any()):
            sel += run.groups * qbytes
    else:
        if j % w.s == 0:
            mid = sum(middle_len(w, n0) for n0 in lens_j) * w.hkv * run.groups
            written = int(run.topk_len.sum() + run.anchor_len.sum())
            if run.reuses and not run.per_step_sets:
                written += int(run.shared_len.sum())
            sel += mid * w.d * e + run.groups * qbytes + written * 4
        for gi in run.shares_at(j):
            sel += int(run.shared_len[gi].sum() + run.topk_len[gi].sum()) * 4
    rows = {}
    seq = run.seq_lens[j].view(w.batch, 1).expand(w.batch, w.hkv).reshape(-1)
    for l in range(run.L):
        if gated:
            pool, plen, urow, utail = run.set_for(l, j)
            pool = pool.reshape(-1, pool.shape[-1])[urow.long()]
            plen = plen.reshape(-1)[urow.long()]
        else:
            pool, plen, tail = run.set_for(l, j)
            pool, plen = pool.reshape(-1, pool.shape[-1]), plen.reshape(-1)
            utail = seq if tail is None else tail.repeat_interleave(w.hkv)
        start = run.psaw_start(l, j)
        if start is not None:
            start = torch.tensor(start, dtype=torch.int32, device=pool.device)
        if start is None:
            rows[l] = int((plen + (seq - utail)).sum())
        else:
            # rows the PSAW mask leaves: set entries and tail positions outside
            # [sink, start)
            lo = w.sink
            hi = start.repeat_interleave(w.hkv).view(-1, 1)
            col = torch.arange(pool.shape[-1], device=pool.device).view(1, -1)
            inset = (col < plen.view(-1, 1)) & (pool < utail.view(-1, 1))
            vis = inset & ((pool < lo) | (pool >= hi))
            t0 = utail.view(-1)
            tail_vis = (seq - torch.maximum(t0, torch.maximum(hi.view(-1), torch.full_like(t0, lo)))
                        ).clamp(min=0) + (torch.minimum(seq, torch.full_like(t0, lo)) - t0).clamp(min=0)
            rows[l] = int(vis.sum() + tail_vis.sum())
        run.attend(l, j)
    return rows, sel


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def allowed_cores():
    """Cores this process may use: its affinity set, capped by
    OMP_NUM_THREADS when that is set (the host's CPU share)."""
    n = len(os.sched_getaffinity(0))
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    return max(1, n)


def _oracle_units(spec, units):
    """Runs the oracle's decode schedule for the given units over one layer
    group: units is [(K, V, qs)] with K[l], V[l] float64 caches per layer of
    the group and qs[(l, j)] the unit's query group; returns nothing (the
    results are discarded, only the time counts)."""
    import oracle as O
    layers, steps, n_ctx_of, gated = spec["layers"], spec["steps"], spec["n_ctx"], spec["tau"]
    for b, K, V, qs in units:
        if gated is not None:
            dec = O.GatedDecodeOracle(spec["sink"], spec["window"], spec["s"], spec["G"], gated,
                                      r=spec["r"], k=spec["k"], k_num=spec["k_num"],
                                      k_den=spec["k_den"], dilate_m=spec["dilate_m"])
        else:
            dec = O.DecodeOracle(spec["sink"], spec["window"], spec["s"], spec["G"], r=spec["r"],
                                 k=spec["k"], k_num=spec["k_num"], k_den=spec["k_den"],
                                 dilate_m=spec["dilate_m"])
        for j in range(steps):
            n = n_ctx_of[b] + j + 1
            for l in layers:
                Qg = qs[(l, j)]
                S = dec.step_set(l, j, Qg, K[l], n)
                dec.attend(Qg, K[l][:n], V[l][:n], S)


def _cpu_worker(conn):
    """All-cores leg: receives its units' caches (float32, converted to
    float64 before the clock starts), waits for the start signal, runs the
    oracle on one core and reports its time; repeated per layer group."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1):
        while True:
            msg = conn.recv()
            if msg is None:
                break
            spec, raw = msg
            units = [(b, {l: np.asarray(k, dtype=np.float64) for l, k in K.items()},
                      {l: np.asarray(v, dtype=np.float64) for l, v in V.items()},
                      {key: np.asarray(q, dtype=np.float64) for key, q in qs.items()})
                     for b, K, V, qs in raw]
            del raw
            conn.send("ready")
            conn.recv()
            t0 = time.perf_counter()
            _oracle_units(spec, units)
            conn.send(time.perf_counter() - t0)


def cpu_baseline(run, budget_s):
    """Times the CPU oracle on a bounded sample of the same workload, read
    back from the device: whole layer groups (every (batch, kv-head) unit,
    every decode step of the cycle, in schedule order), group after group
    until about budget_s of one core's time is spent.  Two legs over the same
    sample: one core, and every allowed core (one spawned worker process per
    core, the units dealt round-robin; the clock runs from the start signal
    to the last worker's result, after every worker holds its caches).  Only
    oracle work is timed; scaled per layer-step."""
    import multiprocessing as mp

    import numpy as np
    from threadpoolctl import threadpool_limits

    from paper_2602_08329_amd import synth

    w = run.w
    inp = run.inp
    units = [(b, g) for b in range(w.batch) for g in range(w.hkv)]
    cores = allowed_cores()
    ctx = mp.get_context("spawn")
    pipes, procs = [], []
    for _ in range(cores if cores > 1 else 0):
        parent, child = ctx.Pipe()
        p = ctx.Process(target=_cpu_worker, args=(child,), daemon=True)
        p.start()
        pipes.append(parent)
        procs.append(p)
    spent1 = spent_all = 0.0
    layer_steps = 0
    try:
        for g0 in range(0, run.L, w.G):
            layers = list(range(g0, min(g0 + w.G, run.L)))
            spec = dict(layers=layers, steps=w.steps, n_ctx=list(w.n_ctx), sink=w.sink,
                        window=w.window, s=w.s, G=w.G, r=w.r, k=w.k, k_num=w.k_num, k_den=w.k_den,
                        dilate_m=w.dilate_m, tau=getattr(run, "tau", None))
            qh = {l: inp.q[l].float().cpu().numpy().astype(np.float64) for l in layers}
            data = []
            for (b, g) in units:
                K, V = {}, {}
                for l in layers:
                    K[l], V[l] = synth.gather_unit(inp, l, b, g, w.n_ctx[b] + w.steps)
                qs = {(l, j): qh[l][j, b, g * w.g:(g + 1) * w.g] for l in layers
                      for j in range(w.steps)}
                data.append((b, K, V, qs))
            with threadpool_limits(limits=1):
                t0 = time.perf_counter()
                _oracle_units(spec, data)
                spent1 += time.perf_counter() - t0
            if pipes:
                for i, conn in enumerate(pipes):
                    mine = [(b, {l: x.astype(np.float32) for l, x in K.items()},
                             {l: x.astype(np.float32) for l, x in V.items()},
                             {key: q.astype(np.float32) for key, q in qs.items()})
                            for (b, K, V, qs) in data[i::len(pipes)]]
                    conn.send((spec, mine))
                    del mine
                for conn in pipes:
                    assert conn.recv() == "ready"
                t0 = time.perf_counter()
                for conn in pipes:
                    conn.send("go")
                for conn in pipes:
                    conn.recv()
                spent_all += time.perf_counter() - t0
            layer_steps += len(layers) * w.steps
            del data
            if spent1 >= budget_s:
                break
    finally:
        for conn in pipes:
            try:
                conn.send(None)
            except (BrokenPipeError, OSError):
                pass
        for p in procs:
            p.join(timeout=30)
    us1 = spent1 / layer_steps * 1e6
    sample = (f"{layer_steps // w.steps} of {run.L} layers x {w.steps} decode steps x all "
              f"{len(units)} (batch, kv-head) units, per layer-step; {spent1:.1f} s on one core")
    legs = [{"cores": 1, "value": round(us1, 1)}]
    best = {"value": round(us1, 1), "cores": 1}
    if pipes:
        usn = spent_all / layer_steps * 1e6
        legs.append({"cores": cores, "value": round(usn, 1)})
        best = {"value": round(usn, 1), "cores": cores}
        sample += f", {spent_all:.1f} s on {cores} cores"
    return {"value": best["value"], "unit": "us/layer-step", "cores": best["cores"],
            "kind": "oracle", "sample": sample, "legs": legs, "cpu": cpu_model(),
            "allowed_cores": len(os.sched_getaffinity(0))}


ROOT = os.path.dirname(os.path.abspath(__file__))


def committed_traffic(profile, source):
    """HBM bytes per launch of a kernel measured with rocprofv3 counters
    (FETCH_SIZE and WRITE_SIZE, scaled by a plain-copy calibration) and
    recorded in profiles/<profile>; None when there is no record or the
    kernel's source file (csrc/<source>) changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", profile)
    src = os.path.join(ROOT, "paper_2602_08329_amd", "csrc", source)
    if not os.path.exists(path) or not os.path.exists(src):
        return None
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    fields = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get(f"{source} sha256") != digest:
        return None
    try:
        return int(fields["traffic bytes per launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration():
    """A plain device-to-device copy of 1 GiB, repeated 5 times: the kernel of
    known size against which FETCH_SIZE and WRITE_SIZE are scaled."""
    import torch
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 5
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "ms": round(ms, 4),
                      "gbps": round(2 * n / ms / 1e6, 1)}), flush=True)


PREFILL_METRIC = ("prefill attention µs/layer + TFLOP/s (% of bf16 MFMA peak); "
                  "PSAW speedup vs causal")
MFMA_BF16_PEAK_TFLOPS = 2500.0


def prefill_main(args):
    """Prefill attention of every layer of a LLaMA-2-7B-shaped model (32
    layers, 32 heads, d 128) over seeded synthetic prompts: the layers from
    l_s on under the PSAW mask (Sec. 5.1 defaults, C_sink 16), the others
    causal; timed against all layers causal.  A step is one pass over the 32
    layers.  Flops counted are the useful ones: 4 d per (query, visible key)
    pair per head (q.k and p.v)."""
    import numpy as np
    import torch

    from paper_2602_08329_amd import binding as B
    from paper_2602_08329_amd.schedule import capture_steps, psaw_defaults, psaw_layers

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    B.lib()
    dev = torch.device("cuda:0")
    L, H, d, sink = 32, 32, 128, 16
    Bsz = args.batch or 1
    T = args.nmax or 4096
    K_steps, W_steps = args.steps, args.warmup
    l_s, phi, alpha = psaw_defaults(L)
    gen = torch.Generator(device=dev)
    gen.manual_seed(4242 + T)
    log(f"prefill: {L} layers, batch {Bsz}, {H} heads, d {d}, prompt {T}")
    qs = [torch.randn(Bsz, H, T, d, generator=gen, device=dev).to(torch.bfloat16) for _ in range(L)]
    Ks = [torch.randn(Bsz, H, T, d, generator=gen, device=dev).to(torch.bfloat16) for _ in range(L)]
    Vs = [torch.randn(Bsz, H, T, d, generator=gen, device=dev).to(torch.bfloat16) for _ in range(L)]
    seq = torch.full((Bsz,), T, dtype=torch.int32, device=dev)
    if args.paged:
        # 16-token pages of every prompt in one pool, in a seeded random order
        ps = 16
        npg = (T + ps - 1) // ps
        pgen = torch.Generator(device="cpu")
        pgen.manual_seed(4243 + T)
        perm = torch.randperm(Bsz * npg, generator=pgen).to(dev)
        table = perm.view(Bsz, npg).to(torch.int32)

        def paged(X):
            Xp = torch.zeros(Bsz, H, npg * ps, d, dtype=X.dtype, device=dev)
            Xp[:, :, :T] = X
            pages = Xp.view(Bsz, H, npg, ps, d).permute(0, 2, 1, 3, 4).reshape(Bsz * npg, H, ps, d)
            pool = torch.empty(pages.shape, dtype=X.dtype, device=dev)
            pool[perm.long()] = pages
            return pool

        kvs = [B.KV(paged(Ks[l]), paged(Vs[l]), seq, T, H, table) for l in range(L)]
    else:
        kvs = [B.KV(Ks[l], Vs[l], seq, T, H) for l in range(L)]
    ps = psaw_layers(L, sink, (l_s, phi, alpha))
    # first visible position of every query row of the masking layers, from
    # the library's Eq. psaw (for the useful-flop count and the CPU leg)
    vis = [np.array([B.prhs_psaw_first_visible(ps[l], i + 1) for i in range(T)], dtype=np.int64)
           if l in ps else None for l in range(L)]
    out = torch.empty(Bsz, H, T, d, device=dev)
    lse = torch.empty(Bsz, H, T, device=dev)
    scale = 1.0 / math.sqrt(d)

    def step(psaw):
        for l in range(L):
            B.prhs_prefill_attn(kvs[l], qs[l], scale, out, lse, psaw=ps.get(l) if psaw else None)

    def timed(psaw, label):
        for _ in range(W_steps):
            step(psaw)
        torch.cuda.synchronize()
        graph = None if args.eager else capture_steps(lambda _j: step(psaw), range(K_steps))
        if graph is not None:
            graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        if graph is not None:
            graph.replay()
        else:
            for _ in range(K_steps):
                step(psaw)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        log(f"{label}: {ms / K_steps:.3f} ms/step")
        del graph
        return ms

    workload = f"llama2-7b-prefill-b{Bsz}-{T}" + ("-paged" if args.paged else "")
    ms_psaw = timed(True, "prefill, PSAW on layers > l_s")
    ms_causal = timed(False, "prefill, all layers causal")
    # useful flops: visible (query, key) pairs x 4 d, per head and prompt
    i = np.arange(T, dtype=np.int64)
    pairs_causal = int((i + 1).sum())
    pairs = 0
    for l in range(L):
        if vis[l] is None:
            pairs += pairs_causal
        else:
            v = vis[l]
            se = np.minimum(sink, i + 1)
            pairs += int((se + (i + 1 - np.maximum(v, se))).sum())
    flops = 4.0 * d * H * Bsz * pairs
    flops_causal = 4.0 * d * H * Bsz * pairs_causal * L
    us_layer = ms_psaw * 1e3 / (K_steps * L)
    tflops = flops * K_steps / (ms_psaw * 1e-3) / 1e12
    tflops_causal = flops_causal * K_steps / (ms_causal * 1e-3) / 1e12
    result = {
        "metric": PREFILL_METRIC,
        "value": round(us_layer, 3),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": K_steps,
        "warmup": W_steps,
        "ms_per_step": round(ms_psaw / K_steps, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": workload, "layers": L, "batch": Bsz,
                   "heads": H, "head_dim": d, "prompt": T, "sink": sink,
                   "psaw": {"l_s": l_s, "phi": phi, "alpha": alpha},
                   "launch": "eager" if args.eager else "hip-graph replay"},
        "causal_us_per_layer": round(ms_causal * 1e3 / (K_steps * L), 3),
        "speedup_vs_causal": round(ms_causal / ms_psaw, 3),
        "visible_pair_fraction": round(pairs / (pairs_causal * L), 4),
        "roofline": {"kernel": "attn_prefill_bf16", "bound": "mfma", "achieved": round(tflops, 1),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": committed_traffic(f"attn_prefill_bf16_{workload}.md", "prefill.hip"),
                     "causal_achieved": round(tflops_causal, 1),
                     "note": "useful flops (4 d per visible query-key pair and head) over the "
                             "timed prefill; the kernel issues more (16-column tiles, the "
                             "probabilities' low bf16 part)"},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = prefill_cpu_baseline(qs, Ks, Vs, vis, T, sink, scale, L, H, Bsz,
                                                      args.cpu_seconds)
    print(json.dumps(result), flush=True)


def prefill_cpu_baseline(qs, Ks, Vs, vis, T, sink, scale, L, H, Bsz, budget_s):
    """The oracle's prefill attention for one head of a causal layer and one
    head of the top (pruning) layer, scaled to every head and layer (the
    causal head stands for the layers below l_s, the top-layer head,
    conservatively, for the pruning layers)."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle as O

    rows = T
    times = {}
    with threadpool_limits(limits=1):
        for name, l in (("causal", 0), ("psaw", L - 1)):
            q = qs[l][0, 0].float().cpu().numpy()
            K = Ks[l][0, 0].float().cpu().numpy()
            V = Vs[l][0, 0].float().cpu().numpy()
            v = vis[l]
            # rows sampled evenly until the time budget is half spent
            step = max(1, T // 256)
            t0 = time.perf_counter()
            done = 0
            for i in range(T - 1, -1, -step):
                S = O.prefill_visible_set(i, sink, None if v is None else int(v[i]))
                O.sparse_attention(q[i], K[: i + 1], V[: i + 1], S, scale)
                done += 1
                if time.perf_counter() - t0 > budget_s / 2:
                    break
            dt = time.perf_counter() - t0
            times[name] = dt / done * rows   # per head, all rows
    n_psaw = sum(1 for x in vis if x is not None)
    per_step = (times["causal"] * (L - n_psaw) + times["psaw"] * n_psaw) * H * Bsz
    return {"value": round(per_step * 1e6 / L, 1), "unit": "us/layer", "cores": 1,
            "kind": "oracle", "cpu": cpu_model(),
            "sample": f"every {max(1, T // 256)}-th query row (from the last) of head 0 of layer 0 "
                      f"(causal) and layer {L - 1} (PSAW), scaled to {H} heads x {L} layers"}


def selection_kernels(w, cus):
    """The refresh launches the library picks for this workload (the rule of
    its select_path): one fused kernel when the middle range fits LDS, the
    cache is contiguous bf16 and the rows fill more than half the CUs."""
    rows = w.batch * w.hkv
    fits = w.capacity <= 24576
    if fits and w.dtype == "bf16" and not w.paged and 2 * rows > cus:
        return "select_fused", 1
    if fits:
        return "score + select_keyed", 2
    return "score + select_filter + select_finish", 3


def measure(w, args, dev, K_steps, W_steps, psaw=None, gated=False, tau=None):
    """Times one workload's decode loop (sparse step, selection alone,
    attention alone, one refresh of every group alone, dense) as HIP-graph
    replays and returns (numbers, runner)."""
    import torch

    from paper_2602_08329_amd import synth
    from paper_2602_08329_amd.schedule import DecodeRunner, GatedDecodeRunner, capture_steps

    T = w.steps
    log(f"workload {w.name}: generating inputs on the GPU")
    t0 = time.time()
    inp = synth.generate(w, device=dev)
    torch.cuda.synchronize()
    log(f"inputs ready in {time.time() - t0:.1f} s; "
        f"{sum(x.numel() * x.element_size() for x in inp.K + inp.V) / 2**30:.1f} GiB of KV")
    if gated:
        run = GatedDecodeRunner(inp, dev, tau=tau, psaw=psaw, concurrent=args.concurrent)
    else:
        run = DecodeRunner(inp, dev, per_step_sets=args.per_step_sets, psaw=psaw)

    # one untimed pass over all steps: set sizes and selection bytes
    set_lens = {}
    per = {}
    retrieving = 0
    for j in range(T):
        rows, sel = record_step(run, j, gated)
        if gated:
            retrieving += run.retrieving_units()
        for l, r in rows.items():
            set_lens[(l, j)] = r
        per[j] = dict(attn=sum(attention_bytes(w, r) for r in rows.values()), sel=sel)
    torch.cuda.synchronize()

    def timed(fn, label, order=None):
        """Warm-up steps, then the K timed steps: by default the launches of
        the K steps are captured once into a HIP graph, replayed once
        untimed and once timed, so the region holds the same kernels
        back to back without host launch overhead; with --eager they are
        launched one by one from Python.  HIP events on the launch stream."""
        order = order or (lambda i: i % T)
        for i in range(W_steps):
            fn(order(i))
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        js = [order(W_steps + i) for i in range(K_steps)]
        graph = None
        if not args.eager:
            graph = capture_steps(fn, js)
            graph.replay()
        torch.cuda.synchronize()
        ev0.record()
        t = time.perf_counter()
        if graph is not None:
            graph.replay()
        else:
            for j in js:
                fn(j)
        ev1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t
        ms = ev0.elapsed_time(ev1)
        log(f"{label}: {ms / K_steps:.3f} ms/step (wall {wall * 1e3 / K_steps:.3f} ms/step)")
        del graph
        return ms, js

    log(f"timing {K_steps} sparse decode steps after {W_steps} warm-up steps")
    ms_sparse, js = timed(run.step, "sparse (selection + attention)")
    ms_sel, _ = timed(run.selection_step, "selection only")

    # attention alone: the steps of the last refresh block, cycled, over the
    # sets that block's selection produced (its sets and tails are exactly
    # those of the byte accounting); with the gate, whose decisions are per
    # step, the block's last step repeated
    j_blk = ((T - 1) // w.s) * w.s
    if gated:
        for j in range(j_blk, T):
            run.selection_step(j)
        order = lambda i: T - 1  # noqa: E731
    else:
        run.selection_step(j_blk)
        if args.per_step_sets:   # the shared set is then rebuilt per step; keep the last one
            for j in range(j_blk + 1, T):
                run.selection_step(j)
        order = lambda i: j_blk + i % (T - j_blk)  # noqa: E731

    def attn_only(j):
        for l in range(run.L):
            run.attend(l, j)
    ms_attn, js_attn = timed(attn_only, "attention only", order=order)

    # one refresh of every layer group at the refresh step j_blk, repeated:
    # the selection launches alone, back to back
    refresh = None
    if not gated:
        def refresh_only(_j):
            for gi in range(run.groups):
                run.refresh(gi, j_blk)
        ms_ref, _ = timed(refresh_only, "refresh launches only", order=lambda i: j_blk)
        cus = torch.cuda.get_device_properties(dev).multi_processor_count
        name, nk = selection_kernels(w, cus)
        refresh = dict(kernel=name, launches_per_refresh=nk, groups=run.groups,
                       avg_us=ms_ref * 1e3 / (K_steps * run.groups),
                       avg_bytes=per[j_blk]["sel"] / run.groups)
        if args.per_step_sets:
            refresh = None
        else:
            run.selection_step(j_blk)   # restore the block's sets

    ms_dense, js_dense = timed(run.dense_step, "dense attention")
    dense_total = sum(run.L * dense_bytes(w, run.seq_lens[j].tolist()) for j in js_dense)

    launch_bytes = [attention_bytes(w, set_lens[(l, j)]) for j in js_attn for l in range(run.L)]
    avg_bytes = sum(launch_bytes) / len(launch_bytes)
    avg_dur = ms_attn * 1e-3 / (K_steps * run.L)
    L = run.L
    total_bytes = sum(per[j]["attn"] + per[j]["sel"] for j in js)
    eff_gbps = total_bytes / (ms_sparse * 1e-3) / 1e9
    num = dict(
        workload=w.name, ms_sparse=ms_sparse, us_layer_step=ms_sparse * 1e3 / (K_steps * L),
        eff_gbps=eff_gbps, speedup=ms_dense / ms_sparse,
        dense_us=ms_dense * 1e3 / (K_steps * L),
        dense_gbps=dense_total / (ms_dense * 1e-3) / 1e9,
        sel_us=ms_sel * 1e3 / (K_steps * L), attn_us=ms_attn * 1e3 / (K_steps * L),
        attn_launch=dict(avg_us=avg_dur * 1e6, avg_bytes=avg_bytes, launches=len(launch_bytes)),
        refresh=refresh, retrieving=retrieving, groups=run.groups)
    return num, run


def roofline_of(w, num, copy_traffic=True):
    """Roofline of the dominant kernel: the refresh launch when the
    selection takes more of the step than attention and the refresh is one
    kernel, else the sparse attention launch.  achieved = its algorithmic
    bytes per launch / its average launch duration (HIP events over a loop
    of only those launches)."""
    ref = num["refresh"]
    if ref is not None and num["sel_us"] > num["attn_us"] and ref["launches_per_refresh"] == 1:
        achieved = ref["avg_bytes"] / (ref["avg_us"] * 1e-6) / 1e9
        traffic = committed_traffic(f"{ref['kernel']}_{w.name}_pmc.md", "select.hip")
        return {"kernel": ref["kernel"], "bound": "hbm", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": traffic if copy_traffic else None,
                "avg_launch_us": round(ref["avg_us"], 3), "avg_launch_bytes": int(ref["avg_bytes"]),
                "launches": ref["groups"]}
    a = num["attn_launch"]
    achieved = a["avg_bytes"] / (a["avg_us"] * 1e-6) / 1e9
    kern = "attn_split_bf16" if w.dtype != "f32" else "attn_split_f32"
    traffic = committed_traffic(f"{kern}_{w.name}_pmc.md", "attention.hip")
    return {"kernel": kern + " (sparse)", "bound": "hbm", "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic if copy_traffic else None, "avg_launch_us": round(a["avg_us"], 3),
            "avg_launch_bytes": int(a["avg_bytes"]), "launches": a["launches"]}


def summary_of(w, num):
    """The numbers of one workload as the JSON line reports them."""
    out = {
        "workload": w.name,
        "us_per_layer_step": round(num["us_layer_step"], 3),
        "effective_gbps": round(num["eff_gbps"], 1),
        "pct_hbm_peak": round(100 * num["eff_gbps"] / HBM_PEAK_GBPS, 2),
        "speedup_vs_dense": round(num["speedup"], 3),
        "dense_us_per_layer_step": round(num["dense_us"], 3),
        "dense_gbps": round(num["dense_gbps"], 1),
        "selection_us_per_layer_step": round(num["sel_us"], 3),
        "attention_us_per_layer_step": round(num["attn_us"], 3),
        "attention_launch": {"avg_us": round(num["attn_launch"]["avg_us"], 3),
                             "frac": round(num["attn_launch"]["avg_bytes"]
                                           / (num["attn_launch"]["avg_us"] * 1e-6) / 1e9
                                           / HBM_PEAK_GBPS, 4)},
    }
    if num["refresh"] is not None:
        r = num["refresh"]
        out["refresh_launch"] = {"kernels": r["kernel"], "avg_us": round(r["avg_us"], 3),
                                 "frac": round(r["avg_bytes"] / (r["avg_us"] * 1e-6) / 1e9
                                               / HBM_PEAK_GBPS, 4)}
    return out


HEADLINE = (4, 64, 16384)      # the largest single-GPU workload: GQA sweep, B 64 x nmax 16k
LONG_CONTEXT = (2, 3)          # 32k and 128k (paged) context, the speedup target's range


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", type=int, default=HEADLINE[0], help="workload index 0-5")
    ap.add_argument("--batch", type=int, default=None, help="workloads 4, 5: batch")
    ap.add_argument("--nmax", type=int, default=None, help="workloads 4, 5: max context")
    ap.add_argument("--block", type=int, default=None, help="workload 5: CIS block size s")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-long-context", action="store_true",
                    help="skip the 32k and 128k workloads measured after the headline")
    ap.add_argument("--per-step-sets", action="store_true",
                    help="rebuild the dilated shared set at every step instead of once per refresh")
    ap.add_argument("--psaw", action="store_true",
                    help="progressive sliding attention window on the top layers (Sec. 5.1 "
                         "defaults: l_s = floor(3N/4), phi = 0.7, alpha = 1): CPE with --gate")
    ap.add_argument("--gate", type=float, default=None, metavar="TAU",
                    help="similarity-gated sharing with threshold TAU in [0, 1] instead of the "
                         "fixed refresh period (blocks of refresh_every steps)")
    ap.add_argument("--concurrent", action="store_true",
                    help="with --gate: the sharing units' attention on a second stream beside "
                         "the refresh and the retrieving units' attention")
    ap.add_argument("--eager", action="store_true",
                    help="time eager launches instead of replays of a captured HIP graph")
    ap.add_argument("--paged", action="store_true",
                    help="with --prefill: the prompts' K/V in a paged cache (16-token pages, "
                         "seeded random page order)")
    ap.add_argument("--prefill", action="store_true",
                    help="prefill attention under the PSAW mask instead of the decode step "
                         "(LLaMA-2-7B shape; --nmax prompt length, --batch prompts)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (HBM counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return

    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the hot path has no multi-GPU mode)", file=sys.stderr)
        sys.exit(2)
    if args.prefill:
        prefill_main(args)
        return

    import torch

    from paper_2602_08329_amd import binding as B
    from paper_2602_08329_amd import synth
    from paper_2602_08329_amd.schedule import psaw_defaults

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    B.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    headline = (args.config == HEADLINE[0] and args.batch is None and args.nmax is None)
    batch = HEADLINE[1] if headline else args.batch
    nmax = HEADLINE[2] if headline else args.nmax
    w = synth.workload(args.config, batch=batch, nmax=nmax, block=args.block)
    K_steps, W_steps = args.steps, args.warmup
    gated = args.gate is not None
    if gated and args.per_step_sets:
        print("--gate and --per-step-sets exclude each other", file=sys.stderr)
        sys.exit(2)
    psaw = psaw_defaults(w.layers) if args.psaw else None
    num, run = measure(w, args, dev, K_steps, W_steps, psaw=psaw, gated=gated, tau=args.gate)
    L = run.L
    result = {
        "metric": METRIC,
        "value": round(num["us_layer_step"], 3),
        "unit": "us/layer-step",
        "n_gpus": 1,
        "steps": K_steps,
        "warmup": W_steps,
        "ms_per_step": round(num["ms_sparse"] / K_steps, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name, "layers": w.layers, "batch": w.batch, "q_heads": w.hq,
            "kv_heads": w.hkv, "head_dim": w.d, "context": max(w.n_ctx),
            "context_per_sequence": "uniform in [nmax/2, nmax - 16]" if w.k_den else "fixed",
            "k": w.k if not w.k_den else f"{w.k_num}/{w.k_den} n", "window": w.window,
            "sink": w.sink, "refresh_every": w.s, "layer_group": w.G, "dilate_r": w.r,
            "paged": w.paged, "decode_steps_cycled": w.steps,
            "shared_sets": (("similarity gate, concurrent branches" if args.concurrent else
                             "similarity gate") if gated else
                            "per step" if args.per_step_sets else "per refresh + decoded tail"),
            "psaw": ({"l_s": psaw[0], "phi": psaw[1], "alpha": psaw[2]} if psaw else None),
            "launch": "eager" if args.eager else "hip-graph replay",
        },
        "effective_gbps": round(num["eff_gbps"], 1),
        "pct_hbm_peak": round(100 * num["eff_gbps"] / HBM_PEAK_GBPS, 2),
        "speedup_vs_dense": round(num["speedup"], 3),
        "dense_us_per_layer_step": round(num["dense_us"], 3),
        "dense_gbps": round(num["dense_gbps"], 1),
        "selection_us_per_layer_step": round(num["sel_us"], 3),
        "attention_us_per_layer_step": round(num["attn_us"], 3),
        "roofline": roofline_of(w, num),
    }
    s_ = summary_of(w, num)
    for key in ("attention_launch", "refresh_launch"):
        if key in s_:
            result[key] = s_[key]
    if gated:
        result["gate"] = {"tau": args.gate,
                          "retrieval_ratio": round(num["retrieving"]
                                                   / (num["groups"] * w.batch * w.hkv * w.steps), 4),
                          "note": "retrieving (anchor layer, kv head) units over all of them, "
                                  "measured over the decode-step cycle"}
    if not args.no_cpu_baseline:
        log(f"timing the CPU oracle for about {args.cpu_seconds:.0f} s on one core, then on "
            f"{allowed_cores()} cores")
        result["cpu_baseline"] = cpu_baseline(run, args.cpu_seconds)
    del run
    torch.cuda.empty_cache()
    if headline and not args.no_long_context and not gated and not args.per_step_sets:
        result["long_context"] = []
        for c in LONG_CONTEXT:
            wl = synth.workload(c)
            nl, rl = measure(wl, args, dev, K_steps, W_steps, psaw=psaw)
            result["long_context"].append(summary_of(wl, nl))
            del rl
            torch.cuda.empty_cache()
    result["stream_reference"] = {"torch_sum_gbps": torch_sum_gbps()}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
