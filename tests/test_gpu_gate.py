"""GPU parity of the similarity-gated schedule (Sec. 4.1, Similarity
Criteria) against the oracle: the gate's decisions bit for bit, and the whole
gated decode schedule (sets bit-exact, outputs within tolerance, the same
retrieval counts) on cut-down and full-size paper-shaped workloads.  Queries
lie on the j/16 grid, so the cosine decisions are exact on both sides."""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2602_08329_amd import binding as B
from paper_2602_08329_amd import synth
from paper_2602_08329_amd.schedule import GatedDecodeRunner

pytestmark = pytest.mark.gpu
DEV = "cuda"
TOL = {"bf16": 2e-3, "f32": 1e-5}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def on_grid(x):
    return torch.clamp(torch.round(x * 16), -255, 255) / 16


def gate_queries(S, Bsz, Hq, d, seed, spread):
    """Queries of S block steps: a base direction per head plus growing
    noise, so that similarity decays along the block; on the grid."""
    g = torch.Generator().manual_seed(seed)
    base = torch.randn(Bsz, Hq, d, generator=g)
    qs = []
    for t in range(S):
        qs.append(on_grid(base + spread * t * torch.randn(Bsz, Hq, d, generator=g)))
    return qs


@pytest.mark.parametrize("dtype,hq,hkv,d,tau,spread", [
    ("bf16", 8, 2, 128, 0.8, 0.25),
    ("bf16", 32, 32, 128, 0.9, 0.2),
    ("f32", 4, 4, 64, 0.7, 0.3),
    ("bf16", 16, 1, 128, 0.5, 0.5),
])
def test_gate_decisions_match_oracle(dtype, hq, hkv, d, tau, spread):
    S, Bsz = 6, 3
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    qs = [q.to(tdt) for q in gate_queries(S, Bsz, hq, d, 7 + hq, spread)]
    U = Bsz * hkv
    G = hq // hkv
    ref_q = torch.zeros(S, Bsz, hq, d, dtype=tdt, device=DEV)
    ref_valid = torch.full((S, U), 7, dtype=torch.int32, device=DEV)   # stale garbage
    slot_lens = torch.full((S, Bsz), -1, dtype=torch.int32, device=DEV)
    outs = [torch.full((U,), -9, dtype=torch.int32, device=DEV) for _ in range(4)]
    lens0 = [500, 700, 900]
    anchors = {u: [] for u in range(U)}
    mixed = set()
    for t in range(S):
        lens = torch.tensor([n + t for n in lens0], dtype=torch.int32, device=DEV)
        q = qs[t].to(DEV)
        B.prhs_gate(q, lens, tau, t, ref_q, ref_valid, slot_lens, *outs, hkv)
        torch.cuda.synchronize()
        choice, row_a, row_o, tail = (o.cpu().numpy() for o in outs)
        rv = ref_valid.cpu().numpy()
        sl = slot_lens.cpu().numpy()
        assert np.array_equal(sl[t], [n + t for n in lens0])
        assert torch.equal(ref_q[t].cpu(), qs[t])
        for u in range(U):
            b, g = divmod(u, hkv)
            Qg = qs[t][b, g * G:(g + 1) * G].float().numpy()
            src = None if t == 0 else O.gate_choice(Qg, anchors[u], tau)
            want = -1 if src is None else src
            assert choice[u] == want, f"slot {t} unit {u}: choice {choice[u]} != {want}"
            mixed.add(want)
            assert rv[t, u] == (1 if src is None else 0)
            if src is None:
                anchors[u].append((t, Qg))
                assert row_a[u] == t * U + u and row_o[u] == (S + t) * U + u
                assert tail[u] == lens0[b] + t
            else:
                assert row_a[u] == (S + src) * U + u and row_o[u] == row_a[u]
                assert tail[u] == lens0[b] + src
    assert len(mixed) > 1, "the case should mix sharing and retrieval"


def test_gate_extreme_thresholds():
    S, Bsz, hq, hkv, d = 4, 2, 8, 2, 128
    qs = [q.abs().to(torch.bfloat16) for q in gate_queries(S, Bsz, hq, d, 3, 0.5)]
    U = Bsz * hkv
    for tau, expect in ((1.0, [-1, -1, -1]), (0.0, [0, 0, 0])):
        ref_q = torch.zeros(S, Bsz, hq, d, dtype=torch.bfloat16, device=DEV)
        ref_valid = torch.zeros(S, U, dtype=torch.int32, device=DEV)
        slot_lens = torch.zeros(S, Bsz, dtype=torch.int32, device=DEV)
        outs = [torch.zeros(U, dtype=torch.int32, device=DEV) for _ in range(4)]
        lens = torch.tensor([100, 200], dtype=torch.int32, device=DEV)
        got = []
        for t in range(S):
            B.prhs_gate(qs[t].to(DEV), lens, tau, t, ref_q, ref_valid, slot_lens, *outs, hkv)
            torch.cuda.synchronize()
            got.append(outs[0].cpu().numpy().tolist())
        assert got[0] == [-1] * U
        for t in range(1, S):
            assert got[t] == [expect[t - 1]] * U, (tau, t, got[t])


def run_gated(w, tau, steps, units_out, layers=None, units_set=None, psaw=None):
    inp = synth.generate(w, device=DEV, layers=layers)
    L = len(inp.K)
    run = GatedDecodeRunner(inp, DEV, tau=tau, psaw=psaw)
    units = [(b, g) for b in range(w.batch) for g in range(w.hkv)]
    units_set = units if units_set is None else units_set
    dec = {u: O.GatedDecodeOracle(w.sink, w.window, w.s, w.G, tau, r=w.r, k=w.k, k_num=w.k_num,
                                  k_den=w.k_den, dilate_m=w.dilate_m) for u in units_set}
    # with PSAW the sets are compared before the mask and the outputs after it
    out = torch.empty(w.batch, w.hq, w.d, device=DEV)
    lse = torch.empty(w.batch, w.hq, device=DEV)
    cache = {}
    worst = 0.0
    gpu_retrievals = 0
    for j in steps:
        run.selection_step(j)
        torch.cuda.synchronize()
        gpu_retrievals += int((run.choice.view(run.groups, w.batch, w.hkv).cpu().numpy()[
            :, [b for b, _ in units_set], [g for _, g in units_set]] < 0).sum())
        for l in range(L):
            out.fill_(float("nan"))
            run.attend(l, j, out, lse)
            pool, plen, rows, tail = run.set_for(l, j)
            torch.cuda.synchronize()
            pool_h = pool.reshape(-1, pool.shape[-1]).cpu().numpy()
            plen_h = plen.reshape(-1).cpu().numpy()
            rows_h, tail_h = rows.cpu().numpy(), tail.cpu().numpy()
            y = out.cpu().numpy()
            for (b, g) in units_set:
                u = b * w.hkv + g
                n = w.n_ctx[b] + j + 1
                Qg = synth.query_group(inp, l, j, b, g)
                K_sel = synth.gather_unit(inp, l, b, g, n)[0] if l % w.G == 0 else None
                S = dec[(b, g)].step_set(l, j, Qg, K_sel, n)
                r, t0 = rows_h[u], tail_h[u]
                base = pool_h[r, : plen_h[r]]
                got = np.concatenate([base[base < t0], np.arange(t0, n)])
                assert np.array_equal(got, S), f"l{l} j{j} b{b} g{g}: set differs"
                if psaw is not None:
                    S = O.psaw_restrict(S, O.psaw_visible_start(l, L, n, w.sink, *psaw), w.sink, n)
                if (b, g) in units_out:
                    key = (l, b, g)
                    if key not in cache:
                        cache[key] = synth.gather_unit(inp, l, b, g, w.n_ctx[b] + w.steps)
                    K, V = cache[key]
                    for i in range(w.g):
                        h = g * w.g + i
                        yr, _ = O.sparse_attention(Qg[i], K[:n], V[:n], S)
                        e = np.abs(y[b, h] - yr).max() / max(np.abs(yr).max(), 1e-30)
                        worst = max(worst, e)
                        assert e <= TOL[w.dtype], f"l{l} j{j} b{b} h{h}: rel err {e:.3e}"
    oracle_retrievals = sum(dec[u].retrievals for u in units_set)
    assert gpu_retrievals == oracle_retrievals
    decisions = sum(dec[u].decisions for u in units_set)
    print(f"{w.name} tau {tau}: retrieval ratio {oracle_retrievals / decisions:.3f}, "
          f"worst rel err {worst:.2e}")
    return oracle_retrievals / decisions


def test_gated_schedule_config1_cut():
    w = synth.workload(1).replace(layers=8, batch=2, n_ctx=(2048, 1500))
    ratio = run_gated(w, 0.8, range(w.steps), {(0, 0), (1, 17)},
                      units_set=[(b, g) for b in range(2) for g in (0, 5, 17, 31)])
    assert 1 / w.s <= ratio <= 1


def test_gated_schedule_fused_rows():
    # 5 sequences x 32 kv heads = 160 rows, more than half the CUs: the gated
    # refresh on the single-launch path, non-retrieving rows exiting at once
    w = synth.workload(1).replace(layers=4, batch=5, n_ctx=(1500, 900, 1200, 700, 1100), steps=8)
    ratio = run_gated(w, 0.8, range(w.steps), {(0, 0), (4, 31)},
                      units_set=[(b, g) for b in range(5) for g in (0, 13, 31)])
    assert 1 / w.s <= ratio <= 1


def test_gated_schedule_config0_full():
    w = synth.workload(0)
    run_gated(w, 0.85, range(w.steps), {(0, g) for g in range(w.hkv)})


def test_gated_schedule_config3_cut_paged():
    w = synth.workload(3).replace(layers=2, n_ctx=(20000,), heavy=100)
    run_gated(w, 0.8, range(w.steps), {(0, 0), (0, 7)})


def test_gated_schedule_config4_cut_ragged():
    w = synth.workload(4, batch=4, nmax=4096).replace(layers=2)
    run_gated(w, 0.6, range(w.steps), {(b, 3) for b in range(4)})


def test_gated_schedule_config2_full_size():
    # the full 32k shape on the layers of one group, steps of one block
    w = synth.workload(2)
    run_gated(w, 0.8, range(8), {(0, 0), (3, 7)}, layers=4,
              units_set=[(b, g) for b in range(4) for g in (0, 3, 7)])


def test_gated_schedule_config1_cut_cpe():
    # CPE: the similarity gate with PSAW on the top layers
    w = synth.workload(1).replace(layers=8, batch=2, n_ctx=(2048, 1500))
    run_gated(w, 0.8, range(8), {(0, 0), (1, 17)}, psaw=(6, 0.3, 1.0),
              units_set=[(b, g) for b in range(2) for g in (0, 17)])


def test_pool_attention_row_outside_pool_is_empty():
    lens = (300, 40)
    inp = synth.random_inputs(2, 4, 2, 128, lens, seed=61, device=DEV)
    kv = B.KV(inp.K[0], inp.V[0], torch.tensor(lens, dtype=torch.int32, device=DEV),
              inp.w.capacity, 4)
    # rows of capacity 64 holding 16 sorted entries (room for the tails)
    vals = torch.sort(torch.arange(6 * 16, dtype=torch.int32, device=DEV).view(6, 16) % 37,
                      dim=1).values
    pool = torch.full((6, 64), -5, dtype=torch.int32, device=DEV)
    pool[:, :16] = vals
    plen = torch.full((6,), 16, dtype=torch.int32, device=DEV)
    rows = torch.tensor([2, -1, 6, 5], dtype=torch.int32, device=DEV)
    tail = torch.tensor([300, 300, 40, 30], dtype=torch.int32, device=DEV)
    out = torch.full((2, 4, 128), float("nan"), device=DEV)
    lse = torch.full((2, 4), float("nan"), device=DEV)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv, None, 64), DEV)
    B.prhs_pool_decode_attn(kv, inp.q[0, 0], pool, plen, rows, tail, 0.1, out, lse, ws)
    torch.cuda.synchronize()
    y, ls = out.cpu().numpy(), lse.cpu().numpy()
    # units (0, 1) and (1, 0): row outside the pool, empty tail -> empty set
    assert np.all(y[0, 2:] == 0) and np.all(np.isneginf(ls[0, 2:]))
    assert np.all(y[1, :2] == 0) and np.all(np.isneginf(ls[1, :2]))
    # unit (1, 1): row 5 below position 30, then the tail [30, 40)
    P = vals[5].cpu().numpy()
    S = sorted(set(P[P < 30].tolist()) | set(range(30, 40)))
    K, V = synth.gather_unit(inp, 0, 1, 1, 40)
    Qg = synth.query_group(inp, 0, 0, 1, 1)
    for i in range(2):
        yr, _ = O.sparse_attention(Qg[i], K, V, S, 0.1)
        assert np.abs(y[1, 2 + i] - yr).max() <= 2e-3 * np.abs(yr).max()


@pytest.mark.parametrize("dtype,hq,hkv,tau", [("bf16", 8, 2, 0.8), ("f32", 4, 4, 0.7),
                                               ("bf16", 32, 8, 0.9)])
def test_gate_decisions_off_grid(dtype, hq, hkv, tau):
    # queries off the grid: the gate's fp32 sums are no longer exact, so a
    # decision may differ from the exact one only where some query head's
    # exact cosine lies within 1e-4 of tau (fp32 rounding of d = 128 sums
    # moves a cosine by about 3 gamma_d = 2.3e-5 at most).  The reference
    # follows the gate's own retrievals, so later steps compare like for like.
    S, Bsz, d = 6, 3, 128
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g_ = torch.Generator().manual_seed(5 + hq)
    base = torch.randn(Bsz, hq, d, generator=g_)
    qs = [(base + 0.3 * t * torch.randn(Bsz, hq, d, generator=g_)).to(tdt) for t in range(S)]
    U, G = Bsz * hkv, hq // hkv
    ref_q = torch.zeros(S, Bsz, hq, d, dtype=tdt, device=DEV)
    ref_valid = torch.zeros(S, U, dtype=torch.int32, device=DEV)
    slot_lens = torch.zeros(S, Bsz, dtype=torch.int32, device=DEV)
    outs = [torch.zeros(U, dtype=torch.int32, device=DEV) for _ in range(4)]
    lens = torch.tensor([700, 800, 900], dtype=torch.int32, device=DEV)
    anchors = {u: [] for u in range(U)}

    def cosines(a, b):
        a, b = np.atleast_2d(a), np.atleast_2d(b)
        return (a * b).sum(1) / np.sqrt((a * a).sum(1) * (b * b).sum(1))

    for t in range(S):
        B.prhs_gate(qs[t].to(DEV), lens, tau, t, ref_q, ref_valid, slot_lens, *outs, hkv)
        torch.cuda.synchronize()
        choice = outs[0].cpu().numpy()
        for u in range(U):
            b, g = divmod(u, hkv)
            Qg = qs[t][b, g * G:(g + 1) * G].double().numpy()
            c = int(choice[u])
            if t == 0:
                assert c == -1
            assert c == -1 or any(st == c for st, _ in anchors[u]), f"slot {t} unit {u}: {c}"
            # the gate's choice c implies: slot c similar (c >= 0) and every
            # later anchor not similar (every anchor when c = -1); where the
            # exact decision differs, some head's cosine must sit at tau
            for st, Qr in anchors[u]:
                if c >= 0 and st < c:
                    continue
                if O.group_similar(Qg, Qr, tau) != (st == c):
                    margin = np.abs(cosines(Qg, Qr) - tau).min()
                    assert margin <= 1e-4, f"slot {t} unit {u} anchor {st}: margin {margin:.2e}"
            if c == -1:
                anchors[u].append((t, Qg))


@pytest.mark.parametrize("case", ["fused-rows", "radix-paged", "psaw"])
def test_concurrent_step_equals_sequential(case):
    # GatedDecodeRunner.step runs the sharing units' attention on a second
    # stream beside the gate + refresh + retrieving units' attention: every
    # layer's outputs equal, bit for bit, those of the same work run one
    # launch after another, at every step of two blocks (the gate in the
    # refresh launch on the fused path; a gate launch first otherwise)
    psaw = None
    if case == "fused-rows":
        w = synth.workload(1).replace(layers=4, batch=5, n_ctx=(1500, 900, 1200, 700, 1100), steps=8)
    elif case == "radix-paged":
        w = synth.workload(3).replace(layers=2, n_ctx=(30000,), heavy=100, steps=16)
    else:
        w = synth.workload(1).replace(layers=8, batch=2, n_ctx=(2048, 1500), steps=8)
        psaw = (6, 0.3, 1.0)
    inp = synth.generate(w, device=DEV)
    L = len(inp.K)
    seq = GatedDecodeRunner(inp, DEV, tau=0.8, psaw=psaw)
    con = GatedDecodeRunner(inp, DEV, tau=0.8, psaw=psaw, concurrent=True)
    mk = lambda: [(torch.full((w.batch, w.hq, w.d), float("nan"), device=DEV),  # noqa: E731
                   torch.full((w.batch, w.hq), float("nan"), device=DEV)) for _ in range(L)]
    mixed = False
    for j in range(w.steps):
        a, b = mk(), mk()
        seq.selection_step(j)
        for l in range(L):
            seq.attend(l, j, *a[l])
        con.step(j, b)
        torch.cuda.synchronize()
        c = seq.choice.cpu().numpy()
        assert np.array_equal(c, con.choice.cpu().numpy()), f"step {j}: decisions differ"
        assert np.array_equal(c, con.side_choice.cpu().numpy()), f"step {j}: side decisions differ"
        mixed |= bool((c < 0).any() and (c >= 0).any())
        for l in range(L):
            for x, y in zip(a[l], b[l]):
                xh, yh = x.cpu().numpy(), y.cpu().numpy()
                assert not np.isnan(yh).any(), f"step {j} layer {l}: unit not attended"
                assert np.array_equal(xh, yh), f"step {j} layer {l}: outputs differ"
    assert mixed, "the case should mix sharing and retrieving units"
