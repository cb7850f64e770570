"""HIP-graph replay of whole decode steps.

The launches of a decode cycle (selection, reuse-set construction and
attention of every layer) are captured once into a HIP graph and replayed
several times, with eager work and synchronisations in between; every
replay must reproduce the eager outputs bit for bit.  The benchmark times
such replays, so this pins that the captured launches compute what the
eager ones do (no launch in the path records anything that a replay would
not redo)."""

import pytest
import torch

from paper_2602_08329_amd import binding as B
from paper_2602_08329_amd import synth
from paper_2602_08329_amd.schedule import DecodeRunner, GatedDecodeRunner, capture_steps

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def _cycle(run, steps, bufs):
    for j in steps:
        run.step(j, outs=[bufs[(l, j)] for l in range(run.L)])


def _check_graph(w, runner, replays=3):
    inp = synth.generate(w, device=DEV)
    run = runner(inp)
    steps = list(range(w.steps))
    bufs = {(l, j): (torch.empty(w.batch, w.hq, w.d, device=DEV),
                     torch.empty(w.batch, w.hq, device=DEV))
            for l in range(run.L) for j in steps}

    def poison():
        for o, s in bufs.values():
            o.fill_(float("nan"))
            s.fill_(float("nan"))

    poison()
    _cycle(run, steps, bufs)
    torch.cuda.synchronize()
    ref = {k: (o.clone(), s.clone()) for k, (o, s) in bufs.items()}
    assert all(torch.isfinite(o).all() for o, _ in ref.values())

    g = capture_steps(lambda j: run.step(j, outs=[bufs[(l, j)] for l in range(run.L)]), steps)
    torch.cuda.synchronize()
    spare = (torch.empty(w.batch, w.hq, w.d, device=DEV), torch.empty(w.batch, w.hq, device=DEV))
    for rep in range(replays):
        poison()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, (o, s) in bufs.items():
            assert torch.equal(o, ref[k][0]), f"replay {rep}: output of (layer, step) {k} differs"
            assert torch.equal(s, ref[k][1]), f"replay {rep}: lse of (layer, step) {k} differs"
        # eager work between replays
        run.step(0, outs=[spare] * run.L)
        torch.cuda.synchronize()
    del g


@pytest.mark.parametrize("mode", ["shared", "per_step", "psaw", "gated", "gated_fused",
                                  "gated_concurrent"])
def test_graph_replay_config1_cut(mode):
    # 4 layers in one group of 4, blocks of 4 steps; the gated step runs its
    # sharing units on a second stream inside the graph; with 5 sequences
    # (160 rows) the gate runs inside the fused refresh launch
    w = synth.workload(1).replace(layers=4, batch=2, n_ctx=(2048, 1500), steps=8)
    if mode in ("gated_fused", "gated_concurrent"):
        w = w.replace(batch=5, n_ctx=(2048, 1500, 900, 1700, 1200))
    if mode.startswith("gated"):
        conc = mode == "gated_concurrent"
        runner = lambda inp: GatedDecodeRunner(inp, DEV, tau=0.8, concurrent=conc)  # noqa: E731
    elif mode == "psaw":
        runner = lambda inp: DecodeRunner(inp, DEV, psaw=(2, 0.3, 1.0))  # noqa: E731
    else:
        runner = lambda inp: DecodeRunner(inp, DEV, per_step_sets=mode == "per_step")  # noqa: E731
    _check_graph(w, runner)


def test_graph_replay_config3_cut_paged():
    # multi-launch refresh path (clear, score, filter, finish) on a paged cache
    w = synth.workload(3).replace(layers=2, n_ctx=(40000,), heavy=100, steps=8)
    _check_graph(w, lambda inp: DecodeRunner(inp, DEV))
