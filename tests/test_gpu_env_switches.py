"""The library's tuning switches change how the work is laid out, never what
is computed: the same inputs, each in a fresh process (the switches are read
once per process), under every forced selection path (PRHS_SELECT_PATH) and
several split geometries (PRHS_ATTN_GROUPS, PRHS_ATTN_WAVES) give identical
top-k, anchor and shared sets, attention outputs bit for bit equal wherever
the split geometry is the same, and outputs within tolerance of the oracle
everywhere."""

import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_2602_08329_amd import synth
from tests.env_switch_child import LENS, STEP

pytestmark = pytest.mark.gpu
CHILD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "env_switch_child.py")

VARIANTS = [
    {},
    {"PRHS_SELECT_PATH": "fused"},
    {"PRHS_SELECT_PATH": "keyed"},
    {"PRHS_SELECT_PATH": "split"},
    {"PRHS_SELECT_PATH": "fused", "PRHS_SELECT_BALANCE": "0"},
    {"PRHS_ATTN_GROUPS": "64"},
    {"PRHS_ATTN_GROUPS": "1024"},
    {"PRHS_ATTN_WAVES": "1"},
    {"PRHS_ATTN_WAVES": "8"},
]


def test_switches_change_layout_not_results(tmp_path):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    base = {k: v for k, v in os.environ.items() if not k.startswith("PRHS_")}
    res = []
    for i, var in enumerate(VARIANTS):
        path = str(tmp_path / f"v{i}.npz")
        print(f"variant {var}", flush=True)
        r = subprocess.run([sys.executable, "-u", CHILD, path], env=dict(base, **var),
                           capture_output=True, text=True, timeout=180)
        assert r.returncode == 0, (var, r.stdout[-2000:], r.stderr[-2000:])
        res.append(dict(np.load(path)))
    ref = res[0]
    for var, got in zip(VARIANTS[1:], res[1:]):
        for key in ("tlen", "clen", "hlen"):
            assert np.array_equal(got[key], ref[key]), (var, key)
        for key, lk in (("topk", "tlen"), ("cset", "clen"), ("hset", "hlen")):
            for b in range(4):
                for g in range(8):
                    n = ref[lk][b, g]
                    assert np.array_equal(got[key][b, g, :n], ref[key][b, g, :n]), (var, key, b, g)
        if not any(k.startswith("PRHS_ATTN") for k in var):
            assert np.array_equal(got["out"], ref["out"]) and np.array_equal(got["lse"], ref["lse"])
    # every variant's outputs against the oracle over the shared set plus tail
    inp = synth.random_inputs(4, 32, 8, 128, LENS, seed=321, grid=True, steps=STEP + 1)
    for b in range(4):
        n = LENS[b] + STEP
        for g in (0, 3, 7):
            K, V = synth.gather_unit(inp, 0, b, g, n)
            Qg = synth.query_group(inp, 0, STEP, b, g)
            S = np.concatenate([ref["hset"][b, g, : ref["hlen"][b, g]], np.arange(LENS[b], n)])
            for i in range(4):
                yr, lr = O.sparse_attention(Qg[i], K, V, S)
                for var, got in zip(VARIANTS, res):
                    y = got["out"][b, g * 4 + i]
                    err = np.abs(y - yr).max() / np.abs(yr).max()
                    assert err <= 2e-3, (var, b, g, i, err)
                    assert abs(got["lse"][b, g * 4 + i] - lr) <= 1e-4 * max(1.0, abs(lr))
