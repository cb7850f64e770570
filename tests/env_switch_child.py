"""Child process of test_gpu_env_switches: one refresh (prhs_select_shared)
and one reuse-step attention (prhs_reuse_decode_attn) on fixed seeded inputs,
under whatever PRHS_* tuning switches the environment sets; saves every
output to the .npz file named on the command line."""

import math
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2602_08329_amd import binding as B  # noqa: E402
from paper_2602_08329_amd import synth  # noqa: E402

LENS = (6000, 9000, 3000, 12000)
STEP = 3


def main(path):
    env = {k: v for k, v in os.environ.items() if k.startswith("PRHS_")}
    print(f"[child] switches {env}", flush=True)
    dev = torch.device("cuda:0")
    inp = synth.random_inputs(4, 32, 8, 128, LENS, seed=321, grid=True, steps=STEP + 1,
                              device=dev)
    p = B.params(k=300, sink=4, window=32, dilate_r=1, refresh_every=4)
    cap = inp.w.capacity
    n0 = torch.tensor(LENS, dtype=torch.int32, device=dev)
    kv0 = B.KV(inp.K[0], inp.V[0], n0, cap, 32)
    k_cap, set_cap = B.prhs_max_topk(p, cap), B.prhs_set_capacity(p, cap)
    i32 = dict(dtype=torch.int32, device=dev)
    topk, tlen = torch.zeros(4, 8, k_cap, **i32), torch.zeros(4, 8, **i32)
    cset, clen = torch.zeros(4, 8, set_cap, **i32), torch.zeros(4, 8, **i32)
    hset, hlen = torch.zeros(4, 8, set_cap, **i32), torch.zeros(4, 8, **i32)
    ws = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SELECT, kv0, p), dev)
    B.prhs_select_shared(kv0, inp.q[0, 0], p, topk, tlen, cset, clen, hset, hlen, ws)
    n = torch.tensor([x + STEP for x in LENS], dtype=torch.int32, device=dev)
    kv = B.KV(inp.K[0], inp.V[0], n, cap, 32)
    out = torch.full((4, 32, 128), float("nan"), device=dev)
    lse = torch.full((4, 32), float("nan"), device=dev)
    wsa = B.workspace(B.prhs_workspace_size(B.PRHS_OP_SPARSE_ATTN, kv, p, set_cap), dev)
    B.prhs_reuse_decode_attn(kv, inp.q[0, STEP], hset, hlen, n0, 1 / math.sqrt(128), out, lse, wsa)
    torch.cuda.synchronize()
    np.savez(path, topk=topk.cpu().numpy(), tlen=tlen.cpu().numpy(), cset=cset.cpu().numpy(),
             clen=clen.cpu().numpy(), hset=hset.cpu().numpy(), hlen=hlen.cpu().numpy(),
             out=out.cpu().numpy(), lse=lse.cpu().numpy())
    print("[child] done", flush=True)


if __name__ == "__main__":
    main(sys.argv[1])
