"""Write the oracle's full-size backward samples used by the GPU parity tests.

For workload w (1..4) with seed w, the oracle (fp64, CPU) runs the forward and
backward of every batch row of one sampled head h* = H // 2, so the summed
init gradients of that head are complete.  Stored (float32, .npz):
  pairs                     the (b, h*) chains
  rows                      sampled token indices (chunk and shard edges plus
                            seeded random positions)
  o, dq, dk, dv             [B][len(rows)][d] at those tokens
  dlr, dmom, ddecay         [M][B][len(rows)]
  dW1, dW2                  [M][hid][d], [M][d][hid] of head h*
Only `oracle/` and the seeded input generator are called.

Usage: python tests/golden/make_golden.py 1 2 3 4
"""
import os
import sys
import time

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle as O  # noqa: E402
from paper_2511_07343_amd.inputs import WORKLOADS, make_inputs  # noqa: E402


def sample_rows(cfg, n_random=448, seed=7):
    edges = set()
    steps = [cfg.C_G] + [c for c, _ in cfg.locals_] + [s for _, s in cfg.locals_]
    for st in steps:
        for t0 in range(0, cfg.L, st):
            edges.update((t0, t0 + st - 1))
    edges = sorted(e for e in edges if 0 <= e < cfg.L)
    rng = np.random.default_rng(seed)
    if len(edges) > 256:
        edges = sorted(rng.choice(edges, 256, replace=False).tolist())
    rnd = rng.choice(cfg.L, n_random, replace=False).tolist()
    return np.array(sorted(set(edges) | set(rnd)), dtype=np.int64)


def make(idx):
    cfg = WORKLOADS[idx]
    torch.set_num_threads(max(1, len(os.sched_getaffinity(0))))
    inp = make_inputs(cfg, idx)
    h = cfg.H // 2
    pairs = [(b, h) for b in range(cfg.B)]
    t0 = time.time()
    r = O.backward_pairs(inp, cfg, pairs)
    rows = sample_rows(cfg)
    out = dict(pairs=np.array(pairs), rows=rows)
    for n in ("o", "dq", "dk", "dv"):
        out[n] = r[n].numpy()[:, rows].astype(np.float32)
    for n in ("dlr", "dmom", "ddecay"):
        out[n] = r[n].numpy()[:, :, rows].astype(np.float32)
    out["dW1"] = r["dW1"].numpy().sum(1).astype(np.float32)
    out["dW2"] = r["dW2"].numpy().sum(1).astype(np.float32)
    path = os.path.join(HERE, f"workload{idx}_bwd.npz")
    np.savez_compressed(path, **out)
    print(f"workload {idx}: {time.time() - t0:.0f} s -> {path}", flush=True)


if __name__ == "__main__":
    for a in sys.argv[1:]:
        make(int(a))
