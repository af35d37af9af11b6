"""Write the oracle's full-size samples used by the GPU parity tests.

Two files per workload w (1..4), seed w, written by the fp64 oracle on the CPU:

* ``workload{w}_bwd.npz``: the workload as stated.  The oracle runs the
  forward and backward of every batch row of the sampled heads (h* = H // 2;
  workload 1 also head 0), so the summed init gradients of those heads are
  complete.
* ``workload{w}_global32.npz`` (``--global-fp32``): that global-only shape
  with fp32 inputs (no bf16 rounding), for the fp32 bound chunk by chunk.
* ``workload{w}_intra.npz`` (``--intra``): the workload with the global
  memory read at V_t after each token's update (the intra-chunk reading).
* ``workload{w}_global.npz``: the same shape with the global memory alone
  (no local memory; its own seeded draw).  The global memory's outputs shrink
  by orders of magnitude from one 2048-token chunk to the next under the
  stated decay range, so the GPU test compares this file chunk by chunk, each
  global chunk against its own largest value; it also holds the final global
  state of every sampled chain.

Stored (float32, .npz):
  pairs                     the (b, h) chains
  rows                      sampled token indices (chunk and shard edges plus
                            seeded random positions)
  o, dq, dk, dv             [P][len(rows)][d] at those tokens
  dlr, dmom, ddecay         [M][P][len(rows)]
  dW1, dW2                  [M][len(heads)][hid][d], [M][len(heads)][d][hid]
  heads                     the sampled heads (dW1 / dW2 are summed over their chains)
  final_state               [P][4][hid*d] (global file only): V1, V2, S1, S2
Only `oracle/` and the seeded input generator are called.

Usage: python tests/golden/make_golden.py 1 2 3 4 [--global-only | --full-only | --global-fp32 | --intra]
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
from paper_2511_07343_amd.inputs import F32, WORKLOADS, make_inputs  # noqa: E402


def global_only(cfg):
    return cfg.replace(locals_=(), name=cfg.name + " global only")


def sampled_heads(idx, cfg, variant="bwd"):
    return (0, cfg.H // 2) if (idx == 1 and variant == "bwd") else (cfg.H // 2,)


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


def make(idx, variant):
    cfg = WORKLOADS[idx] if variant == "bwd" else global_only(WORKLOADS[idx])
    if variant == "global32":   # the same global-only shape with fp32 inputs
        cfg = cfg.replace(dtype=F32, name=cfg.name + " fp32")
    if variant == "intra":      # the workload with the global memory's intra-chunk reading
        cfg = WORKLOADS[idx].replace(global_intra=1, name=WORKLOADS[idx].name + " global intra")
    torch.set_num_threads(max(1, len(os.sched_getaffinity(0))))
    inp = make_inputs(cfg, idx)
    heads = sampled_heads(idx, cfg, variant)
    pairs = [(b, h) for h in heads for b in range(cfg.B)]
    t0 = time.time()
    r = O.backward_pairs(inp, cfg, pairs)
    rows = sample_rows(cfg)
    out = dict(pairs=np.array(pairs), rows=rows, heads=np.array(heads))
    for n in ("o", "dq", "dk", "dv"):
        out[n] = r[n].numpy()[:, rows].astype(np.float32)
    for n in ("dlr", "dmom", "ddecay"):
        out[n] = r[n].numpy()[:, :, rows].astype(np.float32)
    for n in ("dW1", "dW2"):
        full = r[n].numpy()
        out[n] = np.stack([full[:, [i for i, p in enumerate(pairs) if p[1] == h]].sum(1)
                           for h in heads], 1).astype(np.float32)
    if variant.startswith("global") or variant == "intra":
        _, fin = O.forward_pairs(inp, cfg, pairs, with_final=True)
        out["final_state"] = np.stack([f.numpy().reshape(len(pairs), -1) for f in fin],
                                      1).astype(np.float32)
    path = os.path.join(HERE, f"workload{idx}_{variant}.npz")
    np.savez_compressed(path, **out)
    print(f"workload {idx} {variant}: {time.time() - t0:.0f} s -> {path}", flush=True)


if __name__ == "__main__":
    args = [a for a in sys.argv[1:] if not a.startswith("--")]
    variants = ["bwd", "global"]
    if "--global-only" in sys.argv:
        variants = ["global"]
    if "--full-only" in sys.argv:
        variants = ["bwd"]
    if "--global-fp32" in sys.argv:
        variants = ["global32"]
    if "--intra" in sys.argv:
        variants = ["intra"]
    for a in args:
        for v in variants:
            make(int(a), v)
