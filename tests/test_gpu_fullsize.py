"""Full-size parity of tnt_mem_fwd / tnt_mem_bwd against stored oracle samples.

tests/golden/workload{w}_bwd.npz holds the fp64 oracle's layer output and
gradients for workload w with seed w, written by tests/golden/make_golden.py
(which calls only the oracle and the seeded input generator): every batch row
of head h* = H // 2 at sampled token rows (chunk and shard edges plus seeded
random positions), and that head's complete init gradients.  The GPU runs the
whole workload, every chain, in the launch configuration bench.py times; the
sampled entries are compared with the bound of the small parity tests:
max |gpu - oracle| / max |oracle| over the samples <= 2e-2 (bf16 inputs).
"""
import os

import numpy as np
import pytest
import torch

from paper_2511_07343_amd import tnt
from paper_2511_07343_amd.inputs import WORKLOADS, make_inputs, max_rel_err

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))
TOL = 2e-2


def golden(w):
    return np.load(os.path.join(HERE, "golden", f"workload{w}_bwd.npz"))


@pytest.mark.parametrize("w", [1, 2, 3, 4])
def test_fullsize_against_oracle_samples(w):
    cfg = WORKLOADS[w]
    print(f"\n[case] workload {w}: {cfg.name}", flush=True)
    ref = golden(w)
    hs = cfg.H // 2
    assert np.array_equal(ref["pairs"][:, 1], np.full(cfg.B, hs))
    rows = torch.as_tensor(ref["rows"])
    inp = make_inputs(cfg, w)
    x = tnt.device_inputs(inp, cfg)
    o, saved, _ = tnt.forward(cfg, x, save=True)
    g = tnt.backward(cfg, x, x["dO"], saved=saved)
    torch.cuda.synchronize()
    got = {"o": o[:, hs].float().cpu()[:, rows]}
    for n in ("dq", "dk", "dv"):
        got[n] = g[n][:, hs].float().cpu()[:, rows]
    for n in ("dlr", "dmom", "ddecay"):
        got[n] = g[n][:, :, hs].float().cpu()[:, :, rows]
    for n in ("dW1", "dW2"):
        got[n] = g[n][:, hs].float().cpu()
    bad = []
    for n, v in got.items():
        v = v.numpy()
        assert v.shape == ref[n].shape, (n, v.shape, ref[n].shape)
        e = max_rel_err(v, ref[n])
        print(f"  {n:7s} max rel err {e:.3e}", flush=True)
        if not np.isfinite(v).all() or e > TOL:
            bad.append((n, e))
    assert not bad, bad
