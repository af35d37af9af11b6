"""GPU parity of the global memory's intra-chunk reading (global_intra = 1:
each token reads the global memory at V_t after its own update, gradients at
the chunk-entry state; the Sec. 2.2 chunkwise retrieval rule applied to the
global memory) against the fp64 oracle's flag of the same name.

On the GPU that memory runs as a local-style walk with no reset and no Q-K
projection, in sub-chunks of at most 64 tokens whose gradients are taken at
the entry state of their C_G chunk (C_G = 96, 128, 256 below take 2 to 4
sub-chunks per gradient point; C_G <= 64 one).  Forward output, final global
state and every gradient, element by element; bounds as for the other parity
tests (1e-4 fp32, 2e-2 bf16).
"""
import os

import numpy as np
import pytest
import torch

import oracle as O
from paper_2511_07343_amd import tnt
from paper_2511_07343_amd.inputs import (ACT_GELU, ACT_SILU, BF16, F32, WORKLOADS, make_inputs,
                                         max_rel_err, small_config)
from parity_log import check_err

pytestmark = pytest.mark.gpu
GRADS = ["dq", "dk", "dv", "dlr", "dmom", "ddecay", "dW1", "dW2"]


def tol(cfg):
    return 2e-2 if cfg.dtype == BF16 else 1e-4


CASES = [
    small_config(F32, ACT_GELU, B=2, H=2, L=128, d=16, hid=32, C_G=32, locals_=((8, 32),),
                 global_intra=1, name="intra f32 C_G=32 (one sub-chunk)"),
    small_config(F32, ACT_SILU, B=1, H=2, L=192, d=16, hid=32, C_G=96, locals_=((16, 64),),
                 global_intra=1, name="intra f32 C_G=96 (2 x 48)"),
    small_config(F32, ACT_SILU, B=2, H=1, L=256, d=32, hid=64, C_G=128, locals_=(),
                 global_intra=1, name="intra f32 global only C_G=128 (2 x 64)"),
    small_config(BF16, ACT_SILU, B=1, H=2, L=512, d=64, hid=256, C_G=256, locals_=((32, 128),),
                 global_intra=1, name="intra bf16 d64 h256 C_G=256 (4 x 64)"),
]


@pytest.mark.parametrize("cfg", CASES, ids=lambda c: c.name)
def test_global_intra_forward_backward(cfg):
    inp = make_inputs(cfg, 701)
    print(f"\n[case] {cfg.name}", flush=True)
    x = tnt.device_inputs(inp, cfg)
    o, saved, fin = tnt.forward(cfg, x, save=True, final_state=True)
    g = tnt.backward(cfg, x, x["dO"], saved=saved)
    torch.cuda.synchronize()
    pairs = O.all_pairs(cfg)
    ref_o, rfin = O.forward_pairs(inp, cfg, pairs, with_final=True)
    r = O.backward_pairs(inp, cfg, pairs)
    B, H, L, d = cfg.B, cfg.H, cfg.L, cfg.d
    want = {"o": ref_o.numpy().reshape(B, H, L, d)}
    for n in ("dq", "dk", "dv"):
        want[n] = r[n].numpy().reshape(B, H, L, d)
    for n in ("dlr", "dmom", "ddecay"):
        want[n] = r[n].numpy().reshape(cfg.M, B, H, L)
    want["dW1"] = O.reduce_init_grads(r["dW1"], pairs, H).numpy()
    want["dW2"] = O.reduce_init_grads(r["dW2"], pairs, H).numpy()
    got = {"o": o.float().cpu().numpy()}
    got.update({k: v.float().cpu().numpy() for k, v in g.items()})
    bad = []
    for n in ["o"] + GRADS:
        e = max_rel_err(got[n], want[n])
        print(f"  {n:7s} max rel err {e:.3e}", flush=True)
        if not np.isfinite(got[n]).all() or not check_err(f"intra {cfg.name}", n, e, tol(cfg)):
            bad.append((n, e))
    rf = np.stack([t.numpy().reshape(len(pairs), -1) for t in rfin], 1)
    e = max_rel_err(fin.cpu().numpy().reshape(len(pairs), 4, -1), rf)
    print(f"  final state max rel err {e:.3e}", flush=True)
    if not check_err(f"intra {cfg.name}", "final_state", e, tol(cfg)):
        bad.append(("final_state", e))
    assert not bad, bad


def test_global_intra_differs_from_chunk_entry_reading():
    """The two readings give different outputs (the flag reaches the GPU path)
    and the no-save forward equals the saved one."""
    cfg = CASES[1]
    inp = make_inputs(cfg, 702)
    x = tnt.device_inputs(inp, cfg)
    a, _, _ = tnt.forward(cfg, x, save=True)
    b, _, _ = tnt.forward(cfg.replace(global_intra=0), x, save=True)
    c, _, _ = tnt.forward(cfg, x, save=False)
    torch.cuda.synchronize()
    assert max_rel_err(a.cpu().numpy(), b.cpu().numpy()) > 1e-3
    assert torch.equal(a, c)


def test_global_intra_workload1_against_oracle_samples():
    """Workload 1 (B2 H4 L2048 d64 h256, C_G 256 = 4 sub-chunks of 64, local
    (16, 256)) with the intra-chunk reading, every chain on the GPU, compared
    at the stored oracle samples (tests/golden/workload1_intra.npz: every batch
    row of head 2, sampled token rows, that head's init gradients and the final
    global state)."""
    cfg = WORKLOADS[1].replace(global_intra=1, name=WORKLOADS[1].name + " global intra")
    ref = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                               "workload1_intra.npz"))
    print(f"\n[case] {cfg.name}", flush=True)
    x = tnt.device_inputs(make_inputs(cfg, 1), cfg)
    o, saved, fin = tnt.forward(cfg, x, save=True, final_state=True)
    g = tnt.backward(cfg, x, x["dO"], saved=saved)
    torch.cuda.synchronize()
    pairs = ref["pairs"]
    bi, hi = torch.as_tensor(pairs[:, 0]), torch.as_tensor(pairs[:, 1])
    rows = torch.as_tensor(ref["rows"])
    got = {"o": o.float()[bi, hi].cpu()[:, rows].numpy()}
    for n in ("dq", "dk", "dv"):
        got[n] = g[n].float()[bi, hi].cpu()[:, rows].numpy()
    bad = []
    for n in ("o", "dq", "dk", "dv"):
        e = max_rel_err(got[n], ref[n])
        print(f"  {n:7s} max rel err {e:.3e}", flush=True)
        if not np.isfinite(got[n]).all() or not check_err("intra w1", n, e, 2e-2):
            bad.append((n, e))
    for n in ("dlr", "dmom", "ddecay"):
        mine = g[n][:, bi, hi].float().cpu()[:, :, rows].numpy()
        for m in range(cfg.M):
            e = max_rel_err(mine[m], ref[n][m])
            print(f"  {n:7s} memory {m} max rel err {e:.3e}", flush=True)
            if not np.isfinite(mine[m]).all() or not check_err("intra w1", f"{n}[m{m}]", e, 2e-2):
                bad.append((n, m, e))
    heads = ref["heads"].tolist()
    for n in ("dW1", "dW2"):
        mine = g[n][:, heads].float().cpu().numpy()
        for m in range(cfg.M):
            e = max_rel_err(mine[m], ref[n][m])
            print(f"  {n:7s} memory {m} max rel err {e:.3e}", flush=True)
            if not np.isfinite(mine[m]).all() or not check_err("intra w1", f"{n}[m{m}]", e, 2e-2):
                bad.append((n, m, e))
    f = fin[bi, hi].cpu().numpy()
    e = max_rel_err(f, ref["final_state"])
    print(f"  final state max rel err {e:.3e}", flush=True)
    if not check_err("intra w1", "final_state", e, 2e-2):
        bad.append(("final_state", e))
    assert not bad, bad
