"""Full-size parity of tnt_mem_fwd / tnt_mem_bwd against stored oracle samples.

tests/golden/workload{w}_bwd.npz holds the fp64 oracle's layer output and
gradients for workload w with seed w, written by tests/golden/make_golden.py
(which calls only the oracle and the seeded input generator): every batch row
of the sampled heads at sampled token rows (chunk and shard edges plus seeded
random positions), and those heads' complete init gradients.  The GPU runs the
whole workload, every chain, in the launch configuration bench.py times; the
sampled entries are compared with the bound of the small parity tests:
max |gpu - oracle| / max |oracle| <= 2e-2 (bf16 inputs), taken per tensor and,
for the per-memory tensors (gate and init gradients), per memory.

tests/golden/workload{w}_global.npz holds the same shape with the global
memory alone.  Under the stated decay range its outputs shrink by orders of
magnitude from one global chunk to the next, so a whole-tensor maximum would
hide every chunk after the first: this file is compared chunk by chunk, each
global chunk's sampled rows against that chunk's own largest value, and the
final global state of every sampled chain is compared too.
"""
import os

import numpy as np
import pytest
import torch

from paper_2511_07343_amd import tnt
from paper_2511_07343_amd.inputs import WORKLOADS, make_inputs, max_rel_err
from parity_log import check_err, record

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))
TOL = 2e-2
# Per global chunk, the momentum and decay gradients of the late chunks are
# sums of per-token adjoint dot products of both signs, taken from bf16
# operands (relative rounding 2^-9 each); normalised by their own chunk's
# largest value they sit at 1e-2 to 2e-2 in bf16 (the same kernels in fp32
# mode stay at the fp32 bound per chunk, test_fullsize_global_fp32_every_chunk),
# so the chunk-by-chunk view of those two uses twice the tensor bound.  Every
# tensor is also held to TOL over the whole tensor (the stated metric).
TOL_GATE_CHUNK = 4e-2
# The gate gradients of a chunk are sums of adjoint x state products; once a
# chunk's gradients are below 1e-9 of the tensor's largest value (workload 4's
# eight 4096-token chunks reach 1e-19) their relative precision says more about
# fp32 arithmetic on such products than about the chunk chain, so the chunk-wise
# bound applies to chunks above that scale; the rest are recorded, not bounded
# (and stay inside the whole-tensor bound).
GATE_SCALE_FLOOR = 1e-9


def golden(name):
    return np.load(os.path.join(HERE, "golden", name))


def heads_of(ref, cfg):
    return tuple(ref["heads"].tolist()) if "heads" in ref else (cfg.H // 2,)


def init_grads(ref, name, nheads):
    g = ref[name]
    return g if g.ndim == 4 else g[:, None]      # [M][heads][...]


def run_layer(cfg, w, final=False):
    inp = make_inputs(cfg, w)
    x = tnt.device_inputs(inp, cfg)
    o, saved, fin = tnt.forward(cfg, x, save=True, final_state=final)
    g = tnt.backward(cfg, x, x["dO"], saved=saved)
    torch.cuda.synchronize()
    return o, g, fin


def gather(o, g, pairs, rows):
    b = torch.as_tensor(pairs[:, 0])
    h = torch.as_tensor(pairs[:, 1])
    rows = torch.as_tensor(rows)
    got = {"o": o.float()[b, h].cpu()[:, rows]}
    for n in ("dq", "dk", "dv"):
        got[n] = g[n].float()[b, h].cpu()[:, rows]
    for n in ("dlr", "dmom", "ddecay"):
        got[n] = g[n][:, b, h].float().cpu()[:, :, rows]
    return {k: v.numpy() for k, v in got.items()}


@pytest.mark.parametrize("w", [1, 2, 3, 4])
def test_fullsize_against_oracle_samples(w):
    cfg = WORKLOADS[w]
    case = f"fullsize w{w}"
    print(f"\n[case] workload {w}: {cfg.name}", flush=True)
    ref = golden(f"workload{w}_bwd.npz")
    heads = heads_of(ref, cfg)
    o, g, _ = run_layer(cfg, w)
    got = gather(o, g, ref["pairs"], ref["rows"])
    bad = []
    for n in ("o", "dq", "dk", "dv"):
        e = max_rel_err(got[n], ref[n])
        print(f"  {n:7s} max rel err {e:.3e}", flush=True)
        if not np.isfinite(got[n]).all() or not check_err(case, n, e, TOL):
            bad.append((n, e))
    for n in ("dlr", "dmom", "ddecay"):
        for m in range(cfg.M):                    # each memory against its own scale
            e = max_rel_err(got[n][m], ref[n][m])
            print(f"  {n:7s} memory {m} max rel err {e:.3e}", flush=True)
            if not np.isfinite(got[n][m]).all() or not check_err(case, f"{n}[m{m}]", e, TOL):
                bad.append((n, m, e))
    for n in ("dW1", "dW2"):
        want = init_grads(ref, n, len(heads))
        mine = g[n][:, list(heads)].float().cpu().numpy()
        for m in range(cfg.M):
            e = max_rel_err(mine[m], want[m])
            print(f"  {n:7s} memory {m} max rel err {e:.3e}", flush=True)
            if not np.isfinite(mine[m]).all() or not check_err(case, f"{n}[m{m}]", e, TOL):
                bad.append((n, m, e))
    assert not bad, bad


@pytest.mark.parametrize("w", [1, 2, 3, 4])
def test_fullsize_global_memory_every_chunk(w):
    """The global memory alone at full size, every global chunk normalised on
    its own: the multi-chunk carry of the fixed-size global kernels (C_G =
    2048 / 4096 with their split partial sums) and the global share of the gate
    and init gradients are checked in every chunk, not just the first."""
    cfg = WORKLOADS[w].replace(locals_=(), name=WORKLOADS[w].name + " global only")
    global_every_chunk(cfg, w, f"workload{w}_global.npz", f"fullsize global-only w{w}", TOL, TOL,
                       TOL_GATE_CHUNK)


def test_fullsize_global_fp32_every_chunk():
    """The pre-training shape's global memory alone in fp32 (runtime-sized
    kernels, same chunk chain): every global chunk, gate gradients included,
    within the fp32 bound of its own chunk's scale."""
    from paper_2511_07343_amd.inputs import F32
    cfg = WORKLOADS[2].replace(locals_=(), dtype=F32, name=WORKLOADS[2].name + " global only fp32")
    global_every_chunk(cfg, 2, "workload2_global32.npz", "fullsize global-only fp32 w2", 1e-4, 1e-4,
                       1e-4)


def global_every_chunk(cfg, w, fname, case, tol, chunk_tol, gate_chunk_tol):
    print(f"\n[case] workload {w} global memory alone: {cfg.name}", flush=True)
    ref = golden(fname)
    heads = heads_of(ref, cfg)
    o, g, fin = run_layer(cfg, w, final=True)
    rows = ref["rows"]
    got = gather(o, g, ref["pairs"], rows)
    chunk_of = rows // cfg.C_G
    bad = []
    for n in ("o", "dq", "dk", "dv", "dlr", "dmom", "ddecay"):
        e = max_rel_err(got[n], ref[n])          # the whole tensor, the stated metric
        if not np.isfinite(got[n]).all() or not check_err(case, n, e, tol):
            bad.append((n, e))
        bound = chunk_tol if n not in ("dmom", "ddecay") else gate_chunk_tol
        gate = n in ("dlr", "dmom", "ddecay")
        scale = float(np.abs(ref[n]).max())
        worst = 0.0
        for c in range(cfg.L // cfg.C_G):
            sel = chunk_of == c
            if not sel.any():
                continue
            a = got[n][..., sel, :] if n in ("o", "dq", "dk", "dv") else got[n][..., sel]
            b = ref[n][..., sel, :] if n in ("o", "dq", "dk", "dv") else ref[n][..., sel]
            e = max_rel_err(a, b)
            if gate and float(np.abs(b).max()) < GATE_SCALE_FLOOR * scale:
                record(case, f"{n}[chunk {c}] (below 1e-9 of the tensor scale, not bounded)", e,
                       float("nan"))
                continue
            worst = max(worst, e)
            if not np.isfinite(a).all() or not check_err(case, f"{n}[chunk {c}]", e, bound):
                bad.append((n, c, e))
        print(f"  {n:7s} whole {max_rel_err(got[n], ref[n]):.3e} worst chunk {worst:.3e}",
              flush=True)
    for n in ("dW1", "dW2"):
        want = init_grads(ref, n, len(heads))
        mine = g[n][:, list(heads)].float().cpu().numpy()
        e = max_rel_err(mine, want)
        print(f"  {n:7s} max rel err {e:.3e}", flush=True)
        if not np.isfinite(mine).all() or not check_err(case, n, e, tol):
            bad.append((n, e))
    pairs = ref["pairs"]
    mine = fin[torch.as_tensor(pairs[:, 0]), torch.as_tensor(pairs[:, 1])].cpu().numpy()
    for j, nm in enumerate(("V1", "V2", "S1", "S2")):
        e = max_rel_err(mine[:, j], ref["final_state"][:, j])
        print(f"  final {nm} max rel err {e:.3e}", flush=True)
        if not np.isfinite(mine[:, j]).all() or not check_err(case, f"final {nm}", e, tol):
            bad.append((nm, e))
    assert not bad, bad
