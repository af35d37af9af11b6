"""GPU parity at the small chunk sizes of the fine-tuning stage (Sec. 4.2 and
its tables: local chunks of 1, 2 and 4 tokens) and at a global chunk of one
token, forward and backward, element by element against the fp64 oracle.

A local chunk shorter than the 16-row MFMA tile is padded to one tile with
masked rows (eta = 0, alpha = 0, beta = 1 on the padding), so these cases run
the same kernels as the 16-token chunks with 15, 14 or 12 dead rows per tile.

The per-token check compares the GPU layer at C_L = 1 with the oracle's
token-by-token recurrence (Sec. 2.1, with the local reset), which does not go
through the oracle's chunkwise code at all.

Tolerance as elsewhere: max_i |gpu - oracle| / max_i |oracle| <= 1e-4 (fp32
inputs) or 2e-2 (bf16 inputs).
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2511_07343_amd import tnt
from parity_log import check_err
from paper_2511_07343_amd.inputs import (ACT_GELU, ACT_SILU, BF16, F32, make_inputs, max_rel_err,
                                         small_config)

pytestmark = pytest.mark.gpu
torch.set_num_threads(4)
GRADS = ["dq", "dk", "dv", "dlr", "dmom", "ddecay", "dW1", "dW2"]


def tol(cfg):
    return 2e-2 if cfg.dtype == BF16 else 1e-4


CASES = [
    small_config(F32, ACT_GELU, B=1, H=2, L=48, d=16, hid=32, C_G=16, locals_=((1, 16),),
                 name="f32 C_L=1 S_L=16"),
    small_config(F32, ACT_SILU, B=2, H=1, L=48, d=16, hid=32, C_G=24, locals_=((2, 24), (4, 16)),
                 name="f32 C_L=2,4 two locals"),
    small_config(F32, ACT_GELU, B=1, H=1, L=32, d=16, hid=32, C_G=1, locals_=((4, 16),),
                 name="f32 C_G=1 C_L=4"),
    small_config(BF16, ACT_SILU, B=1, H=2, L=64, d=64, hid=256, C_G=32, locals_=((1, 32),),
                 name="bf16 d64 h256 C_L=1"),
    small_config(BF16, ACT_SILU, B=1, H=1, L=96, d=64, hid=256, C_G=48, locals_=((2, 48), (4, 32)),
                 name="bf16 d64 h256 C_L=2,4"),
]


def oracle_grads(cfg, inp):
    pairs = O.all_pairs(cfg)
    r = O.backward_pairs(inp, cfg, pairs)
    B, H, L, d = cfg.B, cfg.H, cfg.L, cfg.d
    out = {n: r[n].numpy().reshape(B, H, L, d) for n in ("dq", "dk", "dv")}
    for n in ("dlr", "dmom", "ddecay"):
        out[n] = r[n].numpy().reshape(cfg.M, B, H, L)
    out["dW1"] = O.reduce_init_grads(r["dW1"], pairs, H).numpy()
    out["dW2"] = O.reduce_init_grads(r["dW2"], pairs, H).numpy()
    return out


@pytest.mark.parametrize("cfg", CASES, ids=lambda c: c.name)
def test_small_chunks_forward_backward(cfg):
    inp = make_inputs(cfg, 301)
    print(f"\n[case] {cfg.name}", flush=True)
    x = tnt.device_inputs(inp, cfg)
    o, saved, _ = tnt.forward(cfg, x, save=True)
    g = tnt.backward(cfg, x, x["dO"], saved=saved)
    torch.cuda.synchronize()
    got = {k: v.float().cpu().numpy() for k, v in g.items()}
    got["o"] = o.float().cpu().numpy()
    ref = oracle_grads(cfg, inp)
    ref["o"] = O.forward_pairs(inp, cfg, O.all_pairs(cfg)).numpy().reshape(got["o"].shape)
    bad = []
    for n in ["o"] + GRADS:
        e = max_rel_err(got[n], ref[n])
        print(f"  {n:7s} max rel err {e:.3e}", flush=True)
        if not np.isfinite(got[n]).all() or not check_err(f"small chunks {cfg.name}", n, e, tol(cfg)):
            bad.append((n, e))
    assert not bad, bad


@pytest.mark.parametrize("dtype,d,hid", [(F32, 16, 32), (BF16, 64, 256)], ids=["f32", "bf16"])
def test_local_chunk_one_equals_token_recurrence(dtype, d, hid):
    """One local memory at C_L = 1 (no global memory) on the GPU against the
    token-by-token recurrence with the state reset every S_L tokens."""
    S = 16
    cfg = small_config(dtype, ACT_SILU, B=1, H=2, L=48, d=d, hid=hid, C_G=48, locals_=((1, S),),
                       has_global=0, name=f"local only C_L=1 d{d}")
    inp = make_inputs(cfg, 302)
    print(f"\n[case] {cfg.name}", flush=True)
    x = tnt.device_inputs(inp, cfg)
    o, _, _ = tnt.forward(cfg, x, save=False)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()
    pairs = O.all_pairs(cfg)
    c = O.gather_pairs(inp, pairs)
    with torch.no_grad():
        ref, _ = O.sequential(c["q"], c["k"], c["v"], c["lr"][0], c["mom"][0], c["decay"][0],
                              c["W1"][0], c["W2"][0], "silu", reset=S, qk_proj=True)
    ref = ref.numpy().reshape(got.shape)
    e = max_rel_err(got, ref)
    print(f"  o max rel err {e:.3e}", flush=True)
    assert check_err(f"C_L=1 vs token recurrence {cfg.name}", "o", e, tol(cfg))
