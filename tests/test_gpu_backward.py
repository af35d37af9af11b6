"""GPU parity of tnt_mem_bwd against autograd through the fp64 oracle.

Every gradient tensor (dq, dk, dv, dlr, dmom, ddecay, dW1_init, dW2_init) is
compared element by element; tolerance as for the forward: max_i |gpu - oracle|
/ max_i |oracle| <= 1e-4 (fp32 inputs) or 2e-2 (bf16 inputs).
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2511_07343_amd import tnt
from paper_2511_07343_amd.inputs import (ACT_GELU, ACT_SILU, BF16, F32, QK_CHUNK, WORKLOADS,
                                         make_inputs, max_rel_err, small_config)
from parity_log import check_err

pytestmark = pytest.mark.gpu
torch.set_num_threads(4)
GRADS = ["dq", "dk", "dv", "dlr", "dmom", "ddecay", "dW1", "dW2"]


def tol(cfg):
    return 2e-2 if cfg.dtype == BF16 else 1e-4


def gpu_backward(cfg, inp, use_saved=True):
    x = tnt.device_inputs(inp, cfg)
    o, saved, _ = tnt.forward(cfg, x, save=use_saved)
    g = tnt.backward(cfg, x, x["dO"], saved=saved if use_saved else None)
    torch.cuda.synchronize()
    return {k: v.float().cpu().numpy() for k, v in g.items()}


def oracle_backward(cfg, inp):
    pairs = O.all_pairs(cfg)
    r = O.backward_pairs(inp, cfg, pairs)
    B, H, L, d = cfg.B, cfg.H, cfg.L, cfg.d
    out = {}
    for n in ("dq", "dk", "dv"):
        out[n] = r[n].numpy().reshape(B, H, L, d)
    for n in ("dlr", "dmom", "ddecay"):
        out[n] = r[n].numpy().reshape(cfg.M, B, H, L)
    out["dW1"] = O.reduce_init_grads(r["dW1"], pairs, H).numpy()
    out["dW2"] = O.reduce_init_grads(r["dW2"], pairs, H).numpy()
    return out


def check(cfg, got, ref, names=GRADS, case=None):
    bad = []
    for n in names:
        e = max_rel_err(got[n], ref[n])
        print(f"  {n:7s} max rel err {e:.3e}", flush=True)
        if not np.isfinite(got[n]).all() or not check_err(case or f"bwd {cfg.name}", n, e, tol(cfg)):
            bad.append((n, e))
    assert not bad, bad


SMALL = [
    WORKLOADS[0],
    small_config(F32, ACT_GELU, B=2, H=2, L=64, d=16, hid=32, C_G=32, locals_=((8, 32),),
                 name="f32 tiny two chunks"),
    small_config(F32, ACT_SILU, B=1, H=2, L=96, d=32, hid=64, C_G=48,
                 locals_=((12, 48), (16, 32)), name="f32 two locals ragged"),
    small_config(F32, ACT_SILU, B=1, H=1, L=64, d=16, hid=32, C_G=16, locals_=((8, 32),),
                 qk_scope=QK_CHUNK, name="f32 chunk-scope QK"),
    small_config(F32, ACT_GELU, B=1, H=2, L=64, d=16, hid=32, C_G=16, locals_=((16, 32),),
                 qk_proj=0, name="f32 no QK projection"),
    small_config(F32, ACT_GELU, B=1, H=1, L=64, d=16, hid=32, C_G=64, locals_=((16, 64),),
                 has_global=0, name="f32 locals only"),
    small_config(F32, ACT_SILU, B=2, H=1, L=64, d=16, hid=32, C_G=16, locals_=(),
                 name="f32 global only"),
    small_config(BF16, ACT_SILU, B=1, H=2, L=128, d=64, hid=256, C_G=64, locals_=((32, 64),),
                 name="bf16 d64 h256"),
    small_config(BF16, ACT_SILU, B=1, H=1, L=128, d=128, hid=512, C_G=128,
                 locals_=((64, 128),), name="bf16 d128 h512"),
    small_config(BF16, ACT_SILU, B=1, H=2, L=256, d=64, hid=256, C_G=128,
                 locals_=((64, 128),), name="bf16 d64 h256 C64"),
    small_config(BF16, ACT_SILU, B=1, H=1, L=192, d=64, hid=256, C_G=96,
                 locals_=((48, 96),), name="bf16 d64 h256 C48 ragged"),
]


@pytest.mark.parametrize("cfg", SMALL, ids=lambda c: c.name)
def test_backward_small_all_chains(cfg):
    inp = make_inputs(cfg, 0 if cfg is WORKLOADS[0] else 201)
    print(f"\n[case] {cfg.name}", flush=True)
    got = gpu_backward(cfg, inp)
    ref = oracle_backward(cfg, inp)
    check(cfg, got, ref)


@pytest.mark.parametrize("cfg", [SMALL[2], SMALL[7], SMALL[9]], ids=lambda c: c.name)
def test_backward_recompute_equals_saved(cfg):
    """tnt_mem_bwd without the saved buffer recomputes the same states (the
    bf16 d64 h256 shapes take the fixed-size forward walk, the chunk-parallel
    retrieval and the three-pass backward from a recomputed saved area) and
    gives the same bits as with the forward's buffer, within the bound of the
    oracle."""
    inp = make_inputs(cfg, 202)
    print(f"\n[case] recompute {cfg.name}", flush=True)
    a = gpu_backward(cfg, inp, use_saved=True)
    b = gpu_backward(cfg, inp, use_saved=False)
    for n in GRADS:
        assert np.array_equal(a[n], b[n]), n
    check(cfg, b, oracle_backward(cfg, inp), case=f"bwd recompute {cfg.name}")


def test_backward_deterministic():
    cfg = SMALL[7]
    inp = make_inputs(cfg, 203)
    a = gpu_backward(cfg, inp)
    b = gpu_backward(cfg, inp)
    for n in GRADS:
        assert np.array_equal(a[n], b[n]), n


@pytest.mark.parametrize("cfg", [WORKLOADS[0], SMALL[2], SMALL[7]], ids=lambda c: c.name)
def test_backward_generic_kernels(cfg):
    """The runtime-sized kernels against the oracle (the fixed-size ones are
    what the default path takes for these shapes)."""
    inp = make_inputs(cfg, 204)
    print(f"\n[case] generic {cfg.name}", flush=True)
    with tnt.kernel_family(tnt.FAMILY_GENERIC):
        got = gpu_backward(cfg, inp)
    check(cfg, got, oracle_backward(cfg, inp), case=f"bwd generic {cfg.name}")


@pytest.mark.parametrize("cfg", [WORKLOADS[0], SMALL[3], SMALL[7], SMALL[9], SMALL[10]],
                         ids=lambda c: c.name)
def test_backward_single_walk(cfg):
    """The fixed-size local backward as one reverse walk per unit (the default
    splits it into a chunk-parallel pass, the walk of the carried adjoint and a
    chunk-parallel gate pass)."""
    inp = make_inputs(cfg, 205)
    print(f"\n[case] single walk {cfg.name}", flush=True)
    with tnt.kernel_family(tnt.FAMILY_SINGLE_WALK):
        got = gpu_backward(cfg, inp)
    check(cfg, got, oracle_backward(cfg, inp), case=f"bwd single walk {cfg.name}")


def test_saved_buffer_from_another_family_is_refused():
    """A saved buffer written under one kernel family (which decides which
    fp32 state slots the forward writes) is refused by a backward under
    another: TNT_ERR_ARG before anything is enqueued, never a computation on
    unwritten slots."""
    cfg = SMALL[9]  # bf16 d64 h256 C64: the default forward keeps a two-slot ring
    x = tnt.device_inputs(make_inputs(cfg, 206), cfg)
    o, saved, _ = tnt.forward(cfg, x, save=True)
    with tnt.kernel_family(tnt.FAMILY_SINGLE_WALK):
        with pytest.raises(tnt.TntError) as ei:
            tnt.backward(cfg, x, x["dO"], saved=saved)
    assert ei.value.status == 7
    torch.cuda.synchronize()
    g = tnt.backward(cfg, x, x["dO"], saved=saved)   # the writing family still works
    torch.cuda.synchronize()
    assert all(torch.isfinite(v.float()).all() for v in g.values())
