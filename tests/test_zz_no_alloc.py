"""tnt_mem_fwd_noalloc (forward on the library's static workspace) against
tnt_mem_fwd, through the C ABI: two calls in a row, the second on a smaller
input, each compared with tnt_mem_fwd on the same inputs (the same kernels:
outputs and final state bit for bit) and with the fp64 oracle within the bf16
bound; an oversized configuration is refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2511_07343_amd import tnt
from paper_2511_07343_amd.inputs import ACT_SILU, BF16, WORKLOADS, make_inputs, max_rel_err, small_config
from parity_log import check_err

pytestmark = pytest.mark.gpu

BIG = small_config(BF16, ACT_SILU, B=2, H=2, L=512, d=64, hid=256, C_G=128,
                   locals_=((32, 128), (16, 64)), name="noalloc bf16 B2 H2 L512 two locals")
SMALL = small_config(BF16, ACT_SILU, B=1, H=2, L=128, d=64, hid=256, C_G=64,
                     locals_=((16, 64),), name="noalloc bf16 B1 H2 L128")


def _noalloc(cfg, x):
    o = torch.empty_like(x["q"])
    fin = torch.empty(cfg.B, cfg.H, 4, cfg.hid * cfg.d, dtype=torch.float32, device=o.device)
    st = tnt.tnt_mem_fwd_noalloc(cfg, x["q"], x["k"], x["v"], x["lr"], x["mom"], x["decay"],
                                 x["W1"], x["W2"], o, fin)
    assert st == 0, tnt.strerror(st)
    return o, fin


def test_noalloc_forward_matches_tnt_mem_fwd_two_calls():
    outs = []
    for cfg, seed in ((BIG, 601), (SMALL, 602)):   # the second call is the smaller one
        print(f"\n[case] {cfg.name}", flush=True)
        assert tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_FWD_MIN) <= tnt.NOALLOC_WORKSPACE_BYTES
        inp = make_inputs(cfg, seed)
        x = tnt.device_inputs(inp, cfg)
        o_na, fin_na = _noalloc(cfg, x)
        torch.cuda.synchronize()
        o_ref, _, fin_ref = tnt.forward(cfg, x, save=False, final_state=True)
        torch.cuda.synchronize()
        assert torch.equal(o_na, o_ref)
        assert torch.equal(fin_na, fin_ref)
        ref = O.forward_pairs(inp, cfg, O.all_pairs(cfg)).numpy().reshape(o_na.shape)
        e = max_rel_err(o_na.float().cpu().numpy(), ref)
        print(f"  o vs oracle {e:.3e}", flush=True)
        assert check_err(f"noalloc {cfg.name}", "o", e, 2e-2)
        outs.append(o_na)
    assert np.isfinite(outs[1].float().cpu().numpy()).all()


def test_noalloc_rejects_oversized_config():
    cfg = WORKLOADS[2]   # forward workspace ~785 MiB
    assert tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_FWD_MIN) > tnt.NOALLOC_WORKSPACE_BYTES
    p = 256
    assert tnt.tnt_mem_fwd_noalloc(cfg, p, p, p, p, p, p, p, p, p, None, stream=0) == 4
