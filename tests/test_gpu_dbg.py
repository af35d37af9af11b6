"""GPU check of one chunk's inner-gradient quantities (tnt_dbg_chunk_grads)
against the oracle's inner_grad: the per-token gradients rebuilt from the
GPU's Zk, R, D1 (u1_t = D1_t k_t^T, u2_t = R_t s(Zk_t)^T, with s evaluated in
fp64 on the GPU's Zk) are compared element by element with the fp64 chain-rule
gradients at the same weights.  Tolerance: max |gpu - oracle| / max |oracle|
<= 1e-4 (fp32 inputs) or 2e-2 (bf16 inputs, the keys and values are the
bf16-rounded ones on both sides)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2511_07343_amd import tnt
from parity_log import check_err
from paper_2511_07343_amd.inputs import (ACT_GELU, ACT_SILU, BF16, F32, make_inputs, max_rel_err,
                                         small_config)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg,b,h,t0,C", [
    (small_config(F32, ACT_GELU, B=2, H=2, L=64, d=16, hid=32, C_G=16, locals_=((8, 32),),
                  name="f32 d16 h32"), 1, 1, 24, 8),
    (small_config(BF16, ACT_SILU, B=1, H=2, L=128, d=64, hid=256, C_G=64, locals_=((64, 128),),
                  name="bf16 d64 h256"), 0, 1, 64, 64),
    (small_config(BF16, ACT_GELU, B=1, H=1, L=64, d=128, hid=512, C_G=32, locals_=((16, 32),),
                  name="bf16 d128 h512"), 0, 0, 16, 16),
], ids=lambda c: c.name if hasattr(c, "name") else str(c))
def test_chunk_grads_match_oracle_inner_grad(cfg, b, h, t0, C):
    inp = make_inputs(cfg, 501)
    print(f"\n[case] dbg chunk grads {cfg.name} chain ({b},{h}) tokens {t0}..{t0 + C}", flush=True)
    x = tnt.device_inputs(inp, cfg)
    m = cfg.M - 1  # the last memory's init weights for that head
    W1 = x["W1"][m, h].contiguous()
    W2 = x["W2"][m, h].contiguous()
    dev = x["q"].device
    Zk = torch.empty(C, cfg.hid, dtype=torch.float32, device=dev)
    R = torch.empty(C, cfg.d, dtype=torch.float32, device=dev)
    D1 = torch.empty(C, cfg.hid, dtype=torch.float32, device=dev)
    st = tnt.tnt_dbg_chunk_grads(cfg, b, h, t0, C, x["k"], x["v"], W1, W2, Zk, R, D1)
    assert st == 0, tnt.strerror(st)
    torch.cuda.synchronize()
    # fp64 oracle at the same (device-rounded) keys and values
    k = x["k"][b, h, t0:t0 + C].double().cpu()
    v = x["v"][b, h, t0:t0 + C].double().cpu()
    W1d, W2d = W1.double().cpu(), W2.double().cpu()
    kind = {ACT_GELU: "gelu", ACT_SILU: "silu"}[cfg.act]
    g1, g2 = O.inner_grad(W1d[None], W2d[None], k[None], v[None], kind)
    g1, g2 = g1[0].numpy(), g2[0].numpy()
    zk, r, d1 = Zk.double().cpu(), R.double().cpu(), D1.double().cpu()
    u1 = (d1[:, :, None] * k[:, None, :]).numpy()
    u2 = (r[:, :, None] * O.act(zk, kind)[:, None, :]).numpy()
    zref = (k @ W1d.T).numpy()
    tol = 2e-2 if cfg.dtype == BF16 else 1e-4
    for name, got, ref in (("Zk", zk.numpy(), zref), ("u1", u1, g1), ("u2", u2, g2)):
        e = max_rel_err(got, ref)
        print(f"  {name} max rel err {e:.3e}", flush=True)
        assert np.isfinite(got).all() and check_err(f"chunk grads {cfg.name}", name, e, tol), (name, e)
