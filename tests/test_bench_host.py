"""Host-side checks of bench.py: the one-GPU refusal, the algorithmic FLOP and
byte counts it divides by, and the committed counter summaries it reads."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2511_07343_amd.inputs import WORKLOADS  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_step_flops_workload2():
    """5.88e11 FLOP per fwd+bwd step at the headline workload: the per-token
    counts of the global (18dh + 36dh) and local memory (forward and backward
    formulas at C = 64) times B*H*L token-heads, less the last global chunk's
    chunk gradients and carry (14dh per token of that chunk), which feed only
    the final state."""
    cfg = WORKLOADS[2]
    d, h, C = cfg.d, cfg.hid, 64
    per_tok = (18 + 36) * d * h
    per_tok += 22 * d * h + 4 * C * (d + h) + 4 * d * d + 4 * C * d
    per_tok += 44 * d * h + 8 * C * h + 8 * C * d + 8 * C * d + 6 * d * d
    last = 14 * d * h * cfg.B * cfg.H * cfg.C_G
    assert bench.step_flops(cfg) == per_tok * cfg.B * cfg.H * cfg.L - last
    assert bench.step_flops(cfg) == pytest.approx(5.88e11, rel=2e-3)


def test_hbm_bytes_workload2():
    cfg = WORKLOADS[2]
    chains = cfg.B * cfg.H
    assert bench.hbm_bytes(cfg, "global_scan") == chains * (cfg.L * 36 + (cfg.L // cfg.C_G) * 16)
    st = 4 * cfg.hid * cfg.d * 4
    # operands, entry and exit state, and the next chunk's four bf16 state copies
    assert bench.hbm_bytes(cfg, "global_carry") == \
        chains * ((2 * cfg.hid + 4 * cfg.d) * cfg.C_G * 2 + 2 * st + 4 * cfg.hid * cfg.d * 2)
    assert bench.hbm_bytes(cfg, "local_bwd") is None


def test_committed_summaries_parse():
    """The committed traffic and MFMA summaries carry an entry for every launch
    label bench.py reports, with positive figures."""
    path = os.path.join(ROOT, "profiles", bench.TRAFFIC_FILE[2])
    labels = {}
    for line in open(path):
        t = line.split()
        if t and t[0] == "launch":
            labels[t[1]] = float(t[9])
    for lab in bench.LAUNCH_SOURCES:
        assert labels.get(lab, 0) > 0, lab
    mf = os.path.join(ROOT, "profiles", bench.MFMA_FILE[2])
    steps = [line.split() for line in open(mf) if line.startswith("step sha256")]
    assert len(steps) == 1 and float(steps[0][5]) > 0


def test_local_carry_bytes_workload2():
    """The local state carry's algorithmic bytes at the pre-training shape, by hand:
    128 units x 32 chunks, each reading K and V (64 x 64 bf16) and three gates
    (64 fp32), writing the bf16 entry state (4 x 256 x 64 + 64 x 64)."""
    cfg = WORKLOADS[2]
    per_chunk = 2 * 64 * 64 * 2 + 3 * 64 * 4 + (4 * 256 * 64 + 64 * 64) * 2
    cb = bench.local_carry_bytes(cfg)
    assert cb["alg_bytes"] == 128 * 32 * per_chunk == 640679936
    assert cb["spilled_state_bytes"] == 128 * 32 * 2 * 4 * 256 * 64 * 4
    assert bench.hbm_bytes(cfg, "local_carry") == cb["alg_bytes"]
