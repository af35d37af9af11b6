"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

from paper_2511_07343_amd import tnt
from paper_2511_07343_amd.inputs import WORKLOADS, small_config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "tnt.h")).read()
    return sorted(set(re.findall(r"\b(tnt_[a-z_]+)\s*\(", src)))


def test_header_symbols_exported():
    L = tnt.lib()
    names = _declared()
    assert set(tnt.EXPORTED) <= set(names)
    for n in names:
        assert hasattr(L, n), n


def _param_counts():
    src = open(os.path.join(ROOT, "include", "tnt.h")).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    out = {}
    for m in re.finditer(r"\b(tnt_[a-z_]+)\s*\(([^;{]*?)\)\s*;", src, re.S):
        args = m.group(2).strip()
        out[m.group(1)] = 0 if args in ("", "void") else args.count(",") + 1
    return out


def test_binding_argument_counts_match_header():
    L = tnt.lib()
    counts = _param_counts()
    for name in tnt.EXPORTED:
        fn = getattr(L, name)
        assert len(fn.argtypes) == counts[name], name


def test_abi_version():
    assert tnt.lib().tnt_abi_version() == 2


def test_strerror_names():
    for s in range(8):
        assert tnt.strerror(s)


@pytest.mark.parametrize("cfg", WORKLOADS, ids=lambda c: c.name.split()[0] + str(c.L))
def test_workspace_sizes_positive(cfg):
    assert tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_FWD_MIN) > 0
    # the full forward workspace adds the no-save two-pass forward's state copies
    assert tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_FWD) >= \
        tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_FWD_MIN)
    assert tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_BWD) > \
        tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_FWD_MIN)
    assert tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_BWD_RECOMPUTE) >= \
        tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_BWD) + tnt.tnt_mem_saved_size(cfg)
    assert tnt.tnt_mem_saved_size(cfg) > 0


def _fwd_status(cfg, ptr=256, ws=1 << 40):
    p = ptr
    return tnt.tnt_mem_fwd(cfg, p, p, p, p, p, p, p, p, p, None, None, p, ws_bytes=ws, stream=0)


@pytest.mark.parametrize("bad,code", [
    (dict(L=100), 2),                      # L % C_G
    (dict(locals_=((8, 12),)), 2),         # S_L % C_L
    (dict(locals_=((8, 48),)), 2),         # L % S_L
    (dict(d=24), 3),
    (dict(hid=48), 3),
    (dict(locals_=((80, 160),), L=320, C_G=64), 3),
    (dict(act=5), 7),
    (dict(qk_scope=2), 7),
    (dict(B=0), 2),
    (dict(has_global=0, locals_=()), 2),
    (dict(global_intra=2), 7),
])
def test_validation_codes(bad, code):
    cfg = small_config(L=64, C_G=16, locals_=((8, 32),)).replace(**bad)
    assert _fwd_status(cfg) == code


def test_null_and_alignment_and_workspace():
    cfg = small_config(L=64, C_G=16, locals_=((8, 32),))
    assert _fwd_status(cfg, ptr=0) == 1
    assert _fwd_status(cfg, ptr=258) == 5
    assert _fwd_status(cfg, ws=16) == 4
    # final_state without a global memory is a shape error
    c = tnt.to_c(cfg.replace(has_global=0))
    st = tnt.lib().tnt_mem_fwd(ctypes.byref(c), *([256] * 9), 256, None, 0, 256, 1 << 40, None)
    assert st == 2


def test_saved_buffer_size_and_record_checked_before_launch():
    """A saved buffer smaller than tnt_mem_saved_size is refused by the
    forward (TNT_ERR_WORKSPACE); a backward given a buffer that no forward of
    this process wrote for this configuration and kernel family is refused
    (TNT_ERR_ARG).  Both before anything is enqueued (no GPU here)."""
    cfg = small_config(L=64, C_G=16, locals_=((8, 32),))
    p = 256
    need = tnt.tnt_mem_saved_size(cfg)
    st = tnt.tnt_mem_fwd(cfg, p, p, p, p, p, p, p, p, p, None, p, p, ws_bytes=1 << 40, stream=0,
                         saved_bytes=need - 16)
    assert st == 4
    args = [p] * 10
    st = tnt.tnt_mem_bwd(cfg, *args[:9], 4096, *([p] * 8), p, ws_bytes=1 << 40, stream=0,
                         saved_bytes=need)
    assert st == 7


def test_kernel_family_setting():
    assert tnt.tnt_set_kernel_family(-1) == -1
    assert tnt.tnt_set_kernel_family(3) == -1
    prev = tnt.tnt_set_kernel_family(tnt.FAMILY_GENERIC)
    assert prev == tnt.FAMILY_DEFAULT
    assert tnt.tnt_set_kernel_family(prev) == tnt.FAMILY_GENERIC


def test_saved_size_reserves_only_the_fp32_ring():
    """At the pre-training workload the default family's local walk keeps its
    fp32 carry in a two-slot ring per unit (the backward reads the compute-type
    copies), so the saved buffer reserves two fp32 slots per unit instead of one
    per chunk boundary: 128 units x 31 slots x 256 KB less than the families
    that read every fp32 slot."""
    cfg = WORKLOADS[2]
    small = tnt.tnt_mem_saved_size(cfg)
    with tnt.kernel_family(tnt.FAMILY_SINGLE_WALK):
        full = tnt.tnt_mem_saved_size(cfg)
    units = cfg.B * cfg.H * (cfg.L // cfg.locals_[0][1])
    chunks = cfg.locals_[0][1] // cfg.locals_[0][0]
    slot = 4 * cfg.hid * cfg.d * 4
    assert full - small == units * (chunks + 1 - 2) * slot
    assert full - small > 1.0e9


# ---------------------------------------------------------------- step-wise entry points
def test_state_size_formula():
    cfg = WORKLOADS[3]  # global + two locals, d 64, hid 256
    M = cfg.has_global + len(cfg.locals_)
    per = 6 * cfg.hid * cfg.d + cfg.d * cfg.d
    G = cfg.hid // min(64, cfg.hid)
    scratch = -(-(2 * cfg.hid + cfg.d + 3 * G * cfg.d) // 64) * 64
    assert tnt.tnt_mem_state_size(cfg) == M * cfg.B * cfg.H * (per + scratch) * 4


def test_state_size_ignores_L():
    """The step-wise calls take an open-ended sequence: L need not be a
    multiple of the chunk or shard sizes."""
    cfg = small_config(L=1)
    assert tnt.tnt_mem_state_size(cfg) > 0
    assert tnt.tnt_mem_state_size(small_config(d=24)) == 0


@pytest.mark.parametrize("bad,code", [
    (dict(locals_=((8, 12),)), 2),         # S_L % C_L
    (dict(d=24), 3),
    (dict(act=5), 7),
    (dict(B=0), 2),
])
def test_step_rejects_bad_config(bad, code):
    import dataclasses
    cfg = dataclasses.replace(small_config(), **bad)
    p = 256
    assert tnt.tnt_mem_step(cfg, 0, 4, p, p, p, p, p, p, p, p, p, p, stream=0) == code
    assert tnt.tnt_mem_state_init(cfg, p, p, p, stream=0) == code


def test_step_rejects_bad_arguments():
    cfg = small_config()
    p = 256
    assert tnt.tnt_mem_step(cfg, -1, 4, p, p, p, p, p, p, p, p, p, p, stream=0) == 2
    assert tnt.tnt_mem_step(cfg, 0, -1, p, p, p, p, p, p, p, p, p, p, stream=0) == 2
    assert tnt.tnt_mem_step(cfg, 0, 4, p, p, p, p, p, p, p, p, None, p, stream=0) == 1
    assert tnt.tnt_mem_step(cfg, 0, 4, p + 8, p, p, p, p, p, p, p, p, p, stream=0) == 5
    assert tnt.tnt_mem_state_init(cfg, p, p, None, stream=0) == 1
    # T == 0 enqueues nothing and succeeds without touching the pointers
    assert tnt.tnt_mem_step(cfg, 0, 0, p, p, p, p, p, p, p, p, p, p, stream=0) == 0


def test_state_from_fwd_validation():
    cfg = small_config()  # has a global memory
    p = 256
    assert tnt.tnt_mem_state_from_fwd(cfg, None, p, p, p, stream=0) == 1
    import dataclasses
    assert tnt.tnt_mem_state_from_fwd(dataclasses.replace(cfg, L=100), p, p, p, p, stream=0) == 2
    assert tnt.tnt_mem_state_from_fwd(cfg, p + 4, p, p, p, stream=0) == 5


def test_dbg_chunk_grads_validation():
    cfg = small_config()  # B1 H2 L64
    p = 256
    args = (p,) * 7
    assert tnt.tnt_dbg_chunk_grads(cfg, 1, 0, 0, 8, *args, stream=0) == 2     # b >= B
    assert tnt.tnt_dbg_chunk_grads(cfg, 0, 2, 0, 8, *args, stream=0) == 2     # h >= H
    assert tnt.tnt_dbg_chunk_grads(cfg, 0, 0, 60, 8, *args, stream=0) == 2    # t0 + C > L
    assert tnt.tnt_dbg_chunk_grads(cfg, 0, 0, 0, 65, *args, stream=0) == 2    # C > 64
    assert tnt.tnt_dbg_chunk_grads(cfg, 0, 0, 0, 8, None, *args[1:], stream=0) == 1


def test_global_intra_limits():
    """The intra-chunk reading of the global memory runs as one more local-style
    memory: with four locals it is unsupported, and the step-wise calls do not
    take it (chunk-parallel calls only)."""
    cfg = small_config(L=64, C_G=16, locals_=((8, 32),), global_intra=1)
    assert tnt.tnt_mem_workspace_size(cfg, tnt.TNT_WS_FWD) > 0
    assert tnt.tnt_mem_saved_size(cfg) > 0
    full = cfg.replace(locals_=((8, 32),) * 4)
    assert _fwd_status(full) == 3
    assert tnt.tnt_mem_state_size(cfg) == 0
    p = 256
    assert tnt.tnt_mem_step(cfg, 0, 4, p, p, p, p, p, p, p, p, p, p, stream=0) == 3
    assert tnt.tnt_mem_state_from_fwd(cfg, p, p, p, p, stream=0) == 3
    # without a global memory the flag is ignored
    assert tnt.tnt_mem_saved_size(cfg.replace(has_global=0)) == \
        tnt.tnt_mem_saved_size(cfg.replace(has_global=0, global_intra=0))
