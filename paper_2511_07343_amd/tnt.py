"""ctypes binding of ``libtnt.so`` (see ``include/tnt.h``).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  Torch tensors provide device memory and the current HIP stream.
The functions named like the C entry points take tensors for the pointer
arguments; ``forward`` / ``backward`` also allocate outputs and workspaces.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import torch

from .inputs import BF16, LayerConfig

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtnt.so")
_lib = None

TNT_MAX_LOCAL = 4
TNT_WS_FWD, TNT_WS_BWD, TNT_WS_BWD_RECOMPUTE, TNT_WS_FWD_MIN = 0, 1, 2, 3
STATUS = {0: "TNT_OK", 1: "TNT_ERR_NULL", 2: "TNT_ERR_SHAPE", 3: "TNT_ERR_UNSUPPORTED",
          4: "TNT_ERR_WORKSPACE", 5: "TNT_ERR_ALIGN", 6: "TNT_ERR_HIP", 7: "TNT_ERR_ARG"}
EXPORTED = ["tnt_mem_workspace_size", "tnt_mem_saved_size", "tnt_mem_fwd", "tnt_mem_bwd",
            "tnt_strerror", "tnt_abi_version", "tnt_timing_enable", "tnt_timing_read",
            "tnt_mem_state_size", "tnt_mem_state_init", "tnt_mem_step", "tnt_mem_state_from_fwd",
            "tnt_dbg_chunk_grads", "tnt_set_kernel_family", "tnt_mem_fwd_noalloc"]
NOALLOC_WORKSPACE_BYTES = 128 << 20
FAMILY_DEFAULT, FAMILY_GENERIC, FAMILY_SINGLE_WALK = 0, 1, 2


class TntError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {STATUS.get(status, status)} ({strerror(status)})")
        self.status = status


class tnt_config(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("L", ctypes.c_int32),
                ("d", ctypes.c_int32), ("hid", ctypes.c_int32),
                ("has_global", ctypes.c_int32), ("C_G", ctypes.c_int32),
                ("n_local", ctypes.c_int32),
                ("C_L", ctypes.c_int32 * TNT_MAX_LOCAL), ("S_L", ctypes.c_int32 * TNT_MAX_LOCAL),
                ("act", ctypes.c_int32), ("qk_proj", ctypes.c_int32),
                ("qk_scope", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("global_intra", ctypes.c_int32)]


def lib(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the library; raises if it has not been built (no fallback)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or _LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2511_07343_amd.build`")
    L = ctypes.CDLL(p)
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
    cp = ctypes.POINTER(tnt_config)
    L.tnt_mem_workspace_size.argtypes = [cp, ctypes.c_int]
    L.tnt_mem_workspace_size.restype = sz
    L.tnt_mem_saved_size.argtypes = [cp]
    L.tnt_mem_saved_size.restype = sz
    L.tnt_mem_fwd.argtypes = [cp] + [vp] * 11 + [sz, vp, sz, vp]
    L.tnt_mem_fwd.restype = ctypes.c_int
    L.tnt_mem_bwd.argtypes = [cp] + [vp] * 10 + [sz] + [vp] * 9 + [sz, vp]
    L.tnt_mem_bwd.restype = ctypes.c_int
    L.tnt_mem_state_size.argtypes = [cp]
    L.tnt_mem_state_size.restype = sz
    L.tnt_mem_state_init.argtypes = [cp, vp, vp, vp, vp]
    L.tnt_mem_state_init.restype = ctypes.c_int
    L.tnt_mem_step.argtypes = [cp, ctypes.c_int64, i32] + [vp] * 11
    L.tnt_dbg_chunk_grads.argtypes = [cp, i32, i32, i32, i32] + [vp] * 8
    L.tnt_dbg_chunk_grads.restype = ctypes.c_int
    L.tnt_mem_state_from_fwd.argtypes = [cp] + [vp] * 5
    L.tnt_mem_state_from_fwd.restype = ctypes.c_int
    L.tnt_mem_step.restype = ctypes.c_int
    L.tnt_strerror.argtypes = [ctypes.c_int]
    L.tnt_strerror.restype = ctypes.c_char_p
    L.tnt_abi_version.argtypes = []
    L.tnt_abi_version.restype = i32
    L.tnt_mem_fwd_noalloc.argtypes = [cp] + [vp] * 11
    L.tnt_mem_fwd_noalloc.restype = ctypes.c_int
    L.tnt_set_kernel_family.argtypes = [i32]
    L.tnt_set_kernel_family.restype = i32
    L.tnt_timing_enable.argtypes = [i32]
    L.tnt_timing_enable.restype = i32
    L.tnt_timing_read.argtypes = [i32, ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(i32)]
    L.tnt_timing_read.restype = i32
    if path is None:
        _lib = L
    return L


def to_c(cfg: LayerConfig) -> tnt_config:
    c = tnt_config()
    c.B, c.H, c.L, c.d, c.hid = cfg.B, cfg.H, cfg.L, cfg.d, cfg.hid
    c.has_global, c.C_G, c.n_local = cfg.has_global, cfg.C_G, len(cfg.locals_)
    for i, (cl, sl) in enumerate(cfg.locals_):
        c.C_L[i], c.S_L[i] = cl, sl
    c.act, c.qk_proj, c.qk_scope, c.dtype = cfg.act, cfg.qk_proj, cfg.qk_scope, cfg.dtype
    c.global_intra = getattr(cfg, "global_intra", 0)
    return c


def strerror(status: int) -> str:
    return lib().tnt_strerror(status).decode()


def _p(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def tnt_mem_workspace_size(cfg: LayerConfig, kind: int) -> int:
    return lib().tnt_mem_workspace_size(ctypes.byref(to_c(cfg)), kind)


def tnt_mem_saved_size(cfg: LayerConfig) -> int:
    return lib().tnt_mem_saved_size(ctypes.byref(to_c(cfg)))


def _nbytes(t, given):
    if given is not None:
        return given
    if t is None or isinstance(t, int):
        return 0
    return t.numel() * t.element_size()


def tnt_mem_fwd(cfg, q, k, v, lr, mom, decay, W1_init, W2_init, o, final_state, saved,
                workspace, ws_bytes=None, stream=None, saved_bytes=None) -> int:
    ws_bytes = _nbytes(workspace, ws_bytes)
    c = to_c(cfg)
    return lib().tnt_mem_fwd(ctypes.byref(c), _p(q), _p(k), _p(v), _p(lr), _p(mom), _p(decay),
                             _p(W1_init), _p(W2_init), _p(o), _p(final_state), _p(saved),
                             _nbytes(saved, saved_bytes), _p(workspace), ws_bytes,
                             _stream(stream))


def tnt_mem_bwd(cfg, q, k, v, lr, mom, decay, W1_init, W2_init, dO, saved, dq, dk, dv, dlr,
                dmom, ddecay, dW1_init, dW2_init, workspace, ws_bytes=None, stream=None,
                saved_bytes=None) -> int:
    ws_bytes = _nbytes(workspace, ws_bytes)
    c = to_c(cfg)
    return lib().tnt_mem_bwd(ctypes.byref(c), _p(q), _p(k), _p(v), _p(lr), _p(mom), _p(decay),
                             _p(W1_init), _p(W2_init), _p(dO), _p(saved),
                             _nbytes(saved, saved_bytes), _p(dq), _p(dk), _p(dv), _p(dlr),
                             _p(dmom), _p(ddecay), _p(dW1_init), _p(dW2_init), _p(workspace),
                             ws_bytes, _stream(stream))


def tnt_mem_fwd_noalloc(cfg, q, k, v, lr, mom, decay, W1_init, W2_init, o, final_state,
                        stream=None) -> int:
    c = to_c(cfg)
    return lib().tnt_mem_fwd_noalloc(ctypes.byref(c), _p(q), _p(k), _p(v), _p(lr), _p(mom),
                                     _p(decay), _p(W1_init), _p(W2_init), _p(o),
                                     _p(final_state), _stream(stream))


def tnt_set_kernel_family(family: int) -> int:
    return lib().tnt_set_kernel_family(family)


class kernel_family:
    """Context manager: run the enclosed calls under another kernel family
    (tnt_set_kernel_family), restoring the previous one on exit."""

    def __init__(self, family: int):
        self.family = family
        self.prev = None

    def __enter__(self):
        self.prev = tnt_set_kernel_family(self.family)
        if self.prev < 0:
            raise ValueError(f"unknown kernel family {self.family}")
        return self

    def __exit__(self, *exc):
        tnt_set_kernel_family(self.prev)
        return False


def tnt_mem_state_size(cfg: LayerConfig) -> int:
    return lib().tnt_mem_state_size(ctypes.byref(to_c(cfg)))


def tnt_mem_state_init(cfg, W1_init, W2_init, state, stream=None) -> int:
    c = to_c(cfg)
    return lib().tnt_mem_state_init(ctypes.byref(c), _p(W1_init), _p(W2_init), _p(state),
                                    _stream(stream))


def tnt_dbg_chunk_grads(cfg, b, h, t0, C, k, v, W1, W2, Zk, R, D1, stream=None) -> int:
    c = to_c(cfg)
    return lib().tnt_dbg_chunk_grads(ctypes.byref(c), b, h, t0, C, _p(k), _p(v), _p(W1), _p(W2),
                                     _p(Zk), _p(R), _p(D1), _stream(stream))


def tnt_mem_state_from_fwd(cfg, final_state, W1_init, W2_init, state, stream=None) -> int:
    c = to_c(cfg)
    return lib().tnt_mem_state_from_fwd(ctypes.byref(c), _p(final_state), _p(W1_init),
                                        _p(W2_init), _p(state), _stream(stream))


def tnt_mem_step(cfg, pos, T, q, k, v, lr, mom, decay, W1_init, W2_init, state, o,
                 stream=None) -> int:
    c = to_c(cfg)
    return lib().tnt_mem_step(ctypes.byref(c), pos, T, _p(q), _p(k), _p(v), _p(lr), _p(mom),
                              _p(decay), _p(W1_init), _p(W2_init), _p(state), _p(o),
                              _stream(stream))


def tnt_timing_enable(on: bool) -> int:
    return lib().tnt_timing_enable(1 if on else 0)


def tnt_timing_read(max_entries: int = 64) -> Dict[str, tuple]:
    """{kernel name: (total ms, launches)} of the launches recorded while
    timing was enabled; clears the record."""
    names = ctypes.create_string_buffer(32 * max_entries)
    ms = (ctypes.c_double * max_entries)()
    cnt = (ctypes.c_int32 * max_entries)()
    n = lib().tnt_timing_read(max_entries, names, ms, cnt)
    if n < 0:
        raise RuntimeError("tnt_timing_read: HIP error")
    out = {}
    for i in range(n):
        nm = names.raw[32 * i: 32 * i + 32].split(b"\0", 1)[0].decode()
        out[nm] = (ms[i], cnt[i])
    return out


# --------------------------------------------------------------------------
# allocating wrappers
# --------------------------------------------------------------------------
def io_dtype(cfg: LayerConfig):
    return torch.bfloat16 if cfg.dtype == BF16 else torch.float32


def device_inputs(inp, cfg: LayerConfig, device="cuda") -> Dict[str, torch.Tensor]:
    """Copy host arrays (``inputs.LayerInputs``) to the device in the ABI's dtypes."""
    io = io_dtype(cfg)
    t = lambda a, dt: torch.from_numpy(a).to(device=device, dtype=dt).contiguous()
    return dict(q=t(inp.q, io), k=t(inp.k, io), v=t(inp.v, io), dO=t(inp.dO, io),
                lr=t(inp.lr, torch.float32), mom=t(inp.mom, torch.float32),
                decay=t(inp.decay, torch.float32), W1=t(inp.W1, torch.float32),
                W2=t(inp.W2, torch.float32))


def _bytes(n: int, device) -> torch.Tensor:
    return torch.empty(max(n, 16), dtype=torch.uint8, device=device)


def forward(cfg: LayerConfig, x: Dict[str, torch.Tensor], save: bool = True,
            final_state: bool = False, workspace: Optional[torch.Tensor] = None,
            stream=None):
    """Run tnt_mem_fwd; returns (o, saved or None, final_state or None)."""
    dev = x["q"].device
    o = torch.empty_like(x["q"])
    saved = _bytes(tnt_mem_saved_size(cfg), dev) if save else None
    fin = (torch.empty(cfg.B, cfg.H, 4, cfg.hid * cfg.d, dtype=torch.float32, device=dev)
           if final_state else None)
    if workspace is None:
        workspace = _bytes(tnt_mem_workspace_size(cfg, TNT_WS_FWD), dev)
    st = tnt_mem_fwd(cfg, x["q"], x["k"], x["v"], x["lr"], x["mom"], x["decay"], x["W1"],
                     x["W2"], o, fin, saved, workspace, stream=stream)
    if st != 0:
        raise TntError(st, "tnt_mem_fwd")
    return o, saved, fin


def backward(cfg: LayerConfig, x: Dict[str, torch.Tensor], dO: torch.Tensor,
             saved: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
             stream=None) -> Dict[str, torch.Tensor]:
    """Run tnt_mem_bwd; returns the gradients of sum(dO * o)."""
    dev = x["q"].device
    g = dict(dq=torch.empty_like(x["q"]), dk=torch.empty_like(x["k"]),
             dv=torch.empty_like(x["v"]), dlr=torch.empty_like(x["lr"]),
             dmom=torch.empty_like(x["mom"]), ddecay=torch.empty_like(x["decay"]),
             dW1=torch.empty_like(x["W1"]), dW2=torch.empty_like(x["W2"]))
    if workspace is None:
        kind = TNT_WS_BWD if saved is not None else TNT_WS_BWD_RECOMPUTE
        workspace = _bytes(tnt_mem_workspace_size(cfg, kind), dev)
    st = tnt_mem_bwd(cfg, x["q"], x["k"], x["v"], x["lr"], x["mom"], x["decay"], x["W1"],
                     x["W2"], dO, saved, g["dq"], g["dk"], g["dv"], g["dlr"], g["dmom"],
                     g["ddecay"], g["dW1"], g["dW2"], workspace, stream=stream)
    if st != 0:
        raise TntError(st, "tnt_mem_bwd")
    return g


def step_forward(cfg: LayerConfig, x: Dict[str, torch.Tensor], pieces, state=None, pos: int = 0,
                 stream=None):
    """Feed the sequence in ``x`` through tnt_mem_step in consecutive pieces of
    the given lengths (starting at token ``pos`` of ``x`` with ``state``, or
    from a fresh state); returns (o of the fed tokens [B,H,sum(pieces),d], state)."""
    dev = x["q"].device
    if state is None:
        state = _bytes(tnt_mem_state_size(cfg), dev)
        st = tnt_mem_state_init(cfg, x["W1"], x["W2"], state, stream=stream)
        if st != 0:
            raise TntError(st, "tnt_mem_state_init")
    outs = []
    t0 = pos
    for T in pieces:
        sl = slice(t0, t0 + T)
        # fresh copies: a slice that is already contiguous would be an offset
        # view, not 16-byte aligned in general
        cp = lambda t: t.clone(memory_format=torch.contiguous_format)
        q, k, v = (cp(x[n][:, :, sl]) for n in ("q", "k", "v"))
        lr, mom, dec = (cp(x[n][..., sl]) for n in ("lr", "mom", "decay"))
        o = torch.empty_like(q)
        st = tnt_mem_step(cfg, t0, T, q, k, v, lr, mom, dec, x["W1"], x["W2"], state, o,
                          stream=stream)
        if st != 0:
            raise TntError(st, "tnt_mem_step")
        outs.append(o)
        t0 += T
    return torch.cat(outs, 2), state
