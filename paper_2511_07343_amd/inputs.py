"""Seeded synthetic workloads for the TNT memory layer.

This module holds the shapes of the five workloads and the seeded generator
that draws their inputs.  It contains none of the method's arithmetic: it only
draws random numbers, normalises q/k (and v for the fp32 smoke shape) to unit
length and rounds to bf16 where the workload computes in bf16.  Both the HIP
path (through the tests and the benchmark) and the fp64 oracle are fed from
here; neither of them imports the other.

Draw order for a workload with seed ``s`` (fixed, so every consumer sees the
same numbers):

1. ``rng = numpy.random.default_rng(s)``; q, k, v ~ N(0, 1), shape [B,H,L,d],
   drawn in that order.
2. q and k are divided by their per-token L2 norm (v too when ``norm_v``).
3. For each memory m (memory 0 is the global one when present), in order:
   lr ~ U(0.01, 0.1), mom ~ U(0.8, 0.95), decay ~ U(0, 0.01), shape [B,H,L].
4. For each memory: W1 ~ N(0, 2/(d+h)) shape [H,h,d], then W2 ~ N(0, 2/(d+h))
   shape [H,d,h] (Xavier-normal).
5. dO ~ N(0, 1), shape [B,H,L,d], from ``default_rng(s + 1000)``.
6. For bf16 workloads q, k, v and dO are rounded to bf16 (nearest-even) after
   normalisation; gates and initial weights stay fp32.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Tuple

import numpy as np

ACT_GELU = 0
ACT_SILU = 1
F32 = 0
BF16 = 1
QK_SHARD = 0
QK_CHUNK = 1


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """Shape and schedule of one TNT memory layer call.

    ``locals_`` lists (C_L, S_L) per local memory.  Memory 0 is the global
    memory when ``has_global``; local memory i is memory ``has_global + i``.
    """

    B: int
    H: int
    L: int
    d: int
    hid: int
    C_G: int
    locals_: Tuple[Tuple[int, int], ...]
    act: int = ACT_SILU
    dtype: int = BF16
    has_global: int = 1
    qk_proj: int = 1
    qk_scope: int = QK_SHARD
    norm_v: bool = False
    name: str = ""
    # retrieval of the global memory: 0 = at the chunk-entry state (Sec. 4.1.2
    # box), 1 = after each token's own update (Sec. 2.2 chunkwise retrieval)
    global_intra: int = 0

    @property
    def n_local(self) -> int:
        return len(self.locals_)

    @property
    def M(self) -> int:
        return self.has_global + self.n_local

    @property
    def tokens(self) -> int:
        return self.B * self.L

    def replace(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


# The five workloads.  Shapes follow the paper's efficiency setup (global chunk
# 2048, local shards 2048/4096, 2k-32k contexts) at single-layer scale.
WORKLOADS: List[LayerConfig] = [
    LayerConfig(B=1, H=1, L=256, d=16, hid=32, C_G=64, locals_=((8, 64),),
                act=ACT_GELU, dtype=F32, norm_v=True,
                name="fp32 smoke B1 H1 L256 d16 h32 CG64 CL8 SL64"),
    LayerConfig(B=2, H=4, L=2048, d=64, hid=256, C_G=256, locals_=((16, 256),),
                act=ACT_SILU, dtype=BF16,
                name="bf16 B2 H4 L2048 d64 h256 CG256 CL16 SL256"),
    LayerConfig(B=4, H=8, L=8192, d=64, hid=256, C_G=2048, locals_=((64, 2048),),
                act=ACT_SILU, dtype=BF16,
                name="bf16 pre-train B4 H8 L8192 d64 h256 CG2048 CL64 SL2048"),
    LayerConfig(B=4, H=8, L=8192, d=64, hid=256, C_G=2048,
                locals_=((16, 1024), (32, 1024)), act=ACT_SILU, dtype=BF16,
                name="bf16 two locals B4 H8 L8192 d64 h256 CG2048 CL16,32 SL1024"),
    LayerConfig(B=1, H=16, L=32768, d=128, hid=512, C_G=4096, locals_=((64, 4096),),
                act=ACT_SILU, dtype=BF16,
                name="bf16 long B1 H16 L32768 d128 h512 CG4096 CL64 SL4096"),
]


@dataclasses.dataclass
class LayerInputs:
    """Host arrays of one call (numpy).  Floating arrays are float32; for bf16
    workloads q/k/v/dO hold bf16-representable float32 values."""

    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    lr: np.ndarray      # [M,B,H,L]
    mom: np.ndarray     # [M,B,H,L]
    decay: np.ndarray   # [M,B,H,L]
    W1: np.ndarray      # [M,H,hid,d]
    W2: np.ndarray      # [M,H,d,hid]
    dO: np.ndarray      # [B,H,L,d]


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    nan = np.isnan(x)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out


def _unit(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def make_inputs(cfg: LayerConfig, seed: int,
                lr_range=(0.01, 0.1), mom_range=(0.8, 0.95),
                decay_range=(0.0, 0.01)) -> LayerInputs:
    """Draw the inputs of ``cfg`` with ``seed`` in the fixed order above."""
    B, H, L, d, h, M = cfg.B, cfg.H, cfg.L, cfg.d, cfg.hid, cfg.M
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, H, L, d))
    k = rng.standard_normal((B, H, L, d))
    v = rng.standard_normal((B, H, L, d))
    q = _unit(q)
    k = _unit(k)
    if cfg.norm_v:
        v = _unit(v)
    lr = np.empty((M, B, H, L))
    mom = np.empty((M, B, H, L))
    decay = np.empty((M, B, H, L))
    for m in range(M):
        lr[m] = rng.uniform(lr_range[0], lr_range[1], (B, H, L))
        mom[m] = rng.uniform(mom_range[0], mom_range[1], (B, H, L))
        decay[m] = rng.uniform(decay_range[0], decay_range[1], (B, H, L))
    std = np.sqrt(2.0 / (d + h))
    W1 = np.empty((M, H, h, d))
    W2 = np.empty((M, H, d, h))
    for m in range(M):
        W1[m] = rng.normal(0.0, std, (H, h, d))
        W2[m] = rng.normal(0.0, std, (H, d, h))
    dO = np.random.default_rng(seed + 1000).standard_normal((B, H, L, d))
    f32 = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    q, k, v, dO = f32(q), f32(k), f32(v), f32(dO)
    if cfg.dtype == BF16:
        q, k, v, dO = round_bf16(q), round_bf16(k), round_bf16(v), round_bf16(dO)
    return LayerInputs(q=q, k=k, v=v, lr=f32(lr), mom=f32(mom), decay=f32(decay),
                       W1=f32(W1), W2=f32(W2), dO=dO)


def workload(idx: int) -> LayerConfig:
    return WORKLOADS[idx]


def max_rel_err(x: np.ndarray, ref: np.ndarray) -> float:
    """max_i |x_i - ref_i| / max_i |ref_i| (0 when both are all zero)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(x - ref))) if ref.size else 0.0
    if den == 0.0:
        return num
    return num / den


def small_config(dtype: int = F32, act: int = ACT_GELU, *, B=1, H=2, L=64, d=16,
                 hid=32, C_G=16, locals_=((8, 32),), has_global=1, qk_proj=1,
                 qk_scope=QK_SHARD, norm_v=False, global_intra=0,
                 name: Optional[str] = None) -> LayerConfig:
    """A small shape for CPU tests and multi-tile GPU parity cases."""
    return LayerConfig(B=B, H=H, L=L, d=d, hid=hid, C_G=C_G, locals_=tuple(locals_),
                       act=act, dtype=dtype, has_global=has_global, qk_proj=qk_proj,
                       qk_scope=qk_scope, norm_v=norm_v, global_intra=global_intra,
                       name=name or f"small B{B} H{H} L{L} d{d} h{hid}")
