"""Plain fp64 CPU oracle of one TNT memory layer (forward and backward).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  It shares
no code with the HIP path and imports nothing from the package.

What it computes (paper: "TNT: Improving Chunkwise Training for Test-Time
Memorization", arXiv 2511.07343), per (batch, head) chain, in fp64:

* Memory module f(W, x) = W2 sigma(W1 x), W1 in R^{h x d}, W2 in R^{d x h}
  (Sec. 2.1, "deep memory modules"; no bias / residual / norm).
* Inner loss l(W; k, v) = (1/d) ||f(W, k) - v||^2, the mean squared error that
  Sec. 2.1 names, averaged over the d output components, and its gradient
  u = grad_W l (``inner_grad``).
* Chunkwise rule (Sec. 2.2, chunkwise compression / retrieval equations): every
  token of a chunk takes its gradient at the chunk-entry state.
* Momentum and decay (App. D defers the gating to Titans): with u_t taken at
  the chunk-entry state, S_t = beta_t S_{t-1} - eta_t u_t and
  W_t = (1 - alpha_t) W_{t-1} + S_t.  beta = alpha = 0 is the paper's plain rule.
* Global memory (Sec. 4.1.1 box, global update; App. E general form): chunks
  of C_G, state carried across chunks, never reset; retrieval at the
  chunk-entry state V_{xi(t, C_G)} (Sec. 4.1.2 box; App. E retrieval rule).
  ``intra=True`` takes the other reading: the chunkwise retrieval rule of
  Sec. 2.2 applied to the global memory, o_t = f(V_t, q_t) with V_t the state
  after token t's own update (gradients still at the chunk-entry state).
* Local memories (Sec. 4.1.1 box, local update; App. E): chunks of C_L, state
  reset to the learned init (and momentum to zero) every S_L tokens; retrieval
  at W_t, i.e. after token t's own update (Sec. 2.1 / 2.2 retrieval rules).
* Q-K projection (Sec. 4.1.2; App. C): local memory i is queried at
  x_t = M_t q_t, M_t = sum of k k^T / ||k||^2 over the tokens since the last
  shard start up to and including t (the appendix's running sum with reset);
  ``qk_scope='chunk'`` takes the sum from the chunk start instead, which is the
  literal reading of the retrieval box.
* Output o_t = f(V_{xi(t,C_G)}, q_t) + sum_i f(W^(i)_t, x^(i)_t)
  (Sec. 4.1.2 box; App. E generalised retrieval rule).

Tokens are 0-indexed: the chunk of size C holding token t starts at
xi(t, C) = t - (t mod C) (Sec. 1, notation).  The backward pass is autograd of
sum <dO, o> through this forward, with full second-order terms (the inner
gradient is differentiated, never stopped); chunk-level checkpointing only
bounds memory.

Every function here is pinned by tests under ``tests/test_oracle_*.py``
(finite differences, closed forms, the per-token rule, brute-force sums,
shard isolation, gradcheck).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch
import torch.utils.checkpoint as _ckpt

DT = torch.float64
_SQRT2 = math.sqrt(2.0)
_INV_SQRT_2PI = 1.0 / math.sqrt(2.0 * math.pi)


# --------------------------------------------------------------------------
# activation and memory module (Sec. 2.1)
# --------------------------------------------------------------------------
def act(z: torch.Tensor, kind: str) -> torch.Tensor:
    """sigma(z): exact (erf) GELU or SiLU."""
    if kind == "gelu":
        return 0.5 * z * (1.0 + torch.erf(z / _SQRT2))
    if kind == "silu":
        return z * torch.sigmoid(z)
    raise ValueError(kind)


def act_grad(z: torch.Tensor, kind: str) -> torch.Tensor:
    """sigma'(z), written out by hand (differentiable, so the outer backward
    sees second-order terms)."""
    if kind == "gelu":
        cdf = 0.5 * (1.0 + torch.erf(z / _SQRT2))
        pdf = torch.exp(-0.5 * z * z) * _INV_SQRT_2PI
        return cdf + z * pdf
    if kind == "silu":
        s = torch.sigmoid(z)
        return s + z * s * (1.0 - s)
    raise ValueError(kind)


def memory_fn(W1: torch.Tensor, W2: torch.Tensor, x: torch.Tensor, kind: str) -> torch.Tensor:
    """f(W, x) = W2 sigma(W1 x); W1 [...,h,d], W2 [...,d,h], x [...,d] -> [...,d]."""
    z = torch.einsum("...hd,...d->...h", W1, x)
    return torch.einsum("...dh,...h->...d", W2, act(z, kind))


def recall_loss(W1, W2, k, v, kind) -> torch.Tensor:
    """l(W; k, v) = (1/d) ||f(W, k) - v||^2 (mean over the last axis)."""
    e = memory_fn(W1, W2, k, kind) - v
    return (e * e).mean(-1)


def inner_grad(W1, W2, k, v, kind) -> Tuple[torch.Tensor, torch.Tensor]:
    """u = grad_W (1/d) ||f(W,k) - v||^2 written out by the chain rule.

    z = W1 k, a = sigma(z), y = W2 a, r = (2/d) (y - v);
    dl/dW2 = r a^T;  dl/dW1 = ((W2^T r) * sigma'(z)) k^T.
    Leading axes broadcast (W [P,1,h,d] with k [P,C,d] gives one gradient
    per token, all at the same W).
    """
    z = torch.einsum("...hd,...d->...h", W1, k)
    a = act(z, kind)
    y = torch.einsum("...dh,...h->...d", W2, a)
    r = (2.0 / v.shape[-1]) * (y - v)
    g2 = r[..., :, None] * a[..., None, :]
    back = torch.einsum("...dh,...d->...h", W2, r) * act_grad(z, kind)
    g1 = back[..., :, None] * k[..., None, :]
    return g1, g2


def _bc(x: torch.Tensor) -> torch.Tensor:
    return x[:, None, None]


def _gated_step(W1, W2, S1, S2, g1, g2, eta, beta, alpha):
    """One token of the gated inner optimiser (momentum S, decay alpha)."""
    S1 = _bc(beta) * S1 - _bc(eta) * g1
    S2 = _bc(beta) * S2 - _bc(eta) * g2
    W1 = _bc(1.0 - alpha) * W1 + S1
    W2 = _bc(1.0 - alpha) * W2 + S2
    return W1, W2, S1, S2


# --------------------------------------------------------------------------
# global memory (Sec. 4.1.1 global update, Sec. 4.1.2 retrieval at V_xi)
# --------------------------------------------------------------------------
def _global_retrieve(V1, V2, q, kind):
    """f(V_hat, q_t) for every token of a chunk, V_hat = chunk-entry state."""
    z = torch.einsum("phd,pcd->pch", V1, q)
    return torch.einsum("pdh,pch->pcd", V2, act(z, kind))


def _global_accumulate(V1, V2, S1, S2, V1h, V2h, k, v, eta, beta, alpha, kind):
    """Gated accumulation of the tokens of (part of) a global chunk, every
    gradient taken at the chunk-entry state (V1h, V2h)."""
    g1, g2 = inner_grad(V1h[:, None], V2h[:, None], k, v, kind)
    for i in range(k.shape[1]):
        V1, V2, S1, S2 = _gated_step(V1, V2, S1, S2, g1[:, i], g2[:, i],
                                     eta[:, i], beta[:, i], alpha[:, i])
    return V1, V2, S1, S2


def _global_accumulate_intra(V1, V2, S1, S2, V1h, V2h, q, k, v, eta, beta, alpha, kind):
    """As ``_global_accumulate``, and after each token's update the memory is
    read at the updated state: o_t = f(V_t, q_t) (Sec. 2.2 chunkwise retrieval
    rule, the intra-chunk reading of the global memory)."""
    g1, g2 = inner_grad(V1h[:, None], V2h[:, None], k, v, kind)
    outs = []
    for i in range(k.shape[1]):
        V1, V2, S1, S2 = _gated_step(V1, V2, S1, S2, g1[:, i], g2[:, i],
                                     eta[:, i], beta[:, i], alpha[:, i])
        outs.append(memory_fn(V1, V2, q[:, i], kind))
    return V1, V2, S1, S2, torch.stack(outs, 1)


def global_memory(q, k, v, eta, beta, alpha, W1, W2, C_G: int, kind: str,
                  ckpt: bool = False, block: int = 64, states: Optional[list] = None,
                  intra: bool = False):
    """Global memory of every chain.  q,k,v [P,L,d]; gates [P,L]; W1 [P,h,d].

    Returns (o [P,L,d], (V1, V2, S1, S2) after the last token).  When
    ``states`` is a list, the chunk-entry states are appended to it.  A chunk's
    tokens are accumulated in sub-blocks of ``block`` tokens (a bound on the
    size of the batched gradient only: every sub-block takes its gradients at
    the chunk-entry state).  ``intra``: retrieval after each token's update
    instead of at the chunk-entry state.
    """
    P, L, d = q.shape
    if L % C_G:
        raise ValueError("L must be a multiple of C_G")
    V1, V2 = W1, W2
    S1 = torch.zeros_like(W1)
    S2 = torch.zeros_like(W2)
    outs = []
    for n in range(L // C_G):
        t0 = n * C_G
        V1h, V2h = V1, V2
        if states is not None:
            states.append((V1, V2, S1, S2))
        if not intra:
            outs.append(_global_retrieve(V1h, V2h, q[:, t0:t0 + C_G], kind))
        for b0 in range(t0, t0 + C_G, block):
            b1 = min(b0 + block, t0 + C_G)
            if intra:
                args = (V1, V2, S1, S2, V1h, V2h, q[:, b0:b1], k[:, b0:b1], v[:, b0:b1],
                        eta[:, b0:b1], beta[:, b0:b1], alpha[:, b0:b1], kind)
                fn = _global_accumulate_intra
            else:
                args = (V1, V2, S1, S2, V1h, V2h, k[:, b0:b1], v[:, b0:b1],
                        eta[:, b0:b1], beta[:, b0:b1], alpha[:, b0:b1], kind)
                fn = _global_accumulate
            res = (_ckpt.checkpoint(fn, *args, use_reentrant=False) if ckpt else fn(*args))
            V1, V2, S1, S2 = res[:4]
            if intra:
                outs.append(res[4])
    return torch.cat(outs, 1), (V1, V2, S1, S2)


# --------------------------------------------------------------------------
# local memories (Sec. 4.1.1 local update with reset, Sec. 4.1.2 Q-K projection)
# --------------------------------------------------------------------------
def _local_chunk(W1, W2, S1, S2, Mq, q, k, v, eta, beta, alpha, kind, qk_proj):
    """One local chunk: gradients at the chunk-entry state, per-token gated
    update, Q-K running sum including token t, retrieval at W_t."""
    g1, g2 = inner_grad(W1[:, None], W2[:, None], k, v, kind)   # all at the entry state
    outs = []
    for i in range(k.shape[1]):
        W1, W2, S1, S2 = _gated_step(W1, W2, S1, S2, g1[:, i], g2[:, i],
                                     eta[:, i], beta[:, i], alpha[:, i])
        kt = k[:, i]
        Mq = Mq + kt[:, :, None] * kt[:, None, :] / (kt * kt).sum(-1)[:, None, None]
        x = torch.einsum("pde,pe->pd", Mq, q[:, i]) if qk_proj else q[:, i]
        outs.append(memory_fn(W1, W2, x, kind))
    return W1, W2, S1, S2, Mq, torch.stack(outs, 1)


def local_memory(q, k, v, eta, beta, alpha, W1i, W2i, C_L: int, S_L: int, kind: str,
                 qk_proj: bool = True, qk_scope: str = "shard", ckpt: bool = False,
                 shards: Optional[Sequence[int]] = None, final: Optional[list] = None):
    """One local memory over every chain.  Returns o [P,L,d] (zero outside the
    requested ``shards`` when a subset is given)."""
    P, L, d = q.shape
    if L % S_L or S_L % C_L:
        raise ValueError("need S_L | L and C_L | S_L")
    wanted = set(range(L // S_L)) if shards is None else set(shards)
    per_shard = []
    for s in range(L // S_L):
        if s not in wanted:
            per_shard.append(torch.zeros(P, S_L, d, dtype=q.dtype))
            continue
        W1, W2 = W1i, W2i                      # reset to the learned init
        S1 = torch.zeros_like(W1i)
        S2 = torch.zeros_like(W2i)
        Mq = torch.zeros(P, d, d, dtype=q.dtype)
        chunks = []
        for c0 in range(s * S_L, (s + 1) * S_L, C_L):
            if qk_scope == "chunk":
                Mq = torch.zeros(P, d, d, dtype=q.dtype)
            sl = slice(c0, c0 + C_L)
            args = (W1, W2, S1, S2, Mq, q[:, sl], k[:, sl], v[:, sl],
                    eta[:, sl], beta[:, sl], alpha[:, sl], kind, qk_proj)
            if ckpt:
                W1, W2, S1, S2, Mq, o = _ckpt.checkpoint(_local_chunk, *args, use_reentrant=False)
            else:
                W1, W2, S1, S2, Mq, o = _local_chunk(*args)
            chunks.append(o)
        per_shard.append(torch.cat(chunks, 1))
        if final is not None:
            final.append((W1, W2, S1, S2, Mq))
    return torch.cat(per_shard, 1)


# --------------------------------------------------------------------------
# the layer
# --------------------------------------------------------------------------
_ACT_NAMES = {0: "gelu", 1: "silu"}


def _kind(cfg) -> str:
    a = getattr(cfg, "act")
    return _ACT_NAMES[a] if isinstance(a, int) else a


def _intra(cfg) -> bool:
    return bool(getattr(cfg, "global_intra", 0))


def _scope(cfg) -> str:
    s = getattr(cfg, "qk_scope", 0)
    return {0: "shard", 1: "chunk"}[s] if isinstance(s, int) else s


def layer_forward(q, k, v, lr, mom, decay, W1, W2, cfg, ckpt: bool = False,
                  shards: Optional[Sequence[int]] = None, with_final: bool = False):
    """o for every chain.  q,k,v [P,L,d]; lr/mom/decay [M,P,L] (eta, beta,
    alpha); W1 [M,P,h,d], W2 [M,P,d,h] (the head's init for every chain).

    ``cfg`` supplies C_G, locals_ = ((C_L, S_L), ...), act, has_global,
    qk_proj, qk_scope and optionally global_intra (the global memory's
    retrieval reading).  Memory 0 is the global memory when has_global.
    ``shards`` restricts the local memories to some shards (for sampling; the
    output is then only meaningful on those shards and without the global).
    """
    kind = _kind(cfg)
    o = torch.zeros_like(q)
    m = 0
    final = None
    if cfg.has_global:
        og, final = global_memory(q, k, v, lr[0], mom[0], decay[0], W1[0], W2[0],
                                  cfg.C_G, kind, ckpt=ckpt, intra=_intra(cfg))
        o = o + og
        m = 1
    for (C_L, S_L) in cfg.locals_:
        o = o + local_memory(q, k, v, lr[m], mom[m], decay[m], W1[m], W2[m], C_L, S_L, kind,
                             qk_proj=bool(cfg.qk_proj), qk_scope=_scope(cfg), ckpt=ckpt,
                             shards=shards)
        m += 1
    if with_final:
        return o, final
    return o


def layer_backward(q, k, v, lr, mom, decay, W1, W2, dO, cfg, ckpt: bool = True):
    """Gradients of sum <dO, o> with respect to every input.  Returns a dict
    with dq, dk, dv [P,L,d], dlr, dmom, ddecay [M,P,L], dW1 [M,P,h,d],
    dW2 [M,P,d,h] (per chain: the caller sums chains that share a head) and o.

    ``ckpt=False``: one autograd pass through the whole forward (memory grows
    with L).  ``ckpt=True``: the same gradients segment by segment -- a forward
    without autograd stores the state entering each segment (a global chunk's
    sub-block, a local chunk), then the segments are walked in reverse and each
    one is differentiated by autograd of the same per-token code, the
    adjoint of its exit state flowing into its entry state."""
    if not ckpt:
        leaves = [t.detach().clone().requires_grad_(True) for t in (q, k, v, lr, mom, decay, W1, W2)]
        o = layer_forward(*leaves, cfg)
        grads = torch.autograd.grad((o * dO).sum(), leaves)
        names = ["dq", "dk", "dv", "dlr", "dmom", "ddecay", "dW1", "dW2"]
        out = {n: g.detach() for n, g in zip(names, grads)}
        out["o"] = o.detach()
        return out
    kind = _kind(cfg)
    out = dict(dq=torch.zeros_like(q), dk=torch.zeros_like(k), dv=torch.zeros_like(v),
               dlr=torch.zeros_like(lr), dmom=torch.zeros_like(mom),
               ddecay=torch.zeros_like(decay), dW1=torch.zeros_like(W1),
               dW2=torch.zeros_like(W2), o=torch.zeros_like(q))
    m = 0
    if cfg.has_global:
        _global_backward(q, k, v, lr[0], mom[0], decay[0], W1[0], W2[0], dO, cfg.C_G, kind, out, 0,
                         intra=_intra(cfg))
        m = 1
    for (C_L, S_L) in cfg.locals_:
        _local_backward(q, k, v, lr[m], mom[m], decay[m], W1[m], W2[m], dO, C_L, S_L, kind,
                        bool(cfg.qk_proj), _scope(cfg), out, m)
        m += 1
    return out


def _vjp(fn, args, diff, grad_outs):
    """Evaluate fn(*args) with autograd on the positions `diff` of args and
    return (outputs, grads of sum_i <grad_outs[i], outputs[i]> for each diff
    position); grad_outs entries may be None (no incoming gradient)."""
    args = list(args)
    leaves = []
    for i in diff:
        args[i] = args[i].detach().requires_grad_(True)
        leaves.append(args[i])
    with torch.enable_grad():
        outs = fn(*args)
        pairs = [(o, g) for o, g in zip(outs, grad_outs) if g is not None]
        gs = torch.autograd.grad([o for o, _ in pairs], leaves, [g for _, g in pairs],
                                 allow_unused=True)
    gs = [torch.zeros_like(x) if g is None else g for g, x in zip(gs, leaves)]
    return [o.detach() for o in outs], gs


def _global_backward(q, k, v, eta, beta, alpha, W1, W2, dO, C_G, kind, out, m, block=64,
                     intra=False):
    P, L, d = q.shape
    V1, V2 = W1, W2
    S1 = torch.zeros_like(W1)
    S2 = torch.zeros_like(W2)
    chunks = []
    with torch.no_grad():
        for n in range(L // C_G):
            t0 = n * C_G
            blocks = []
            V1h, V2h = V1, V2                      # chunk-entry state
            for b0 in range(t0, t0 + C_G, block):
                b1 = min(b0 + block, t0 + C_G)
                blocks.append((b0, b1, V1, V2, S1, S2))
                V1, V2, S1, S2 = _global_accumulate(V1, V2, S1, S2, V1h, V2h, k[:, b0:b1],
                                                    v[:, b0:b1], eta[:, b0:b1], beta[:, b0:b1],
                                                    alpha[:, b0:b1], kind)
            chunks.append((t0, blocks))
    dV1, dV2 = torch.zeros_like(W1), torch.zeros_like(W2)
    dS1, dS2 = torch.zeros_like(W1), torch.zeros_like(W2)
    for t0, blocks in reversed(chunks):
        V1h, V2h = chunks_entry(blocks)
        dV1h, dV2h = torch.zeros_like(W1), torch.zeros_like(W2)
        for (b0, b1, a1, a2, s1, s2) in reversed(blocks):
            if intra:
                # the sub-block's outputs f(V_t, q_t) receive dO as well
                args = (a1, a2, s1, s2, V1h, V2h, q[:, b0:b1], k[:, b0:b1], v[:, b0:b1],
                        eta[:, b0:b1], beta[:, b0:b1], alpha[:, b0:b1], kind)
                o, g = _vjp(_global_accumulate_intra, args, range(12),
                            (dV1, dV2, dS1, dS2, dO[:, b0:b1]))
                out["o"][:, b0:b1] += o[4]
                out["dq"][:, b0:b1] += g[6]
                g = g[:6] + g[7:]
            else:
                args = (a1, a2, s1, s2, V1h, V2h, k[:, b0:b1], v[:, b0:b1], eta[:, b0:b1],
                        beta[:, b0:b1], alpha[:, b0:b1], kind)
                _, g = _vjp(_global_accumulate, args, range(11), (dV1, dV2, dS1, dS2))
            dV1, dV2, dS1, dS2 = g[0], g[1], g[2], g[3]
            dV1h = dV1h + g[4]
            dV2h = dV2h + g[5]
            out["dk"][:, b0:b1] += g[6]
            out["dv"][:, b0:b1] += g[7]
            out["dlr"][m, :, b0:b1] += g[8]
            out["dmom"][m, :, b0:b1] += g[9]
            out["ddecay"][m, :, b0:b1] += g[10]
        if not intra:
            sl = slice(t0, t0 + C_G)
            o, g = _vjp(lambda a, b, x, kd: (_global_retrieve(a, b, x, kd),),
                        (V1h, V2h, q[:, sl], kind), range(3), (dO[:, sl],))
            out["o"][:, sl] += o[0]
            dV1h = dV1h + g[0]
            dV2h = dV2h + g[1]
            out["dq"][:, sl] += g[2]
        # the chunk-entry state is both the running state and V_hat
        dV1 = dV1 + dV1h
        dV2 = dV2 + dV2h
    out["dW1"][m] += dV1
    out["dW2"][m] += dV2


def chunks_entry(blocks):
    """(V1, V2) entering the chunk whose sub-blocks are listed."""
    return blocks[0][2], blocks[0][3]


def _local_backward(q, k, v, eta, beta, alpha, W1i, W2i, dO, C_L, S_L, kind, qk_proj, qk_scope,
                    out, m):
    P, L, d = q.shape
    for s in range(L // S_L):
        W1, W2 = W1i, W2i
        S1 = torch.zeros_like(W1i)
        S2 = torch.zeros_like(W2i)
        Mq = torch.zeros(P, d, d, dtype=q.dtype)
        entries = []
        with torch.no_grad():
            for c0 in range(s * S_L, (s + 1) * S_L, C_L):
                if qk_scope == "chunk":
                    Mq = torch.zeros(P, d, d, dtype=q.dtype)
                entries.append((c0, W1, W2, S1, S2, Mq))
                sl = slice(c0, c0 + C_L)
                W1, W2, S1, S2, Mq, _ = _local_chunk(W1, W2, S1, S2, Mq, q[:, sl], k[:, sl], v[:, sl],
                                                     eta[:, sl], beta[:, sl], alpha[:, sl], kind,
                                                     qk_proj)
        dW1, dW2 = torch.zeros_like(W1i), torch.zeros_like(W2i)
        dS1, dS2 = torch.zeros_like(W1i), torch.zeros_like(W2i)
        dM = torch.zeros(P, d, d, dtype=q.dtype)
        for (c0, a1, a2, s1, s2, mq) in reversed(entries):
            sl = slice(c0, c0 + C_L)
            args = (a1, a2, s1, s2, mq, q[:, sl], k[:, sl], v[:, sl], eta[:, sl], beta[:, sl],
                    alpha[:, sl], kind, qk_proj)
            gM = None if qk_scope == "chunk" else dM
            o, g = _vjp(_local_chunk, args, range(11), (dW1, dW2, dS1, dS2, gM, dO[:, sl]))
            out["o"][:, sl] += o[5]
            dW1, dW2, dS1, dS2 = g[0], g[1], g[2], g[3]
            dM = g[4] if qk_scope != "chunk" else torch.zeros_like(dM)
            out["dq"][:, sl] += g[5]
            out["dk"][:, sl] += g[6]
            out["dv"][:, sl] += g[7]
            out["dlr"][m, :, sl] += g[8]
            out["dmom"][m, :, sl] += g[9]
            out["ddecay"][m, :, sl] += g[10]
        out["dW1"][m] += dW1
        out["dW2"][m] += dW2


# --------------------------------------------------------------------------
# the per-token rule (Sec. 2.1 compression / retrieval equations)
# --------------------------------------------------------------------------
def sequential(q, k, v, eta, beta, alpha, W1, W2, kind: str, reset: Optional[int] = None,
               qk_proj: bool = False, retrieve_first: bool = False):
    """Token-by-token deep memory with no chunking: each gradient is taken at
    the current state W_{t-1}.  ``reset`` re-initialises W, S (and the Q-K sum)
    every ``reset`` tokens; ``retrieve_first`` reads f(W_{t-1}, q_t) before the
    update (what a chunk of one token gives under the global retrieval rule)."""
    P, L, d = q.shape
    outs = []
    for t in range(L):
        if t == 0 or (reset is not None and t % reset == 0):
            Wa, Wb = W1, W2
            Sa = torch.zeros_like(W1)
            Sb = torch.zeros_like(W2)
            Mq = torch.zeros(P, d, d, dtype=q.dtype)
        if retrieve_first:
            outs.append(memory_fn(Wa, Wb, q[:, t], kind))
        ga, gb = inner_grad(Wa, Wb, k[:, t], v[:, t], kind)
        Sa = _bc(beta[:, t]) * Sa - _bc(eta[:, t]) * ga
        Sb = _bc(beta[:, t]) * Sb - _bc(eta[:, t]) * gb
        Wa = _bc(1.0 - alpha[:, t]) * Wa + Sa
        Wb = _bc(1.0 - alpha[:, t]) * Wb + Sb
        kt = k[:, t]
        Mq = Mq + torch.einsum("pd,pe->pde", kt, kt) / (kt * kt).sum(-1)[:, None, None]
        if not retrieve_first:
            x = torch.einsum("pde,pe->pd", Mq, q[:, t]) if qk_proj else q[:, t]
            outs.append(memory_fn(Wa, Wb, x, kind))
    return torch.stack(outs, 1), (Wa, Wb, Sa, Sb)


# --------------------------------------------------------------------------
# helpers to feed full [B,H,L,d] arrays (numpy) for a list of (b, h) chains
# --------------------------------------------------------------------------
def gather_pairs(inp, pairs: Sequence[Tuple[int, int]]):
    """Pick the chains ``pairs`` out of full-size numpy arrays and return fp64
    torch tensors in the oracle's per-chain layout."""
    b = np.array([p[0] for p in pairs])
    h = np.array([p[1] for p in pairs])
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))
    return dict(
        q=t(inp.q[b, h]), k=t(inp.k[b, h]), v=t(inp.v[b, h]),
        lr=t(inp.lr[:, b, h]), mom=t(inp.mom[:, b, h]), decay=t(inp.decay[:, b, h]),
        W1=t(inp.W1[:, h]), W2=t(inp.W2[:, h]), dO=t(inp.dO[b, h]),
    )


def forward_pairs(inp, cfg, pairs, with_final: bool = False):
    g = gather_pairs(inp, pairs)
    with torch.no_grad():
        return layer_forward(g["q"], g["k"], g["v"], g["lr"], g["mom"], g["decay"],
                             g["W1"], g["W2"], cfg, with_final=with_final)


def backward_pairs(inp, cfg, pairs):
    g = gather_pairs(inp, pairs)
    return layer_backward(g["q"], g["k"], g["v"], g["lr"], g["mom"], g["decay"],
                          g["W1"], g["W2"], g["dO"], cfg)


def all_pairs(cfg) -> List[Tuple[int, int]]:
    return [(b, h) for b in range(cfg.B) for h in range(cfg.H)]


def reduce_init_grads(dW: torch.Tensor, pairs, H: int) -> torch.Tensor:
    """Sum per-chain init gradients [M,P,...] over the chains of each head
    -> [M,H,...] (the init is shared across batch and shards)."""
    out = torch.zeros((dW.shape[0], H) + tuple(dW.shape[2:]), dtype=dW.dtype)
    for i, (_, h) in enumerate(pairs):
        out[:, h] += dW[:, i]
    return out
