"""Gradient oracle of the pruned layer stack -- TEST INFRASTRUCTURE.

Only the tests may import this module. It is the reference for the backward
pass through the pruned forward (the fine-tuning step of Eq. 3 trains
through it): a plain float64 PyTorch (CPU) re-implementation of the forward
with every pruning point's kept rows held fixed -- the selection is a
discrete choice and carries no gradient -- differentiated by autograd.

Because the kept rows are fixed, the function is an ordinary composition of
differentiable steps: rows a pruning layer drops still feed that layer's
attention as keys and values, so they receive gradient through it (and
through the layers before it); the rows it keeps continue. Its forward is
pinned to the NumPy oracle (identical outputs), its gradients to finite
differences.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from oracle import zsa_oracle as O

WEIGHTS = ["norm1_w", "norm1_b", "w_qkv", "b_qkv", "w_o", "b_o",
           "norm2_w", "norm2_b", "w_up", "b_up", "w_down", "b_down"]


def _rope(x, pos, n_heads, theta):
    n, d = x.shape
    hd = d // n_heads
    half = hd // 2
    i = torch.arange(half, dtype=torch.float64)
    ang = pos.to(torch.float64)[:, None] * theta ** (-2.0 * i / hd)[None, :]
    c, s = torch.cos(ang), torch.sin(ang)
    parts = []
    for h in range(n_heads):
        a = x[:, h * hd:h * hd + half]
        b = x[:, h * hd + half:(h + 1) * hd]
        parts += [a * c - b * s, b * c + a * s]
    return torch.cat(parts, dim=1)


def _attention(q, k, v, n_heads, n_kv, causal):
    n, d = q.shape
    hd = d // n_heads
    group = n_heads // n_kv
    outs = []
    for h in range(n_heads):
        g = h // group
        S = q[:, h * hd:(h + 1) * hd] @ k[:, g * hd:(g + 1) * hd].T / math.sqrt(hd)
        if causal:
            S = S.masked_fill(torch.ones(n, n, dtype=torch.bool).triu(1), float("-inf"))
        outs.append(torch.softmax(S, dim=1) @ v[:, g * hd:(g + 1) * hd])
    return torch.cat(outs, dim=1)


def _layer(x, pos, w, cfg: O.LayerCfg, kept: Optional[torch.Tensor]):
    """One block on one sequence; with ``kept`` only those output rows."""
    d = cfg.d_model
    kvd = cfg.kv_heads * (d // cfg.n_heads)
    lin = lambda a, W, b: a @ W.T + (b if b is not None else 0.0)
    if cfg.kind == O.ENCODER:
        h = torch.nn.functional.layer_norm(x, (d,), w["norm1_w"], w["norm1_b"], cfg.norm_eps)
    else:
        h = x * torch.rsqrt((x * x).mean(dim=1, keepdim=True) + cfg.norm_eps) * w["norm1_w"]
    qkv = lin(h, w["w_qkv"], w["b_qkv"])
    q, k, v = qkv[:, :d], qkv[:, d:d + kvd], qkv[:, d + kvd:d + 2 * kvd]
    if cfg.kind == O.DECODER:
        q = _rope(q, pos, cfg.n_heads, cfg.rope_theta)
        k = _rope(k, pos, cfg.kv_heads, cfg.rope_theta)
    o = _attention(q, k, v, cfg.n_heads, cfg.kv_heads, cfg.causal)
    if kept is not None:          # the row-wise rest of the block runs on kept rows
        x, o = x[kept], o[kept]
    x1 = x + lin(o, w["w_o"], w["b_o"])
    if cfg.kind == O.ENCODER:
        h2 = torch.nn.functional.layer_norm(x1, (d,), w["norm2_w"], w["norm2_b"], cfg.norm_eps)
        f = torch.nn.functional.gelu(lin(h2, w["w_up"], w["b_up"]))
    else:
        h2 = x1 * torch.rsqrt((x1 * x1).mean(dim=1, keepdim=True) + cfg.norm_eps) * w["norm2_w"]
        z = lin(h2, w["w_up"], w["b_up"])
        f = torch.nn.functional.silu(z[:, 0::2]) * z[:, 1::2]
    return x1 + lin(f, w["w_down"], w["b_down"])


def forward(x, pos, weights, cfg: O.LayerCfg, prune_after: Sequence[int],
            kept: Dict[int, np.ndarray]):
    """The pruned stack on ONE sequence with fixed kept sets (kept[layer] =
    local indices among the rows entering that layer). Tensors in, tensor
    out (float64, autograd-tracked)."""
    cur, cpos = x, pos
    for l, w in enumerate(weights, start=1):
        kl = torch.as_tensor(np.asarray(kept[l], dtype=np.int64)) if l in set(prune_after) else None
        cur = _layer(cur, cpos, w, cfg, kl)
        if kl is not None:
            cpos = cpos[kl]
    return cur


def stack_backward(x: np.ndarray, pos: np.ndarray, weights: Sequence[Dict], cfg: O.LayerCfg,
                   prune_after: Sequence[int], kept: Dict[int, np.ndarray], dy: np.ndarray):
    """Gradients of sum(out * dy) for one sequence: returns (out, dx, grads)
    with grads[l][name] for every weight present (float64 NumPy)."""
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    post = torch.as_tensor(np.asarray(pos, dtype=np.int64))
    wts: List[Dict[str, Optional[torch.Tensor]]] = []
    for w in weights:
        wts.append({k: (None if w.get(k) is None else
                        torch.tensor(w[k], dtype=torch.float64, requires_grad=True))
                    for k in WEIGHTS})
    out = forward(xt, post, wts, cfg, prune_after, kept)
    (out * torch.as_tensor(dy, dtype=torch.float64)).sum().backward()
    grads = [{k: (None if t is None else t.grad.numpy().copy()) for k, t in w.items()} for w in wts]
    return out.detach().numpy(), xt.grad.numpy().copy(), grads
