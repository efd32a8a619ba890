"""An independent float64 PyTorch (CPU) formulation of the server block, used
only to cross-check the oracle.  It shares no code with the oracle: LayerNorm,
linear layers and the tanh GeLU are torch library routines, the rotary
encoding is complex multiplication, attention is torch's
scaled_dot_product_attention with an explicit boolean mask per sequence, and
every gradient comes from autograd."""

from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def _mask(L: int, prefix):
    i = torch.arange(L)[:, None]
    j = torch.arange(L)[None, :]
    causal = j <= i
    if prefix is None:
        return causal
    in_prefix = (i < prefix) & (j < prefix)
    return causal | in_prefix


def _rotate(x: torch.Tensor, pos: torch.Tensor, r: int, base: float) -> torch.Tensor:
    """x [L, nh, d]: leading r dims of each head as r/2 complex numbers
    (x[i], x[i + r/2]) multiplied by exp(i * p * theta_i)."""
    half = r // 2
    theta = base ** (-(2.0 * torch.arange(half, dtype=torch.float64)) / r)
    ang = pos.to(torch.float64)[:, None] * theta[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]
    z = torch.complex(x[..., :half], x[..., half:r]) * rot
    return torch.cat([z.real, z.imag, x[..., r:]], dim=-1)


def _glm_pos(L: int, P: int):
    """GLM 2-D positions of one sequence with a P-token context: the first
    counter freezes at the [gMASK] position after the context, the second
    counts the span after it (vectorised, independent of the oracle)."""
    t = torch.arange(L)
    m = max(P - 1, 0)
    p1 = torch.where(t < P, t, torch.full_like(t, m))
    p2 = torch.clamp(t - P + 1, min=0)
    return p1, p2


def block(p, x, cu_seqlens, prefix_len, shape):
    """One block; with "prefix_k" / "prefix_v" in p ([L_p, H], not rotated)
    the P-tuning v2 prefix is concatenated in front of every sequence's keys
    and values and is visible to every query.  shape.residual_alpha > 0:
    ChatGLM-6B's residual on the normalised input; shape.rotary_2d: the
    second half of every head rotated by the GLM block position."""
    alpha = float(getattr(shape, "residual_alpha", 0.0))
    two_d = bool(getattr(shape, "rotary_2d", False))
    r = shape.rotary_dim
    T, H = x.shape
    nh = shape.num_heads
    d = H // nh
    u = F.layer_norm(x, (H,), p["ln1_g"], p["ln1_b"], shape.ln_eps)
    qkv = F.linear(u, p["w_qkv"], p["b_qkv"])
    q, k, v = qkv.split(H, dim=1)
    outs = []
    for s in range(len(cu_seqlens) - 1):
        r0, r1 = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
        L = r1 - r0
        pre = None if prefix_len is None else int(prefix_len[s])
        qs, ks = q[r0:r1].reshape(L, nh, d), k[r0:r1].reshape(L, nh, d)
        if two_d:
            p1, p2 = _glm_pos(L, L if pre is None else pre)
            qs = torch.cat([_rotate(qs[..., :r], p1, r, shape.rope_base),
                            _rotate(qs[..., r:], p2, r, shape.rope_base)], dim=-1)
            ks = torch.cat([_rotate(ks[..., :r], p1, r, shape.rope_base),
                            _rotate(ks[..., r:], p2, r, shape.rope_base)], dim=-1)
        else:
            pos = torch.arange(L)
            qs = _rotate(qs, pos, r, shape.rope_base)
            ks = _rotate(ks, pos, r, shape.rope_base)
        vs = v[r0:r1].reshape(L, nh, d)
        mask = _mask(L, pre)
        if "prefix_k" in p:
            Lp = p["prefix_k"].shape[0]
            ks = torch.cat([p["prefix_k"].reshape(Lp, nh, d), ks], dim=0)
            vs = torch.cat([p["prefix_v"].reshape(Lp, nh, d), vs], dim=0)
            mask = torch.cat([torch.ones(L, Lp, dtype=torch.bool), mask], dim=1)
        o = F.scaled_dot_product_attention(qs.transpose(0, 1), ks.transpose(0, 1), vs.transpose(0, 1),
                                           attn_mask=mask)
        outs.append(o.transpose(0, 1).reshape(L, H))
    o = torch.cat(outs, dim=0)
    h = (alpha * u if alpha else x) + F.linear(o, p["w_o"], p["b_o"])
    w = F.layer_norm(h, (H,), p["ln2_g"], p["ln2_b"], shape.ln_eps)
    g = F.gelu(F.linear(w, p["w_1"], p["b_1"]), approximate="tanh")
    return (alpha * w if alpha else h) + F.linear(g, p["w_2"], p["b_2"])


def stack_fwd_bwd(layers, x, dy, batch, shape):
    """Returns y, dx and per-layer grads (numpy float64) via autograd."""
    tl = [{k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in lp.items()}
          for lp in layers]
    tx = torch.tensor(np.asarray(x, np.float64), requires_grad=True)
    cur = tx
    pre = batch.prefix_len if batch.mask == "prefix" else None
    for lp in tl:
        cur = block(lp, cur, batch.cu_seqlens, pre, shape)
    (cur * torch.tensor(np.asarray(dy, np.float64))).sum().backward()
    grads = [{k: v.grad.numpy() for k, v in lp.items()} for lp in tl]
    return cur.detach().numpy(), tx.grad.numpy(), grads
