"""Plain numpy definition of one server-held block and of the block stack.

Test infrastructure only (see the package docstring).  Every function names
the passage it follows.  ``batch`` and ``shape`` are plain records with the
attributes used below (cu_seqlens, client_seq_ptr, mask, prefix_len;
hidden, num_heads, rotary_dim, rope_base, ln_eps); nothing from the HIP
library is used.
"""

from __future__ import annotations

import math
from typing import Callable, Dict, List, Optional, Sequence, Union

import numpy as np

GELU_C = math.sqrt(2.0 / math.pi)
GELU_A = 0.044715

PARAMS = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2",
          "ln1_g", "ln1_b", "ln2_g", "ln2_b")


# ----------------------------------------------------------------------------
# Client batching (Section 3.3): packing, boundaries
# ----------------------------------------------------------------------------

def client_token_ranges(cu_seqlens: np.ndarray, client_seq_ptr: np.ndarray) -> np.ndarray:
    """[C, 2] int64: first and one-past-last packed row of each client.

    Client-batch training concatenates each client's smashed data into one
    batch (Section 3.3); client c owns sequences client_seq_ptr[c] ..
    client_seq_ptr[c+1]-1, and sequence s owns rows cu_seqlens[s] ..
    cu_seqlens[s+1]-1.
    """
    C = len(client_seq_ptr) - 1
    out = np.zeros((C, 2), np.int64)
    for c in range(C):
        out[c, 0] = int(cu_seqlens[int(client_seq_ptr[c])])
        out[c, 1] = int(cu_seqlens[int(client_seq_ptr[c + 1])])
    return out


def pack_clients(client_tensors: Sequence[np.ndarray], cu_seqlens: np.ndarray,
                 client_seq_ptr: np.ndarray) -> np.ndarray:
    """Stack the clients' smashed data into one packed [T, H] batch.

    Each client sends a sequence-first tensor [L_max_c, B_c, H] (the paper's
    {seqlength, batchsize, hiddensize} layout, Section 3.3), padded to the
    client's longest sequence; sequence b of client c has length
    cu_seqlens[s+1]-cu_seqlens[s] with s = client_seq_ptr[c] + b.  Rows are
    ordered client, then sequence, then position.
    """
    T = int(cu_seqlens[-1])
    H = client_tensors[0].shape[2] if len(client_tensors) else 0
    out = np.zeros((T, H), dtype=client_tensors[0].dtype if len(client_tensors) else np.float32)
    for c, xc in enumerate(client_tensors):
        for b in range(int(client_seq_ptr[c + 1]) - int(client_seq_ptr[c])):
            s = int(client_seq_ptr[c]) + b
            r0, r1 = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
            for p in range(r1 - r0):
                out[r0 + p, :] = xc[p, b, :]
    return out


def unpack_clients(packed: np.ndarray, cu_seqlens: np.ndarray, client_seq_ptr: np.ndarray,
                   fill: float = 0.0) -> List[np.ndarray]:
    """Inverse of ``pack_clients``: per-client [L_max_c, B_c, H] tensors, with
    positions beyond a sequence's length set to ``fill``."""
    outs = []
    H = packed.shape[1]
    for c in range(len(client_seq_ptr) - 1):
        s0, s1 = int(client_seq_ptr[c]), int(client_seq_ptr[c + 1])
        Lmax = max(int(cu_seqlens[s + 1]) - int(cu_seqlens[s]) for s in range(s0, s1))
        xc = np.full((Lmax, s1 - s0, H), fill, dtype=packed.dtype)
        for b, s in enumerate(range(s0, s1)):
            r0, r1 = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
            for p in range(r1 - r0):
                xc[p, b, :] = packed[r0 + p, :]
        outs.append(xc)
    return outs


def positions(cu_seqlens: np.ndarray) -> np.ndarray:
    """Position of every packed row inside its own sequence (0-based, restarts
    at each sequence): the positions a client would use on its own data."""
    T = int(cu_seqlens[-1])
    pos = np.zeros(T, np.int64)
    for s in range(len(cu_seqlens) - 1):
        r0, r1 = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
        pos[r0:r1] = np.arange(r1 - r0)
    return pos


def glm_positions(batch):
    """GLM 2-D positions of every packed row (ChatGLM-6B's blank infilling,
    which the paper's base model uses; not given in the paper).  Sequence s
    has a context of P_s tokens (the prefix-LM prefix; the whole sequence
    when the batch is causal) ending with the [gMASK] token at M_s =
    max(P_s - 1, 0).  The first position counts context tokens and stays at
    M_s after the context: p1 = t for t < P_s, else M_s.  The second
    (block) position is 0 in the context and counts the generated span from
    1: p2 = 0 for t < P_s, else t - P_s + 1."""
    cu = batch.cu_seqlens
    T = int(cu[-1])
    p1 = np.zeros(T, np.int64)
    p2 = np.zeros(T, np.int64)
    for s in range(len(cu) - 1):
        r0, r1 = int(cu[s]), int(cu[s + 1])
        L = r1 - r0
        P = int(batch.prefix_len[s]) if getattr(batch, "mask", "causal") == "prefix" else L
        M = max(P - 1, 0)
        for t in range(L):
            p1[r0 + t] = t if t < P else M
            p2[r0 + t] = 0 if t < P else t - P + 1
    return p1, p2


# ----------------------------------------------------------------------------
# LayerNorm (pre-LN reading; biased variance, eps inside the square root)
# ----------------------------------------------------------------------------

def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float):
    """y = (x - mean) / sqrt(var + eps) * g + b over the hidden dimension.
    Returns (y, xhat, rstd)."""
    mu = x.mean(axis=1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    return xhat * g + b, xhat, rstd


def layer_norm_backward(dy: np.ndarray, xhat: np.ndarray, rstd: np.ndarray, g: np.ndarray):
    """Gradient of ``layer_norm``: returns (dx, dg, db).

    With dxhat = dy * g:  dx = rstd * (dxhat - mean(dxhat) - xhat * mean(dxhat * xhat)).
    """
    dxhat = dy * g
    dg = (dy * xhat).sum(axis=0)
    db = dy.sum(axis=0)
    dx = rstd * (dxhat - dxhat.mean(axis=1, keepdims=True)
                 - xhat * (dxhat * xhat).mean(axis=1, keepdims=True))
    return dx, dg, db


# ----------------------------------------------------------------------------
# GeLU (tanh form)
# ----------------------------------------------------------------------------

def gelu(z: np.ndarray) -> np.ndarray:
    """0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))  (z^3 as z z z)."""
    return 0.5 * z * (1.0 + np.tanh(GELU_C * (z + GELU_A * (z * z * z))))


def gelu_grad(z: np.ndarray) -> np.ndarray:
    """d gelu / dz = 0.5 (1 + t) + 0.5 z (1 - t^2) sqrt(2/pi) (1 + 3 * 0.044715 z^2),
    t = tanh(sqrt(2/pi) (z + 0.044715 z^3))."""
    t = np.tanh(GELU_C * (z + GELU_A * (z * z * z)))
    return 0.5 * (1.0 + t) + 0.5 * z * (1.0 - t * t) * GELU_C * (1.0 + 3.0 * GELU_A * z * z)


# ----------------------------------------------------------------------------
# Rotary position encoding on the leading half of each head
# ----------------------------------------------------------------------------

def rope_tables(pos: np.ndarray, rotary_dim: int, base: float, dtype=np.float64):
    """cos and sin of p * theta_i, theta_i = base^(-2 i / r), i < r/2, shape [T, r/2].
    Angles are formed in float64 whatever the working dtype."""
    half = rotary_dim // 2
    inv = base ** (-(2.0 * np.arange(half, dtype=np.float64)) / rotary_dim)
    ang = pos.astype(np.float64)[:, None] * inv[None, :]
    return np.cos(ang).astype(dtype), np.sin(ang).astype(dtype)


def rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray, rotary_dim: int,
         inverse: bool = False) -> np.ndarray:
    """Rotate dims [0, r) of every head of x [T, n_h, d] pairwise (i, i + r/2):
        x'[i]       = x[i] cos - x[i + r/2] sin
        x'[i + r/2] = x[i + r/2] cos + x[i] sin
    dims [r, d) pass through.  ``inverse`` applies the transpose rotation
    (angle -p theta), which is the backward of the forward rotation."""
    half = rotary_dim // 2
    out = x.copy()
    c = cos[:, None, :]
    s = -sin[:, None, :] if inverse else sin[:, None, :]
    a = x[:, :, :half]
    b = x[:, :, half:rotary_dim]
    out[:, :, :half] = a * c - b * s
    out[:, :, half:rotary_dim] = b * c + a * s
    return out


# ----------------------------------------------------------------------------
# Attention: per sequence and head, explicit L x L scores
# ----------------------------------------------------------------------------

def allowed_mask(L: int, prefix: Optional[int]) -> np.ndarray:
    """[L, L] bool: query i may attend key j.  Causal: j <= i.  Prefix-LM with
    a bidirectional prefix of P tokens: j <= max(i, P - 1).  Keys of other
    sequences (hence of other clients) are never visible."""
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    if prefix is None:
        return j <= i
    return j <= np.maximum(i, int(prefix) - 1)


def _seq_prefix(batch, s: int) -> Optional[int]:
    if getattr(batch, "mask", "causal") == "prefix":
        return int(batch.prefix_len[s])
    return None


def _scores_probs(qs: np.ndarray, ks: np.ndarray, allowed: np.ndarray, scale: float):
    """S = q k^T * scale with disallowed entries at -inf; P = row softmax."""
    S = (qs @ ks.T) * scale
    S = np.where(allowed, S, -np.inf)
    m = S.max(axis=1, keepdims=True)
    e = np.exp(S - m)
    e = np.where(allowed, e, 0.0)
    P = e / e.sum(axis=1, keepdims=True)
    return P


def _prefix_head(pk: Optional[np.ndarray], h: int, d: int, dtype) -> np.ndarray:
    """Prefix rows of head h ([L_p, d]); an empty array when there is none."""
    if pk is None:
        return np.zeros((0, d), dtype)
    return pk[:, h]


def attention_forward(q: np.ndarray, k: np.ndarray, v: np.ndarray, batch,
                      pk: Optional[np.ndarray] = None, pv: Optional[np.ndarray] = None) -> np.ndarray:
    """o = softmax_mask(q k'^T / sqrt(d)) v' for every sequence and head
    (Appendix A gives the softmax(Q K^T / sqrt(d_h)) form).  q, k, v, o:
    [T, n_h, d].  With P-tuning v2 (Appendix A, P-tuning v2 section) the
    block's prefix keys and values pk, pv [L_p, n_h, d] are spliced in front:
    K' = [pk; k], V' = [pv; v], the prefix visible to every query of every
    sequence; the sequence's own keys keep their causal / prefix-LM mask."""
    T, nh, d = q.shape
    scale = 1.0 / math.sqrt(d)
    o = np.zeros_like(q)
    cu = batch.cu_seqlens
    for s in range(len(cu) - 1):
        r0, r1 = int(cu[s]), int(cu[s + 1])
        L = r1 - r0
        for h in range(nh):
            pkh = _prefix_head(pk, h, d, q.dtype)
            pvh = _prefix_head(pv, h, d, q.dtype)
            allowed = np.concatenate([np.ones((L, len(pkh)), bool), allowed_mask(L, _seq_prefix(batch, s))], axis=1)
            P = _scores_probs(q[r0:r1, h], np.concatenate([pkh, k[r0:r1, h]]), allowed, scale)
            o[r0:r1, h] = P @ np.concatenate([pvh, v[r0:r1, h]])
    return o


def attention_backward(q: np.ndarray, k: np.ndarray, v: np.ndarray, do: np.ndarray, batch,
                       pk: Optional[np.ndarray] = None, pv: Optional[np.ndarray] = None):
    """Gradient of ``attention_forward`` given do; P is recomputed.
        dV' = P^T dO,  dP = dO V'^T,  D_i = sum_j P_ij dP_ij,
        dS = P (dP - D),  dQ = dS K' / sqrt(d),  dK' = dS^T Q / sqrt(d).
    Returns (dq, dk, dv), plus (dpk, dpv) summed over all sequences when a
    prefix is given."""
    T, nh, d = q.shape
    scale = 1.0 / math.sqrt(d)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    Lp = 0 if pk is None else pk.shape[0]
    dpk = np.zeros((Lp, nh, d), q.dtype)
    dpv = np.zeros((Lp, nh, d), q.dtype)
    cu = batch.cu_seqlens
    for s in range(len(cu) - 1):
        r0, r1 = int(cu[s]), int(cu[s + 1])
        L = r1 - r0
        allowed = np.concatenate([np.ones((L, Lp), bool), allowed_mask(L, _seq_prefix(batch, s))], axis=1)
        for h in range(nh):
            kk = np.concatenate([_prefix_head(pk, h, d, q.dtype), k[r0:r1, h]])
            vv = np.concatenate([_prefix_head(pv, h, d, q.dtype), v[r0:r1, h]])
            qs, dos = q[r0:r1, h], do[r0:r1, h]
            P = _scores_probs(qs, kk, allowed, scale)
            dvv = P.T @ dos
            dP = dos @ vv.T
            D = (P * dP).sum(axis=1, keepdims=True)
            dS = P * (dP - D)
            dq[r0:r1, h] = (dS @ kk) * scale
            dkk = (dS.T @ qs) * scale
            dk[r0:r1, h] = dkk[Lp:]
            dv[r0:r1, h] = dvv[Lp:]
            dpk[:, h] += dkk[:Lp]
            dpv[:, h] += dvv[:Lp]
    if pk is None:
        return dq, dk, dv
    return dq, dk, dv, dpk, dpv


def attention_query_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, rows: np.ndarray,
                         prefix: Optional[int] = None, pk: Optional[np.ndarray] = None,
                         pv: Optional[np.ndarray] = None, do: Optional[np.ndarray] = None):
    """The attention of ``attention_forward`` / ``attention_backward`` for a
    few query rows of ONE sequence, for sequences too long for the L x L
    score matrix: q, k, v [L, n_h, d] are that sequence's rows, ``rows`` the
    query indices, ``prefix`` its prefix-LM length (None: causal), pk, pv the
    P-tuning v2 prefix [L_p, n_h, d] (Appendix A; visible to every query).

    Forward: o [len(rows), n_h, d] and lse [len(rows), n_h], the natural-log
    sum over the visible keys of exp(q k'/sqrt(d)).  With ``do`` (the output
    gradient of the given rows, [len(rows), n_h, d]; every other query row
    of the sequence has a zero output gradient) also the gradients, by the
    same equations as ``attention_backward``: dq of the given rows, dk, dv
    [L, n_h, d] of the whole sequence, and dpk, dpv [L_p, n_h, d].  Query rows
    with a zero output gradient have dP = 0 and D = 0, hence dS = 0: they add
    nothing, so these are the whole sequence's gradients."""
    L, nh, d = q.shape
    scale = 1.0 / math.sqrt(d)
    rows = np.asarray(rows, np.int64)
    Lp = 0 if pk is None else pk.shape[0]
    j = np.arange(L)[None, :]
    i = rows[:, None]
    own = j <= (i if prefix is None else np.maximum(i, int(prefix) - 1))
    allowed = np.concatenate([np.ones((len(rows), Lp), bool), own], axis=1)
    o = np.zeros((len(rows), nh, d), q.dtype)
    lse = np.zeros((len(rows), nh), q.dtype)
    grads = do is not None
    if grads:
        dq = np.zeros((len(rows), nh, d), q.dtype)
        dk, dv = np.zeros_like(k), np.zeros_like(v)
        dpk = np.zeros((Lp, nh, d), q.dtype)
        dpv = np.zeros((Lp, nh, d), q.dtype)
    for h in range(nh):
        kk = np.concatenate([_prefix_head(pk, h, d, q.dtype), k[:, h]])
        vv = np.concatenate([_prefix_head(pv, h, d, q.dtype), v[:, h]])
        S = np.where(allowed, (q[rows, h] @ kk.T) * scale, -np.inf)
        m = S.max(axis=1, keepdims=True)
        e = np.where(allowed, np.exp(S - m), 0.0)
        ssum = e.sum(axis=1, keepdims=True)
        P = e / ssum
        o[:, h] = P @ vv
        lse[:, h] = (m + np.log(ssum))[:, 0]
        if grads:
            dP = do[:, h] @ vv.T
            D = (P * dP).sum(axis=1, keepdims=True)
            dS = P * (dP - D)
            dq[:, h] = (dS @ kk) * scale
            dkk = (dS.T @ q[rows, h]) * scale
            dvv = P.T @ do[:, h]
            dk[:, h], dv[:, h] = dkk[Lp:], dvv[Lp:]
            dpk[:, h], dpv[:, h] = dkk[:Lp], dvv[:Lp]
    if not grads:
        return o, lse
    return o, lse, dq, dk, dv, dpk, dpv


# ----------------------------------------------------------------------------
# One block (Section 3.1: an LLM-Block is self-attention followed by an FFN)
# ----------------------------------------------------------------------------

def _cast(p: Dict[str, np.ndarray], dtype) -> Dict[str, np.ndarray]:
    return {k: np.asarray(v, dtype=dtype) for k, v in p.items()}


def _rotate_qk(x: np.ndarray, tables, shape, inverse: bool = False) -> np.ndarray:
    """The block's rotary encoding of q or k [T, n_h, d]: dims [0, r) by the
    first table; with GLM 2-D positions also dims [r, 2r) by the second."""
    r = shape.rotary_dim
    out = rope(x, tables[0], tables[1], r, inverse)
    if len(tables) == 4:
        out[:, :, r:2 * r] = rope(x[:, :, r:2 * r], tables[2], tables[3], r, inverse)
    return out


def block_forward(p: Dict[str, np.ndarray], x: np.ndarray, batch, shape, dtype=np.float64):
    """One pre-LN block:
        u = LN1(x);  qkv = u W_qkv^T + b_qkv;  q, k rotated (first half of each head)
        h = x + attn(q, k, v) W_o^T + b_o
        w = LN2(h);  z = w W_1^T + b_1;  g = gelu(z)
        y = h + g W_2^T + b_2
    ChatGLM-6B's variant (shape.residual_alpha = alpha > 0) feeds the
    normalised input forward instead: h = alpha u + attn(...) W_o^T + b_o and
    y = alpha w + g W_2^T + b_2.  With shape.rotary_2d the second half of each
    head is rotated too, by the GLM block position (``glm_positions``).
    Returns (y, cache) with everything the backward uses."""
    p = _cast(p, dtype)
    x = np.asarray(x, dtype=dtype)
    T, H = x.shape
    nh = shape.num_heads
    d = H // nh
    eps = shape.ln_eps
    alpha = float(getattr(shape, "residual_alpha", 0.0))
    if getattr(shape, "rotary_2d", False):
        p1, p2 = glm_positions(batch)
        tables = rope_tables(p1, shape.rotary_dim, shape.rope_base, dtype) + \
            rope_tables(p2, shape.rotary_dim, shape.rope_base, dtype)
    else:
        tables = rope_tables(positions(batch.cu_seqlens), shape.rotary_dim, shape.rope_base, dtype)

    u, xhat1, rstd1 = layer_norm(x, p["ln1_g"], p["ln1_b"], eps)
    qkv = u @ p["w_qkv"].T + p["b_qkv"]
    q = qkv[:, 0:H].reshape(T, nh, d)
    k = qkv[:, H:2 * H].reshape(T, nh, d)
    v = qkv[:, 2 * H:3 * H].reshape(T, nh, d)
    qr = _rotate_qk(q, tables, shape)
    kr = _rotate_qk(k, tables, shape)
    # P-tuning v2 prefix (Appendix A): learned keys / values [L_p, H] spliced
    # in front of every sequence's own; they carry no position, so they are
    # not rotated
    pk, pv = _prefix_kv(p, nh, d)
    o = attention_forward(qr, kr, v, batch, pk, pv).reshape(T, H)
    h = (alpha * u if alpha else x) + o @ p["w_o"].T + p["b_o"]
    w, xhat2, rstd2 = layer_norm(h, p["ln2_g"], p["ln2_b"], eps)
    z = w @ p["w_1"].T + p["b_1"]
    g = gelu(z)
    y = (alpha * w if alpha else h) + g @ p["w_2"].T + p["b_2"]
    cache = dict(x=x, u=u, xhat1=xhat1, rstd1=rstd1, qr=qr, kr=kr, v=v, o=o, h=h,
                 w=w, xhat2=xhat2, rstd2=rstd2, z=z, g=g, tables=tables, pk=pk, pv=pv)
    return y, cache


def _prefix_kv(p: Dict[str, np.ndarray], nh: int, d: int):
    """The block's P-tuning v2 prefix as [L_p, n_h, d] arrays, or (None, None)."""
    if "prefix_k" not in p:
        return None, None
    return p["prefix_k"].reshape(-1, nh, d), p["prefix_v"].reshape(-1, nh, d)


def zero_prefix_grads(num_prefix: int, hidden: int, dtype=np.float64) -> Dict[str, np.ndarray]:
    return {"prefix_k": np.zeros((num_prefix, hidden), dtype), "prefix_v": np.zeros((num_prefix, hidden), dtype)}


def zero_grads(shape, dtype=np.float64) -> Dict[str, np.ndarray]:
    H, F = shape.hidden, shape.ffn_hidden
    shp = {"w_qkv": (3 * H, H), "b_qkv": (3 * H,), "w_o": (H, H), "b_o": (H,),
           "w_1": (F, H), "b_1": (F,), "w_2": (H, F), "b_2": (H,),
           "ln1_g": (H,), "ln1_b": (H,), "ln2_g": (H,), "ln2_b": (H,)}
    return {k: np.zeros(v, dtype) for k, v in shp.items()}


def block_backward(p: Dict[str, np.ndarray], cache, dy: np.ndarray, batch, shape,
                   grads: Dict[str, np.ndarray], dtype=np.float64) -> np.ndarray:
    """Backward of ``block_forward``: returns dx and adds every parameter
    gradient named in ``grads`` into it (sum over all tokens of all clients).
    The server returns dx to the client in split learning (Section 3.1).
    With P-tuning v2 the block weights are frozen and only the prefix is
    trained (Section 3.1, Appendix A): pass grads holding just "prefix_k" and
    "prefix_v" and no weight-gradient product is formed (likewise for any
    weight left out of grads)."""
    p = _cast(p, dtype)
    dy = np.asarray(dy, dtype=dtype)
    c = cache
    T, H = dy.shape
    nh = shape.num_heads
    d = H // nh
    grads = _Sink(grads)
    alpha = float(getattr(shape, "residual_alpha", 0.0))

    # y = h + g W_2^T + b_2   (ChatGLM-6B: y = alpha w + g W_2^T + b_2)
    if grads.wants("w_2"):
        grads["w_2"] += dy.T @ c["g"]
    grads["b_2"] += dy.sum(axis=0)
    dg = dy @ p["w_2"]
    dz = dg * gelu_grad(c["z"])
    # z = w W_1^T + b_1
    if grads.wants("w_1"):
        grads["w_1"] += dz.T @ c["w"]
    grads["b_1"] += dz.sum(axis=0)
    dw = dz @ p["w_1"]
    if alpha:
        dw = dw + alpha * dy
    # w = LN2(h); h also feeds y directly (plain residual)
    dh_ln, dg2, db2 = layer_norm_backward(dw, c["xhat2"], c["rstd2"], p["ln2_g"])
    grads["ln2_g"] += dg2
    grads["ln2_b"] += db2
    dh = dh_ln if alpha else dy + dh_ln
    # h = x + o W_o^T + b_o
    if grads.wants("w_o"):
        grads["w_o"] += dh.T @ c["o"]
    grads["b_o"] += dh.sum(axis=0)
    do = (dh @ p["w_o"]).reshape(T, nh, d)
    if c["pk"] is None:
        dqr, dkr, dv = attention_backward(c["qr"], c["kr"], c["v"], do, batch)
    else:
        dqr, dkr, dv, dpk, dpv = attention_backward(c["qr"], c["kr"], c["v"], do, batch, c["pk"], c["pv"])
        grads["prefix_k"] += dpk.reshape(-1, H)
        grads["prefix_v"] += dpv.reshape(-1, H)
    dq = _rotate_qk(dqr, c["tables"], shape, inverse=True)
    dk = _rotate_qk(dkr, c["tables"], shape, inverse=True)
    dqkv = np.concatenate([dq.reshape(T, H), dk.reshape(T, H), dv.reshape(T, H)], axis=1)
    # qkv = u W_qkv^T + b_qkv
    if grads.wants("w_qkv"):
        grads["w_qkv"] += dqkv.T @ c["u"]
    grads["b_qkv"] += dqkv.sum(axis=0)
    du = dqkv @ p["w_qkv"]
    if alpha:
        du = du + alpha * dh
    # u = LN1(x); x also feeds h directly (plain residual)
    dx_ln, dg1, db1 = layer_norm_backward(du, c["xhat1"], c["rstd1"], p["ln1_g"])
    grads["ln1_g"] += dg1
    grads["ln1_b"] += db1
    return dx_ln if alpha else dh + dx_ln


class _Sink:
    """grads[name] += value for the names the caller asked for; others are
    dropped (frozen parameters)."""

    def __init__(self, grads: Dict[str, np.ndarray]):
        self.g = grads

    def wants(self, k) -> bool:
        return k in self.g

    def __getitem__(self, k):
        return self.g[k] if k in self.g else _Discard()

    def __setitem__(self, k, v):
        if k in self.g:
            self.g[k] = v


class _Discard:
    def __iadd__(self, other):
        return self


# ----------------------------------------------------------------------------
# The server stack (Section 3.1: h_{N-2} = Block_(1,N-2)(h_0))
# ----------------------------------------------------------------------------

LayerSource = Union[Sequence[Dict[str, np.ndarray]], Callable[[int], Dict[str, np.ndarray]]]


def _layer(layers: LayerSource, l: int) -> Dict[str, np.ndarray]:
    return layers(l) if callable(layers) else layers[l]


def stack_forward(layers: LayerSource, num_layers: int, x: np.ndarray, batch, shape,
                  dtype=np.float64, keep: str = "inputs"):
    """x_0 = x, x_l = Block_l(x_{l-1}), output x_N.  ``layers`` is a list of
    parameter dicts or a function l -> dict (lets a caller produce layers one
    at a time).  keep = "inputs" stores only each block's input (the backward
    recomputes the block); "caches" stores each block's whole forward cache
    (no recompute, more memory); "none" stores nothing."""
    xs = []
    cur = np.asarray(x, dtype=dtype)
    for l in range(num_layers):
        if keep == "inputs":
            xs.append(cur)
        cur, cache = block_forward(_layer(layers, l), cur, batch, shape, dtype)
        if keep == "caches":
            xs.append(cache)
    return cur, xs


def stack_backward(layers: LayerSource, num_layers: int, xs: List[np.ndarray], dy: np.ndarray,
                   batch, shape, grads: Optional[List[Dict[str, np.ndarray]]] = None,
                   dtype=np.float64):
    """Backward through blocks N..1: each block's forward is recomputed from
    its stored input (or taken from its stored cache, keep="caches"), then
    its backward runs; the dx of block l is the dy of block l-1.  Returns
    (dx, grads) with grads[l] accumulated (+=)."""
    if grads is None:
        grads = [zero_grads(shape, dtype) for _ in range(num_layers)]
    cur = np.asarray(dy, dtype=dtype)
    for l in reversed(range(num_layers)):
        p = _layer(layers, l)
        if isinstance(xs[l], dict):
            cache = xs[l]
        else:
            _, cache = block_forward(p, xs[l], batch, shape, dtype)
        cur = block_backward(p, cache, cur, batch, shape, grads[l], dtype)
    return cur, grads
