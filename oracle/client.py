"""The client side of the split model around the server stack.

Test infrastructure only (see the package docstring).

Section 3.1 (Model Split): the client holds the embedding layer, block 0,
block N-1 and the final linear layer.  It computes the smashed data
h_0 = Block_0(Embedding(x)), sends it to the server, receives
h_{N-2} = Block_(1,N-2)(h_0), and finishes with
y' = Linear(Block_{N-1}(h_{N-2})) and the cross-entropy loss against the
next-token labels y.  The backward runs the same chain in reverse: the client
returns dL/dh_{N-2} to the server and receives dL/dh_0.

Readings: the final linear layer maps hidden to vocabulary logits with no
bias and, by default, no final normalisation (the paper's formula applies
Linear directly to Block_{N-1}'s output; ChatGLM-6B's final LayerNorm in
front of it is optional: "final_ln_g" / "final_ln_b" in the client dict);
the loss is the sum over labelled tokens of log-sum-exp(logits) -
logit[label], a negative label marking a token without a target; the gradient of the loss is scaled by a caller-chosen
factor (1 / number of labelled tokens gives the mean).
"""

from __future__ import annotations

from typing import Dict, Optional, Sequence, Tuple

import numpy as np

from .block import layer_norm, layer_norm_backward, stack_backward, stack_forward


def embedding_forward(table: np.ndarray, ids: np.ndarray, dtype=np.float64) -> np.ndarray:
    """Embedding(x): row ids[t] of the [V, H] table for every token t."""
    return np.asarray(table, dtype)[np.asarray(ids, np.int64)]


def embedding_backward(ids: np.ndarray, dh: np.ndarray, vocab: int, dtype=np.float64) -> np.ndarray:
    """Gradient of the table: row v is the sum of dh over the tokens whose id
    is v (tokens in order)."""
    dtable = np.zeros((vocab, dh.shape[1]), dtype)
    for t, v in enumerate(np.asarray(ids, np.int64)):
        dtable[v] += dh[t]
    return dtable


def lm_head_forward(h: np.ndarray, w: np.ndarray, labels: np.ndarray, dtype=np.float64):
    """y' = h W^T (W [V, H]) and the per-token cross-entropy
    loss_t = logsumexp(y'_t) - y'_t[label_t] (0 where label_t < 0).
    Returns (logits, lse, loss_tok, loss_sum)."""
    h = np.asarray(h, dtype)
    logits = h @ np.asarray(w, dtype).T
    mx = logits.max(axis=1, keepdims=True)
    lse = (mx + np.log(np.exp(logits - mx).sum(axis=1, keepdims=True)))[:, 0]
    labels = np.asarray(labels, np.int64)
    loss = np.zeros(h.shape[0], dtype)
    ok = labels >= 0
    loss[ok] = lse[ok] - logits[np.nonzero(ok)[0], labels[ok]]
    return logits, lse, loss, loss.sum()


def lm_head_backward(h: np.ndarray, w: np.ndarray, logits: np.ndarray, lse: np.ndarray, labels: np.ndarray,
                     grad_scale: float, dtype=np.float64) -> Tuple[np.ndarray, np.ndarray]:
    """d(grad_scale * loss_sum): dlogits = grad_scale (softmax - onehot(label))
    on labelled rows, 0 on the others; dh = dlogits W, dW = dlogits^T h.
    Returns (dh, dW)."""
    labels = np.asarray(labels, np.int64)
    p = np.exp(np.asarray(logits, dtype) - np.asarray(lse, dtype)[:, None])
    ok = labels >= 0
    p[~ok] = 0.0
    p[np.nonzero(ok)[0], labels[ok]] -= 1.0
    dlogits = grad_scale * p
    return dlogits @ np.asarray(w, dtype), dlogits.T @ np.asarray(h, dtype)


def split_step(client: Dict, server_layers: Sequence[Dict], ids: np.ndarray, labels: np.ndarray, batch, shape,
               grad_scale: float, num_server: Optional[int] = None, train_weights: bool = True,
               dtype=np.float64) -> Dict:
    """One training step of the whole split model (Section 3.1) on one
    client batch (Section 3.3).  ``client`` holds "embedding" [V, H],
    "block0" and "block_last" (parameter dicts of the client's two blocks)
    and "lm_head" [V, H]; ``shape`` describes one block.  With
    train_weights=False every weight is frozen (P-tuning v2) and only prefix
    gradients (present when the blocks carry "prefix_k"/"prefix_v") are
    formed.  Returns the forward tensors at each boundary and every
    gradient."""
    from .block import zero_grads, zero_prefix_grads
    n_srv = len(server_layers) if num_server is None else num_server

    def grads_for(layers):
        out = []
        for lp in layers:
            g = dict(zero_grads(shape, dtype)) if train_weights else {}
            if "prefix_k" in lp:
                g.update(zero_prefix_grads(lp["prefix_k"].shape[0], shape.hidden, dtype))
            out.append(g)
        return out

    e = embedding_forward(client["embedding"], ids, dtype)
    h0, xs0 = stack_forward([client["block0"]], 1, e, batch, shape, dtype=dtype)
    hs, xss = stack_forward(server_layers, n_srv, h0, batch, shape, dtype=dtype)
    hl, xsl = stack_forward([client["block_last"]], 1, hs, batch, shape, dtype=dtype)
    final_ln = "final_ln_g" in client
    hn = hl
    if final_ln:
        hn, xhat, rstd = layer_norm(hl, np.asarray(client["final_ln_g"], dtype),
                                    np.asarray(client["final_ln_b"], dtype), shape.ln_eps)
    logits, lse, loss_tok, loss_sum = lm_head_forward(hn, client["lm_head"], labels, dtype)
    dhl, dw_head = lm_head_backward(hn, client["lm_head"], logits, lse, labels, grad_scale, dtype)
    if final_ln:
        dhl, dg_ln, db_ln = layer_norm_backward(dhl, xhat, rstd, np.asarray(client["final_ln_g"], dtype))
    dhs, g_last = stack_backward([client["block_last"]], 1, xsl, dhl, batch, shape,
                                 grads_for([client["block_last"]]), dtype=dtype)
    dh0, g_srv = stack_backward(server_layers, n_srv, xss, dhs, batch, shape, grads_for(server_layers[:n_srv]),
                                dtype=dtype)
    de, g_0 = stack_backward([client["block0"]], 1, xs0, dh0, batch, shape, grads_for([client["block0"]]),
                             dtype=dtype)
    out = {"h0": h0, "h_server": hs, "logits": logits, "lse": lse, "loss_tok": loss_tok, "loss_sum": loss_sum,
           "d_h_server": dhs, "d_h0": dh0, "d_embedded": de,
           "grads_block_last": g_last[0], "grads_server": g_srv, "grads_block0": g_0[0]}
    if train_weights:
        out["grad_lm_head"] = dw_head
        if final_ln:
            out["grad_final_ln_g"], out["grad_final_ln_b"] = dg_ln, db_ln
        out["grad_embedding"] = embedding_backward(ids, de, client["embedding"].shape[0], dtype)
    return out
