"""Pins of the oracle's client side (Section 3.1, Model Split): the embedding
gather and its scatter-add gradient, the final linear layer with the
cross-entropy loss, and one whole split training step, against torch library
routines (F.embedding, F.linear, F.cross_entropy) driven by autograd, closed
forms and finite differences."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import client as oc
from tests import torch_block
from tests.test_oracle_pins import TINY, _tiny_batch, _tiny_layers, rel_l2

V = 50


def _ids_labels(b, seed, vocab=V):
    """Token ids with repeats; labels = next token inside each sequence, the
    last token of a sequence unlabelled (-100)."""
    g = np.random.default_rng(seed)
    ids = g.integers(0, vocab, b.total_tokens).astype(np.int32)
    ids[:4] = 7  # a repeated id
    labels = np.full(b.total_tokens, -100, np.int32)
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        labels[r0:r1 - 1] = ids[r0 + 1:r1]
    return ids, labels


def test_embedding_vs_torch():
    g = np.random.default_rng(0)
    table = g.standard_normal((V, 16))
    ids = np.array([3, 7, 7, 0, 49, 7, 3], np.int32)
    dh = g.standard_normal((len(ids), 16))
    tt = torch.tensor(table, requires_grad=True)
    out = F.embedding(torch.tensor(ids, dtype=torch.long), tt)
    (out * torch.tensor(dh)).sum().backward()
    assert np.array_equal(oc.embedding_forward(table, ids), out.detach().numpy())
    assert rel_l2(oc.embedding_backward(ids, dh, V), tt.grad.numpy()) < 1e-15
    # untouched rows stay zero; a thrice-used row is the sum of its three rows
    dt = oc.embedding_backward(ids, dh, V)
    assert not dt[[1, 2, 48]].any()
    assert np.allclose(dt[7], dh[1] + dh[2] + dh[5], rtol=0, atol=1e-15)


@pytest.mark.parametrize("scale", [1.0, 0.125])
def test_lm_head_vs_torch_cross_entropy(scale):
    g = np.random.default_rng(1)
    T, H = 13, 16
    h = g.standard_normal((T, H))
    w = g.standard_normal((V, H)) * 0.5
    labels = g.integers(0, V, T).astype(np.int32)
    labels[[2, 5]] = -100
    th = torch.tensor(h, requires_grad=True)
    tw = torch.tensor(w, requires_grad=True)
    logits = F.linear(th, tw)
    per = F.cross_entropy(logits, torch.tensor(labels, dtype=torch.long), ignore_index=-100, reduction="none")
    (per.sum() * scale).backward()
    lg, lse, loss_tok, loss_sum = oc.lm_head_forward(h, w, labels)
    assert rel_l2(lg, logits.detach().numpy()) < 1e-15
    assert rel_l2(loss_tok, per.detach().numpy()) < 1e-14
    assert math.isclose(loss_sum, float(per.sum().detach()), rel_tol=1e-14)
    assert np.allclose(lse, torch.logsumexp(logits, 1).detach().numpy(), rtol=1e-15, atol=0)
    dh, dw = oc.lm_head_backward(h, w, lg, lse, labels, scale)
    assert rel_l2(dh, th.grad.numpy()) < 1e-14
    assert rel_l2(dw, tw.grad.numpy()) < 1e-14


def test_lm_head_closed_forms():
    """Zero weights give uniform logits: every labelled token costs log V,
    dlogits = scale (1/V - onehot), so dh = 0 and dW = dlogits^T h.  Two
    classes: the loss is the softplus of the logit margin."""
    g = np.random.default_rng(2)
    T, H = 6, 8
    h = g.standard_normal((T, H))
    labels = np.array([0, 3, -1, 49, 10, 10], np.int32)
    lg, lse, loss_tok, loss_sum = oc.lm_head_forward(h, np.zeros((V, H)), labels)
    ok = labels >= 0
    assert np.allclose(loss_tok[ok], math.log(V), rtol=1e-15) and loss_tok[~ok].sum() == 0
    assert math.isclose(loss_sum, 5 * math.log(V), rel_tol=1e-14)
    dh, dw = oc.lm_head_backward(h, np.zeros((V, H)), lg, lse, labels, 0.5)
    assert not dh.any()
    d = np.where(ok[:, None], 1.0 / V, 0.0) * np.ones((T, V))
    d[np.nonzero(ok)[0], labels[ok]] -= 1.0
    assert np.allclose(dw, 0.5 * d.T @ h, rtol=1e-13, atol=1e-15)
    # V = 2: loss = log(1 + exp(l_other - l_label))
    w2 = g.standard_normal((2, H))
    _, _, lt, _ = oc.lm_head_forward(h[:1], w2, np.array([1]))
    l0, l1 = h[0] @ w2[0], h[0] @ w2[1]
    assert math.isclose(lt[0], math.log1p(math.exp(l0 - l1)), rel_tol=1e-13)


def test_unlabelled_tokens_contribute_nothing():
    g = np.random.default_rng(3)
    T, H = 9, 8
    h, w = g.standard_normal((T, H)), g.standard_normal((V, H))
    labels = g.integers(0, V, T).astype(np.int32)
    lg, lse, lt, ls = oc.lm_head_forward(h, w, labels)
    dh, dw = oc.lm_head_backward(h, w, lg, lse, labels, 1.0)
    lab2 = labels.copy()
    lab2[4] = -100
    lg2, lse2, lt2, ls2 = oc.lm_head_forward(h, w, lab2)
    dh2, dw2 = oc.lm_head_backward(h, w, lg2, lse2, lab2, 1.0)
    assert lt2[4] == 0 and math.isclose(ls2, ls - lt[4], rel_tol=1e-14)
    assert not dh2[4].any()
    assert np.allclose(np.delete(dh2, 4, 0), np.delete(dh, 4, 0), rtol=0, atol=1e-15)


def _client(seed, with_prefix):
    g = np.random.default_rng(seed)
    blocks = _tiny_layers(seed=seed + 1)
    for lp in blocks:
        if with_prefix:
            lp["prefix_k"] = g.standard_normal((3, TINY.hidden)) * 0.3
            lp["prefix_v"] = g.standard_normal((3, TINY.hidden)) * 0.3
    return {"embedding": g.standard_normal((V, TINY.hidden)), "block0": blocks[0], "block_last": blocks[1],
            "lm_head": g.standard_normal((V, TINY.hidden)) * 0.3}


def _torch_split(client, server, ids, labels, b, scale, train_weights):
    """Independent formulation: torch embedding, the torch block, linear and
    cross-entropy, gradients by autograd."""
    def leaf(a, trainable):
        return torch.tensor(np.asarray(a, np.float64), requires_grad=trainable)
    tc = {"embedding": leaf(client["embedding"], train_weights), "lm_head": leaf(client["lm_head"], train_weights)}
    blocks = {}
    for name, lp in [("block0", client["block0"]), ("block_last", client["block_last"])] + \
            [(f"s{i}", lp) for i, lp in enumerate(server)]:
        blocks[name] = {k: leaf(v, train_weights or k.startswith("prefix_")) for k, v in lp.items()}
    pre = b.prefix_len if b.mask == "prefix" else None
    cur = F.embedding(torch.tensor(ids, dtype=torch.long), tc["embedding"])
    cur = torch_block.block(blocks["block0"], cur, b.cu_seqlens, pre, TINY)
    h0 = cur
    h0.retain_grad()
    for i in range(len(server)):
        cur = torch_block.block(blocks[f"s{i}"], cur, b.cu_seqlens, pre, TINY)
    hs = cur
    hs.retain_grad()
    cur = torch_block.block(blocks["block_last"], cur, b.cu_seqlens, pre, TINY)
    loss = F.cross_entropy(F.linear(cur, tc["lm_head"]), torch.tensor(labels, dtype=torch.long),
                           ignore_index=-100, reduction="sum")
    (loss * scale).backward()
    return loss, h0, hs, tc, blocks


@pytest.mark.parametrize("mask,train_weights", [("causal", True), ("prefix", False)])
def test_split_step_vs_torch_autograd(mask, train_weights):
    """One whole split step (client embedding and block 0, a 2-block server,
    client block N-1, linear, cross-entropy) against torch autograd: loss, the
    gradients at both split boundaries, every trained gradient."""
    b = _tiny_batch(mask)
    client = _client(4, with_prefix=not train_weights)
    server = _tiny_layers(seed=9)
    if not train_weights:
        g = np.random.default_rng(5)
        for lp in server:
            lp["prefix_k"] = g.standard_normal((3, TINY.hidden)) * 0.3
            lp["prefix_v"] = g.standard_normal((3, TINY.hidden)) * 0.3
    ids, labels = _ids_labels(b, 6)
    scale = 1.0 / int((labels >= 0).sum())
    r = oc.split_step(client, server, ids, labels, b, TINY, scale, train_weights=train_weights)
    loss, h0, hs, tc, blocks = _torch_split(client, server, ids, labels, b, scale, train_weights)
    assert math.isclose(r["loss_sum"], float(loss.detach()), rel_tol=1e-12)
    assert rel_l2(r["h0"], h0.detach().numpy()) < 1e-13
    assert rel_l2(r["h_server"], hs.detach().numpy()) < 1e-13
    assert rel_l2(r["d_h0"], h0.grad.numpy()) < 1e-11
    assert rel_l2(r["d_h_server"], hs.grad.numpy()) < 1e-11
    if train_weights:
        assert rel_l2(r["grad_lm_head"], tc["lm_head"].grad.numpy()) < 1e-11
        assert rel_l2(r["grad_embedding"], tc["embedding"].grad.numpy()) < 1e-11
    pairs = [("grads_block0", "block0"), ("grads_block_last", "block_last")] + \
        [(None, f"s{i}") for i in range(len(server))]
    for key, name in pairs:
        mine = r[key] if key else r["grads_server"][int(name[1:])]
        for k, v in mine.items():
            assert rel_l2(v, blocks[name][k].grad.numpy()) < 1e-10, (name, k)
        if not train_weights:
            assert set(mine) == {"prefix_k", "prefix_v"}


def test_split_step_finite_differences():
    """Central differences of scale * loss_sum in float64 for a few entries of
    the embedding table, the final linear layer and block 0's QKV weight."""
    b = _tiny_batch("causal")
    client = _client(7, with_prefix=False)
    server = _tiny_layers(seed=8)[:1]
    ids, labels = _ids_labels(b, 8)
    scale = 0.25
    r = oc.split_step(client, server, ids, labels, b, TINY, scale)
    eps = 1e-6

    def loss_with(path, idx, delta):
        c = {k: (dict(v) if isinstance(v, dict) else v.copy()) for k, v in client.items()}
        tgt = c[path[0]] if len(path) == 1 else c[path[0]]
        if len(path) == 2:
            tgt[path[1]] = tgt[path[1]].copy()
            tgt[path[1]][idx] += delta
        else:
            c[path[0]] = tgt.copy()
            c[path[0]][idx] += delta
        return scale * oc.split_step(c, server, ids, labels, b, TINY, scale)["loss_sum"]

    checks = [(("embedding",), (7, 3), r["grad_embedding"]), (("embedding",), (int(ids[9]), 0), r["grad_embedding"]),
              (("lm_head",), (int(labels[0]), 5), r["grad_lm_head"]), (("lm_head",), (11, 2), r["grad_lm_head"]),
              (("block0", "w_qkv"), (40, 3), r["grads_block0"]["w_qkv"]),
              (("block0", "b_o"), (6,), r["grads_block0"]["b_o"])]
    for path, idx, grad in checks:
        fd = (loss_with(path, idx, eps) - loss_with(path, idx, -eps)) / (2 * eps)
        assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(fd)), (path, idx, fd, grad[idx])
