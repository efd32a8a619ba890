"""Pins of the oracle's P-tuning v2 path (Appendix A, P-tuning v2 section):
learned prefix keys / values spliced in front of every sequence's keys and
values in each block, visible to every query; block weights frozen, only the
prefix trained.  Pinned against brute force, torch autograd of an
independent formulation, a closed form, finite differences, the no-prefix
case and client-batching invariance."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from tests import torch_block
from tests.test_oracle_pins import TINY, _tiny_batch, _tiny_layers, rel_l2

LP = 3  # prefix length used by the small pins


def _prefix(seed, Lp=LP, H=TINY.hidden, std=0.3):
    g = np.random.default_rng(seed)
    return g.standard_normal((Lp, H)) * std, g.standard_normal((Lp, H)) * std


def _brute(q, k, v, pk, pv, batch):
    """Pure-Python loops: query i of a sequence weighs every prefix key and
    its own visible keys."""
    T, nh, d = q.shape
    o = np.zeros_like(q)
    cu = batch.cu_seqlens
    for s in range(len(cu) - 1):
        r0, r1 = int(cu[s]), int(cu[s + 1])
        P = None if batch.mask != "prefix" else int(batch.prefix_len[s])
        for h in range(nh):
            for i in range(r1 - r0):
                keys = [pk[j, h] for j in range(len(pk))]
                vals = [pv[j, h] for j in range(len(pv))]
                for j in range(r1 - r0):
                    if j <= i or (P is not None and j < P):
                        keys.append(k[r0 + j, h])
                        vals.append(v[r0 + j, h])
                sc = [sum(q[r0 + i, h, t] * kk[t] for t in range(d)) / math.sqrt(d) for kk in keys]
                m = max(sc)
                e = [math.exp(x - m) for x in sc]
                z = sum(e)
                for t in range(d):
                    o[r0 + i, h, t] = sum(e[a] * vals[a][t] for a in range(len(vals))) / z
    return o


@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_prefix_attention_brute_force(mask):
    b = _tiny_batch(mask)
    g = np.random.default_rng(11)
    T = b.total_tokens
    q, k, v = (g.standard_normal((T, 2, 4)) for _ in range(3))
    pk, pv = (g.standard_normal((LP, 2, 4)) for _ in range(2))
    o = oracle.attention_forward(q, k, v, b, pk, pv)
    np.testing.assert_allclose(o, _brute(q, k, v, pk, pv, b), rtol=1e-12, atol=1e-12)


def test_empty_prefix_is_plain_attention():
    b = _tiny_batch("prefix")
    g = np.random.default_rng(12)
    T = b.total_tokens
    q, k, v, do = (g.standard_normal((T, 2, 4)) for _ in range(4))
    e = np.zeros((0, 2, 4))
    np.testing.assert_array_equal(oracle.attention_forward(q, k, v, b, e, e), oracle.attention_forward(q, k, v, b))
    dq, dk, dv, dpk, dpv = oracle.attention_backward(q, k, v, do, b, e, e)
    ref = oracle.attention_backward(q, k, v, do, b)
    for a, r in zip((dq, dk, dv), ref):
        np.testing.assert_array_equal(a, r)
    assert dpk.shape == (0, 2, 4) and dpv.shape == (0, 2, 4)


def test_prefix_closed_form():
    """One token, one prefix slot, d = 4 (scale 1/2): q = (2,0,0,0),
    prefix key (1,0,0,0), own key 0 -> scores (1, 0), weights (e, 1)/(e+1)."""
    b = synth.Batch(np.array([0, 1], np.int32), np.array([0, 1], np.int32))
    q = np.array([[[2.0, 0, 0, 0]]])
    k = np.zeros((1, 1, 4))
    v = np.array([[[0.0, 1, 0, 0]]])
    pk = np.array([[[1.0, 0, 0, 0]]])
    pv = np.array([[[1.0, 0, 0, 0]]])
    o = oracle.attention_forward(q, k, v, b, pk, pv)
    e = math.e
    np.testing.assert_allclose(o[0, 0], [e / (e + 1), 1 / (e + 1), 0, 0], rtol=1e-15, atol=1e-15)


def test_prefix_attention_backward_vs_autograd():
    b = synth.make_batch(2, 2, (3, 9), "prefix", 0.25, seed=5)
    g = np.random.default_rng(13)
    T = b.total_tokens
    q, k, v, do = (g.standard_normal((T, 2, 8)) for _ in range(4))
    pk, pv = (g.standard_normal((LP, 2, 8)) for _ in range(2))
    dq, dk, dv, dpk, dpv = oracle.attention_backward(q, k, v, do, b, pk, pv)
    tq, tk, tv, tpk, tpv = (torch.tensor(a, requires_grad=True) for a in (q, k, v, pk, pv))
    outs = []
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        L = r1 - r0
        i = torch.arange(L)[:, None]
        j = torch.arange(L)[None, :]
        m = (j <= i) | ((i < int(b.prefix_len[s])) & (j < int(b.prefix_len[s])))
        m = torch.cat([torch.ones(L, LP, dtype=torch.bool), m], dim=1)
        kk = torch.cat([tpk, tk[r0:r1]], dim=0).transpose(0, 1)
        vv = torch.cat([tpv, tv[r0:r1]], dim=0).transpose(0, 1)
        outs.append(F.scaled_dot_product_attention(tq[r0:r1].transpose(0, 1), kk, vv, attn_mask=m).transpose(0, 1))
    (torch.cat(outs) * torch.tensor(do)).sum().backward()
    for a, ref in ((dq, tq), (dk, tk), (dv, tv), (dpk, tpk), (dpv, tpv)):
        assert rel_l2(a, ref.grad.numpy()) < 1e-12


@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_prefix_stack_vs_torch_autograd(mask):
    b = _tiny_batch(mask)
    layers = _tiny_layers()
    for l, lp in enumerate(layers):
        lp["prefix_k"], lp["prefix_v"] = _prefix(20 + l)
    g = np.random.default_rng(14)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal((b.total_tokens, TINY.hidden))
    y, xs = oracle.stack_forward(layers, TINY.num_layers, x, b, TINY)
    grads = [dict(oracle.zero_grads(TINY), **oracle.zero_prefix_grads(LP, TINY.hidden)) for _ in layers]
    dx, grads = oracle.stack_backward(layers, TINY.num_layers, xs, dy, b, TINY, grads)
    ty, tdx, tg = torch_block.stack_fwd_bwd(layers, x, dy, b, TINY)
    assert rel_l2(y, ty) < 1e-12 and rel_l2(dx, tdx) < 1e-12
    for l in range(TINY.num_layers):
        for k in grads[l]:
            assert rel_l2(grads[l][k], tg[l][k]) < 1e-11, (l, k)


def test_prefix_finite_differences_frozen_weights():
    """Weights frozen (only prefix gradients requested): central differences
    of sum(y * dy) in float64 for every prefix entry of both layers."""
    b = _tiny_batch("causal")
    layers = _tiny_layers()
    for l, lp in enumerate(layers):
        lp["prefix_k"], lp["prefix_v"] = _prefix(30 + l, Lp=2)
    g = np.random.default_rng(15)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal((b.total_tokens, TINY.hidden))
    _, xs = oracle.stack_forward(layers, TINY.num_layers, x, b, TINY)
    grads = [oracle.zero_prefix_grads(2, TINY.hidden) for _ in layers]
    _, grads = oracle.stack_backward(layers, TINY.num_layers, xs, dy, b, TINY, grads)
    assert all(set(gr) == {"prefix_k", "prefix_v"} for gr in grads)

    def f():
        y, _ = oracle.stack_forward(layers, TINY.num_layers, x, b, TINY, keep="none")
        return float((y * dy).sum())

    eps = 1e-5
    for l in range(TINY.num_layers):
        for name in ("prefix_k", "prefix_v"):
            a = layers[l][name]
            num = np.zeros_like(a)
            for idx in np.ndindex(a.shape):
                old = a[idx]
                a[idx] = old + eps
                fp = f()
                a[idx] = old - eps
                fm = f()
                a[idx] = old
                num[idx] = (fp - fm) / (2 * eps)
            assert rel_l2(grads[l][name], num) < 1e-7, (l, name)


def test_prefix_client_batching_invariance():
    """Client batching stays exact with a prefix: each client's rows equal its
    own run, and the prefix gradient is the sum of the clients' gradients."""
    b = synth.make_batch(3, 2, (2, 7), "causal", seed=8)
    layers = _tiny_layers(std=0.1)
    for l, lp in enumerate(layers):
        lp["prefix_k"], lp["prefix_v"] = _prefix(40 + l)
    g = np.random.default_rng(16)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal((b.total_tokens, TINY.hidden))
    y, xs = oracle.stack_forward(layers, 2, x, b, TINY)
    gr = [oracle.zero_prefix_grads(LP, TINY.hidden) for _ in range(2)]
    dx, gr = oracle.stack_backward(layers, 2, xs, dy, b, TINY, gr)
    acc = [oracle.zero_prefix_grads(LP, TINY.hidden) for _ in range(2)]
    ranges = oracle.client_token_ranges(b.cu_seqlens, b.client_seq_ptr)
    for c in range(b.num_clients):
        s0, s1 = int(b.client_seq_ptr[c]), int(b.client_seq_ptr[c + 1])
        r0, r1 = ranges[c]
        cu = (b.cu_seqlens[s0:s1 + 1] - b.cu_seqlens[s0]).astype(np.int32)
        sub = synth.Batch(cu, np.array([0, s1 - s0], np.int32))
        yc, xsc = oracle.stack_forward(layers, 2, x[r0:r1], sub, TINY)
        dxc, acc = oracle.stack_backward(layers, 2, xsc, dy[r0:r1], sub, TINY, acc)
        assert rel_l2(y[r0:r1], yc) < 1e-13 and rel_l2(dx[r0:r1], dxc) < 1e-13
    for l in range(2):
        for k in acc[l]:
            assert rel_l2(gr[l][k], acc[l][k]) < 1e-12, (l, k)
