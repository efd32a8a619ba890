"""Pins of the oracle's ChatGLM-6B-exact block variant (the paper's base
model, Section 4.1.4; the architecture details are ChatGLM-6B's own, not the
paper's): the residual on the normalised input scaled by alpha = sqrt(2 x 28),
GLM 2-D rotary positions, and the final LayerNorm in front of the client's
linear layer.  Pinned against an independent torch formulation with
autograd, hand-derived positions, closed forms, the invariance of 2-D
positions on context-only sequences, and finite differences."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import client as oc
from tests import torch_block
from tests.test_oracle_pins import TINY, _tiny_batch, _tiny_layers, rel_l2

ALPHA = math.sqrt(2 * 28)


def _shape(alpha=ALPHA, two_d=True, base=TINY):
    return synth.StackShape(base.num_layers, base.hidden, base.num_heads, base.ffn_hidden, base.head_dim // 2,
                            base.rope_base, base.ln_eps, alpha, two_d)


def test_glm_positions_by_hand():
    """Two sequences: L = 5 with a 2-token context ([gMASK] at 1), L = 3 with
    a 3-token context (all context); a causal batch counts every token as
    context."""
    b = synth.Batch(np.array([0, 5, 8], np.int32), np.array([0, 2], np.int32), "prefix", np.array([2, 3], np.int32))
    p1, p2 = oracle.glm_positions(b)
    assert p1.tolist() == [0, 1, 1, 1, 1, 0, 1, 2]
    assert p2.tolist() == [0, 0, 1, 2, 3, 0, 0, 0]
    bp0 = synth.Batch(np.array([0, 4], np.int32), np.array([0, 1], np.int32), "prefix", np.array([0], np.int32))
    p1, p2 = oracle.glm_positions(bp0)  # empty context: mask position clamps to 0
    assert p1.tolist() == [0, 0, 0, 0] and p2.tolist() == [1, 2, 3, 4]
    bc = synth.Batch(np.array([0, 4], np.int32), np.array([0, 1], np.int32), "causal", None)
    p1, p2 = oracle.glm_positions(bc)
    assert p1.tolist() == [0, 1, 2, 3] and p2.tolist() == [0, 0, 0, 0]


def test_2d_rotation_closed_form():
    """A key that is e_0 in the second half of head 0, at a token whose block
    position is 2, comes out of the block's rotation as (cos 2, sin 2) on dims
    (r, r + r/2): the lowest frequency pair turns by 2 * theta_0 = 2 rad."""
    sh = _shape(two_d=True)
    r = sh.rotary_dim
    b = synth.Batch(np.array([0, 5], np.int32), np.array([0, 1], np.int32), "prefix", np.array([2], np.int32))
    p1, p2 = oracle.glm_positions(b)
    tables = oracle.rope_tables(p1, r, sh.rope_base) + oracle.rope_tables(p2, r, sh.rope_base)
    x = np.zeros((5, sh.num_heads, sh.head_dim))
    x[:, 0, r] = 1.0
    from oracle.block import _rotate_qk
    y = _rotate_qk(x, tables, sh)
    assert p2[3] == 2
    assert math.isclose(y[3, 0, r], math.cos(2.0), abs_tol=1e-15)
    assert math.isclose(y[3, 0, r + r // 2], math.sin(2.0), abs_tol=1e-15)
    assert not y[3, 0, :r].any()  # the first half is untouched by the second rotation


def test_2d_positions_on_context_only_sequences_change_nothing():
    """Causal batches are all context: block positions are 0, so the 2-D
    rotation equals the 1-D one bit for bit."""
    b = _tiny_batch("causal")
    layers = _tiny_layers()
    x = np.random.default_rng(1).standard_normal((b.total_tokens, TINY.hidden))
    y1, _ = oracle.stack_forward(layers, 2, x, b, _shape(alpha=0.0, two_d=False))
    y2, _ = oracle.stack_forward(layers, 2, x, b, _shape(alpha=0.0, two_d=True))
    assert np.array_equal(y1, y2)


def test_alpha_residual_closed_form():
    """Zero weights and biases, unit gains and zero shifts: h = alpha LN(x)
    and y = alpha LN(h), i.e. y = alpha * n(alpha * n(x)) with n the
    normalisation with eps."""
    sh = _shape(two_d=False)
    b = _tiny_batch("causal")
    H = sh.hidden
    p = {k: np.zeros(s) for k, s in synth.param_shapes(sh).items()}
    p["ln1_g"] = np.ones(H)
    p["ln2_g"] = np.ones(H)
    x = np.random.default_rng(2).standard_normal((b.total_tokens, H)) * 3 + 1

    def n(v):
        c = v - v.mean(axis=1, keepdims=True)
        return c / np.sqrt((c ** 2).mean(axis=1, keepdims=True) + sh.ln_eps)
    y, _ = oracle.block_forward(p, x, b, sh)
    assert np.allclose(y, ALPHA * n(ALPHA * n(x)), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("mask,two_d", [("causal", False), ("prefix", True), ("prefix", False)])
def test_glm_stack_vs_torch_autograd(mask, two_d):
    sh = _shape(two_d=two_d)
    b = _tiny_batch(mask)
    layers = _tiny_layers()
    g = np.random.default_rng(3)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal((b.total_tokens, TINY.hidden))
    y, xs = oracle.stack_forward(layers, 2, x, b, sh)
    dx, grads = oracle.stack_backward(layers, 2, xs, dy, b, sh)
    ty, tdx, tg = torch_block.stack_fwd_bwd(layers, x, dy, b, sh)
    assert rel_l2(y, ty) < 1e-12 and rel_l2(dx, tdx) < 1e-12
    for l in range(2):
        for k in grads[l]:
            assert rel_l2(grads[l][k], tg[l][k]) < 1e-11, (l, k)


def test_glm_block_finite_differences():
    """Central differences of sum(y * dy) for entries of x and of parameters
    the alpha residual routes gradient through (both LayerNorms)."""
    sh = _shape(two_d=True)
    b = _tiny_batch("prefix")
    p = _tiny_layers()[0]
    g = np.random.default_rng(4)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal((b.total_tokens, TINY.hidden))
    _, cache = oracle.block_forward(p, x, b, sh)
    grads = oracle.zero_grads(sh)
    dx = oracle.block_backward(p, cache, dy, b, sh, grads)
    eps = 1e-6

    def f(pp, xx):
        return float((oracle.block_forward(pp, xx, b, sh)[0] * dy).sum())
    for (t, j) in [(0, 0), (5, 7), (11, 31)]:
        xp, xm = x.copy(), x.copy()
        xp[t, j] += eps
        xm[t, j] -= eps
        fd = (f(p, xp) - f(p, xm)) / (2 * eps)
        assert abs(fd - dx[t, j]) <= 1e-6 * max(1.0, abs(fd))
    for k, idx in [("ln1_g", (3,)), ("ln2_b", (9,)), ("ln2_g", (20,)), ("w_qkv", (70, 5))]:
        pp, pm = dict(p), dict(p)
        pp[k], pm[k] = p[k].copy(), p[k].copy()
        pp[k][idx] += eps
        pm[k][idx] -= eps
        fd = (f(pp, x) - f(pm, x)) / (2 * eps)
        assert abs(fd - grads[k][idx]) <= 1e-6 * max(1.0, abs(fd)), (k, fd, grads[k][idx])


def test_final_layernorm_head_vs_torch():
    """The client's final LayerNorm + linear + cross-entropy in the split
    step: loss and gradients against F.layer_norm / F.linear /
    F.cross_entropy with autograd, through a whole split step."""
    sh = _shape(two_d=True)
    b = _tiny_batch("prefix")
    g = np.random.default_rng(5)
    V = 40
    blocks = _tiny_layers(seed=6)
    client = {"embedding": g.standard_normal((V, TINY.hidden)), "block0": blocks[0], "block_last": blocks[1],
              "lm_head": g.standard_normal((V, TINY.hidden)) * 0.3,
              "final_ln_g": 1 + 0.1 * g.standard_normal(TINY.hidden), "final_ln_b": 0.1 * g.standard_normal(TINY.hidden)}
    server = _tiny_layers(seed=7)[:1]
    ids = g.integers(0, V, b.total_tokens).astype(np.int32)
    labels = np.roll(ids, -1).astype(np.int32)
    labels[[3, 7]] = -100
    r = oc.split_step(client, server, ids, labels, b, sh, 0.5)

    def leaf(a):
        return torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    tl = {k: leaf(v) for k, v in client.items() if not isinstance(v, dict)}
    tb = [{k: leaf(v) for k, v in lp.items()} for lp in (blocks[0], server[0], blocks[1])]
    pre = b.prefix_len
    cur = F.embedding(torch.tensor(ids, dtype=torch.long), tl["embedding"])
    for lp in tb:
        cur = torch_block.block(lp, cur, b.cu_seqlens, pre, sh)
    cur = F.layer_norm(cur, (TINY.hidden,), tl["final_ln_g"], tl["final_ln_b"], sh.ln_eps)
    loss = F.cross_entropy(F.linear(cur, tl["lm_head"]), torch.tensor(labels, dtype=torch.long), ignore_index=-100,
                           reduction="sum")
    (0.5 * loss).backward()
    assert math.isclose(r["loss_sum"], float(loss.detach()), rel_tol=1e-12)
    for k in ("lm_head", "embedding", "final_ln_g", "final_ln_b"):
        assert rel_l2(r["grad_" + k], tl[k].grad.numpy()) < 1e-11, k
    assert rel_l2(r["grads_block0"]["w_qkv"], tb[0]["w_qkv"].grad.numpy()) < 1e-10
