"""Pins of the oracle's server update (Adam, Section 4.1.4) and of the
server-hierarchical replica averaging (Section 3.3): torch's own Adam
implementation, closed forms of Adam on constant and alternating gradients
(bias correction and beta1), the first-step sign form, scale invariance, an
arithmetic-series mean, the SGD linearity that ties averaging to client
batching, and a two-step P-tuning training loop against torch autograd with
torch.optim.Adam."""

import math

import numpy as np
import pytest
import torch

import oracle
from tests import torch_block
from tests.test_oracle_pins import TINY, _tiny_batch, _tiny_layers, rel_l2

LR, B1, B2, EPS = oracle.ADAM_LR, oracle.ADAM_BETA1, oracle.ADAM_BETA2, oracle.ADAM_EPS


def test_adam_defaults_follow_the_paper_and_adam():
    assert (LR, B1, B2, EPS) == (2e-2, 0.9, 0.999, 1e-8)


def test_adam_vs_torch_adam():
    """Six steps of seeded gradients: parameters and both moments equal
    torch.optim.Adam (float64, CPU, no weight decay, no amsgrad)."""
    g = np.random.default_rng(0)
    p0 = g.standard_normal(257)
    tp = torch.tensor(p0.copy(), requires_grad=True)
    opt = torch.optim.Adam([tp], lr=LR, betas=(B1, B2), eps=EPS, weight_decay=0.0, foreach=False)
    p, m, v = p0, np.zeros_like(p0), np.zeros_like(p0)
    for t in range(1, 7):
        grad = g.standard_normal(257) * 10.0 ** g.integers(-6, 1)
        tp.grad = torch.tensor(grad)
        opt.step()
        p, m, v = oracle.adam_step(p, grad, m, v, t)
        st = opt.state[tp]
        assert rel_l2(p, tp.detach().numpy()) < 1e-14
        assert rel_l2(m, st["exp_avg"].numpy()) < 1e-14
        assert rel_l2(v, st["exp_avg_sq"].numpy()) < 1e-14


def test_adam_first_step_is_a_signed_step():
    """From zero moments, m_hat = g and v_hat = g^2, so the first step moves
    every entry by lr * g / (|g| + eps)."""
    g = np.array([3.0, -2e-3, 1e-9, 0.0, -7.5])
    p0 = np.array([1.0, 2.0, 3.0, 4.0, 5.0])
    p, m, v = oracle.adam_step(p0, g, np.zeros(5), np.zeros(5), 1)
    assert np.allclose(p, p0 - LR * g / (np.abs(g) + EPS), rtol=0, atol=1e-15)
    assert np.allclose(m, (1 - B1) * g, rtol=1e-15, atol=0)
    assert np.allclose(v, (1 - B2) * g * g, rtol=1e-15, atol=0)


def test_adam_constant_gradient_closed_form():
    """A constant gradient c gives m_t = c (1 - b1^t) and v_t = c^2 (1 - b2^t);
    the bias corrections cancel those factors exactly, so after t steps
    p_t = p_0 - t lr c / (|c| + eps).  Without the corrections the early
    steps would be far smaller."""
    c = np.array([0.5, -4.0, 1e-4])
    p, m, v = np.zeros(3), np.zeros(3), np.zeros(3)
    for t in range(1, 21):
        p, m, v = oracle.adam_step(p, c, m, v, t)
        assert np.allclose(m, c * (1 - B1 ** t), rtol=1e-13, atol=0)
        assert np.allclose(v, c * c * (1 - B2 ** t), rtol=1e-12, atol=0)
        assert np.allclose(p, -t * LR * c / (np.abs(c) + EPS), rtol=1e-12, atol=0)


def test_adam_alternating_gradient_closed_form():
    """g_t = c (-1)^t: m_t = (1 - b1) c (-1)^t (1 - (-b1)^t) / (1 + b1) (a
    geometric series) and v_hat = c^2, so the step at t is
    -lr (1 - b1)(-1)^t (1 - (-b1)^t) / ((1 + b1)(1 - b1^t)) * sign(c)
    (eps = 0 here so the form is exact).  This fixes beta1's role in m."""
    c = 0.3
    p = m = v = np.zeros(1)
    prev = 0.0
    for t in range(1, 12):
        p, m, v = oracle.adam_step(p, np.array([c * (-1) ** t]), m, v, t, eps=0.0)
        m_exp = (1 - B1) * c * (-1) ** t * (1 - (-B1) ** t) / (1 + B1)
        assert math.isclose(m[0], m_exp, rel_tol=1e-13)
        step = -LR * (1 - B1) * (-1) ** t * (1 - (-B1) ** t) / ((1 + B1) * (1 - B1 ** t))
        assert math.isclose(p[0] - prev, step, rel_tol=1e-12)
        prev = p[0]


def test_adam_scale_invariance_without_eps():
    """With eps = 0 the update is invariant to rescaling every gradient by
    the same positive factor (Adam paper, Section 2.1)."""
    g = np.random.default_rng(3)
    grads = [g.standard_normal(64) for _ in range(4)]
    p0 = g.standard_normal(64)
    ra = rb = (p0, np.zeros(64), np.zeros(64))
    for t, gr in enumerate(grads, 1):
        ra = oracle.adam_step(*ra[:1], gr, *ra[1:], t, eps=0.0)
        rb = oracle.adam_step(*rb[:1], 1e5 * gr, *rb[1:], t, eps=0.0)
    assert rel_l2(ra[0], rb[0]) < 1e-14


def test_adam_zero_gradient_leaves_everything():
    p0 = np.array([1.5, -2.0])
    p, m, v = oracle.adam_step(p0, np.zeros(2), np.zeros(2), np.zeros(2), 1)
    assert np.array_equal(p, p0) and not m.any() and not v.any()
    with pytest.raises(ValueError):
        oracle.adam_step(p0, np.zeros(2), np.zeros(2), np.zeros(2), 0)


def test_average_arithmetic_series_and_symmetry():
    """Replicas r_k = a + k d (k = 0..M-1) average to a + (M - 1) d / 2; the
    mean does not depend on the replicas' order; M copies of one tensor
    average to it."""
    g = np.random.default_rng(5)
    a, d = g.standard_normal(33), g.standard_normal(33)
    for M in (1, 2, 3, 10):
        reps = [a + k * d for k in range(M)]
        assert np.allclose(oracle.average_replicas(reps), a + (M - 1) * d / 2, rtol=1e-13, atol=1e-14)
        perm = g.permutation(M)
        assert np.allclose(oracle.average_replicas([reps[i] for i in perm]), oracle.average_replicas(reps),
                           rtol=1e-14, atol=1e-15)
        assert np.allclose(oracle.average_replicas([a] * M), a, rtol=1e-15, atol=0)
    with pytest.raises(ValueError):
        oracle.average_replicas([])


def test_average_of_sgd_replicas_is_client_batch_sgd():
    """One plain gradient step per replica from a common start, then the
    average, equals one step on the client batch with the mean of the
    per-client gradients.  The per-client gradients come from the oracle's
    stack on each client alone; their sum equals the client-batched gradient
    (the client-batching invariance), which ties the two parallel strategies
    of Section 3.3 together at period 1."""
    b = _tiny_batch("causal")
    layers = _tiny_layers()
    g = np.random.default_rng(6)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal((b.total_tokens, TINY.hidden))
    ranges = oracle.client_token_ranges(b.cu_seqlens, b.client_seq_ptr)
    per_client = []
    for c in range(b.num_clients):
        s0, s1 = int(b.client_seq_ptr[c]), int(b.client_seq_ptr[c + 1])
        r0, r1 = ranges[c]
        cu = (b.cu_seqlens[s0:s1 + 1] - b.cu_seqlens[s0]).astype(np.int32)
        sub = type(b)(cu, np.array([0, s1 - s0], np.int32), b.mask, None)
        _, xs = oracle.stack_forward(layers, TINY.num_layers, x[r0:r1], sub, TINY)
        _, gr = oracle.stack_backward(layers, TINY.num_layers, xs, dy[r0:r1], sub, TINY)
        per_client.append(gr)
    _, xs = oracle.stack_forward(layers, TINY.num_layers, x, b, TINY)
    _, batched = oracle.stack_backward(layers, TINY.num_layers, xs, dy, b, TINY)
    lr, M = 0.1, b.num_clients
    for l in range(TINY.num_layers):
        for k in ("w_qkv", "b_o", "ln2_g"):
            replicas = [layers[l][k] - lr * per_client[c][l][k] for c in range(M)]
            assert rel_l2(oracle.average_replicas(replicas), layers[l][k] - lr * batched[l][k] / M) < 1e-13


def test_ptuning_training_loop_vs_torch_adam():
    """Two P-tuning v2 training steps on the tiny stack (weights frozen, the
    prefix trained with Adam at lr 2e-2): the oracle's forward, backward and
    Adam steps against torch autograd of the independent block formulation
    driven by torch.optim.Adam."""
    b = _tiny_batch("prefix")
    layers = _tiny_layers()
    g = np.random.default_rng(8)
    Lp = 3
    for lp in layers:
        lp["prefix_k"] = g.standard_normal((Lp, TINY.hidden)) * 0.3
        lp["prefix_v"] = g.standard_normal((Lp, TINY.hidden)) * 0.3
    xs_in = [g.standard_normal((b.total_tokens, TINY.hidden)) for _ in range(2)]
    dys = [g.standard_normal((b.total_tokens, TINY.hidden)) for _ in range(2)]
    names = ("prefix_k", "prefix_v")

    # torch: frozen weights, trainable prefix tensors
    tl = [{k: torch.tensor(v, requires_grad=k in names) for k, v in lp.items()} for lp in layers]
    opt = torch.optim.Adam([lp[k] for lp in tl for k in names], lr=LR, betas=(B1, B2), eps=EPS, foreach=False)
    for x, dy in zip(xs_in, dys):
        opt.zero_grad()
        cur = torch.tensor(x)
        for lp in tl:
            cur = torch_block.block(lp, cur, b.cu_seqlens, b.prefix_len, TINY)
        (cur * torch.tensor(dy)).sum().backward()
        opt.step()

    # oracle
    cur_layers = [dict(lp) for lp in layers]
    state = [{k: (np.zeros_like(lp[k]), np.zeros_like(lp[k])) for k in names} for lp in layers]
    for t, (x, dy) in enumerate(zip(xs_in, dys), 1):
        _, xs = oracle.stack_forward(cur_layers, TINY.num_layers, x, b, TINY)
        grads = [oracle.zero_prefix_grads(Lp, TINY.hidden) for _ in layers]
        _, grads = oracle.stack_backward(cur_layers, TINY.num_layers, xs, dy, b, TINY, grads)
        for l, lp in enumerate(cur_layers):
            for k in names:
                m, v = state[l][k]
                lp[k], m, v = oracle.adam_step(lp[k], grads[l][k], m, v, t)
                state[l][k] = (m, v)
    for l in range(TINY.num_layers):
        for k in names:
            assert rel_l2(cur_layers[l][k], tl[l][k].detach().numpy()) < 1e-12, (l, k)
        assert cur_layers[l]["w_qkv"] is layers[l]["w_qkv"]
