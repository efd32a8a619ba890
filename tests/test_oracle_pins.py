"""Pins of the CPU oracle against things other than itself: brute force,
library routines, closed forms, finite differences and the invariants that
the paper's client-batch method implies (Section 3.3: stacking clients into
one batch changes nothing per client)."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from tests import torch_block

TINY = synth.StackShape(num_layers=2, hidden=32, num_heads=4, ffn_hidden=128, rotary_dim=4)


def _tiny_batch(mask="causal"):
    # clients with sequence lengths {3, 5} and {4}
    cu = np.array([0, 3, 8, 12], np.int32)
    csp = np.array([0, 2, 3], np.int32)
    pre = np.array([1, 2, 2], np.int32) if mask == "prefix" else None
    return synth.Batch(cu, csp, mask, pre)


def _tiny_layers(shape=TINY, seed=0, std=0.2):
    # larger std than the workloads so every term matters in finite differences
    return [{k: v.astype(np.float64) for k, v in synth.layer_params(shape, l, seed=seed, bf16=False,
                                                                      std=std).items()}
            for l in range(shape.num_layers)]


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


# ---------------------------------------------------------------------------
# Attention: brute force, library, special cases
# ---------------------------------------------------------------------------

def _brute_attention(q, k, v, L, prefix):
    """Pure-Python loops: for each query, exp-weights over the keys it may see."""
    nh, d = q.shape[1], q.shape[2]
    o = np.zeros_like(q)
    for h in range(nh):
        for i in range(L):
            vis = [j for j in range(L) if j <= i or (prefix is not None and j < prefix)]
            s = [sum(q[i, h, t] * k[j, h, t] for t in range(d)) / math.sqrt(d) for j in vis]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for t in range(d):
                o[i, h, t] = sum(e[a] * v[vis[a], h, t] for a in range(len(vis))) / z
    return o


@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_attention_brute_force(mask):
    b = _tiny_batch(mask)
    g = np.random.default_rng(1)
    T = b.total_tokens
    q, k, v = (g.standard_normal((T, 2, 5)) for _ in range(3))
    o = oracle.attention_forward(q, k, v, b)
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        pre = int(b.prefix_len[s]) if mask == "prefix" else None
        ref = _brute_attention(q[r0:r1], k[r0:r1], v[r0:r1], r1 - r0, pre)
        np.testing.assert_allclose(o[r0:r1], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_attention_vs_torch_sdpa(mask):
    b = synth.make_batch(2, 2, (5, 19), mask, 0.25, seed=3)
    g = np.random.default_rng(2)
    T = b.total_tokens
    q, k, v = (g.standard_normal((T, 3, 16)) for _ in range(3))
    o = oracle.attention_forward(q, k, v, b)
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        L = r1 - r0
        i = torch.arange(L)[:, None]
        j = torch.arange(L)[None, :]
        m = j <= i
        if mask == "prefix":
            P = int(b.prefix_len[s])
            m = m | ((i < P) & (j < P))
        t = lambda a: torch.tensor(a[r0:r1]).transpose(0, 1)
        ref = F.scaled_dot_product_attention(t(q), t(k), t(v), attn_mask=m).transpose(0, 1).numpy()
        assert rel_l2(o[r0:r1], ref) < 1e-12


def test_attention_special_cases():
    g = np.random.default_rng(4)
    # L = 1: the only visible key is the query's own -> o = v exactly
    b1 = synth.Batch(np.array([0, 1, 2], np.int32), np.array([0, 2], np.int32))
    q, k, v = (g.standard_normal((2, 2, 8)) for _ in range(3))
    np.testing.assert_array_equal(oracle.attention_forward(q, k, v, b1), v)
    # q = 0: uniform weights -> o_i = mean of v_0..v_i (causal)
    b = synth.Batch(np.array([0, 6], np.int32), np.array([0, 1], np.int32))
    q = np.zeros((6, 1, 4))
    k, v = g.standard_normal((6, 1, 4)), g.standard_normal((6, 1, 4))
    o = oracle.attention_forward(q, k, v, b)
    ref = np.cumsum(v, axis=0) / np.arange(1, 7)[:, None, None]
    np.testing.assert_allclose(o, ref, rtol=1e-13, atol=1e-13)
    # prefix covering the whole sequence: plain bidirectional attention
    bp = synth.Batch(np.array([0, 6], np.int32), np.array([0, 1], np.int32), "prefix",
                     np.array([6], np.int32))
    q = g.standard_normal((6, 1, 4))
    o = oracle.attention_forward(q, k, v, bp)
    ref = F.scaled_dot_product_attention(*(torch.tensor(a).transpose(0, 1) for a in (q, k, v)))
    np.testing.assert_allclose(o, ref.transpose(0, 1).numpy(), rtol=1e-12, atol=1e-12)
    # prefix of 0 or 1 tokens is the causal mask
    for P in (0, 1):
        bp.prefix_len = np.array([P], np.int32)
        np.testing.assert_array_equal(oracle.attention_forward(q, k, v, bp),
                                      oracle.attention_forward(q, k, v, b))


def test_attention_backward_vs_autograd():
    b = synth.make_batch(2, 2, (3, 9), "prefix", 0.25, seed=5)
    g = np.random.default_rng(6)
    T = b.total_tokens
    q, k, v, do = (g.standard_normal((T, 2, 8)) for _ in range(4))
    dq, dk, dv = oracle.attention_backward(q, k, v, do, b)
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    outs = []
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        L = r1 - r0
        i = torch.arange(L)[:, None]
        j = torch.arange(L)[None, :]
        m = (j <= i) | ((i < int(b.prefix_len[s])) & (j < int(b.prefix_len[s])))
        sl = lambda a: a[r0:r1].transpose(0, 1)
        outs.append(F.scaled_dot_product_attention(sl(tq), sl(tk), sl(tv), attn_mask=m).transpose(0, 1))
    (torch.cat(outs) * torch.tensor(do)).sum().backward()
    for a, ref in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        assert rel_l2(a, ref.numpy()) < 1e-12


@pytest.mark.parametrize("mask", ["causal", "prefix"])
@pytest.mark.parametrize("num_prefix", [0, 3])
def test_attention_query_rows_vs_torch_autograd(mask, num_prefix):
    """The few-rows attention of one long sequence against torch SDPA with an
    explicit mask and autograd: o and the log-sum-exp of the chosen rows, and
    with a zero output gradient on every other row, dq of the rows and dk, dv
    and the prefix gradients of the whole sequence."""
    g = np.random.default_rng(7)
    L, nh, d = 37, 2, 8
    P = 9 if mask == "prefix" else None
    q, k, v = (g.standard_normal((L, nh, d)) for _ in range(3))
    pk, pv = (g.standard_normal((num_prefix, nh, d)) if num_prefix else None for _ in range(2))
    rows = np.array([0, 5, 8, 9, 20, 35, 36])
    do = g.standard_normal((len(rows), nh, d))
    o, lse, dq, dk, dv, dpk, dpv = oracle.attention_query_rows(q, k, v, rows, P, pk, pv, do)
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    tpk, tpv = (torch.tensor(a if num_prefix else np.zeros((0, nh, d)), requires_grad=True) for a in (pk, pv))
    i = torch.arange(L)[:, None]
    j = torch.arange(L)[None, :]
    m = j <= i if P is None else (j <= i) | (j < P)
    m = torch.cat([torch.ones((L, num_prefix), dtype=torch.bool), m], dim=1)
    kk, vv = torch.cat([tpk, tk]).transpose(0, 1), torch.cat([tpv, tv]).transpose(0, 1)
    ref = F.scaled_dot_product_attention(tq.transpose(0, 1), kk, vv, attn_mask=m).transpose(0, 1)
    S = torch.where(m, (tq.transpose(0, 1) @ kk.transpose(1, 2)) / math.sqrt(d), -torch.inf)
    ref_lse = torch.logsumexp(S, dim=-1).transpose(0, 1)
    assert rel_l2(o, ref.detach().numpy()[rows]) < 1e-12
    assert rel_l2(lse, ref_lse.detach().numpy()[rows]) < 1e-12
    full_do = torch.zeros((L, nh, d), dtype=torch.float64)
    full_do[rows] = torch.tensor(do)
    (ref * full_do).sum().backward()
    assert rel_l2(dq, tq.grad.numpy()[rows]) < 1e-12
    assert rel_l2(dk, tk.grad.numpy()) < 1e-12 and rel_l2(dv, tv.grad.numpy()) < 1e-12
    if num_prefix:
        assert rel_l2(dpk, tpk.grad.numpy()) < 1e-12 and rel_l2(dpv, tpv.grad.numpy()) < 1e-12


# ---------------------------------------------------------------------------
# LayerNorm, GeLU, rotary
# ---------------------------------------------------------------------------

def test_layer_norm_and_gelu_vs_torch():
    g = np.random.default_rng(7)
    x = g.standard_normal((9, 24)) * 3 + 1
    ga, be = g.standard_normal(24), g.standard_normal(24)
    y, xhat, rstd = oracle.layer_norm(x, ga, be, 1e-5)
    ref = F.layer_norm(torch.tensor(x), (24,), torch.tensor(ga), torch.tensor(be), 1e-5).numpy()
    assert rel_l2(y, ref) < 1e-13
    z = np.linspace(-8, 8, 1001)
    tz = torch.tensor(z, requires_grad=True)
    gz = F.gelu(tz, approximate="tanh")
    gz.sum().backward()
    np.testing.assert_allclose(oracle.gelu(z), gz.detach().numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(oracle.gelu_grad(z), tz.grad.numpy(), rtol=1e-12, atol=1e-14)
    # layer norm backward against autograd
    tx = torch.tensor(x, requires_grad=True)
    tg = torch.tensor(ga, requires_grad=True)
    tb = torch.tensor(be, requires_grad=True)
    dy = g.standard_normal(x.shape)
    (F.layer_norm(tx, (24,), tg, tb, 1e-5) * torch.tensor(dy)).sum().backward()
    dx, dga, dbe = oracle.layer_norm_backward(dy, xhat, rstd, ga)
    assert rel_l2(dx, tx.grad.numpy()) < 1e-12
    assert rel_l2(dga, tg.grad.numpy()) < 1e-12
    assert rel_l2(dbe, tb.grad.numpy()) < 1e-12


def test_rope_closed_form():
    """Head dim 8, r = 4 (pairs (0,2), (1,3)), base 10000, position 1:
    theta_0 = 1, theta_1 = 10000^(-1/2) = 0.01.  Unit vector e_0 goes to
    (cos 1, 0, sin 1, 0, ...); e_3 goes to (0, -sin .01, 0, cos .01, ...);
    dims 4..7 are untouched."""
    cos, sin = oracle.rope_tables(np.array([1]), 4, 10000.0)
    np.testing.assert_allclose(cos[0], [math.cos(1.0), math.cos(0.01)], rtol=1e-15)
    x = np.zeros((1, 2, 8))
    x[0, 0, 0] = 1.0
    x[0, 1, 3] = 1.0
    x[0, :, 4:] = 7.0
    y = oracle.rope(x, cos, sin, 4)
    np.testing.assert_allclose(y[0, 0, :4], [math.cos(1), 0, math.sin(1), 0], atol=1e-15)
    np.testing.assert_allclose(y[0, 1, :4], [0, -math.sin(0.01), 0, math.cos(0.01)], atol=1e-15)
    np.testing.assert_array_equal(y[0, :, 4:], 7.0)


def test_rope_invariants():
    g = np.random.default_rng(8)
    pos = np.arange(40)
    cos, sin = oracle.rope_tables(pos, 16, 10000.0)
    q = g.standard_normal((40, 3, 32))
    k = g.standard_normal((40, 3, 32))
    qr, kr = oracle.rope(q, cos, sin, 16), oracle.rope(k, cos, sin, 16)
    # position 0 is the identity; norms are preserved; inverse undoes it
    np.testing.assert_array_equal(qr[0], q[0])
    np.testing.assert_allclose(np.linalg.norm(qr, axis=2), np.linalg.norm(q, axis=2), rtol=1e-13)
    np.testing.assert_allclose(oracle.rope(qr, cos, sin, 16, inverse=True), q, atol=1e-13)
    # relative position: q_i . k_j depends only on i - j
    c2, s2 = oracle.rope_tables(pos + 17, 16, 10000.0)
    q2, k2 = oracle.rope(q, c2, s2, 16), oracle.rope(k, c2, s2, 16)
    np.testing.assert_allclose(np.einsum("ihd,jhd->hij", qr, kr), np.einsum("ihd,jhd->hij", q2, k2),
                               atol=1e-11)


def test_positions_reset_per_sequence():
    cu = np.array([0, 3, 3 + 5, 12], np.int32)
    np.testing.assert_array_equal(oracle.positions(cu), [0, 1, 2, 0, 1, 2, 3, 4, 0, 1, 2, 3])


# ---------------------------------------------------------------------------
# Whole block and stack: library cross-check and finite differences
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_stack_vs_torch_autograd(mask):
    b = _tiny_batch(mask)
    layers = _tiny_layers()
    g = np.random.default_rng(9)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal(x.shape)
    y, xs = oracle.stack_forward(layers, 2, x, b, TINY)
    dx, grads = oracle.stack_backward(layers, 2, xs, dy, b, TINY)
    ty, tdx, tgrads = torch_block.stack_fwd_bwd(layers, x, dy, b, TINY)
    assert rel_l2(y, ty) < 1e-12
    assert rel_l2(dx, tdx) < 1e-11
    for l in range(2):
        for k in oracle.block.PARAMS:
            assert rel_l2(grads[l][k], tgrads[l][k]) < 1e-10, (l, k)


@pytest.mark.slow
def test_stack_finite_differences():
    """Central differences of L = sum(y * dy) in float64 for every dx entry
    and up to 200 random entries of every parameter tensor of both layers."""
    b = _tiny_batch("prefix")
    layers = _tiny_layers()
    g = np.random.default_rng(10)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal(x.shape)
    y, xs = oracle.stack_forward(layers, 2, x, b, TINY)
    dx, grads = oracle.stack_backward(layers, 2, xs, dy, b, TINY)

    def loss(xx, ll):
        yy, _ = oracle.stack_forward(ll, 2, xx, b, TINY, keep="none")
        return float((yy * dy).sum())

    eps = 1e-5

    def check(an, fd):
        assert abs(an - fd) <= 2e-7 + 1e-6 * abs(an), (an, fd)

    for idx in np.ndindex(*x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        check(dx[idx], (loss(xp, layers) - loss(xm, layers)) / (2 * eps))
    for l in range(2):
        for k in oracle.block.PARAMS:
            arr = layers[l][k]
            flat = np.arange(arr.size)
            pick = flat if arr.size <= 200 else g.choice(flat, 200, replace=False)
            for f in pick:
                idx = np.unravel_index(f, arr.shape)
                lp = [dict(d) for d in layers]
                lm = [dict(d) for d in layers]
                lp[l][k] = arr.copy()
                lm[l][k] = arr.copy()
                lp[l][k][idx] += eps
                lm[l][k][idx] -= eps
                check(grads[l][k][idx], (loss(x, lp) - loss(x, lm)) / (2 * eps))


# ---------------------------------------------------------------------------
# Invariants of client batching and of the stack
# ---------------------------------------------------------------------------

def _fwd_bwd(layers, x, dy, b, shape=TINY):
    y, xs = oracle.stack_forward(layers, shape.num_layers, x, b, shape)
    dx, grads = oracle.stack_backward(layers, shape.num_layers, xs, dy, b, shape)
    return y, dx, grads


@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_I1_batched_equals_sequential_clients(mask):
    """Section 3.3: the server stacks the clients' smashed data into one batch.
    Per client, the stacked run must equal running that client alone; the
    batched weight gradient is the sum of the per-client ones."""
    b = _tiny_batch(mask)
    layers = _tiny_layers()
    g = np.random.default_rng(11)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal(x.shape)
    y, dx, grads = _fwd_bwd(layers, x, dy, b)
    acc = [oracle.zero_grads(TINY) for _ in range(2)]
    for c in range(b.num_clients):
        sub, rows = b.subset_clients([c])
        yc, dxc, gc = _fwd_bwd(layers, x[rows], dy[rows], sub)
        assert rel_l2(y[rows], yc) < 1e-14
        assert rel_l2(dx[rows], dxc) < 1e-13
        for l in range(2):
            for k in acc[l]:
                acc[l][k] += gc[l][k]
    for l in range(2):
        for k in acc[l]:
            assert rel_l2(grads[l][k], acc[l][k]) < 1e-12


def test_I2_client_isolation():
    """Poisoning one client's input with NaN leaves every other client's
    output and input gradient bit-for-bit unchanged."""
    b = _tiny_batch("causal")
    layers = _tiny_layers()
    g = np.random.default_rng(12)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal(x.shape)
    y, dx, _ = _fwd_bwd(layers, x, dy, b)
    r0, r1 = b.client_rows(1)
    x2 = x.copy()
    x2[r0:r1] = np.nan
    with np.errstate(invalid="ignore"):
        y2, dx2, _ = _fwd_bwd(layers, x2, dy, b)
    np.testing.assert_array_equal(y2[:r0], y[:r0])
    np.testing.assert_array_equal(dx2[:r0], dx[:r0])
    assert np.isnan(y2[r0:r1]).all()


def test_I3_causality():
    """Outside the prefix, output row i does not depend on rows j > i."""
    b = synth.Batch(np.array([0, 10], np.int32), np.array([0, 1], np.int32), "prefix",
                    np.array([3], np.int32))
    layers = _tiny_layers()
    g = np.random.default_rng(13)
    x = g.standard_normal((10, TINY.hidden))
    y, _ = oracle.stack_forward(layers, 2, x, b, TINY)
    x2 = x.copy()
    x2[6:] += g.standard_normal((4, TINY.hidden))
    y2, _ = oracle.stack_forward(layers, 2, x2, b, TINY)
    np.testing.assert_array_equal(y2[:6], y[:6])
    # a change inside the prefix reaches every earlier prefix row
    x3 = x.copy()
    x3[2] += 1.0
    y3, _ = oracle.stack_forward(layers, 2, x3, b, TINY)
    assert np.all(np.abs(y3[:2] - y[:2]).max(axis=1) > 0)


def test_I4_varlen_equals_padded():
    """Packed ragged sequences equal the same sequences padded to a common
    length with padded keys masked out (compared on valid rows)."""
    b = _tiny_batch("causal")
    g = np.random.default_rng(14)
    T = b.total_tokens
    q, k, v = (g.standard_normal((T, 2, 8)) for _ in range(3))
    o = oracle.attention_forward(q, k, v, b)
    Lmax = b.max_seqlen
    for s in range(b.num_seqs):
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        L = r1 - r0
        pad = lambda a: np.concatenate([a[r0:r1], g.standard_normal((Lmax - L, 2, 8))])
        tq, tk, tv = (torch.tensor(pad(a)).transpose(0, 1) for a in (q, k, v))
        i = torch.arange(Lmax)[:, None]
        j = torch.arange(Lmax)[None, :]
        m = (j <= i) & (j < L)
        ref = F.scaled_dot_product_attention(tq, tk, tv, attn_mask=m).transpose(0, 1).numpy()
        assert rel_l2(o[r0:r1], ref[:L]) < 1e-12


def test_I5_stack_is_composition_of_blocks():
    """Section 3.1: the server computes Block_(1,N-2), the composition of
    single blocks; a 2-block stack equals two chained single-block runs."""
    b = _tiny_batch("prefix")
    layers = _tiny_layers()
    g = np.random.default_rng(15)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal(x.shape)
    y, dx, grads = _fwd_bwd(layers, x, dy, b)
    one = synth.StackShape(1, TINY.hidden, TINY.num_heads, TINY.ffn_hidden, TINY.rotary_dim)
    y0, _ = oracle.stack_forward([layers[0]], 1, x, b, one)
    y1, _ = oracle.stack_forward([layers[1]], 1, y0, b, one)
    np.testing.assert_array_equal(y1, y)
    d1, g1 = oracle.stack_backward([layers[1]], 1, [y0], dy, b, one)
    d0, g0 = oracle.stack_backward([layers[0]], 1, [x], d1, b, one)
    np.testing.assert_array_equal(d0, dx)
    for k in g0[0]:
        np.testing.assert_array_equal(g0[0][k], grads[0][k])
        np.testing.assert_array_equal(g1[0][k], grads[1][k])


def test_I7_recompute_matches_stored_cache():
    b = _tiny_batch("causal")
    p = _tiny_layers()[0]
    g = np.random.default_rng(16)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal(x.shape)
    y, cache = oracle.block_forward(p, x, b, TINY)
    gr = oracle.zero_grads(TINY)
    dx = oracle.block_backward(p, cache, dy, b, TINY, gr)
    one = synth.StackShape(1, TINY.hidden, TINY.num_heads, TINY.ffn_hidden, TINY.rotary_dim)
    dx2, gr2 = oracle.stack_backward([p], 1, [x], dy, b, one)
    np.testing.assert_array_equal(dx, dx2)
    for k in gr:
        np.testing.assert_array_equal(gr[k], gr2[0][k])
    # the two-block stack: stored caches (no recompute) give the same bits
    layers = _tiny_layers()
    y1, xs = oracle.stack_forward(layers, 2, x, b, TINY)
    y2, caches = oracle.stack_forward(layers, 2, x, b, TINY, keep="caches")
    np.testing.assert_array_equal(y1, y2)
    dx1, g1 = oracle.stack_backward(layers, 2, xs, dy, b, TINY)
    dx3, g3 = oracle.stack_backward(layers, 2, caches, dy, b, TINY)
    np.testing.assert_array_equal(dx1, dx3)
    for l in range(2):
        for k in g1[l]:
            np.testing.assert_array_equal(g1[l][k], g3[l][k])
    # weights left out of grads: the same dx, and no product is formed
    dx4, g4 = oracle.stack_backward(layers, 2, caches, dy, b, TINY, grads=[{}, {"b_o": np.zeros(TINY.hidden)}])
    np.testing.assert_array_equal(dx1, dx4)
    np.testing.assert_array_equal(g4[1]["b_o"], g1[1]["b_o"])


def test_I8_zero_output_projections_is_identity():
    """With W_o = b_o = W_2 = b_2 = 0 each block is the identity: y = x and
    dx = dy exactly; only the gradients of W_o, b_o, W_2, b_2 are non-zero."""
    b = _tiny_batch("prefix")
    layers = _tiny_layers()
    for lp in layers:
        for k in ("w_o", "b_o", "w_2", "b_2"):
            lp[k] = np.zeros_like(lp[k])
    g = np.random.default_rng(17)
    x = g.standard_normal((b.total_tokens, TINY.hidden))
    dy = g.standard_normal(x.shape)
    y, dx, grads = _fwd_bwd(layers, x, dy, b)
    np.testing.assert_array_equal(y, x)
    np.testing.assert_array_equal(dx, dy)
    for l in range(2):
        for k, v in grads[l].items():
            if k in ("w_o", "b_o", "w_2", "b_2"):
                assert np.abs(v).max() > 0
            else:
                assert np.abs(v).max() == 0, k


# ---------------------------------------------------------------------------
# Packing and client boundaries
# ---------------------------------------------------------------------------

def test_pack_unpack_and_client_ranges():
    b = synth.make_batch(3, 2, (2, 6), seed=4)
    g = np.random.default_rng(18)
    per = []
    for c in range(b.num_clients):
        s0, s1 = int(b.client_seq_ptr[c]), int(b.client_seq_ptr[c + 1])
        Lmax = int(b.seqlens[s0:s1].max())
        per.append(g.standard_normal((Lmax, s1 - s0, 3)))
    packed = oracle.pack_clients(per, b.cu_seqlens, b.client_seq_ptr)
    back = oracle.unpack_clients(packed, b.cu_seqlens, b.client_seq_ptr)
    for c, (a, r) in enumerate(zip(per, back)):
        s0 = int(b.client_seq_ptr[c])
        for bb in range(a.shape[1]):
            L = int(b.seqlens[s0 + bb])
            np.testing.assert_array_equal(r[:L, bb], a[:L, bb])
            assert (r[L:, bb] == 0).all()
    rng_ = oracle.client_token_ranges(b.cu_seqlens, b.client_seq_ptr)
    for c in range(b.num_clients):
        assert tuple(rng_[c]) == b.client_rows(c)
    assert rng_[0, 0] == 0 and rng_[-1, 1] == b.total_tokens
    assert (rng_[1:, 0] == rng_[:-1, 1]).all()
