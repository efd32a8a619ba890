"""GPU parity of the server update through the C ABI: the Adam step
(Section 4.1.4; Adam paper Algorithm 1) and the server-hierarchical replica
averaging (Section 3.3) against the float64 oracle, element by element on
the same host-drawn fp32 inputs, including ragged tails, the bf16 compute
copy (exact round-to-nearest-even of the updated fp32 values) and the fused
gradient clear; then whole training loops (forward, backward, Adam,
averaging) run independently by the GPU and the oracle from the same
inputs.  Adam's first steps are close to lr * sign(g), so the loops use an
epsilon of a tenth of the gradients' root mean square (taken from the
oracle's gradients): that keeps the update Lipschitz in g, so the two loops'
rounding differences cannot flip whole steps."""

import numpy as np
import pytest

import oracle
import synth
from paper_2406_14898_amd import flglm as F

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

LR, B1, B2, EPS = oracle.ADAM_LR, oracle.ADAM_BETA1, oracle.ADAM_BETA2, oracle.ADAM_EPS


def _grad(g, n):
    """Gradients spanning nine decades, with exact zeros and both signs."""
    a = g.standard_normal(n) * 10.0 ** g.integers(-8, 2, n)
    a[g.random(n) < 0.01] = 0.0
    return a.astype(np.float32)


def _h(t):
    return t.detach().cpu().numpy()


def check_adam(p0, g0, m0, v0, step, p1, m1, v1, lr=LR, b1=B1, b2=B2, eps=EPS):
    """GPU results (p1, m1, v1, fp32) against the oracle from the same fp32
    inputs.  Bounds: a few fp32 roundings of each term that enters."""
    pr, mr, vr = oracle.adam_step(p0.astype(np.float64), g0, m0, v0, step, lr, b1, b2, eps)
    g64 = g0.astype(np.float64)
    tol_m = 1e-6 * (b1 * np.abs(m0) + (1 - b1) * np.abs(g64)) + 1e-37
    tol_v = 1e-6 * vr + 1e-37
    assert np.all(np.abs(m1 - mr) <= tol_m), np.max(np.abs(m1 - mr) / tol_m)
    assert np.all(np.abs(v1 - vr) <= tol_v), np.max(np.abs(v1 - vr) / tol_v)
    # the update's size from the oracle's moments, plus the error m carries in
    upd = np.abs(pr - p0)
    tol_p = 5e-7 * np.abs(pr) + 1e-5 * upd + lr * tol_m / (1 - b1 ** step) / (np.sqrt(vr / (1 - b2 ** step)) + eps)
    tol_p = tol_p + 1e-30
    assert np.all(np.abs(p1 - pr) <= tol_p), np.max(np.abs(p1 - pr) / tol_p)


@pytest.mark.parametrize("n", [1, 3, 4, 5, 2047, 2048 * 3 + 5, (1 << 20) + 7])
@pytest.mark.parametrize("bf16_copy,zero_grad", [(True, True), (False, False)])
def test_adam_matches_oracle(n, bf16_copy, zero_grad):
    """Steps 1, 2 and 3, each from a host-drawn state (zero moments at step
    1, nonnegative second moments later)."""
    g = np.random.default_rng(n)
    p16 = torch.full((n,), 7.0, dtype=torch.bfloat16, device="cuda") if bf16_copy else None
    for step in (1, 2, 3):
        p0 = g.standard_normal(n).astype(np.float32)
        m0 = np.zeros(n, np.float32) if step == 1 else (g.standard_normal(n) * 1e-3).astype(np.float32)
        v0 = np.zeros(n, np.float32) if step == 1 else (g.random(n) * 1e-6).astype(np.float32)
        gr = _grad(g, n)
        p, m, v, tg = (torch.from_numpy(a.copy()).cuda() for a in (p0, m0, v0, gr))
        F.fl_adam_step(p, tg, m, v, p16, n, step, LR, B1, B2, EPS, zero_grad)
        torch.cuda.synchronize()
        check_adam(p0, gr, m0, v0, step, _h(p), _h(m), _h(v))
        if bf16_copy:
            bits = _h(p16.view(torch.int16)).view(np.uint16)
            assert np.array_equal(bits, synth.bf16_bits(_h(p)))
        if zero_grad:
            assert not _h(tg).any()
        else:
            assert np.array_equal(_h(tg), gr)


@pytest.mark.parametrize("step", [1, 7, 1000, 100000])
def test_adam_late_steps_and_hyper_parameters(step):
    """Arbitrary time steps from a nonzero state (bias corrections near 1
    late in training) and non-default hyper-parameters."""
    n = 4099
    g = np.random.default_rng(step)
    p0 = g.standard_normal(n).astype(np.float32)
    m0 = (g.standard_normal(n) * 1e-2).astype(np.float32)
    v0 = (np.abs(g.standard_normal(n)) * 1e-4).astype(np.float32)
    gr = _grad(g, n)
    for lr, b1, b2, eps in ((LR, B1, B2, EPS), (1e-3, 0.5, 0.9, 1e-3), (0.1, 0.0, 0.0, 0.0)):
        if b1 == 0.0 and step > 1:
            continue
        p, m, v = (torch.from_numpy(a.copy()).cuda() for a in (p0, m0, v0))
        F.fl_adam_step(p, torch.from_numpy(gr).cuda(), m, v, None, n, step, lr, b1, b2, eps)
        torch.cuda.synchronize()
        if eps == 0.0:
            ok = gr != 0  # 0/0 where both moments vanish
            pr, _, _ = oracle.adam_step(p0[ok], gr[ok], m0[ok], v0[ok], step, lr, b1, b2, eps)
            assert np.allclose(_h(p)[ok], pr, rtol=2e-6, atol=1e-6 * lr)
        else:
            check_adam(p0, gr, m0, v0, step, _h(p), _h(m), _h(v), lr, b1, b2, eps)


@pytest.mark.parametrize("M", [1, 2, 3, 10, 32])
@pytest.mark.parametrize("n", [1, 4, 7, 4099, (1 << 20) + 3])
def test_average_matches_oracle(M, n):
    g = np.random.default_rng(M * 7919 + n)
    reps = [(g.standard_normal(n) * 10.0 ** g.integers(-3, 3)).astype(np.float32) for _ in range(M)]
    tr = [torch.from_numpy(r).cuda() for r in reps]
    t16 = [torch.zeros(n, dtype=torch.bfloat16, device="cuda") for _ in range(M)] if M % 2 else None
    F.fl_average_replicas(tr, t16, n)
    torch.cuda.synchronize()
    ref = oracle.average_replicas(reps)
    out = [_h(t) for t in tr]
    for o in out[1:]:
        assert np.array_equal(o, out[0])  # every replica holds the same values
    bound = 2e-7 * M * np.max(np.abs(np.stack(reps)), axis=0) + 1e-38
    assert np.all(np.abs(out[0] - ref) <= bound)
    if t16 is not None:
        want = synth.bf16_bits(out[0])
        for t in t16:
            assert np.array_equal(_h(t.view(torch.int16)).view(np.uint16), want)


def test_average_identical_replicas_is_exact():
    """M copies of bf16-exact values (8 significant bits): every partial sum
    k x needs at most 13 bits, so the fp32 sum is exact and the one correctly
    rounded division returns x itself."""
    n = 1000
    x = synth.bf16_round(np.random.default_rng(1).standard_normal(n).astype(np.float32))
    for M in (2, 3, 4, 7, 8, 16, 31, 32):
        tr = [torch.from_numpy(x.copy()).cuda() for _ in range(M)]
        F.fl_average_replicas(tr, None, n)
        torch.cuda.synchronize()
        assert all(np.array_equal(_h(t), x) for t in tr), M


# ---------------------------------------------------------------------------
# Training steps through the stack: forward, backward, update, averaging
# ---------------------------------------------------------------------------

from paper_2406_14898_amd import BatchDesc, ParamArena, ServerStack, average  # noqa: E402
from tests.gpu_helpers import dev, host, rel_l2  # noqa: E402

TINY_W = synth.WORKLOADS["tiny_2blk_fp32"]
SH = TINY_W.shape


def _stack(dt, num_prefix=0):
    return ServerStack(SH.num_layers, SH.hidden, SH.num_heads, SH.ffn_hidden, SH.rotary_dim, dt, SH.rope_base,
                       SH.ln_eps, num_prefix)


def _fwd_bwd(ss, batch, params, grads, x, dy):
    bd = BatchDesc.from_batch(batch)
    saved, ws = ss.buffers(bd, False)
    y, dx = torch.empty_like(x), torch.empty_like(x)
    ss.forward(bd, params, x, y, saved, ws)
    ss.backward(bd, params, grads, x, saved, dy, dx, ws)
    torch.cuda.synchronize()
    return host(y), host(dx)


def _rms(arrs):
    return float(np.sqrt(np.mean(np.concatenate([np.ravel(a) for a in arrs]) ** 2)))


def test_training_steps_fp32_full_weights():
    """Two training steps of the tiny fp32 stack with every weight trained:
    GPU (forward, backward, one Adam launch over the whole parameter arena,
    gradients cleared in the same pass) and the oracle (the same steps in
    float64) from the same initial weights and batches.  Compared after each
    step: y, dx, every gradient, and the updated weights (1e-4)."""
    b = TINY_W.batch()
    pnames = list(synth.param_shapes(SH))
    names = [(f"{l}.{k}", s) for l in range(SH.num_layers) for k, s in synth.param_shapes(SH).items()]
    arena = ParamArena(names, bf16_copy=False)
    ref = [synth.layer_params(SH, l, seed=0, bf16=False) for l in range(SH.num_layers)]
    arena.load({f"{l}.{k}": torch.from_numpy(v).cuda() for l in range(SH.num_layers) for k, v in ref[l].items()})
    ref = [{k: v.astype(np.float64) for k, v in lp.items()} for lp in ref]
    state = [{k: (np.zeros_like(v), np.zeros_like(v)) for k, v in lp.items()} for lp in ref]
    pv, gv = arena.compute_views(), arena.grad_views()
    params = [{k: pv[f"{l}.{k}"] for k in pnames} for l in range(SH.num_layers)]
    grads = [{k: gv[f"{l}.{k}"] for k in pnames} for l in range(SH.num_layers)]
    ss = _stack("f32")
    eps = None
    for step in (1, 2):
        x = synth.activations(b.total_tokens, SH.hidden, seed=10 + step, bf16=False)
        dy = synth.upstream_grad(b.total_tokens, SH.hidden, seed=10 + step, std=TINY_W.dy_std, bf16=False)
        y, dx = _fwd_bwd(ss, b, params, grads, dev(x, "f32"), dev(dy, "f32"))
        yo, xs = oracle.stack_forward(ref, SH.num_layers, x, b, SH)
        dxo, go = oracle.stack_backward(ref, SH.num_layers, xs, dy, b, SH)
        assert rel_l2(y, yo) < 1e-4 and rel_l2(dx, dxo) < 1e-4
        for l in range(SH.num_layers):
            for k in pnames:
                assert rel_l2(host(grads[l][k]), go[l][k]) < 1e-4, (step, l, k)
        if eps is None:
            eps = 0.1 * _rms([go[l][k] for l in range(SH.num_layers) for k in pnames])
        arena.adam_step(eps=eps, zero_grad=True)
        for l in range(SH.num_layers):
            for k in pnames:
                m, v = state[l][k]
                ref[l][k], m, v = oracle.adam_step(ref[l][k], go[l][k], m, v, step, eps=eps)
                state[l][k] = (m, v)
        torch.cuda.synchronize()
        assert not _h(arena.grad).any()
        for l in range(SH.num_layers):
            for k in pnames:
                assert rel_l2(host(params[l][k]), ref[l][k]) < 1e-4, (step, l, k)
    ss.close()


def test_server_hierarchical_ptuning_bf16():
    """Server-hierarchical P-tuning v2 (Section 3.3, Appendix A): two server
    replicas share the frozen bf16 weights; each trains its own prefix on its
    own client's sequences for a period of two Adam steps, then the prefixes
    are averaged.  The oracle runs the same period in float64 (its forward
    reads the prefixes rounded to bf16, as the GPU's compute copy holds
    them).  Compared: the prefix gradients of every step, the prefixes after
    every step and after the average (bf16 tolerance), the bf16 copies
    (exact rounding of the GPU's own fp32 masters), the replicas' equality
    after averaging, and that the Adam moments stay with their replica."""
    Lp = 8
    b = synth.make_batch(2, 2, (40, 90), seed=3)
    weights = [synth.layer_params(SH, l, seed=0) for l in range(SH.num_layers)]
    wdev = [{k: dev(v, "bf16") for k, v in lp.items()} for lp in weights]
    keys = ("prefix_k", "prefix_v")
    names = [(f"{l}.{k}", (Lp, SH.hidden)) for l in range(SH.num_layers) for k in keys]
    arenas, refs, states = [], [], []
    for r in range(2):
        init = [synth.prefix_params(SH, l, Lp, seed=r, bf16=True, std=0.5) for l in range(SH.num_layers)]
        a = ParamArena(names, bf16_copy=True)
        a.load({f"{l}.{k}": torch.from_numpy(init[l][k]).cuda() for l in range(SH.num_layers) for k in keys})
        arenas.append(a)
        refs.append([{k: init[l][k].astype(np.float64) for k in keys} for l in range(SH.num_layers)])
        states.append([{k: (np.zeros((Lp, SH.hidden)), np.zeros((Lp, SH.hidden))) for k in keys}
                       for _ in range(SH.num_layers)])
    ss = _stack("bf16", Lp)
    eps = None
    for step in (1, 2):
        for r, a in enumerate(arenas):
            sub, _ = b.subset_clients([r])
            r0, r1 = b.client_rows(r)
            x = synth.activations(b.total_tokens, SH.hidden, seed=20 + step)[r0:r1]
            dy = synth.upstream_grad(b.total_tokens, SH.hidden, seed=20 + step, std=1e-2)[r0:r1]
            pv, gv = a.compute_views(), a.grad_views()
            params = [dict(wdev[l], prefix_k=pv[f"{l}.prefix_k"], prefix_v=pv[f"{l}.prefix_v"])
                      for l in range(SH.num_layers)]
            grads = [{k: gv[f"{l}.{k}"] for k in keys} for l in range(SH.num_layers)]
            _fwd_bwd(ss, sub, params, grads, dev(x, "bf16"), dev(dy, "bf16"))
            cur = [dict(weights[l], **{k: synth.bf16_round(refs[r][l][k].astype(np.float32)) for k in keys})
                   for l in range(SH.num_layers)]
            _, xs = oracle.stack_forward(cur, SH.num_layers, x, sub, SH)
            zg = [oracle.zero_prefix_grads(Lp, SH.hidden) for _ in range(SH.num_layers)]
            _, go = oracle.stack_backward(cur, SH.num_layers, xs, dy, sub, SH, zg)
            for l in range(SH.num_layers):
                for k in keys:
                    assert rel_l2(host(grads[l][k]), go[l][k]) < 2e-2, (step, r, l, k)
            if eps is None:
                eps = 0.1 * _rms([go[l][k] for l in range(SH.num_layers) for k in keys])
            a.adam_step(eps=eps, zero_grad=True)
            for l in range(SH.num_layers):
                for k in keys:
                    m, v = states[r][l][k]
                    refs[r][l][k], m, v = oracle.adam_step(refs[r][l][k], go[l][k], m, v, step, eps=eps)
                    states[r][l][k] = (m, v)
            torch.cuda.synchronize()
            mv = a.master_views()
            for l in range(SH.num_layers):
                for k in keys:
                    assert rel_l2(host(mv[f"{l}.{k}"]), refs[r][l][k]) < 2e-2, (step, r, l, k)
            assert np.array_equal(_h(a.compute.view(torch.int16)).view(np.uint16), synth.bf16_bits(_h(a.master)))
    moments = [_h(a.exp_avg).copy() for a in arenas]
    average(arenas)
    torch.cuda.synchronize()
    for a, mom in zip(arenas, moments):
        assert np.array_equal(_h(a.master), _h(arenas[0].master))
        assert np.array_equal(_h(a.compute.view(torch.int16)).view(np.uint16), synth.bf16_bits(_h(a.master)))
        assert np.array_equal(_h(a.exp_avg), mom)  # moments stay with their replica
    mv = arenas[0].master_views()
    for l in range(SH.num_layers):
        for k in keys:
            want = oracle.average_replicas([refs[0][l][k], refs[1][l][k]])
            assert rel_l2(host(mv[f"{l}.{k}"]), want) < 2e-2, (l, k)
    ss.close()
