"""GPU parity of ChatGLM-6B's own block variant (alpha-scaled residual on the
normalised input, GLM 2-D rotary positions) and of the final LayerNorm in
front of the client's linear layer, through the C ABI against the oracle:
the residual-scaling GEMM epilogues, block stacks in fp32 and bf16 (causal
and prefix-LM batches, with and without a P-tuning prefix), whole split
steps with the final LayerNorm, and one block at the full ChatGLM-6B shape."""

import math

import numpy as np
import pytest

import oracle
import synth
from oracle import client as oc
from paper_2406_14898_amd import BatchDesc, SplitModel
from paper_2406_14898_amd import flglm as F

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from tests.gpu_helpers import TOL, dev, host, rel_l2, rnd  # noqa: E402
from tests.stack_runner import GpuStack  # noqa: E402

ALPHA = math.sqrt(2 * 28)
TINY = synth.WORKLOADS["tiny_2blk_fp32"].shape


def _glm(base, two_d=True, alpha=ALPHA):
    return synth.StackShape(base.num_layers, base.hidden, base.num_heads, base.ffn_hidden, base.head_dim // 2,
                            base.rope_base, base.ln_eps, alpha, two_d)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_residual_scale_epilogues(dt):
    """NT + bias + alpha R and NN + alpha R (the input-gradient epilogue of
    the alpha residual) against float64 products."""
    code = F.FL_BF16 if dt == "bf16" else F.FL_F32
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    M, N, K = 300, 512, 256
    A, B = rnd((M, K), 1, 1.0, dt), rnd((N, K), 2, 1.0, dt)
    bias, R = rnd((N,), 3, 1.0, dt), rnd((M, N), 4, 1.0, dt)
    C = torch.empty((M, N), dtype=tdt, device="cuda")
    F.fl_test_gemm(code, F.FL_GEMM_NT, F.FL_EPI_BIAS_RES, dev(A, dt), dev(B, dt), C, M, N, K, K, K, N,
                   bias=dev(bias, dt), R=dev(R, dt), ldr=N, res_scale=ALPHA)
    ref = A.astype(np.float64) @ B.T.astype(np.float64) + bias + ALPHA * R
    torch.cuda.synchronize()
    assert rel_l2(host(C), ref) < TOL[dt]
    B2 = rnd((K, N), 5, 1.0, dt)
    C2 = torch.empty((M, N), dtype=tdt, device="cuda")
    F.fl_test_gemm(code, F.FL_GEMM_NN, F.FL_EPI_RES, dev(A, dt), dev(B2, dt), C2, M, N, K, K, N, N, R=dev(R, dt),
                   ldr=N, res_scale=-0.5)
    ref2 = A.astype(np.float64) @ B2.astype(np.float64) - 0.5 * R
    torch.cuda.synchronize()
    assert rel_l2(host(C2), ref2) < TOL[dt]


def _batch(mask):
    return synth.make_batch(2, 2, (40, 90), mask=mask, seed=5)


@pytest.mark.parametrize("dt,mask,two_d,num_prefix", [
    ("f32", "prefix", True, 0), ("f32", "causal", False, 0), ("f32", "prefix", False, 0),
    ("bf16", "prefix", True, 0), ("bf16", "causal", True, 0), ("bf16", "prefix", True, 16)])
def test_glm_stack_matches_oracle(dt, mask, two_d, num_prefix):
    """Two ChatGLM-6B-style blocks (alpha = sqrt(56)), forward and backward:
    y, dx and every gradient (P-tuning: prefix gradients with frozen
    weights)."""
    sh = _glm(TINY, two_d)
    b = _batch(mask)
    bf = dt == "bf16"
    layers = [synth.layer_params(sh, l, seed=0, bf16=bf) for l in range(2)]
    if num_prefix:
        for l, lp in enumerate(layers):
            lp.update(synth.prefix_params(sh, l, num_prefix, seed=0, bf16=bf, std=0.5))
    x = synth.activations(b.total_tokens, sh.hidden, seed=1, bf16=bf)
    dy = synth.upstream_grad(b.total_tokens, sh.hidden, seed=1, bf16=bf, std=1.0)
    g = GpuStack(sh, layers, dt, num_prefix)
    frozen = num_prefix > 0
    res = g.to_host(g.run(b, x, dy, frozen=frozen))
    g.close()
    yo, xs = oracle.stack_forward(layers, 2, x, b, sh)
    grads = [oracle.zero_prefix_grads(num_prefix, sh.hidden) for _ in range(2)] if frozen else None
    dxo, go = oracle.stack_backward(layers, 2, xs, dy, b, sh, grads)
    tol = TOL[dt]
    errs = {"y": rel_l2(res["y"], yo), "dx": rel_l2(res["dx"], dxo)}
    for l in range(2):
        for k, v in go[l].items():
            errs[f"{l}.{k}"] = rel_l2(res["grads"][l][k], v)
    bad = {k: v for k, v in errs.items() if not v < tol}
    print(f"[glm] {sorted(errs.items(), key=lambda kv: -kv[1])[:8]}", flush=True)
    assert not bad, bad


def test_glm_recompute_is_bitwise_identical():
    sh = _glm(TINY, True)
    b = _batch("prefix")
    layers = [synth.layer_params(sh, l, seed=0) for l in range(2)]
    x = synth.activations(b.total_tokens, sh.hidden, seed=2)
    dy = synth.upstream_grad(b.total_tokens, sh.hidden, seed=2, std=1.0)
    g = GpuStack(sh, layers, "bf16")
    a = g.to_host(g.run(b, x, dy, recompute=False))
    r = g.to_host(g.run(b, x, dy, recompute=True))
    g.close()
    assert np.array_equal(a["y"], r["y"]) and np.array_equal(a["dx"], r["dx"])
    for l in range(2):
        for k in a["grads"][l]:
            assert np.array_equal(a["grads"][l][k], r["grads"][l][k]), (l, k)


@pytest.mark.parametrize("dt,frozen", [("f32", False), ("bf16", True)])
def test_glm_split_step_with_final_layernorm(dt, frozen):
    """The whole split model with ChatGLM-6B's blocks and its final LayerNorm
    before the linear layer (prefix-LM batch, 2-D positions)."""
    sh = _glm(TINY, True)
    b = _batch("prefix")
    T, V = b.total_tokens, 1000
    bf = dt == "bf16"
    num_prefix = 8 if frozen else 0
    layers = [synth.layer_params(sh, l, seed=1, bf16=bf) for l in range(4)]
    if num_prefix:
        for l, lp in enumerate(layers):
            lp.update(synth.prefix_params(sh, l, num_prefix, seed=1, bf16=bf, std=0.5))
    g = np.random.default_rng(3)
    lng = 1 + 0.1 * g.standard_normal(sh.hidden).astype(np.float32)
    lnb = 0.1 * g.standard_normal(sh.hidden).astype(np.float32)
    if bf:
        lng, lnb = synth.bf16_round(lng), synth.bf16_round(lnb)
    client = {"embedding": rnd((V, sh.hidden), 4, 1.0, dt), "block0": layers[0], "block_last": layers[3],
              "lm_head": rnd((V, sh.hidden), 5, 0.05, dt), "final_ln_g": lng, "final_ln_b": lnb}
    ids, labels = synth.token_ids(b, V, seed=6)
    scale = 1.0 / int((labels >= 0).sum())
    m = SplitModel(sh.hidden, sh.num_heads, sh.ffn_hidden, sh.rotary_dim, 2, V, dt, sh.rope_base, sh.ln_eps,
                   num_prefix, sh.residual_alpha, sh.rotary_2d)
    bd = BatchDesc.from_batch(b)
    buf = m.buffers(bd, recompute=False)
    dl = [{k: dev(v, dt) for k, v in lp.items()} for lp in layers]
    params = {"embedding": dev(client["embedding"], dt), "lm_head": dev(client["lm_head"], dt), "block0": dl[0],
              "server": dl[1:3], "block_last": dl[3], "final_ln_g": dev(lng, dt), "final_ln_b": dev(lnb, dt)}

    def gz(d):
        return {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in d.items()
                if not frozen or k.startswith("prefix_")}
    grads = {"block0": gz(dl[0]), "server": [gz(d) for d in dl[1:3]], "block_last": gz(dl[3])}
    if not frozen:
        for k, shp in (("embedding", (V, sh.hidden)), ("lm_head", (V, sh.hidden)), ("final_ln_g", (sh.hidden,)),
                       ("final_ln_b", (sh.hidden,))):
            grads[k] = torch.zeros(shp, device="cuda")
    m.step(bd, ids, labels, params, grads, scale, buf)
    torch.cuda.synchronize()
    ref = oc.split_step(client, layers[1:3], ids, labels, b, sh, scale, train_weights=not frozen)
    m.close()
    tol = TOL[dt]
    errs = {"loss_tok": rel_l2(host(buf["loss_tok"]), ref["loss_tok"]),
            "d_h_server": rel_l2(host(buf["d_hs"]), ref["d_h_server"]), "d_h0": rel_l2(host(buf["d_h0"]), ref["d_h0"]),
            "h_server": rel_l2(host(buf["hs"]), ref["h_server"])}
    if not frozen:
        for k in ("lm_head", "embedding", "final_ln_g", "final_ln_b"):
            errs[k] = rel_l2(host(grads[k]), ref["grad_" + k])
    for name, key in (("block0", "grads_block0"), ("block_last", "grads_block_last")):
        for k, v in ref[key].items():
            errs[f"{name}.{k}"] = rel_l2(host(grads[name][k]), v)
    bad = {k: v for k, v in errs.items() if not v < tol}
    print(f"[glm] {sorted(errs.items(), key=lambda kv: -kv[1])[:8]}", flush=True)
    assert not bad, bad


def test_glm_block_full_shape():
    """One ChatGLM-6B-shaped block with its own residual and 2-D positions on
    a ragged prefix-LM batch (context 25 %): y, dx and the weight gradients."""
    base = synth.WORKLOADS["chatglm6b_1blk_fwd_4x4x512"].shape
    sh = _glm(base, True)
    b = synth.Batch(np.array([0, 100, 357], np.int32), np.array([0, 1, 2], np.int32), "prefix",
                    np.array([25, 64], np.int32))
    lp = synth.layer_params(sh, 0, seed=0)
    x = synth.activations(b.total_tokens, sh.hidden, seed=3)
    dy = synth.upstream_grad(b.total_tokens, sh.hidden, seed=3, std=1e-2)
    g = GpuStack(sh, [lp], "bf16")
    res = g.to_host(g.run(b, x, dy))
    g.close()
    yo, xs = oracle.stack_forward([lp], 1, x, b, sh)
    dxo, go = oracle.stack_backward([lp], 1, xs, dy, b, sh)
    errs = {"y": rel_l2(res["y"], yo), "dx": rel_l2(res["dx"], dxo)}
    for k, v in go[0].items():
        errs[k] = rel_l2(res["grads"][0][k], v)
    print(f"[glm] full-shape block: {errs}", flush=True)
    assert all(v < TOL["bf16"] for v in errs.values()), errs
