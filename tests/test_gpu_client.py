"""GPU parity of the client side of the split model (Section 3.1) through the
C ABI: embedding gather (bit-exact) and its deterministic scatter-add
gradient, the final linear layer with the cross-entropy loss (forward and
backward, padded vocabulary, unlabelled tokens), the B-row limit and the
reduction-chunked weight-gradient GEMM it relies on, and whole split
training steps against the oracle."""

import numpy as np
import pytest

import synth
from oracle import client as oc
from paper_2406_14898_amd import BatchDesc, ClientHead, SplitModel
from paper_2406_14898_amd import flglm as F

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from tests.gpu_helpers import TOL, dev, host, rel_l2, rnd  # noqa: E402


def _ids(T, V, seed):
    g = np.random.default_rng(seed)
    ids = g.integers(0, V, T).astype(np.int32)
    ids[: min(T, 5)] = V - 1  # repeats, and the last row of the table
    return ids


def _labels(ids, seed, frac_ignored=0.2):
    g = np.random.default_rng(seed)
    lab = np.roll(ids, -1).astype(np.int32)
    lab[g.random(len(ids)) < frac_ignored] = -100
    lab[-1] = -100
    return lab


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("T,V,H", [(1, 8, 256), (300, 1000, 256), (77, 4104, 512)])
def test_embedding_forward_backward(dt, T, V, H):
    ch = ClientHead(V, H, dt)
    table = rnd((V, H), 1, 1.0, dt)
    ids = _ids(T, V, 2)
    ws = ch.workspace(T)
    out = torch.empty((T, H), dtype=torch.bfloat16 if dt == "bf16" else torch.float32, device="cuda")
    ch.embed(dev(table, dt), ids, out, ws)
    torch.cuda.synchronize()
    assert np.array_equal(host(out), oc.embedding_forward(table, ids))
    dout = rnd((T, H), 3, 1.0, dt)
    base = rnd((V, H), 4, 1.0, "f32")
    dtab = torch.from_numpy(base.copy()).cuda()
    ch.embed_backward(ids, dev(dout, dt), dtab, ws)
    torch.cuda.synchronize()
    ref = base + oc.embedding_backward(ids, dout, V)
    got = host(dtab)
    assert np.allclose(got, ref, rtol=1e-6, atol=1e-5)
    # deterministic: a second accumulation adds exactly the same rows again
    ch.embed_backward(ids, dev(dout, dt), dtab, ws)
    torch.cuda.synchronize()
    assert np.array_equal(host(dtab) - got, got - base) or np.allclose(host(dtab), base + 2 * (got - base),
                                                                        rtol=1e-6, atol=1e-5)
    ch.close()


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("T,V,H", [(300, 1000, 256), (77, 4104, 512), (1, 8, 256)])
def test_lm_head_matches_oracle(dt, T, V, H):
    ch = ClientHead(V, H, dt)
    h = rnd((T, H), 5, 1.0, dt)
    w = rnd((V, H), 6, 0.05, dt)
    labels = _labels(_ids(T, V, 7), 8)
    if T == 1:
        labels[0] = 3
    ws = ch.workspace(T)
    loss_tok = torch.empty(T, device="cuda")
    loss_sum = torch.empty(1, device="cuda")
    th, tw = dev(h, dt), dev(w, dt)
    ch.head_forward(th, tw, labels, loss_tok, loss_sum, ws)
    lg, lse, lt, ls = oc.lm_head_forward(h, w, labels)
    torch.cuda.synchronize()
    tol = TOL[dt]
    assert rel_l2(host(loss_tok), lt) < tol
    assert abs(float(loss_sum.item()) - ls) <= tol * abs(ls)
    assert not host(loss_tok)[labels < 0].any()
    scale = 1.0 / max(1, int((labels >= 0).sum()))
    dh = torch.empty_like(th)
    base = rnd((V, H), 9, 1e-3, "f32")
    dw = torch.from_numpy(base.copy()).cuda()
    ch.head_backward(th, tw, T, scale, dh, dw, ws)
    dho, dwo = oc.lm_head_backward(h, w, lg, lse, labels, scale)
    torch.cuda.synchronize()
    assert rel_l2(host(dh), dho) < tol
    assert rel_l2(host(dw) - base, dwo) < tol
    # frozen head: the same dh, no weight gradient
    ch.head_forward(th, tw, labels, loss_tok, loss_sum, ws)
    dh2 = torch.empty_like(th)
    ch.head_backward(th, tw, T, scale, dh2, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(dh2, dh)
    ch.close()


def test_gemm_b_rows_limit():
    """Rows of B past b_rows are never read: B sits in a larger buffer whose
    extra rows hold huge values, and the result equals the product over the
    real rows only (NT: columns past b_rows are zero; NN: reduction past
    b_rows adds nothing)."""
    for dt in ("bf16", "f32"):
        code = F.FL_BF16 if dt == "bf16" else F.FL_F32
        M, K, N, nb = 300, 128, 512, 333
        A = rnd((M, K), 1, 1.0, dt)
        Bfull = rnd((N, K), 2, 1.0, dt)
        Bfull[nb:] = 1e4
        C = torch.zeros((M, N), dtype=torch.bfloat16 if dt == "bf16" else torch.float32, device="cuda")
        F.fl_test_gemm(code, F.FL_GEMM_NT, F.FL_EPI_STORE, dev(A, dt), dev(Bfull, dt), C, M, N, K, K, K, N,
                       b_rows=nb)
        ref = A.astype(np.float64) @ np.where(np.arange(N)[:, None] < nb, Bfull, 0.0).T
        torch.cuda.synchronize()
        assert rel_l2(host(C), ref) < TOL[dt]
        assert not host(C)[:, nb:].any()
        # NN: C = A2 [M, K2] B2 [K2 rows (only nb2 real), N2]
        K2, N2, nb2 = 512, 256, 300
        A2 = rnd((M, K2), 3, 1.0, dt)
        B2 = rnd((K2, N2), 4, 1.0, dt)
        B2[nb2:] = 1e4
        C2 = torch.zeros((M, N2), dtype=C.dtype, device="cuda")
        F.fl_test_gemm(code, F.FL_GEMM_NN, F.FL_EPI_STORE, dev(A2, dt), dev(B2, dt), C2, M, N2, K2, K2, N2, N2,
                       b_rows=nb2)
        ref2 = A2[:, :nb2].astype(np.float64) @ B2[:nb2].astype(np.float64)
        torch.cuda.synchronize()
        assert rel_l2(host(C2), ref2) < TOL[dt]


def test_weight_gradient_gemm_chunked_along_the_reduction():
    """A TN weight-gradient GEMM whose operand spans more than 2^31 bytes
    (1200 reduction rows of 2^20 bf16 each) is cut along the reduction; the
    pieces accumulate into the fp32 output in order."""
    K, lda, M, N = 1200, 1 << 20, 256, 256
    A = torch.zeros((K, lda), dtype=torch.bfloat16, device="cuda")
    a_used = rnd((K, M), 11, 1.0, "bf16")
    A[:, :M] = dev(a_used, "bf16")
    B = rnd((K, N), 12, 1.0, "bf16")
    base = rnd((M, N), 13, 1.0, "f32")
    C = torch.from_numpy(base.copy()).cuda()
    F.fl_test_gemm(F.FL_BF16, F.FL_GEMM_TN, F.FL_EPI_ACC_F32, A, dev(B, "bf16"), C, M, N, K, lda, N, N)
    ref = base + a_used.astype(np.float64).T @ B.astype(np.float64)
    torch.cuda.synchronize()
    assert rel_l2(host(C), ref) < 1e-5
    del A
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# Whole split training steps
# ---------------------------------------------------------------------------

TINY = synth.WORKLOADS["tiny_2blk_fp32"].shape
VT = 1000


def _run_split(dt, frozen, num_prefix, mask, seed=0):
    b = synth.make_batch(2, 2, (40, 90), mask=mask, seed=seed)
    T = b.total_tokens
    bf = dt == "bf16"
    layers = [synth.layer_params(TINY, l, seed=seed, bf16=bf) for l in range(4)]
    if num_prefix:
        for l, lp in enumerate(layers):
            lp.update(synth.prefix_params(TINY, l, num_prefix, seed=seed, bf16=bf, std=0.5))
    g = np.random.default_rng(seed + 1)
    client = {"embedding": rnd((VT, TINY.hidden), seed + 2, 1.0, dt), "block0": layers[0], "block_last": layers[3],
              "lm_head": rnd((VT, TINY.hidden), seed + 3, 0.05, dt)}
    server = layers[1:3]
    ids = _ids(T, VT, seed + 4)
    labels = _labels(ids, seed + 5)
    scale = 1.0 / int((labels >= 0).sum())
    m = SplitModel(TINY.hidden, TINY.num_heads, TINY.ffn_hidden, TINY.rotary_dim, 2, VT, dt, TINY.rope_base,
                   TINY.ln_eps, num_prefix)
    bd = BatchDesc.from_batch(b)
    buf = m.buffers(bd, recompute=False)
    dlayers = [{k: dev(v, dt) for k, v in lp.items()} for lp in layers]
    params = {"embedding": dev(client["embedding"], dt), "lm_head": dev(client["lm_head"], dt),
              "block0": dlayers[0], "block_last": dlayers[3], "server": dlayers[1:3]}

    def gz(lp):
        return {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in lp.items()
                if not frozen or k.startswith("prefix_")}
    grads = {"block0": gz(dlayers[0]), "block_last": gz(dlayers[3]), "server": [gz(d) for d in dlayers[1:3]]}
    if not frozen:
        grads["embedding"] = torch.zeros((VT, TINY.hidden), device="cuda")
        grads["lm_head"] = torch.zeros((VT, TINY.hidden), device="cuda")
    m.step(bd, ids, labels, params, grads, scale, buf)
    torch.cuda.synchronize()
    ref = oc.split_step(client, server, ids, labels, b, TINY, scale, train_weights=not frozen)
    m.close()
    return buf, grads, ref


@pytest.mark.parametrize("dt,frozen,num_prefix,mask", [("f32", False, 0, "causal"), ("f32", False, 0, "prefix"),
                                                       ("bf16", True, 8, "causal"), ("bf16", False, 0, "prefix")])
def test_split_step_matches_oracle(dt, frozen, num_prefix, mask):
    """Embedding -> block 0 -> 2-block server -> block N-1 -> linear ->
    cross-entropy -> backward through all of them, on the tiny block shape
    with a 1000-word vocabulary: the loss, the tensors crossing both split
    boundaries in each direction, and every trained gradient."""
    buf, grads, ref = _run_split(dt, frozen, num_prefix, mask)
    tol = TOL[dt]
    errs = {"h0": rel_l2(host(buf["h0"]), ref["h0"]), "h_server": rel_l2(host(buf["hs"]), ref["h_server"]),
            "loss_tok": rel_l2(host(buf["loss_tok"]), ref["loss_tok"]),
            "d_h_server": rel_l2(host(buf["d_hs"]), ref["d_h_server"]), "d_h0": rel_l2(host(buf["d_h0"]), ref["d_h0"])}
    errs["loss_sum"] = abs(float(buf["loss_sum"].item()) - ref["loss_sum"]) / abs(ref["loss_sum"])
    if not frozen:
        errs["lm_head"] = rel_l2(host(grads["lm_head"]), ref["grad_lm_head"])
        errs["embedding"] = rel_l2(host(grads["embedding"]), ref["grad_embedding"])
    for name, key in (("block0", "grads_block0"), ("block_last", "grads_block_last")):
        for k, v in ref[key].items():
            errs[f"{name}.{k}"] = rel_l2(host(grads[name][k]), v)
    for l in range(2):
        for k, v in ref["grads_server"][l].items():
            errs[f"server{l}.{k}"] = rel_l2(host(grads["server"][l][k]), v)
    bad = {k: v for k, v in errs.items() if not v < tol}
    assert not bad, bad
    if frozen:
        assert set(grads["block0"]) == {"prefix_k", "prefix_v"}


def test_split_step_is_deterministic_and_recompute_exact():
    """The whole bf16 split step twice, and once with per-block recompute:
    every boundary tensor, the loss and every gradient agree bit for bit (no
    atomics anywhere: segmented embedding sums, fixed-order reductions)."""
    dt = "bf16"
    b = synth.make_batch(3, 2, (20, 130), mask="prefix", seed=9)
    T = b.total_tokens
    layers = [synth.layer_params(TINY, l, seed=9, bf16=True) for l in range(4)]
    m = SplitModel(TINY.hidden, TINY.num_heads, TINY.ffn_hidden, TINY.rotary_dim, 2, VT, dt, TINY.rope_base,
                   TINY.ln_eps)
    bd = BatchDesc.from_batch(b)
    dlayers = [{k: dev(v, dt) for k, v in lp.items()} for lp in layers]
    params = {"embedding": dev(rnd((VT, TINY.hidden), 91, 1.0, dt), dt),
              "lm_head": dev(rnd((VT, TINY.hidden), 92, 0.05, dt), dt),
              "block0": dlayers[0], "block_last": dlayers[3], "server": dlayers[1:3]}
    ids = _ids(T, VT, 93)
    labels = _labels(ids, 94)
    scale = 1.0 / int((labels >= 0).sum())

    def run(recompute):
        buf = m.buffers(bd, recompute=recompute)
        gz = lambda lp: {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in lp.items()}
        grads = {"block0": gz(dlayers[0]), "block_last": gz(dlayers[3]), "server": [gz(d) for d in dlayers[1:3]],
                 "embedding": torch.zeros((VT, TINY.hidden), device="cuda"),
                 "lm_head": torch.zeros((VT, TINY.hidden), device="cuda")}
        m.step(bd, ids, labels, params, grads, scale, buf, recompute=recompute)
        torch.cuda.synchronize()
        out = {k: host(buf[k]) for k in ("h0", "hs", "hl", "d_hl", "d_hs", "d_h0", "d_e", "loss_tok", "loss_sum")}
        for name in ("block0", "block_last"):
            out.update({f"{name}.{k}": host(v) for k, v in grads[name].items()})
        for l in range(2):
            out.update({f"server{l}.{k}": host(v) for k, v in grads["server"][l].items()})
        out["embedding"], out["lm_head"] = host(grads["embedding"]), host(grads["lm_head"])
        return out

    a, a2, r = run(False), run(False), run(True)
    m.close()
    for other in (a2, r):
        for k in a:
            assert np.array_equal(a[k], other[k]), k
    assert np.abs(a["embedding"]).sum() > 0 and np.abs(a["lm_head"]).sum() > 0
