"""Parity at the full ChatGLM-6B block shape (hidden 4096, 32 heads of 128,
FFN 16384), with the batch sizes and launch configuration the benchmark
times.  The GPU runs the whole client batch; the oracle recomputes sampled
sequences on their own, which equals their rows of the batched run because
client batching mixes nothing across sequences (invariant I1, pinned in the
oracle tests).  Weight gradients are checked in full on a small batch at the
same shape.  The 26-block stacks here alternate two generated layers to
keep the host parameter generation bounded; the benchmark's own 26-block
stack runs with 26 distinct layers in test_gpu_fullsize_grads.py, with the
full-batch weight gradients."""

import time

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import dev, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from tests.stack_runner import GpuStack  # noqa: E402

W_FWD = synth.WORKLOADS["chatglm6b_1blk_fwd_4x4x512"]
W_RAGGED = synth.WORKLOADS["chatglm6b_1blk_ragged_8x4"]
W_PREFIX = synth.WORKLOADS["chatglm6b_26blk_prefix_16x2x512"]
W_LONG = synth.WORKLOADS["chatglm6b_26blk_ragged_32x1_recompute"]
ONE = W_FWD.shape
TOL = 2e-2


@pytest.fixture(scope="module")
def layers2():
    t = time.time()
    out = [synth.layer_params(ONE, l, seed=0) for l in range(2)]
    print(f"[fullsize] generated 2 layers in {time.time() - t:.1f}s", flush=True)
    return out


def _seq_batch(b, s):
    """The batch holding only sequence s, and its rows in the packed buffer."""
    r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
    pre = None if b.prefix_len is None else np.array([int(b.prefix_len[s])], np.int32)
    return synth.Batch(np.array([0, r1 - r0], np.int32), np.array([0, 1], np.int32), b.mask, pre), r0, r1


def _shape(n):
    return synth.StackShape(n, ONE.hidden, ONE.num_heads, ONE.ffn_hidden, ONE.rotary_dim)


def test_1blk_fwd_4x4x512_sampled_sequences(layers2):
    """1 block, forward, 4 clients x 4 x 512 tokens, causal."""
    b = W_FWD.batch()
    x = synth.activations(b.total_tokens, ONE.hidden, seed=0)
    g = GpuStack(ONE, [layers2[0]], "bf16")
    y = g.to_host(g.run(b, x, None))["y"]
    g.close()
    for s in (0, b.num_seqs - 1):
        sb, r0, r1 = _seq_batch(b, s)
        yo, _ = oracle.stack_forward([layers2[0]], 1, x[r0:r1], sb, ONE, keep="none")
        err = rel_l2(y[r0:r1], yo)
        print(f"[fullsize] 1 block fwd 4x4x512 seq {s}: rel-L2 {err:.2e}", flush=True)
        assert err < TOL


def test_1blk_ragged_8x4_fwd_bwd_sampled_sequences(layers2):
    """1 block, fwd+bwd, 8 clients x 4 ragged sequences U[128,1024]."""
    b = W_RAGGED.batch()
    x = synth.activations(b.total_tokens, ONE.hidden, seed=0)
    dy = synth.upstream_grad(b.total_tokens, ONE.hidden, seed=0, std=W_RAGGED.dy_std)
    g = GpuStack(ONE, [layers2[0]], "bf16")
    res = g.to_host(g.run(b, x, dy))
    g.close()
    lens = b.seqlens
    for s in (int(np.argmin(lens)), int(np.argmax(lens))):
        sb, r0, r1 = _seq_batch(b, s)
        yo, xs = oracle.stack_forward([layers2[0]], 1, x[r0:r1], sb, ONE)
        dxo, _ = oracle.stack_backward([layers2[0]], 1, xs, dy[r0:r1], sb, ONE)
        ey, edx = rel_l2(res["y"][r0:r1], yo), rel_l2(res["dx"][r0:r1], dxo)
        print(f"[fullsize] 1 block ragged 8x4 seq {s} (L={r1 - r0}): y {ey:.2e} dx {edx:.2e}", flush=True)
        assert ey < TOL and edx < TOL


def test_weight_grads_full_shape(layers2):
    """Every weight gradient against the oracle at the full block shape, on a
    small ragged two-client batch (reduction over 177 tokens, ragged tail)."""
    b = synth.Batch(np.array([0, 100, 177], np.int32), np.array([0, 1, 2], np.int32))
    x = synth.activations(b.total_tokens, ONE.hidden, seed=2)
    dy = synth.upstream_grad(b.total_tokens, ONE.hidden, seed=2, std=1e-2)
    g = GpuStack(ONE, [layers2[1]], "bf16")
    res = g.to_host(g.run(b, x, dy))
    g.close()
    yo, xs = oracle.stack_forward([layers2[1]], 1, x, b, ONE)
    dxo, go = oracle.stack_backward([layers2[1]], 1, xs, dy, b, ONE)
    assert rel_l2(res["y"], yo) < TOL
    assert rel_l2(res["dx"], dxo) < TOL
    for k, v in go[0].items():
        e = rel_l2(res["grads"][0][k], v)
        print(f"[fullsize] grad {k}: rel-L2 {e:.2e}", flush=True)
        assert e < TOL, k


def _stack_sample(w, layers2, sample_seq, recompute):
    b = w.batch()
    n = w.shape.num_layers
    layers = [layers2[l % 2] for l in range(n)]
    x = synth.activations(b.total_tokens, ONE.hidden, seed=0)
    dy = synth.upstream_grad(b.total_tokens, ONE.hidden, seed=0, std=w.dy_std)
    g = GpuStack(w.shape, layers, "bf16")
    t = time.time()
    res = g.run(b, x, dy, recompute=recompute)
    host = {"y": res["y"].float().cpu().numpy(), "dx": res["dx"].float().cpu().numpy()}
    del res
    g.close()
    print(f"[fullsize] {w.name}: GPU run {time.time() - t:.1f}s", flush=True)
    sb, r0, r1 = _seq_batch(b, sample_seq)
    t = time.time()
    # float32 oracle: 26 blocks on one sequence in well under a minute
    yo, xs = oracle.stack_forward(layers, n, x[r0:r1], sb, w.shape, dtype=np.float32)
    dxo, _ = oracle.stack_backward(layers, n, xs, dy[r0:r1], sb, w.shape, dtype=np.float32)
    ey, edx = rel_l2(host["y"][r0:r1], yo), rel_l2(host["dx"][r0:r1], dxo)
    print(f"[fullsize] {w.name} seq {sample_seq} (L={r1 - r0}): y {ey:.2e} dx {edx:.2e} "
          f"(oracle {time.time() - t:.1f}s)", flush=True)
    assert ey < TOL and edx < TOL


def test_26blk_prefix_16x2x512_sampled(layers2):
    """26 blocks, fwd+bwd, 16 clients x 2 x 512 tokens, prefix-LM (25%)."""
    _stack_sample(W_PREFIX, layers2, 0, recompute=False)


def test_26blk_prefix_recompute_is_bitwise_identical(layers2):
    """Per-block recomputation changes no bit of y, dx or any weight gradient
    at the full 26-block shape."""
    b = W_PREFIX.batch()
    n = W_PREFIX.shape.num_layers
    layers = [layers2[l % 2] for l in range(n)]
    x = synth.activations(b.total_tokens, ONE.hidden, seed=0)
    dy = synth.upstream_grad(b.total_tokens, ONE.hidden, seed=0, std=W_PREFIX.dy_std)
    g = GpuStack(W_PREFIX.shape, layers, "bf16")
    a = g.run(b, x, dy, recompute=False)
    ya, dxa = a["y"].clone(), a["dx"].clone()
    ga = [{k: v.clone() for k, v in gg.items()} for gg in a["grads"]]
    del a
    r = g.run(b, x, dy, recompute=True)
    assert torch.equal(r["y"], ya) and torch.equal(r["dx"], dxa)
    for l in (0, n // 2, n - 1):
        for k in ga[l]:
            assert torch.equal(r["grads"][l][k], ga[l][k]), (l, k)
    g.close()


# ---------------------------------------------------------------------------
# P-tuning v2 at the full block shape: 128 prefix rows per block, weights frozen
# ---------------------------------------------------------------------------

NP = synth.WORKLOADS["chatglm6b_26blk_ptuning128_ragged_32x1_recompute"].num_prefix


def _with_prefix(lp, l):
    out = dict(lp)
    out.update(synth.prefix_params(ONE, l, NP, seed=0))
    return out


def test_ptuning_prefix_grads_full_shape(layers2):
    """1 block at the ChatGLM-6B shape, 2 clients / 3 ragged sequences: y, dx
    and both prefix gradients (summed over the sequences) against the oracle;
    no weight gradient is formed."""
    b = synth.Batch(np.array([0, 100, 357, 421], np.int32), np.array([0, 2, 3], np.int32))
    lp = _with_prefix(layers2[0], 0)
    x = synth.activations(b.total_tokens, ONE.hidden, seed=4)
    dy = synth.upstream_grad(b.total_tokens, ONE.hidden, seed=4, std=1e-2)
    g = GpuStack(ONE, [lp], "bf16", NP)
    res = g.to_host(g.run(b, x, dy, frozen=True))
    g.close()
    assert set(res["grads"][0]) == {"prefix_k", "prefix_v"}
    yo, xs = oracle.stack_forward([lp], 1, x, b, ONE)
    dxo, go = oracle.stack_backward([lp], 1, xs, dy, b, ONE, [oracle.zero_prefix_grads(NP, ONE.hidden)])
    errs = {"y": rel_l2(res["y"], yo), "dx": rel_l2(res["dx"], dxo)}
    for k in ("prefix_k", "prefix_v"):
        errs[k] = rel_l2(res["grads"][0][k], go[0][k])
    print(f"[fullsize] ptuning 1 block: {errs}", flush=True)
    assert all(v < TOL for v in errs.values()), errs


def test_ptuning_26_blocks_sampled(layers2):
    """The P-tuning workload (26 blocks, 32 x 1 U[512,2048], recompute,
    frozen weights): the shortest sequence's y and dx against the float32
    oracle."""
    w = synth.WORKLOADS["chatglm6b_26blk_ptuning128_ragged_32x1_recompute"]
    b = w.batch()
    n = w.shape.num_layers
    pl = [_with_prefix(layers2[l], l) for l in range(2)]
    layers = [pl[l % 2] for l in range(n)]
    x = synth.activations(b.total_tokens, ONE.hidden, seed=0)
    dy = synth.upstream_grad(b.total_tokens, ONE.hidden, seed=0, std=w.dy_std)
    g = GpuStack(w.shape, layers, "bf16", NP)
    res = g.run(b, x, dy, recompute=True, frozen=True)
    host = {"y": res["y"].float().cpu().numpy(), "dx": res["dx"].float().cpu().numpy()}
    del res
    g.close()
    s = int(np.argmin(b.seqlens))
    sb, r0, r1 = _seq_batch(b, s)
    yo, xs = oracle.stack_forward(layers, n, x[r0:r1], sb, w.shape, dtype=np.float32)
    grads = [oracle.zero_prefix_grads(NP, ONE.hidden, np.float32) for _ in range(n)]
    dxo, _ = oracle.stack_backward(layers, n, xs, dy[r0:r1], sb, w.shape, grads, dtype=np.float32)
    ey, edx = rel_l2(host["y"][r0:r1], yo), rel_l2(host["dx"][r0:r1], dxo)
    print(f"[fullsize] ptuning 26 blocks seq {s} (L={r1 - r0}): y {ey:.2e} dx {edx:.2e}", flush=True)
    assert ey < TOL and edx < TOL


# ---------------------------------------------------------------------------
# Server update at the full size: every parameter of the 26-block stack
# ---------------------------------------------------------------------------

def _sample_idx(n, k, seed):
    """k sorted indices: random ones plus both ends and the 2^31 / 2^32 marks."""
    g = np.random.default_rng(seed)
    marks = [0, 1, 2, 3, n - 5, n - 4, n - 3, n - 2, n - 1]
    for b in (1 << 31, 1 << 32):
        marks += [b + d for d in range(-4, 4) if 0 <= b + d < n]
    return np.unique(np.concatenate([g.integers(0, n, k), np.array(marks, np.int64)]))


def test_adam_full_stack_sampled():
    """One Adam step over all 5.24e9 parameters of the 26-block ChatGLM-6B
    shaped stack in one launch (indices past 2^32), with the bf16 copy and
    the gradient clear: 200k sampled elements against the oracle."""
    from tests.test_gpu_optim import check_adam
    n = W_LONG.shape.num_layers * W_LONG.shape.params_per_layer()
    assert n > (1 << 32)
    gen = torch.Generator(device="cuda").manual_seed(0)
    p = torch.randn(n, generator=gen, device="cuda")
    gr = torch.randn(n, generator=gen, device="cuda").mul_(1e-3)
    m = torch.randn(n, generator=gen, device="cuda").mul_(1e-4)
    v = torch.rand(n, generator=gen, device="cuda").mul_(1e-6)
    p16 = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    idx = torch.from_numpy(_sample_idx(n, 200_000, 1)).cuda()
    before = [t[idx].cpu().numpy() for t in (p, gr, m, v)]
    from paper_2406_14898_amd import flglm as F
    F.fl_adam_step(p, gr, m, v, p16, n, 5, 2e-2, 0.9, 0.999, 1e-8, True)
    torch.cuda.synchronize()
    after = [t[idx].cpu().numpy() for t in (p, m, v)]
    check_adam(*before, 5, *after)
    assert np.array_equal(p16[idx].view(torch.int16).cpu().numpy().view(np.uint16), synth.bf16_bits(after[0]))
    assert int(torch.count_nonzero(gr)) == 0
    print(f"[fullsize] adam over {n} parameters: sampled {idx.numel()} ok", flush=True)
    del p, gr, m, v, p16
    torch.cuda.empty_cache()


def test_average_full_stack_sampled():
    """Averaging four replicas of every parameter of the 26-block stack (with
    bf16 copies): sampled elements against the oracle, replicas equal."""
    n = W_LONG.shape.num_layers * W_LONG.shape.params_per_layer()
    gen = torch.Generator(device="cuda").manual_seed(1)
    reps = [torch.randn(n, generator=gen, device="cuda") for _ in range(4)]
    c16 = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(4)]
    idx = torch.from_numpy(_sample_idx(n, 200_000, 2)).cuda()
    before = [r[idx].cpu().numpy() for r in reps]
    from paper_2406_14898_amd import flglm as F
    F.fl_average_replicas(reps, c16, n)
    torch.cuda.synchronize()
    ref = oracle.average_replicas(before)
    out = [r[idx].cpu().numpy() for r in reps]
    bound = 8e-7 * np.max(np.abs(np.stack(before)), axis=0) + 1e-38
    for o, c in zip(out, c16):
        assert np.array_equal(o, out[0])
        assert np.array_equal(c[idx].view(torch.int16).cpu().numpy().view(np.uint16), synth.bf16_bits(o))
    assert np.all(np.abs(out[0] - ref) <= bound)
    print(f"[fullsize] average of 4 x {n} parameters: sampled {idx.numel()} ok", flush=True)
    del reps, c16
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# The whole split model at the full block shape and ChatGLM-6B's vocabulary
# ---------------------------------------------------------------------------

WS = synth.WORKLOADS["chatglm6b_28blk_split_ptuning128_ragged_32x1_recompute"]


def test_split_model_full_shape_ptuning(layers2):
    """Client embedding (130528 words) + block 0, one server block, client
    block N-1, final linear layer and cross-entropy, P-tuning v2 (128 prefix
    rows, weights frozen), on a two-client ragged batch: loss, the tensors
    crossing both split boundaries, every prefix gradient, against the
    float64 oracle."""
    from oracle import client as oc
    from paper_2406_14898_amd import BatchDesc, SplitModel
    b = synth.Batch(np.array([0, 100, 357], np.int32), np.array([0, 1, 2], np.int32))
    T, H, V = b.total_tokens, ONE.hidden, WS.vocab
    lays = [_with_prefix(layers2[l % 2], l) for l in range(3)]
    g = np.random.default_rng(5)
    emb = synth.bf16_round(g.standard_normal((V, H), dtype=np.float32))
    head = synth.bf16_round(g.standard_normal((V, H), dtype=np.float32) * np.float32(0.02))
    ids, labels = synth.token_ids(b, V, seed=5)
    scale = 1.0 / int((labels >= 0).sum())
    m = SplitModel(H, ONE.num_heads, ONE.ffn_hidden, ONE.rotary_dim, 1, V, "bf16", ONE.rope_base, ONE.ln_eps, NP)
    bd = BatchDesc.from_batch(b)
    buf = m.buffers(bd, recompute=True)
    dl = [{k: dev(v, "bf16") for k, v in lp.items()} for lp in lays]
    params = {"embedding": dev(emb, "bf16"), "lm_head": dev(head, "bf16"), "block0": dl[0], "server": [dl[1]],
              "block_last": dl[2]}
    gz = [{k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in d.items()
           if k.startswith("prefix_")} for d in dl]
    grads = {"block0": gz[0], "server": [gz[1]], "block_last": gz[2]}
    m.step(bd, ids, labels, params, grads, scale, buf, recompute=True)
    torch.cuda.synchronize()
    got = {k: buf[k].float().cpu().numpy() for k in ("h0", "hs", "d_hs", "d_h0", "loss_tok")}
    got["loss_sum"] = float(buf["loss_sum"].item())
    gg = [{k: v.cpu().numpy() for k, v in d.items()} for d in gz]
    m.close()
    del buf, params
    client = {"embedding": emb, "block0": lays[0], "block_last": lays[2], "lm_head": head}
    t = time.time()
    ref = oc.split_step(client, [lays[1]], ids, labels, b, ONE, scale, train_weights=False)
    errs = {"h0": rel_l2(got["h0"], ref["h0"]), "h_server": rel_l2(got["hs"], ref["h_server"]),
            "d_h_server": rel_l2(got["d_hs"], ref["d_h_server"]), "d_h0": rel_l2(got["d_h0"], ref["d_h0"]),
            "loss_tok": rel_l2(got["loss_tok"], ref["loss_tok"]),
            "loss_sum": abs(got["loss_sum"] - ref["loss_sum"]) / abs(ref["loss_sum"])}
    for i, key in enumerate(("grads_block0", None, "grads_block_last")):
        r = ref[key] if key else ref["grads_server"][0]
        for k in ("prefix_k", "prefix_v"):
            errs[f"{i}.{k}"] = rel_l2(gg[i][k], r[k])
    print(f"[fullsize] split model, oracle {time.time() - t:.0f}s: {errs}", flush=True)
    assert all(v < TOL for v in errs.values()), errs


def test_lm_head_bench_shape_sampled():
    """The final linear layer and loss at the benchmark's shape (41447 tokens,
    130528 words, hidden 4096) with the weight gradient: sampled tokens'
    losses and input-gradient rows against the oracle token by token, the
    loss sum against the per-token losses, and the weight gradient's
    property that each token's softmax-minus-one-hot row sums to zero, so
    sum_v dW[v] = 0 up to the bf16 rounding of the logit gradients."""
    from oracle import client as oc
    from paper_2406_14898_amd import ClientHead
    b = WS.batch()
    T, H, V = b.total_tokens, ONE.hidden, WS.vocab
    gen = torch.Generator(device="cuda").manual_seed(3)
    h = torch.randn((T, H), generator=gen, device="cuda").to(torch.bfloat16)
    w = (torch.randn((V, H), generator=gen, device="cuda") * 0.02).to(torch.bfloat16)
    ids, labels = synth.token_ids(b, V, seed=3)
    n_lab = int((labels >= 0).sum())
    ch = ClientHead(V, H, "bf16")
    ws = ch.workspace(T)
    lt = torch.empty(T, device="cuda")
    ls = torch.empty(1, device="cuda")
    ch.head_forward(h, w, labels, lt, ls, ws)
    dh = torch.empty_like(h)
    dw = torch.zeros((V, H), device="cuda")
    ch.head_backward(h, w, T, 1.0 / n_lab, dh, dw, ws)
    torch.cuda.synchronize()
    sample = np.unique(np.concatenate([np.random.default_rng(4).integers(0, T, 12), [0, T - 1]]))
    sample = sample[labels[sample] >= 0][:10]
    wh = w.float().cpu().numpy()
    hs = h[torch.from_numpy(sample).cuda()].float().cpu().numpy()
    lg, lse, lo, _ = oc.lm_head_forward(hs, wh, labels[sample])
    dho, _ = oc.lm_head_backward(hs, wh, lg, lse, labels[sample], 1.0 / n_lab)
    lt_h = lt.cpu().numpy()
    assert rel_l2(lt_h[sample], lo) < TOL
    assert rel_l2(dh[torch.from_numpy(sample).cuda()].float().cpu().numpy(), dho) < TOL
    assert abs(float(ls.item()) - float(lt_h.astype(np.float64).sum())) <= 1e-5 * abs(float(ls.item()))
    col = dw.sum(dim=0, dtype=torch.float64).cpu().numpy()
    scale_ref = float(torch.linalg.vector_norm(dw, dtype=torch.float64).item()) / np.sqrt(H)
    print(f"[fullsize] lm head T={T} V={V}: sum_v dW rms {np.sqrt(np.mean(col ** 2)):.2e} "
          f"vs column norm {scale_ref:.2e}", flush=True)
    assert np.sqrt(np.mean(col ** 2)) < 2e-2 * scale_ref
    ch.close()
    del ws, h, w, dw
    torch.cuda.empty_cache()


def test_glm_26_blocks_sampled(layers2):
    """The ChatGLM-6B-exact server stack of the GLM benchmark workload (26
    blocks, alpha residual, 2-D positions, prefix-LM batches of 32 x 1
    U[512,2048] with 25 % context, P-tuning v2 with frozen weights,
    recompute): the shortest sequence's y and dx against the float32 oracle.
    The blocks' weights are the plain layers' (the variant changes the
    arithmetic, not the parameters)."""
    w = synth.WORKLOADS["chatglm6b_28blk_split_glm_ptuning128_prefix_32x1_recompute"]
    b = w.batch()
    n = w.shape.num_layers
    pl = [_with_prefix(layers2[l], l) for l in range(2)]
    layers = [pl[l % 2] for l in range(n)]
    x = synth.activations(b.total_tokens, ONE.hidden, seed=0)
    dy = synth.upstream_grad(b.total_tokens, ONE.hidden, seed=0, std=w.dy_std)
    g = GpuStack(w.shape, layers, "bf16", NP)
    res = g.run(b, x, dy, recompute=True, frozen=True)
    host = {"y": res["y"].float().cpu().numpy(), "dx": res["dx"].float().cpu().numpy()}
    del res
    g.close()
    s = int(np.argmin(b.seqlens))
    sb, r0, r1 = _seq_batch(b, s)
    yo, xs = oracle.stack_forward(layers, n, x[r0:r1], sb, w.shape, dtype=np.float32)
    grads = [oracle.zero_prefix_grads(NP, ONE.hidden, np.float32) for _ in range(n)]
    dxo, _ = oracle.stack_backward(layers, n, xs, dy[r0:r1], sb, w.shape, grads, dtype=np.float32)
    ey, edx = rel_l2(host["y"][r0:r1], yo), rel_l2(host["dx"][r0:r1], dxo)
    print(f"[fullsize] GLM 26 blocks seq {s} (L={r1 - r0}, P={int(sb.prefix_len[0])}): y {ey:.2e} dx {edx:.2e}",
          flush=True)
    assert ey < TOL and edx < TOL


def test_long_batch_grads_add_over_client_parts(layers2):
    """A 70000-token batch (35 clients x 2000 tokens, one ChatGLM-6B-shaped
    block): the FFN weight-gradient GEMMs span more than 2^31 bytes along the
    tokens and run cut into pieces.  Client batching mixes nothing across
    clients and the weight gradients are sums over tokens, so the batch's
    gradients equal the sum of three client groups' runs, and its y / dx rows
    equal theirs, up to rounding: a GEMM splits the reduction of its partial
    last round of tiles, which tiles that is depends on the token count, and
    a changed fp32 summation order can move a bf16 intermediate by one unit
    in the last place (2^-8 relative).  The gradients then agree to well
    under 2^-9; a dropped, repeated or misplaced piece of the cut reduction
    (at least 4464 of the 70000 rows) would be off by more than 0.2."""
    b = synth.make_batch(35, 1, 2000, seed=7)
    T = b.total_tokens
    x = synth.activations(T, ONE.hidden, seed=7)
    dy = synth.upstream_grad(T, ONE.hidden, seed=7, std=1e-2)
    g = GpuStack(ONE, [layers2[0]], "bf16")
    full = g.run(b, x, dy, recompute=True)
    y_all, dx_all = full["y"].float().cpu().numpy(), full["dx"].float().cpu().numpy()
    grads_all = {k: v.double().cpu().numpy() for k, v in full["grads"][0].items()}
    del full
    acc = {k: np.zeros_like(v) for k, v in grads_all.items()}
    for part in (range(0, 12), range(12, 24), range(24, 35)):
        sub, rows = b.subset_clients(list(part))
        r = g.run(sub, x[rows], dy[rows], recompute=True)
        assert rel_l2(r["y"].float().cpu().numpy(), y_all[rows]) < 5e-3
        assert rel_l2(r["dx"].float().cpu().numpy(), dx_all[rows]) < 5e-3
        for k, v in r["grads"][0].items():
            acc[k] += v.double().cpu().numpy()
        del r
    g.close()
    errs = {k: rel_l2(grads_all[k], acc[k]) for k in acc}
    print(f"[fullsize] T={T}: batch vs sum of parts: "
          + " ".join(f"{k}={v:.1e}" for k, v in sorted(errs.items())), flush=True)
    assert all(e < 2e-3 for e in errs.values()), errs
    torch.cuda.empty_cache()
