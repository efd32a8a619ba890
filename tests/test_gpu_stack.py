"""Stack-level parity of the HIP path against the oracle (fp32 mode within
1e-4 relative L2, bf16 within 2e-2, per tensor and per client slice), plus
the properties client batching must keep on the GPU: isolation between
clients, invariance to client order, determinism, recompute equivalence and
exact packing."""

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import TOL, dev, host, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from paper_2406_14898_amd import BatchDesc, flglm as F  # noqa: E402
from tests.stack_runner import GpuStack  # noqa: E402

TINY_W = synth.WORKLOADS["tiny_2blk_fp32"]
SHAPE = TINY_W.shape


def _inputs(batch, dt, seed=0, dy_std=1.0, shape=SHAPE):
    bf = dt == "bf16"
    layers = [synth.layer_params(shape, l, seed=seed, bf16=bf) for l in range(shape.num_layers)]
    x = synth.activations(batch.total_tokens, shape.hidden, seed=seed, bf16=bf)
    dy = synth.upstream_grad(batch.total_tokens, shape.hidden, seed=seed, bf16=bf, std=dy_std)
    return layers, x, dy


def _oracle(layers, x, dy, batch, shape=SHAPE):
    y, xs = oracle.stack_forward(layers, shape.num_layers, x, batch, shape)
    dx, grads = oracle.stack_backward(layers, shape.num_layers, xs, dy, batch, shape)
    return y, dx, grads


def _check(res, ref, batch, tol):
    y, dx, grads = ref
    errs = {"y": rel_l2(res["y"], y), "dx": rel_l2(res["dx"], dx)}
    for l, g in enumerate(grads):
        for k, v in g.items():
            errs[f"{l}.{k}"] = rel_l2(res["grads"][l][k], v)
    for c in range(batch.num_clients):
        r0, r1 = batch.client_rows(c)
        errs[f"y[c{c}]"] = rel_l2(res["y"][r0:r1], y[r0:r1])
        errs[f"dx[c{c}]"] = rel_l2(res["dx"][r0:r1], dx[r0:r1])
    bad = {k: v for k, v in errs.items() if not v < tol}
    assert not bad, (bad, max(errs.values()))
    return max(errs.values())


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_tiny_stack_matches_oracle(dt):
    """2 blocks, H 256, 4 heads of 64, FFN 1024, 2 clients x 2 x 64 tokens, causal."""
    b = TINY_W.batch()
    layers, x, dy = _inputs(b, dt)
    g = GpuStack(SHAPE, layers, dt)
    res = g.to_host(g.run(b, x, dy))
    g.close()
    _check(res, _oracle(layers, x, dy, b), b, TOL[dt])


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_ragged_clients_match_oracle(dt, mask):
    """Ragged sequences (1 .. 200 tokens, several 64/128-row tiles and tails)
    across 3 clients, head dim 128."""
    shape = synth.StackShape(num_layers=2, hidden=256, num_heads=2, ffn_hidden=512, rotary_dim=64)
    cu = np.array([0, 1, 67, 200, 400, 529, 530], np.int32)
    csp = np.array([0, 2, 3, 6], np.int32)
    pre = np.array([0, 16, 40, 200, 3, 1], np.int32) if mask == "prefix" else None
    b = synth.Batch(cu, csp, mask, pre)
    layers, x, dy = _inputs(b, dt, seed=3, shape=shape)
    g = GpuStack(shape, layers, dt)
    res = g.to_host(g.run(b, x, dy))
    g.close()
    _check(res, _oracle(layers, x, dy, b, shape), b, TOL[dt])


def test_recompute_and_determinism_bitwise():
    b = synth.make_batch(3, 2, (20, 150), "prefix", seed=5)
    layers, x, dy = _inputs(b, "bf16", seed=5)
    g = GpuStack(SHAPE, layers, "bf16")
    a = g.to_host(g.run(b, x, dy, recompute=False))
    a2 = g.to_host(g.run(b, x, dy, recompute=False))
    r = g.to_host(g.run(b, x, dy, recompute=True))
    g.close()
    for other in (a2, r):
        np.testing.assert_array_equal(other["y"], a["y"])
        np.testing.assert_array_equal(other["dx"], a["dx"])
        for l in range(SHAPE.num_layers):
            for k in a["grads"][l]:
                np.testing.assert_array_equal(other["grads"][l][k], a["grads"][l][k])


def test_client_isolation_nan_poison():
    """A NaN-poisoned client changes no bit of any other client's output or
    input gradient."""
    b = synth.make_batch(3, 2, (30, 90), "causal", seed=6)
    layers, x, dy = _inputs(b, "bf16", seed=6)
    g = GpuStack(SHAPE, layers, "bf16")
    a = g.to_host(g.run(b, x, dy))
    r0, r1 = b.client_rows(1)
    xp = x.copy()
    xp[r0:r1] = np.nan
    p = g.to_host(g.run(b, xp, dy))
    g.close()
    keep = np.r_[0:r0, r1:b.total_tokens]
    np.testing.assert_array_equal(p["y"][keep], a["y"][keep])
    np.testing.assert_array_equal(p["dx"][keep], a["dx"][keep])
    assert np.isnan(p["y"][r0:r1]).all()


def test_client_order_invariance_bitwise():
    """Reordering the clients in the packed batch gives each client the same
    bits of output and input gradient (weight gradients are sums; not
    compared bitwise)."""
    b = synth.make_batch(4, 1, (10, 200), "causal", seed=7)
    layers, x, dy = _inputs(b, "bf16", seed=7)
    g = GpuStack(SHAPE, layers, "bf16")
    a = g.to_host(g.run(b, x, dy))
    order = [2, 0, 3, 1]
    pb, rows = b.subset_clients(order)
    p = g.to_host(g.run(pb, x[rows], dy[rows]))
    g.close()
    np.testing.assert_array_equal(p["y"], a["y"][rows])
    np.testing.assert_array_equal(p["dx"], a["dx"][rows])


def test_weight_grads_accumulate():
    """The backward adds into the caller's gradient buffers."""
    b = TINY_W.batch()
    layers, x, dy = _inputs(b, "f32")
    g = GpuStack(SHAPE, layers, "f32")
    grads = g.zero_grads()
    for gr in grads:
        for t in gr.values():
            t.fill_(0.25)
    res = g.to_host(g.run(b, x, dy, grads=grads))
    g.close()
    _, _, ref = _oracle(layers, x, dy, b)
    for l in range(SHAPE.num_layers):
        for k, v in ref[l].items():
            assert rel_l2(res["grads"][l][k], v + 0.25) < 1e-4, (l, k)


def test_forward_only_matches_saved_forward():
    b = synth.make_batch(2, 3, (5, 70), "prefix", seed=8)
    layers, x, dy = _inputs(b, "bf16", seed=8)
    g = GpuStack(SHAPE, layers, "bf16")
    inf = g.to_host(g.run(b, x, None))
    tr = g.to_host(g.run(b, x, dy))
    g.close()
    np.testing.assert_array_equal(inf["y"], tr["y"])


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_pack_unpack_bit_exact(dt):
    b = synth.make_batch(3, 2, (3, 40), seed=9)
    H = SHAPE.hidden
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    rng = np.random.default_rng(9)
    per = []
    for c in range(b.num_clients):
        s0, s1 = int(b.client_seq_ptr[c]), int(b.client_seq_ptr[c + 1])
        Lmax = int(b.seqlens[s0:s1].max())
        a = rng.standard_normal((Lmax, s1 - s0, H)).astype(np.float32)
        per.append(synth.bf16_round(a) if dt == "bf16" else a)
    ref = oracle.pack_clients(per, b.cu_seqlens, b.client_seq_ptr)
    g = GpuStack(SHAPE, [synth.layer_params(SHAPE, l) for l in range(2)], dt)
    bd = BatchDesc.from_batch(b)
    _, ws = g.ss.buffers(bd, False, with_saved=False)
    dbufs = [dev(a, dt) for a in per]
    packed = torch.full((b.total_tokens, H), float("nan"), dtype=tdt, device="cuda")
    F.fl_pack_clients(g.ss.handle, bd, dbufs, packed, ws, ws.numel())
    outs = [torch.full_like(t, float("nan")) for t in dbufs]
    F.fl_unpack_clients(g.ss.handle, bd, packed, outs, ws, ws.numel())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(packed), ref)
    back = oracle.unpack_clients(ref, b.cu_seqlens, b.client_seq_ptr)
    for o, r in zip(outs, back):
        np.testing.assert_array_equal(host(o), r)
    rng_ = oracle.client_token_ranges(b.cu_seqlens, b.client_seq_ptr)
    for c in range(b.num_clients):
        assert F.fl_client_token_range(bd, c) == tuple(rng_[c])
    g.close()


# ---------------------------------------------------------------------------
# P-tuning v2 (Section 3.1, Appendix A): prefix keys / values per block,
# weights frozen or trained
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("frozen", [True, False])
@pytest.mark.parametrize("mask", ["causal", "prefix"])
@pytest.mark.parametrize("num_prefix", [16, 70])
def test_ptuning_stack_matches_oracle(frozen, mask, num_prefix):
    """bf16, 2 blocks, head dim 128, ragged clients; the prefix gradients are
    the sum over every sequence of every client.  Frozen: only prefix
    gradients are formed (the weight-gradient pointers are NULL)."""
    shape = synth.StackShape(num_layers=2, hidden=256, num_heads=2, ffn_hidden=512, rotary_dim=64)
    cu = np.array([0, 1, 67, 200, 400, 529, 530], np.int32)
    csp = np.array([0, 2, 3, 6], np.int32)
    pre = np.array([0, 16, 40, 200, 3, 1], np.int32) if mask == "prefix" else None
    b = synth.Batch(cu, csp, mask, pre)
    layers, x, dy = _inputs(b, "bf16", seed=5, shape=shape)
    rng = np.random.default_rng(7)
    for lp in layers:
        for k in ("prefix_k", "prefix_v"):
            lp[k] = synth.bf16_round(rng.standard_normal((num_prefix, shape.hidden)).astype(np.float32))
    g = GpuStack(shape, layers, "bf16", num_prefix)
    res = g.to_host(g.run(b, x, dy, frozen=frozen))
    g.close()
    y, xs = oracle.stack_forward(layers, shape.num_layers, x, b, shape)
    want = [oracle.zero_prefix_grads(num_prefix, shape.hidden) for _ in layers]
    if not frozen:
        want = [dict(oracle.zero_grads(shape), **w) for w in want]
    dx, grads = oracle.stack_backward(layers, shape.num_layers, xs, dy, b, shape, want)
    assert all(set(r) == set(w) for r, w in zip(res["grads"], grads))
    _check(res, (y, dx, grads), b, TOL["bf16"])


SHAPES = {
    # widths that are not powers of two, an FFN width other than 4 H, both
    # head dims, and the rotary widths at their ends and in between
    "h768_d128_f2304_r96": synth.StackShape(num_layers=2, hidden=768, num_heads=6, ffn_hidden=2304, rotary_dim=96),
    "h1280_d64_f3328_r64full": synth.StackShape(num_layers=2, hidden=1280, num_heads=20, ffn_hidden=3328,
                                                rotary_dim=64),
    "h512_d128_f1536_r0": synth.StackShape(num_layers=2, hidden=512, num_heads=4, ffn_hidden=1536, rotary_dim=0),
    "h256_d128_f768_r128full": synth.StackShape(num_layers=2, hidden=256, num_heads=2, ffn_hidden=768,
                                                rotary_dim=128),
}


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("name", sorted(SHAPES))
def test_other_block_shapes_match_oracle(name, dt):
    """The stack at block shapes other than the two workload shapes: every
    GEMM width a multiple of 256 but not of 512 somewhere, 9- and 13-tile
    column counts, no rotary at all and rotary over the whole head; a ragged
    prefix-LM batch with a one-token sequence, across three clients."""
    shape = SHAPES[name]
    cu = np.array([0, 1, 70, 203, 260, 389], np.int32)
    csp = np.array([0, 2, 3, 5], np.int32)
    pre = np.array([1, 17, 0, 57, 129], np.int32)
    b = synth.Batch(cu, csp, "prefix", pre)
    layers, x, dy = _inputs(b, dt, seed=11, shape=shape)
    g = GpuStack(shape, layers, dt)
    res = g.to_host(g.run(b, x, dy))
    g.close()
    worst = _check(res, _oracle(layers, x, dy, b, shape), b, TOL[dt])
    print(f"[shapes] {name} {dt}: worst rel-L2 {worst:.2e}", flush=True)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("mask", ["causal", "prefix"])
def test_single_token_batch_matches_oracle(dt, mask):
    """The smallest batch: one client sending one 1-token sequence (T = 1).
    Attention reduces to o = v (the token sees only itself), every GEMM is a
    single ragged row, LayerNorm and the column sums see one row."""
    b = synth.Batch(np.array([0, 1], np.int32), np.array([0, 1], np.int32), mask,
                    np.array([1], np.int32) if mask == "prefix" else None)
    layers, x, dy = _inputs(b, dt, seed=12)
    g = GpuStack(SHAPE, layers, dt)
    res = g.to_host(g.run(b, x, dy))
    g.close()
    _check(res, _oracle(layers, x, dy, b), b, TOL[dt])


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", ["257_one_token_clients", "one_4096_token_sequence"])
def test_extreme_batches_match_oracle(case, dt):
    """257 clients of one token each (T one past a 256-row tile, every
    sequence its own client) and a single 4096-token sequence (rotary angles
    up to position 4095), prefix-LM with a quarter-length context."""
    if case == "257_one_token_clients":
        cu = np.arange(258, dtype=np.int32)
        csp = np.arange(258, dtype=np.int32)
    else:
        cu = np.array([0, 4096], np.int32)
        csp = np.array([0, 1], np.int32)
    pre = (np.diff(cu) // 4).astype(np.int32)
    b = synth.Batch(cu, csp, "prefix", pre)
    layers, x, dy = _inputs(b, dt, seed=13)
    g = GpuStack(SHAPE, layers, dt)
    res = g.to_host(g.run(b, x, dy))
    g.close()
    worst = _check(res, _oracle(layers, x, dy, b), b, TOL[dt])
    print(f"[extreme] {case} {dt}: worst rel-L2 {worst:.2e}", flush=True)


def test_launch_profile_accounts_every_launch():
    """The opt-in launch timing the benchmark reads: one forward (keeping
    intermediates) and one backward of the 2-block stack record every engine
    launch by class, with the algorithmic work of each, and a duration."""
    import bench
    b = synth.make_batch(2, 2, (30, 170), "prefix", seed=14)
    layers, x, dy = _inputs(b, "bf16", seed=14)
    g = GpuStack(SHAPE, layers, "bf16")
    F.fl_stack_profile(g.ss.handle, True)
    g.run(b, x, dy)
    prof = F.profile_table(g.ss.handle)
    F.fl_stack_profile(g.ss.handle, False)
    g.close()
    N = SHAPE.num_layers
    per_block = {"layernorm_fwd": 2, "gemm_nt_bias": 1, "rope_qk": 1, "attn_fwd": 1, "gemm_nt_bias_res": 2,
                 "gemm_nt_bias_gelu": 1, "gemm_tn_acc": 4, "gemm_nn_gelu_bwd": 1, "gemm_nn": 3,
                 "layernorm_bwd": 2, "attn_bwd": 1}
    want = {k: v * N for k, v in per_block.items()}
    want["plan"] = 2
    # column-sum launches: db_1's finish, db_qkv, and the two LayerNorm
    # backward finishes (gain / shift, plus db_o and the block below's db_2);
    # the top block also sums its own dy for db_2
    want["colsum"] = 4 * N + 1
    assert {k: r["launches"] for k, r in prof.items()} == want
    assert all(r["ms"] > 0 for r in prof.values())
    w = synth.WORKLOADS["tiny_2blk_fp32"]
    alg = bench.algorithmic_flops(w, b)
    gemm = sum(r["flops"] for k, r in prof.items() if k.startswith("gemm"))
    attn = sum(r["flops"] for k, r in prof.items() if k.startswith("attn"))
    assert gemm == pytest.approx(alg["gemm"], rel=1e-9)
    assert attn == pytest.approx(alg["attention"], rel=1e-9)


def test_launch_profile_of_chosen_classes():
    """Timing a subset of the classes (the benchmark's timed steps time only
    the dominant one): launches of the other classes carry no record, the
    chosen class's count equals a full profile's, and a zero mask turns
    timing off."""
    b = synth.make_batch(2, 2, (30, 170), "causal", seed=15)
    layers, x, dy = _inputs(b, "bf16", seed=15)
    g = GpuStack(SHAPE, layers, "bf16")
    names = {F.fl_profile_class_name(c): c for c in range(F.FL_PROF_NUM_CLASSES)}
    F.fl_stack_profile(g.ss.handle, True)
    g.run(b, x, dy)
    full = F.profile_table(g.ss.handle)
    mask = (1 << names["gemm_tn_acc"]) | (1 << names["attn_fwd"])
    F.fl_stack_profile_classes(g.ss.handle, mask)
    g.run(b, x, dy)
    some = F.profile_table(g.ss.handle)
    F.fl_stack_profile_classes(g.ss.handle, 0)
    g.run(b, x, dy)
    none = F.profile_table(g.ss.handle)
    g.close()
    assert set(some) == {"gemm_tn_acc", "attn_fwd"}
    assert all(some[k]["launches"] == full[k]["launches"] and some[k]["ms"] > 0 for k in some)
    # records stay until the next enabling call; disabling adds none
    assert none == some
