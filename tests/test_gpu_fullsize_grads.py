"""Gradient parity at the token counts the benchmark runs (Section 3.1: the
server returns dL/dh_0 to every client and updates its own weights; Section
3.3: the clients' smashed data are stacked into one batch).

* One ChatGLM-6B-shaped block over the whole ragged batch of 8 clients x 4
  sequences U[128,1024] (18712 tokens) and over the 32 x 1 U[512,2048] batch
  of the 26-block benchmark (41447 tokens): y and dx, in total and per
  client, and all twelve weight, bias and LayerNorm gradients against the
  float32 oracle over the same batch (the reductions run over every token).
* The 26-block benchmark stack itself (per-block recompute) with 26 distinct
  layers: y and dx of its shortest and its longest sequence against the
  float32 oracle run on those two sequences alone (client batching mixes
  nothing across sequences, invariant I1 of the oracle tests).

Parameters are drawn on the GPU with torch's seeded generator (host draws of
5.2e9 values would take minutes) and copied to the host for the oracle;
activations and upstream gradients are the host draws of the other tests."""

import time

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_helpers import rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from tests.stack_runner import GpuStack  # noqa: E402

W_RAGGED = synth.WORKLOADS["chatglm6b_1blk_ragged_8x4"]
W_LONG = synth.WORKLOADS["chatglm6b_26blk_ragged_32x1_recompute"]
ONE = W_RAGGED.shape
TOL = 2e-2


def _host_layer(lp):
    return {k: v.float().cpu().numpy() for k, v in lp.items()}


def _one_block_all_grads(b, dy_std, seed):
    T, H = b.total_tokens, ONE.hidden
    t0 = time.time()
    lpd = synth.device_layer_params(ONE, 0, seed=seed)
    lp = _host_layer(lpd)
    x = synth.activations(T, H, seed=seed)
    dy = synth.upstream_grad(T, H, seed=seed, std=dy_std)
    g = GpuStack(ONE, [lpd], "bf16")
    res = g.to_host(g.run(b, x, dy))
    g.close()
    del lpd
    print(f"[grads] T={T}: inputs and GPU run {time.time() - t0:.1f}s", flush=True)
    t0 = time.time()
    yo, cache = oracle.block_forward(lp, x, b, ONE, np.float32)
    print(f"[grads] T={T}: float32 oracle forward {time.time() - t0:.1f}s", flush=True)
    go = oracle.zero_grads(ONE, np.float32)
    dxo = oracle.block_backward(lp, cache, dy, b, ONE, go, np.float32)
    del cache
    print(f"[grads] T={T}: float32 oracle {time.time() - t0:.1f}s", flush=True)
    errs = {"y": rel_l2(res["y"], yo), "dx": rel_l2(res["dx"], dxo)}
    per_client = []
    for c in range(b.num_clients):
        r0, r1 = b.client_rows(c)
        per_client.append(max(rel_l2(res["y"][r0:r1], yo[r0:r1]), rel_l2(res["dx"][r0:r1], dxo[r0:r1])))
    errs["worst client y/dx"] = max(per_client)
    for k, v in go.items():
        errs[k] = rel_l2(res["grads"][0][k], v)
    print(f"[grads] T={T}: " + ", ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
    bad = {k: v for k, v in errs.items() if not v < TOL}
    assert not bad, bad


@pytest.mark.timeout(600)
def test_1blk_all_grads_ragged_8x4():
    """One block, the 8 x 4 U[128,1024] batch (18712 tokens)."""
    _one_block_all_grads(W_RAGGED.batch(), W_RAGGED.dy_std, seed=5)


@pytest.mark.timeout(600)
def test_1blk_all_grads_ragged_32x1():
    """One block, the benchmark's 32 x 1 U[512,2048] batch (41447 tokens):
    the weight-gradient GEMMs reduce over 41447 tokens (648 stages)."""
    b = W_LONG.batch()
    assert b.total_tokens == 41447
    _one_block_all_grads(b, W_LONG.dy_std, seed=6)


@pytest.mark.timeout(900)
def test_26blk_ragged_32x1_recompute_distinct_layers():
    """The benchmark's 26-block stack (per-block recompute) with 26 distinct
    layers: y and dx of the shortest and the longest sequence."""
    w = W_LONG
    b = w.batch()
    n = w.shape.num_layers
    T, H = b.total_tokens, ONE.hidden
    t0 = time.time()
    lds = [synth.device_layer_params(ONE, l, seed=0) for l in range(n)]
    x = synth.activations(T, H, seed=0)
    dy = synth.upstream_grad(T, H, seed=0, std=w.dy_std)
    g = GpuStack(w.shape, lds, "bf16")
    res = g.run(b, x, dy, recompute=True)
    y, dx = res["y"].float().cpu().numpy(), res["dx"].float().cpu().numpy()
    del res
    g.close()
    del g
    layers = [_host_layer(lp) for lp in lds]
    del lds
    torch.cuda.empty_cache()
    print(f"[grads] 26 blocks: layers, GPU run, copies {time.time() - t0:.1f}s", flush=True)
    lens = b.seqlens
    picks = [int(np.argmin(lens)), int(np.argmax(lens))]
    # every client holds one sequence: the two picked clients form the batch
    sub, rows = b.subset_clients(picks)
    t0 = time.time()

    def layer(l):  # one progress line per block the oracle takes up
        print(f"[grads] 26 blocks: oracle at block {l} ({time.time() - t0:.0f}s)", flush=True)
        return layers[l]

    yo, caches = oracle.stack_forward(layer, n, x[rows], sub, w.shape, np.float32, keep="caches")
    dxo, _ = oracle.stack_backward(layer, n, caches, dy[rows], sub, w.shape, [{} for _ in range(n)], np.float32)
    del caches
    print(f"[grads] 26 blocks: float32 oracle on sequences {picks} {time.time() - t0:.1f}s", flush=True)
    errs = {}
    for i, s in enumerate(picks):
        a0, a1 = sub.client_rows(i)
        r0, r1 = int(b.cu_seqlens[s]), int(b.cu_seqlens[s + 1])
        errs[f"seq {s} (L={r1 - r0}) y"] = rel_l2(y[r0:r1], yo[a0:a1])
        errs[f"seq {s} (L={r1 - r0}) dx"] = rel_l2(dx[r0:r1], dxo[a0:a1])
    print("[grads] 26 blocks: " + ", ".join(f"{k} {v:.2e}" for k, v in errs.items()), flush=True)
    assert all(v < TOL for v in errs.values()), errs
