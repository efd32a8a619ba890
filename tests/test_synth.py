"""The shared seeded-input module: bf16 encoding, determinism, batch layout."""

import numpy as np
import torch

import synth


def test_bf16_round_matches_torch_rne():
    g = np.random.default_rng(0)
    a = np.concatenate([g.standard_normal(100000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -1e-40, np.inf, -np.inf],
                                 np.float32)])
    ref = torch.tensor(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(synth.bf16_bits(a), ref)
    np.testing.assert_array_equal(synth.bf16_round(a), torch.tensor(a).to(torch.bfloat16).float().numpy())


def test_generators_are_deterministic_and_independent():
    shp = synth.WORKLOADS["tiny_2blk_fp32"].shape
    p0 = synth.layer_params(shp, 0, seed=0)
    p0b = synth.layer_params(shp, 0, seed=0)
    p1 = synth.layer_params(shp, 1, seed=0)
    for k in p0:
        np.testing.assert_array_equal(p0[k], p0b[k])
        assert not np.array_equal(p0[k], p1[k])
    assert abs(float(p0["w_qkv"].std()) - 0.02) < 0.002
    assert abs(float(p0["ln1_g"].mean()) - 1.0) < 0.01
    x = synth.activations(64, 32)
    assert np.array_equal(x, synth.activations(64, 32))
    assert not np.array_equal(x, synth.upstream_grad(64, 32))


def test_workload_batches():
    w = synth.WORKLOADS["chatglm6b_1blk_ragged_8x4"]
    b = w.batch()
    assert b.num_clients == 8 and b.num_seqs == 32
    assert b.seqlens.min() >= 128 and b.seqlens.max() <= 1024
    w4 = synth.WORKLOADS["chatglm6b_26blk_prefix_16x2x512"]
    b4 = w4.batch()
    assert b4.total_tokens == 16384 and (b4.prefix_len == 128).all()
    assert synth.WORKLOADS["chatglm6b_1blk_fwd_4x4x512"].batch().total_tokens == 8192
    assert synth.WORKLOADS["tiny_2blk_fp32"].batch().total_tokens == 256
    sub, rows = b.subset_clients([3, 1])
    assert sub.total_tokens == len(rows)
    r0, r1 = b.client_rows(3)
    np.testing.assert_array_equal(rows[: r1 - r0], np.arange(r0, r1))
