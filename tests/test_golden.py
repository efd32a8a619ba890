"""Oracle against the hand-derived worked examples in tests/golden/."""

import json
import math
import os

import numpy as np
import pytest

import oracle
import synth

CASES = {c["name"]: c for c in json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                                           "worked_examples.json")))["cases"]}
ENV = {"__builtins__": {}, "e": math.e, "pi": math.pi, "sqrt": math.sqrt, "tanh": math.tanh}


def ev(x):
    if isinstance(x, list):
        return np.array([ev(v) for v in x], np.float64)
    return float(eval(x, ENV))


@pytest.mark.parametrize("name", ["attention_causal_two_tokens", "attention_prefix_two_tokens"])
def test_attention_examples(name):
    c = CASES[name]
    pre = None if c["prefix"] is None else np.array([c["prefix"]], np.int32)
    b = synth.Batch(np.array([0, 2], np.int32), np.array([0, 1], np.int32), c["mask"], pre)
    q, k, v = (np.array(c[n], np.float64)[:, None, :] for n in "qkv")
    o = oracle.attention_forward(q, k, v, b)[:, 0, :]
    np.testing.assert_allclose(o, ev(c["o"]), rtol=1e-15, atol=1e-15)


def test_layer_norm_example():
    c = CASES["layer_norm_1234"]
    y, _, _ = oracle.layer_norm(np.array([c["x"]], np.float64), np.array(c["g"], np.float64),
                                np.array(c["b"], np.float64), c["eps"])
    np.testing.assert_allclose(y[0], ev(c["y"]), rtol=1e-14, atol=1e-14)


def test_gelu_example():
    c = CASES["gelu_tanh"]
    z = np.array(c["z"], np.float64)
    np.testing.assert_allclose(oracle.gelu(z), ev(c["gelu"]), rtol=1e-15, atol=1e-16)
    assert oracle.gelu_grad(np.array([0.0]))[0] == ev(c["gelu_grad_at_0"])


def test_block_zero_weights_example():
    c = CASES["block_zero_weights"]
    shape = synth.StackShape(1, c["hidden"], c["num_heads"], c["ffn_hidden"], c["rotary_dim"])
    p = {k: np.zeros_like(v, dtype=np.float64)
         for k, v in synth.layer_params(shape, 0, seed=0, bf16=False).items()}
    p["ln1_g"][:] = 1.0
    p["ln2_g"][:] = 1.0
    p["b_qkv"][:] = np.linspace(-1, 1, p["b_qkv"].size)  # any value: the zero W_o removes it
    p["b_1"][:] = 0.5
    p["b_o"][:] = c["b_o"]
    p["b_2"][:] = c["b_2"]
    cu = np.concatenate([[0], np.cumsum(c["seqlens"])]).astype(np.int32)
    b = synth.Batch(cu, np.array([0, len(c["seqlens"])], np.int32))
    T = int(cu[-1])
    x = np.arange(T, dtype=np.float64)[:, None] - 0.5 * np.arange(c["hidden"])[None, :]
    y, _ = oracle.block_forward(p, x, b, shape)
    np.testing.assert_allclose(y - x, np.broadcast_to(ev(c["y_minus_x"]), x.shape), rtol=0, atol=1e-14)


def test_pack_two_clients_example():
    c = CASES["pack_two_clients"]
    per = [np.array(t, np.float64) for t in c["client_tensors"]]
    cu = np.array(c["cu_seqlens"], np.int32)
    csp = np.array(c["client_seq_ptr"], np.int32)
    packed = oracle.pack_clients(per, cu, csp)
    np.testing.assert_array_equal(packed[:, 0], np.array(c["packed"], np.float64))
    back = oracle.unpack_clients(packed, cu, csp)
    for got, want in zip(back, c["unpacked"]):
        np.testing.assert_array_equal(got, np.array(want, np.float64))
    np.testing.assert_array_equal(oracle.client_token_ranges(cu, csp), np.array(c["client_rows"]))
