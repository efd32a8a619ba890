"""The allocation-free inference forward against the existing one: two calls
in a row (the second on a smaller batch, so the shared scratch array holds
the first call's data), each equal bit for bit to fl_server_stack_forward
with saved = NULL on the same inputs (the stated bar: rel-L2 2e-2 in bf16,
1e-4 in fp32; the kernels being the same, the bits agree)."""

import pytest

import synth
from tests.gpu_helpers import TOL, dev, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from paper_2406_14898_amd import BatchDesc, ServerStack  # noqa: E402
from paper_2406_14898_amd import flglm as F  # noqa: E402

CHATGLM = synth.StackShape(2, 4096, 32, 16384, 64)
TINY = synth.StackShape(2, 256, 4, 1024, 32)


def _regular(ss, bd, params, x):
    _, ws = ss.buffers(bd, False, with_saved=False)
    y = torch.empty_like(x)
    ss.forward(bd, params, x, y, None, ws, False)
    torch.cuda.synchronize()
    return y


def _noalloc(ss, bd, params, x):
    y = torch.empty_like(x)
    F.fl_server_stack_forward_noalloc(ss.handle, bd, [F.layer_params(p) for p in params], x, y)
    return y


@pytest.mark.parametrize("case", ["chatglm_bf16", "tiny_f32", "tiny_bf16_ptuning"])
def test_noalloc_matches_the_regular_forward_twice(case):
    shape = CHATGLM if case.startswith("chatglm") else TINY
    dt = "f32" if case.endswith("f32") else "bf16"
    num_prefix = 24 if case.endswith("ptuning") else 0
    ss = ServerStack(shape.num_layers, shape.hidden, shape.num_heads, shape.ffn_hidden, shape.rotary_dim, dt,
                     num_prefix=num_prefix)
    if shape is CHATGLM:
        params = [synth.device_layer_params(shape, l, seed=11) for l in range(shape.num_layers)]
        big = synth.make_batch(3, 3, (60, 300), "prefix", seed=11)   # ~1600 tokens, 9 sequences
        small = synth.make_batch(2, 1, (90, 200), "causal", seed=12)
    else:
        params = [{k: dev(v, dt) for k, v in synth.layer_params(shape, l, seed=11, bf16=dt == "bf16").items()}
                  for l in range(shape.num_layers)]
        if num_prefix:
            for l, p in enumerate(params):
                p.update({k: dev(v, dt) for k, v in synth.prefix_params(shape, l, num_prefix, seed=11).items()})
        big = synth.make_batch(4, 3, (5, 150), "prefix", seed=13)
        small = synth.make_batch(1, 2, (1, 40), "causal", seed=14)
    assert small.total_tokens < big.total_tokens
    xs = [dev(synth.activations(b.total_tokens, shape.hidden, seed=20 + i, bf16=dt == "bf16"), dt)
          for i, b in enumerate((big, small))]
    bds = [BatchDesc.from_batch(b) for b in (big, small)]
    # the two allocation-free calls back to back, then the regular ones
    ys = [_noalloc(ss, bd, params, x) for bd, x in zip(bds, xs)]
    torch.cuda.synchronize()
    refs = [_regular(ss, bd, params, x) for bd, x in zip(bds, xs)]
    for b, y, r in zip((big, small), ys, refs):
        err = rel_l2(y.float().cpu().numpy(), r.float().cpu().numpy())
        print(f"[noalloc] {case} T={b.total_tokens}: rel-L2 {err:.2e}, bitwise {torch.equal(y, r)}", flush=True)
        assert err < TOL[dt]
        assert torch.equal(y, r)
    ss.close()
