"""Seeded synthetic inputs for the FL-GLM server stack.

This module is shared by the oracle side (tests, CPU baseline) and the HIP
side (tests, bench, smoke).  It holds no arithmetic of the method itself:
only random draws, the fp32 -> bf16 round-to-nearest-even encoding of those
draws, and the packed ragged-batch bookkeeping (which rows belong to which
sequence and client).

Workload shapes follow the paper's setting: ChatGLM-6B has 4096 hidden units
and 32 attention heads per block (Section 4.1.4, Parameter Settings), the
server holds the middle 26 of its 28 blocks (Section 3.1, Model Split), and
client-batch training stacks the smashed data of M clients into one batch
(Section 3.3, Parallel Acceleration).  The paper fixes no sequence lengths
(it adjusted them per dataset), so the lengths below are synthetic stand-ins.

Generator: numpy ``Generator(PCG64(SeedSequence([seed, stream, layer])))``.
Streams: 0 = layer parameters (one generator per layer, so a consumer can
produce the layers one at a time), 1 = input activations x, 2 = upstream
gradient dy, 3 = sequence lengths.  Parameter draw order inside a layer is
W_qkv, b_qkv, W_o, b_o, W_1, b_1, W_2, b_2, ln1_g, ln1_b, ln2_g, ln2_b.
"""

from __future__ import annotations

from dataclasses import dataclass, field
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "STREAM_PARAMS", "STREAM_X", "STREAM_DY", "STREAM_LENS", "STREAM_PREFIX", "STREAM_TOKENS",
    "PARAM_NAMES", "StackShape", "Batch", "Workload", "WORKLOADS",
    "bf16_round", "bf16_bits", "bits_to_f32", "rng", "make_batch",
    "param_shapes", "layer_params", "device_layer_params", "prefix_params", "activations", "upstream_grad", "token_ids",
]

STREAM_PARAMS, STREAM_X, STREAM_DY, STREAM_LENS, STREAM_PREFIX, STREAM_TOKENS = 0, 1, 2, 3, 4, 5

PARAM_NAMES = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2",
               "ln1_g", "ln1_b", "ln2_g", "ln2_b")


# ----------------------------------------------------------------------------
# bf16 encoding (round to nearest, ties to even), bit-exact, vectorised.
# ----------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 array -> uint16 bf16 bit patterns, round-to-nearest-even.

    NaN inputs map to a quiet NaN pattern; no NaN is ever drawn here, the
    branch only keeps the encoding total.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # no overflow for any non-NaN pattern: the largest is 0xFF800000 (-inf)
    r = ((u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def bits_to_f32(b: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> the exactly equal fp32 values."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """fp32 values rounded (RNE) to the nearest bf16, returned as fp32."""
    return bits_to_f32(bf16_bits(a))


def rng(seed: int, stream: int, layer: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, layer])))


# ----------------------------------------------------------------------------
# Shapes and batches
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class StackShape:
    """Shape of the server-held block stack (all blocks identical)."""
    num_layers: int
    hidden: int
    num_heads: int
    ffn_hidden: int
    rotary_dim: int          # rotated leading dims of each head (half the head dim)
    rope_base: float = 10000.0
    ln_eps: float = 1e-5
    residual_alpha: float = 0.0   # > 0: ChatGLM-6B residual alpha * LN(x) + f(LN(x)); 0: x + f(LN(x))
    rotary_2d: bool = False       # GLM 2-D positions: second half of each head rotated by block position

    @property
    def head_dim(self) -> int:
        return self.hidden // self.num_heads

    def params_per_layer(self) -> int:
        H, F = self.hidden, self.ffn_hidden
        return 3 * H * H + 3 * H + H * H + H + F * H + F + H * F + H + 4 * H


@dataclass
class Batch:
    """Packed ragged batch: rows of client c, then its sequences, in order.

    cu_seqlens[s]..cu_seqlens[s+1] are the rows of sequence s;
    client_seq_ptr[c]..client_seq_ptr[c+1] are the sequences of client c.
    prefix_len[s] is the bidirectional prefix of sequence s (prefix-LM mask)
    or None for a causal mask.
    """
    cu_seqlens: np.ndarray            # int32 [S+1]
    client_seq_ptr: np.ndarray        # int32 [C+1]
    mask: str = "causal"              # "causal" | "prefix"
    prefix_len: Optional[np.ndarray] = None   # int32 [S]

    @property
    def num_seqs(self) -> int:
        return len(self.cu_seqlens) - 1

    @property
    def num_clients(self) -> int:
        return len(self.client_seq_ptr) - 1

    @property
    def total_tokens(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def seqlens(self) -> np.ndarray:
        return np.diff(self.cu_seqlens).astype(np.int64)

    @property
    def max_seqlen(self) -> int:
        return int(self.seqlens.max()) if self.num_seqs else 0

    def client_rows(self, c: int) -> Tuple[int, int]:
        s0, s1 = int(self.client_seq_ptr[c]), int(self.client_seq_ptr[c + 1])
        return int(self.cu_seqlens[s0]), int(self.cu_seqlens[s1])

    def subset_clients(self, clients: Sequence[int]) -> Tuple["Batch", np.ndarray]:
        """Batch of only the given clients (in the given order) and the rows
        of the original packed buffer that feed it, in packed order."""
        lens: List[int] = []
        pre: List[int] = []
        csp = [0]
        rows: List[np.ndarray] = []
        for c in clients:
            s0, s1 = int(self.client_seq_ptr[c]), int(self.client_seq_ptr[c + 1])
            for s in range(s0, s1):
                a, b = int(self.cu_seqlens[s]), int(self.cu_seqlens[s + 1])
                lens.append(b - a)
                rows.append(np.arange(a, b))
                if self.prefix_len is not None:
                    pre.append(int(self.prefix_len[s]))
            csp.append(csp[-1] + (s1 - s0))
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        sub = Batch(cu, np.asarray(csp, np.int32), self.mask,
                    np.asarray(pre, np.int32) if self.prefix_len is not None else None)
        return sub, (np.concatenate(rows) if rows else np.zeros(0, np.int64))


def make_batch(num_clients: int, per_client: int, seqlen, mask: str = "causal",
               prefix_frac: float = 0.25, seed: int = 0) -> Batch:
    """Clients x sequences-per-client, lengths fixed (int) or uniform in
    [lo, hi] (tuple, inclusive, drawn client-major from stream 3).  For the
    prefix-LM mask the bidirectional prefix is floor(prefix_frac * L)."""
    n = num_clients * per_client
    if isinstance(seqlen, (tuple, list)):
        lo, hi = int(seqlen[0]), int(seqlen[1])
        lens = rng(seed, STREAM_LENS).integers(lo, hi + 1, size=n).astype(np.int64)
    else:
        lens = np.full(n, int(seqlen), np.int64)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    csp = (np.arange(num_clients + 1) * per_client).astype(np.int32)
    pre = None
    if mask == "prefix":
        pre = np.floor(lens * prefix_frac).astype(np.int32)
    elif mask != "causal":
        raise ValueError(f"unknown mask {mask!r}")
    return Batch(cu, csp, mask, pre)


# ----------------------------------------------------------------------------
# Parameters and activations
# ----------------------------------------------------------------------------

def param_shapes(shape: StackShape) -> Dict[str, Tuple[int, ...]]:
    """Out-features-major weights (y = x W^T + b).  Rows [0,H) of w_qkv are
    the query projection, [H,2H) the key, [2H,3H) the value; head h owns rows
    h*d .. h*d+d-1 inside each."""
    H, F = shape.hidden, shape.ffn_hidden
    return {"w_qkv": (3 * H, H), "b_qkv": (3 * H,), "w_o": (H, H), "b_o": (H,),
            "w_1": (F, H), "b_1": (F,), "w_2": (H, F), "b_2": (H,),
            "ln1_g": (H,), "ln1_b": (H,), "ln2_g": (H,), "ln2_b": (H,)}


def layer_params(shape: StackShape, layer: int, seed: int = 0, bf16: bool = True,
                 std: float = 0.02) -> Dict[str, np.ndarray]:
    """One layer's parameters as fp32 arrays (bf16-exact values when bf16).

    Linear weights and biases ~ N(0, std); LayerNorm gains 1 + N(0, std),
    shifts N(0, std)."""
    g = rng(seed, STREAM_PARAMS, layer)
    out: Dict[str, np.ndarray] = {}
    for name, shp in param_shapes(shape).items():
        a = g.standard_normal(size=shp, dtype=np.float32)
        a *= np.float32(std)
        if name in ("ln1_g", "ln2_g"):
            a += np.float32(1.0)
        out[name] = bf16_round(a) if bf16 else a
    return out


def device_layer_params(shape: StackShape, layer: int, seed: int = 0, bf16: bool = True, std: float = 0.02):
    """One layer's parameters drawn on the GPU (torch's seeded Philox
    generator, seed * 100003 + layer): the distributions of ``layer_params``
    (linear weights and biases N(0, std), LayerNorm gains 1 + N(0, std),
    shifts N(0, std)) in the same draw order, rounded to bf16 (nearest even)
    when bf16.  For full-size stacks, whose host draws would take minutes;
    returns a dict of cuda tensors (not the same values as ``layer_params``)."""
    import torch
    gen = torch.Generator(device="cuda").manual_seed(seed * 100003 + layer)
    out = {}
    for name, shp in param_shapes(shape).items():
        t = torch.randn(shp, generator=gen, device="cuda", dtype=torch.float32) * std
        if name in ("ln1_g", "ln2_g"):
            t += 1.0
        out[name] = t.to(torch.bfloat16) if bf16 else t
    return out


def prefix_params(shape: StackShape, layer: int, num_prefix: int, seed: int = 0, bf16: bool = True,
                  std: float = 1.0) -> Dict[str, np.ndarray]:
    """One layer's P-tuning v2 prefix: "prefix_k", "prefix_v" [num_prefix,
    hidden] ~ N(0, std) (an embedding table's default initialisation; keys
    of the frozen model have a comparable scale)."""
    g = rng(seed, STREAM_PREFIX, layer)
    out: Dict[str, np.ndarray] = {}
    for name in ("prefix_k", "prefix_v"):
        a = g.standard_normal(size=(num_prefix, shape.hidden), dtype=np.float32)
        if std != 1.0:
            a *= np.float32(std)
        out[name] = bf16_round(a) if bf16 else a
    return out


def _normal(seed: int, stream: int, n_rows: int, n_cols: int, std: float, bf16: bool) -> np.ndarray:
    a = rng(seed, stream).standard_normal(size=(n_rows, n_cols), dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return bf16_round(a) if bf16 else a


def activations(total_tokens: int, hidden: int, seed: int = 0, bf16: bool = True,
                std: float = 1.0) -> np.ndarray:
    """Packed smashed activations x [T, H] ~ N(0, std) (stream 1)."""
    return _normal(seed, STREAM_X, total_tokens, hidden, std, bf16)


def upstream_grad(total_tokens: int, hidden: int, seed: int = 0, bf16: bool = True,
                  std: float = 1.0) -> np.ndarray:
    """Upstream gradient dy [T, H] ~ N(0, std) (stream 2)."""
    return _normal(seed, STREAM_DY, total_tokens, hidden, std, bf16)


# ----------------------------------------------------------------------------
# Named workloads
# ----------------------------------------------------------------------------

CHATGLM6B = dict(hidden=4096, num_heads=32, ffn_hidden=16384, rotary_dim=64)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: StackShape
    num_clients: int
    per_client: int
    seqlen: object                 # int or (lo, hi)
    mask: str
    dtype: str                     # "f32" | "bf16"
    backward: bool
    recompute: bool
    dy_std: float
    description: str = ""
    num_prefix: int = 0            # P-tuning v2 prefix length (0: none)
    frozen: bool = False           # weights frozen: no weight gradients
    vocab: int = 0                 # > 0: the whole split model (client blocks, embedding, final linear + loss)

    def batch(self, seed: int = 0) -> Batch:
        return make_batch(self.num_clients, self.per_client, self.seqlen, self.mask, 0.25, seed)


WORKLOADS: Dict[str, Workload] = {
    "tiny_2blk_fp32": Workload(
        "tiny_2blk_fp32",
        StackShape(num_layers=2, hidden=256, num_heads=4, ffn_hidden=1024, rotary_dim=32),
        2, 2, 64, "causal", "f32", True, False, 1.0,
        "2 blocks, H 256, 4 heads x 64, FFN 1024, 2 clients x 2 x 64 tokens, causal, fp32"),
    "chatglm6b_1blk_fwd_4x4x512": Workload(
        "chatglm6b_1blk_fwd_4x4x512",
        StackShape(num_layers=1, **CHATGLM6B),
        4, 4, 512, "causal", "bf16", False, False, 1e-2,
        "1 ChatGLM-6B-shaped block, forward, 4 clients x 4 x 512 tokens, causal, bf16"),
    "chatglm6b_1blk_ragged_8x4": Workload(
        "chatglm6b_1blk_ragged_8x4",
        StackShape(num_layers=1, **CHATGLM6B),
        8, 4, (128, 1024), "causal", "bf16", True, False, 1e-2,
        "1 ChatGLM-6B-shaped block, fwd+bwd, 8 clients x 4 seqs, lengths U[128,1024], causal, bf16"),
    "chatglm6b_26blk_prefix_16x2x512": Workload(
        "chatglm6b_26blk_prefix_16x2x512",
        StackShape(num_layers=26, **CHATGLM6B),
        16, 2, 512, "prefix", "bf16", True, False, 1e-2,
        "26 ChatGLM-6B-shaped blocks, fwd+bwd, 16 clients x 2 x 512 tokens, prefix-LM (25%), bf16"),
    "chatglm6b_26blk_ragged_32x1_recompute": Workload(
        "chatglm6b_26blk_ragged_32x1_recompute",
        StackShape(num_layers=26, **CHATGLM6B),
        32, 1, (512, 2048), "causal", "bf16", True, True, 1e-2,
        "26 ChatGLM-6B-shaped blocks, fwd+bwd with per-block recompute, 32 clients x 1 seq, "
        "lengths U[512,2048], causal, bf16"),
    "chatglm6b_26blk_ptuning128_ragged_32x1_recompute": Workload(
        "chatglm6b_26blk_ptuning128_ragged_32x1_recompute",
        StackShape(num_layers=26, **CHATGLM6B),
        32, 1, (512, 2048), "causal", "bf16", True, True, 1e-2,
        "the 32 x 1 U[512,2048] batch under P-tuning v2: 128 prefix keys / values per block, weights frozen "
        "(input and prefix gradients only), per-block recompute, bf16",
        num_prefix=128, frozen=True),
    "chatglm6b_28blk_split_ptuning128_ragged_32x1_recompute": Workload(
        "chatglm6b_28blk_split_ptuning128_ragged_32x1_recompute",
        StackShape(num_layers=26, **CHATGLM6B),
        32, 1, (512, 2048), "causal", "bf16", True, True, 1e-2,
        "the whole split ChatGLM-6B-shaped model under P-tuning v2 on the 32 x 1 U[512,2048] batch: client "
        "embedding (130528 words) and block 0, 26 server blocks, client block 27, final linear layer and "
        "next-token cross-entropy, forward and backward; 128 prefix rows per block, weights frozen, recompute",
        num_prefix=128, frozen=True, vocab=130528),
    "chatglm6b_28blk_split_glm_ptuning128_prefix_32x1_recompute": Workload(
        "chatglm6b_28blk_split_glm_ptuning128_prefix_32x1_recompute",
        StackShape(num_layers=26, residual_alpha=math.sqrt(2 * 28), rotary_2d=True, **CHATGLM6B),
        32, 1, (512, 2048), "prefix", "bf16", True, True, 1e-2,
        "the whole split model with ChatGLM-6B's own blocks (alpha = sqrt(56) residual, GLM 2-D positions, final "
        "LayerNorm) on GLM blank-infilling batches (32 x 1 U[512,2048], the first 25 % of each sequence the "
        "bidirectional context), P-tuning v2 (128 prefix rows, weights frozen), recompute, bf16",
        num_prefix=128, frozen=True, vocab=130528),
}


def token_ids(batch: Batch, vocab: int, seed: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Synthetic client tokens for the whole split model: ids uniform over the
    vocabulary (stream 5), and next-token labels inside each sequence (the
    last token of a sequence has none: -100)."""
    ids = rng(seed, STREAM_TOKENS).integers(0, vocab, batch.total_tokens).astype(np.int32)
    labels = np.full(batch.total_tokens, -100, np.int32)
    for s in range(batch.num_seqs):
        r0, r1 = int(batch.cu_seqlens[s]), int(batch.cu_seqlens[s + 1])
        labels[r0:r1 - 1] = ids[r0 + 1:r1]
    return ids, labels
