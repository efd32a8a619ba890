"""CPU oracle for the FL-GLM server stack (test infrastructure only).

This package is the plain, slow, obviously correct definition of what the
server computes.  Only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark may import it; the product path (the HIP library and its
Python binding) never does, and this package imports nothing from it.

What it follows:
  * Section 3.1 (Model Split): the server holds blocks 1..N-2 and computes
    h_{N-2} = Block_(1,N-2)(h_0), i.e. the composition of identical
    transformer blocks applied to the smashed data.  Split learning returns
    the gradient of the loss with respect to h_0 to the client.
  * Section 3.1 (last paragraph) and Appendix A (P-tuning v2): each block is
    multi-head self-attention followed by a feed-forward network; attention
    scores are softmax(Q K^T / sqrt(d_h)).
  * Section 3.3 (Parallel Acceleration): client-batch training stacks the
    smashed data of M clients into one batch; nothing mixes across clients.
  * Section 4.1.4 (Parameter Settings) and Section 3.3: the server update
    after the backward (Adam) and the server-hierarchical replica averaging
    (``oracle.optim``).
  * Section 3.1 (Model Split), client side: embedding, block 0, block N-1,
    the final linear layer and the cross-entropy loss (``oracle.client``).
  * Block internals the paper does not give (pre-LN with residual, rotary on
    the first half of each head, tanh GeLU, FFN width, biases, LayerNorm eps)
    follow the readings listed in the design notes (pre-LN residual form,
    rotate-half pairing, base 10000, eps 1e-5, scale 1/sqrt(d), no dropout).

Arithmetic is numpy in the dtype the caller selects (float64 by default;
float32 for the fp32 mode).  Linear layers use numpy matmul; attention builds
the full L x L score matrix of each (sequence, head) with no blocking or
online softmax (``attention_query_rows`` builds the rows of a few queries
of one sequence, for sequences too long for the full matrix).
"""

from .block import (  # noqa: F401
    layer_norm, layer_norm_backward, gelu, gelu_grad, positions, rope_tables,
    rope, glm_positions, allowed_mask, attention_forward, attention_backward, attention_query_rows,
    block_forward,
    block_backward, stack_forward, stack_backward, zero_grads, zero_prefix_grads, client_token_ranges,
    pack_clients, unpack_clients,
)
from .optim import (  # noqa: F401
    ADAM_LR, ADAM_BETA1, ADAM_BETA2, ADAM_EPS, adam_step, average_replicas,
)
from . import client  # noqa: F401,E402
