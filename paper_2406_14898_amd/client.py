"""The client side of the split model (Section 3.1) and one whole split
training step on one GPU, over the C ABI.  torch provides device memory
and the stream only; every step runs in the library's kernels."""

from __future__ import annotations

from typing import Dict, List, Optional

from . import flglm as F
from .stack import ServerStack


class ClientHead:
    """Embedding layer and final linear layer + cross-entropy of the client."""

    def __init__(self, vocab: int, hidden: int, dtype: str = "bf16", ln_eps: float = 1e-5):
        self.vocab, self.hidden = vocab, hidden
        self.dtype = F.FL_BF16 if dtype == "bf16" else F.FL_F32
        self.handle = F.fl_client_create(vocab, hidden, self.dtype, ln_eps)

    def close(self) -> None:
        if self.handle:
            F.fl_client_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass

    def workspace(self, T: int, device="cuda"):
        import torch
        return torch.empty(F.fl_client_workspace_bytes(self.handle, T), dtype=torch.uint8, device=device)

    def embed(self, table, ids, out, ws, stream=None) -> None:
        F.fl_embedding_forward(self.handle, table, ids, out, ws, stream)

    def embed_backward(self, ids, dout, dtable, ws, stream=None) -> None:
        F.fl_embedding_backward(self.handle, ids, dout, dtable, ws, stream)

    def head_forward(self, h, w, labels, loss_tok, loss_sum, ws, stream=None, ln_g=None, ln_b=None) -> None:
        """ln_g / ln_b: the optional final LayerNorm (ChatGLM-6B)."""
        F.fl_lm_head_forward(self.handle, h, w, labels, loss_tok, loss_sum, ws, stream, ln_g, ln_b)

    def head_backward(self, h, w, T: int, grad_scale: float, dh, dw, ws, stream=None, ln_g=None, dln_g=None,
                      dln_b=None) -> None:
        F.fl_lm_head_backward(self.handle, h, w, T, grad_scale, dh, dw, ws, stream, ln_g, dln_g, dln_b)


class SplitModel:
    """The whole split model on one GPU: the client's embedding, block 0,
    block N-1 and final linear layer around the server's block stack, with a
    training step that runs forward, loss and backward through all of them
    (the server's part is what the server runs; the rest is what every
    client runs on its own share of the batch)."""

    def __init__(self, hidden: int, num_heads: int, ffn_hidden: int, rotary_dim: int, num_server: int, vocab: int,
                 dtype: str = "bf16", rope_base: float = 10000.0, ln_eps: float = 1e-5, num_prefix: int = 0,
                 residual_alpha: float = 0.0, rotary_2d: bool = False):
        """residual_alpha / rotary_2d: ChatGLM-6B's own blocks; with them a
        step also takes the final LayerNorm ("final_ln_g" / "final_ln_b" in
        params) when given."""
        args = (hidden, num_heads, ffn_hidden, rotary_dim, dtype, rope_base, ln_eps, num_prefix, residual_alpha,
                rotary_2d)
        self.block0 = ServerStack(1, *args)
        self.server = ServerStack(num_server, *args)
        self.block_last = ServerStack(1, *args)
        self.head = ClientHead(vocab, hidden, dtype, ln_eps)
        self.hidden = hidden

    def close(self) -> None:
        for s in (self.block0, self.server, self.block_last, self.head):
            s.close()

    def buffers(self, batch: F.BatchDesc, recompute: bool, device="cuda") -> Dict:
        """Device buffers for one batch: each stack's saved activations and
        workspace, the client workspace, the activations at every boundary
        and their gradients, the loss outputs."""
        import torch
        T = batch.desc.total_tokens
        dt = torch.bfloat16 if self.head.dtype == F.FL_BF16 else torch.float32
        b = {"T": T}
        for name, st in (("b0", self.block0), ("srv", self.server), ("bl", self.block_last)):
            b[name + "_saved"], b[name + "_ws"] = st.buffers(batch, recompute, device)
        b["client_ws"] = self.head.workspace(T, device)
        for name in ("e", "h0", "hs", "hl", "d_hl", "d_hs", "d_h0", "d_e"):
            b[name] = torch.empty((T, self.hidden), dtype=dt, device=device)
        b["loss_tok"] = torch.empty(T, dtype=torch.float32, device=device)
        b["loss_sum"] = torch.empty(1, dtype=torch.float32, device=device)
        return b

    def step(self, batch: F.BatchDesc, ids, labels, params: Dict, grads: Dict, grad_scale: float, buf: Dict,
             recompute: bool = False, stream=None, marks: Optional[List] = None) -> None:
        """One training step.  params: "embedding" [V, H], "lm_head" [V, H],
        "block0" / "block_last" (one layer's dict), "server" (list of layer
        dicts), optionally "final_ln_g" / "final_ln_b" [H] (ChatGLM-6B's final
        LayerNorm; their gradients in grads, None when frozen).  grads: the same keys with fp32 accumulators (+=); a missing
        or None "embedding" / "lm_head" entry, and block dicts without weight
        keys, mean frozen (P-tuning v2).  marks: when a list, each client-side
        call is bracketed by two timing events on the stream and appended as
        (name, start, end)."""
        T = buf["T"]
        h = self.head

        def timed(name, fn, *a):
            if marks is None:
                return fn(*a)
            import torch
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn(*a)
            e1.record(stream)
            marks.append((name, e0, e1))

        timed("embedding_fwd", h.embed, params["embedding"], ids, buf["e"], buf["client_ws"], stream)
        self.block0.forward(batch, [params["block0"]], buf["e"], buf["h0"], buf["b0_saved"], buf["b0_ws"],
                            recompute, stream)
        self.server.forward(batch, params["server"], buf["h0"], buf["hs"], buf["srv_saved"], buf["srv_ws"],
                            recompute, stream)
        self.block_last.forward(batch, [params["block_last"]], buf["hs"], buf["hl"], buf["bl_saved"], buf["bl_ws"],
                                recompute, stream)
        lg, lb = params.get("final_ln_g"), params.get("final_ln_b")
        timed("lm_head_fwd", h.head_forward, buf["hl"], params["lm_head"], labels, buf["loss_tok"], buf["loss_sum"],
              buf["client_ws"], stream, lg, lb)
        timed("lm_head_bwd", h.head_backward, buf["hl"], params["lm_head"], T, grad_scale, buf["d_hl"],
              grads.get("lm_head"), buf["client_ws"], stream, lg, grads.get("final_ln_g"), grads.get("final_ln_b"))
        self.block_last.backward(batch, [params["block_last"]], [grads["block_last"]], buf["hs"], buf["bl_saved"],
                                 buf["d_hl"], buf["d_hs"], buf["bl_ws"], recompute, stream)
        self.server.backward(batch, params["server"], grads["server"], buf["h0"], buf["srv_saved"], buf["d_hs"],
                             buf["d_h0"], buf["srv_ws"], recompute, stream)
        self.block0.backward(batch, [params["block0"]], [grads["block0"]], buf["e"], buf["b0_saved"], buf["d_h0"],
                             buf["d_e"], buf["b0_ws"], recompute, stream)
        if grads.get("embedding") is not None:
            timed("embedding_bwd", h.embed_backward, ids, buf["d_e"], grads["embedding"], buf["client_ws"], stream)
