"""Convenience wrapper over the C ABI: owns a stack handle and allocates the
saved-activation and workspace buffers with torch (device memory only)."""

from __future__ import annotations

from typing import Dict, Sequence

from . import flglm as F


class ServerStack:
    """FL-GLM server stack (blocks 1..N-2 of the split model) on one GPU."""

    def __init__(self, num_layers: int, hidden: int, num_heads: int, ffn_hidden: int, rotary_dim: int,
                 dtype: str = "bf16", rope_base: float = 10000.0, ln_eps: float = 1e-5, num_prefix: int = 0,
                 residual_alpha: float = 0.0, rotary_2d: bool = False):
        """num_prefix > 0: P-tuning v2 prefix of that many key / value rows per
        block (params then carry "prefix_k" / "prefix_v" [num_prefix, hidden]).
        residual_alpha > 0 / rotary_2d: ChatGLM-6B's own block (alpha-scaled
        residual on the normalised input, GLM 2-D positions)."""
        self.dtype = F.FL_BF16 if dtype == "bf16" else F.FL_F32
        self.num_layers = num_layers
        self.hidden = hidden
        self.num_prefix = num_prefix
        self.handle = F.fl_stack_create(F.stack_desc(num_layers, hidden, num_heads, ffn_hidden, rotary_dim,
                                                     self.dtype, rope_base, ln_eps, num_prefix, residual_alpha,
                                                     rotary_2d))

    def close(self) -> None:
        if self.handle:
            F.fl_stack_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass

    def buffers(self, batch: F.BatchDesc, recompute: bool, device="cuda", with_saved: bool = True):
        """(saved, workspace) as uint8 torch tensors of the sizes the library asks for."""
        import torch
        ws_n = F.fl_stack_workspace_bytes(self.handle, batch, recompute)
        ws = torch.empty(max(ws_n, 1), dtype=torch.uint8, device=device)
        saved = None
        if with_saved:
            sv_n = F.fl_stack_saved_bytes(self.handle, batch, recompute)
            saved = torch.empty(max(sv_n, 256), dtype=torch.uint8, device=device)
        return saved, ws

    def forward(self, batch: F.BatchDesc, params: Sequence[Dict], x, y, saved, workspace, recompute: bool = False,
                stream=None) -> None:
        layers = [F.layer_params(p) for p in params]
        F.fl_server_stack_forward(self.handle, batch, layers, x, y, saved, recompute, workspace,
                                  workspace.numel(), stream)

    def backward(self, batch: F.BatchDesc, params: Sequence[Dict], grads: Sequence[Dict], x, saved, dy, dx,
                 workspace, recompute: bool = False, stream=None) -> None:
        layers = [F.layer_params(p) for p in params]
        gl = [F.layer_grads(g) for g in grads]
        F.fl_server_stack_backward(self.handle, batch, layers, gl, x, saved, dy, dx, recompute, workspace,
                                   workspace.numel(), stream)
