"""Runs the HIP server stack through the C ABI on host arrays and returns
host results; used by the stack-level GPU tests, the smoke check and the
benchmark's parity sampling."""

from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np
import torch

import synth
from paper_2406_14898_amd import BatchDesc, ServerStack
from tests.gpu_helpers import dev, host


class GpuStack:
    def __init__(self, shape: synth.StackShape, layers: List[Dict[str, np.ndarray]], dt: str, num_prefix: int = 0):
        """num_prefix > 0: the layer dicts also carry "prefix_k" / "prefix_v"
        [num_prefix, hidden] (P-tuning v2)."""
        self.shape, self.dt = shape, dt
        self.ss = ServerStack(shape.num_layers, shape.hidden, shape.num_heads, shape.ffn_hidden, shape.rotary_dim,
                              dt, shape.rope_base, shape.ln_eps, num_prefix, shape.residual_alpha, shape.rotary_2d)
        cache = {}  # layers given as the same dict share one device copy
        self.params = []
        for lp in layers:
            if id(lp) not in cache:  # host arrays are uploaded; device tensors used as they are
                cache[id(lp)] = {k: v if isinstance(v, torch.Tensor) else dev(v, dt) for k, v in lp.items()}
            self.params.append(cache[id(lp)])

    def zero_grads(self, frozen: bool = False):
        """fp32 accumulators; frozen: only the prefix ones (weights frozen)."""
        return [{k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in p.items()
                 if not frozen or k.startswith("prefix_")} for p in self.params]

    def run(self, batch: synth.Batch, x: np.ndarray, dy: Optional[np.ndarray], recompute: bool = False,
            grads=None, frozen: bool = False):
        bd = BatchDesc.from_batch(batch)
        saved, ws = self.ss.buffers(bd, recompute, with_saved=dy is not None)
        tx = dev(x, self.dt)
        ty = torch.empty_like(tx)
        self.ss.forward(bd, self.params, tx, ty, saved, ws, recompute)
        out = {"y": ty}
        if dy is not None:
            tdy = dev(dy, self.dt)
            tdx = torch.empty_like(tx)
            g = grads if grads is not None else self.zero_grads(frozen)
            self.ss.backward(bd, self.params, g, tx, saved, tdy, tdx, ws, recompute)
            out["dx"] = tdx
            out["grads"] = g
        torch.cuda.synchronize()
        return out

    @staticmethod
    def to_host(out):
        h = {"y": host(out["y"])}
        if "dx" in out:
            h["dx"] = host(out["dx"])
            h["grads"] = [{k: host(v) for k, v in g.items()} for g in out["grads"]]
        return h

    def close(self):
        self.ss.close()
