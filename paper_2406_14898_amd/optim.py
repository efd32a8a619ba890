"""Flat parameter arenas for the server update (device memory via torch; the
arithmetic is the library's fl_adam_step / fl_average_replicas).

An arena holds a set of named tensors back to back in one fp32 master
buffer, with fp32 gradient and Adam moment buffers of the same layout and,
optionally, a bf16 compute copy.  The per-tensor views are what the stack
reads (the bf16 views, or the fp32 masters for the fp32 stack) and
accumulates into (the gradient views), so one launch updates every tensor.
"""

from __future__ import annotations

from typing import Dict, Iterable, List, Optional, Sequence, Tuple

from . import flglm as F

_ALIGN = 8  # elements: every view starts 16-byte aligned in fp32 and bf16


class ParamArena:
    def __init__(self, shapes: Iterable[Tuple[str, Tuple[int, ...]]], bf16_copy: bool, device="cuda"):
        import torch
        self.names: List[str] = []
        self.offsets: Dict[str, Tuple[int, Tuple[int, ...]]] = {}
        n = 0
        for name, shape in shapes:
            size = 1
            for s in shape:
                size *= int(s)
            self.names.append(name)
            self.offsets[name] = (n, tuple(shape))
            n += (size + _ALIGN - 1) // _ALIGN * _ALIGN
        self.n = n
        z = dict(dtype=torch.float32, device=device)
        self.master = torch.zeros(max(n, _ALIGN), **z)
        self.grad = torch.zeros(max(n, _ALIGN), **z)
        self.exp_avg = torch.zeros(max(n, _ALIGN), **z)
        self.exp_avg_sq = torch.zeros(max(n, _ALIGN), **z)
        self.compute = torch.zeros(max(n, _ALIGN), dtype=torch.bfloat16, device=device) if bf16_copy else None
        self.step_count = 0

    def _view(self, buf, name):
        off, shape = self.offsets[name]
        size = 1
        for s in shape:
            size *= s
        return buf[off:off + size].view(shape)

    def master_views(self) -> Dict[str, "object"]:
        return {k: self._view(self.master, k) for k in self.names}

    def grad_views(self) -> Dict[str, "object"]:
        return {k: self._view(self.grad, k) for k in self.names}

    def compute_views(self) -> Dict[str, "object"]:
        """The tensors the stack reads: the bf16 copy, else the fp32 masters."""
        buf = self.compute if self.compute is not None else self.master
        return {k: self._view(buf, k) for k in self.names}

    def load(self, values: Dict[str, "object"]) -> None:
        """Sets the masters (and the bf16 copy, rounded) from tensors."""
        for k, v in values.items():
            self._view(self.master, k).copy_(v)
        self.refresh_compute()

    def refresh_compute(self) -> None:
        """bf16 copy := the masters rounded to nearest even (after the
        masters were written directly through master_views())."""
        if self.compute is not None:
            self.compute.copy_(self.master)

    def adam_step(self, lr: float = 2e-2, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                  zero_grad: bool = True, stream=None) -> None:
        """One Adam step over every tensor of the arena (time step advances)."""
        self.step_count += 1
        F.fl_adam_step(self.master, self.grad, self.exp_avg, self.exp_avg_sq, self.compute, self.n, self.step_count,
                       lr, beta1, beta2, eps, zero_grad, stream)


def average(arenas: Sequence[ParamArena], stream=None) -> None:
    """Server-hierarchical aggregation: every arena's masters (and bf16
    copies) become the elementwise mean over the arenas."""
    n = arenas[0].n
    if any(a.n != n for a in arenas):
        raise ValueError("arenas differ in layout")
    c16: Optional[list] = [a.compute for a in arenas] if arenas[0].compute is not None else None
    F.fl_average_replicas([a.master for a in arenas], c16, n, stream)
