"""Helpers shared by the GPU parity tests: device upload of bf16-exact host
arrays, downloads, and the relative L2 error."""

from __future__ import annotations

import numpy as np
import torch

import synth
from paper_2406_14898_amd import flglm as F

DTYPES = {"bf16": (F.FL_BF16, torch.bfloat16), "f32": (F.FL_F32, torch.float32)}
TOL = {"bf16": 2e-2, "f32": 1e-4}


def dev(a: np.ndarray, dt: str) -> torch.Tensor:
    """Host fp32 array (bf16-exact when dt == 'bf16') -> device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dt == "bf16":
        # values are already bf16-representable; the cast is exact
        t = t.to(torch.bfloat16)
    return t.cuda()


def dev_i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rnd(shape, seed, std=1.0, dt="bf16"):
    a = np.random.default_rng(seed).standard_normal(shape).astype(np.float32) * np.float32(std)
    return synth.bf16_round(a) if dt == "bf16" else a


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def sync():
    torch.cuda.synchronize()
