"""The README's usage example runs as written (GPU)."""

import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.gpu
def test_readme_example_runs():
    import torch
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```python\n(.*?)```", text, re.S)
    assert len(blocks) == 1
    ns = {}
    exec(compile(blocks[0], "README.md", "exec"), ns)
    y, dx, grads = ns["y"], ns["dx"], ns["grads"]
    assert bool(torch.isfinite(y.float()).all()) and bool(torch.isfinite(dx.float()).all())
    assert all(bool(torch.isfinite(g).all()) for lg in grads for g in lg.values())
    assert float(grads[0]["w_qkv"].abs().sum()) > 0.0
