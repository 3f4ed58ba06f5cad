"""The README's usage example runs as written."""

from __future__ import annotations

import os
import re

import pytest
import torch

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_readme_example_runs():
    text = open(os.path.join(ROOT, "README.md")).read()
    code = re.search(r"```python\n(.*?)```", text, re.S).group(1)
    print("README example", flush=True)
    scope = {}
    exec(compile(code, "README.md", "exec"), scope)
    torch.cuda.synchronize()
    assert all(bool(g.isfinite().all()) for g in scope["grad_shards"])
    assert all(bool(p.float().isfinite().all()) for p in scope["params"])
