"""The usage example in README.md runs as written on the GPU (its comments'
values hold: the prefix match lengths, finite outputs of the stated shapes)."""
import os
import re

import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_readme_usage_example_runs():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with open(os.path.join(ROOT, "README.md")) as f:
        code = re.search(r"## Usage\s+```python\n(.*?)```", f.read(), re.S).group(1)
    ns = {}
    exec(compile(code, "README.md", "exec"), ns)
    torch.cuda.synchronize()
    assert ns["matched"] == 1024
    assert tuple(ns["o"].shape) == (4, 32, 128) and torch.isfinite(ns["o"]).all()
    assert tuple(ns["o_new"].shape) == (100, 32, 128) and torch.isfinite(ns["o_new"]).all()
