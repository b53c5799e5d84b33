"""The README's Python example runs as written (on the GPU) and its outputs have the documented
shapes and types."""
import os
import re

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_readme_python_example():
    import torch
    text = open(os.path.join(ROOT, "README.md")).read()
    block = re.search(r"```python\n(.*?)```", text, re.S).group(1)
    env = {}
    exec(compile(block, "README.md", "exec"), env)  # noqa: S102 - the repository's own README
    torch.cuda.synchronize()
    assert env["y"].shape == (256, 2560) and env["y"].dtype == torch.float32
    assert bool(torch.isfinite(env["y"]).all())
    assert env["yb"].shape == (256, 2560) and env["yb"].dtype == torch.int16
    assert env["dx"].shape == (256, 2048) and env["dw"].shape == (2560, 2048)
    assert env["stats"].shape == (9,) and float(env["stats"][0]) == 256 * 2048
