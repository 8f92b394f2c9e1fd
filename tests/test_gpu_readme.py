"""The usage example of README.md runs as written: its python block is executed
on the GPU, and its streams end where the example leaves them."""
import os
import re

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_readme_example_runs():
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```python\n(.*?)```", text, flags=re.S)
    assert len(blocks) == 1
    env = {}
    exec(compile(blocks[0], "README.md", "exec"), env)
    import torch
    assert env["ring"].seq_len.cpu().tolist() == [6 * 4680]
    assert env["dec"].seq_len.cpu().tolist() == [4] * 32
    assert bool(torch.isfinite(env["out"].float()).all())
    assert bool(torch.isfinite(env["o"].float()).all())
