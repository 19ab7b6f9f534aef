"""The README's Python usage example runs as written on the GPU (MI355X only)."""
import os
import re

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_readme_python_example_runs():
    src = open(os.path.join(ROOT, "README.md"), encoding="utf-8").read()
    blocks = re.findall(r"```python\n(.*?)```", src, re.S)
    assert blocks, "no Python example in the README"
    scope = {}
    exec(compile(blocks[0], "README.md", "exec"), scope)
    out, lens = scope["out"], scope["lens"]
    assert bool(out.isfinite().all())
    assert int(lens.min()) == 1 and int(lens.max()) == 1  # one appended row per sample
