"""The usage example in README.md runs as written and its result is the
approximate sum it claims to be."""

import os
import re

import numpy as np
import pytest

from conftest import ROOT

pytestmark = pytest.mark.gpu


def test_readme_example_runs():
    import torch
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```python\n(.*?)```", text, re.S)
    assert len(blocks) == 1
    scope = {}
    exec(compile(blocks[0], "README.md", "exec"), scope)
    torch.cuda.synchronize()
    grads, out, d = scope["grads"], scope["out"], scope["d"]
    S = grads.double().sum(0).cpu().numpy()
    for i in range(grads.shape[0]):
        e = np.linalg.norm(out[i, :d].double().cpu().numpy() - S) / np.linalg.norm(S)
        assert np.isfinite(e) and e < 1.0, (i, e)
