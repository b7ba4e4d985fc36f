"""The Python example of README.md runs as written and its results agree with
the library's own stage entry points."""

import os
import re

import pytest
import torch

pytestmark = pytest.mark.gpu

README = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "README.md")


def test_readme_python_example_runs(gpu_lib):
    block = re.search(r"```python\n(.*?)```", open(README).read(), re.S).group(1)
    env = {}
    exec(compile(block, "README.md", "exec"), env)
    torch.cuda.synchronize()
    grads, offsets, out, W, G = env["grads"], env["offsets"], env["out"], env["W"], env["G"]
    assert out.shape == (grads.shape[1],) and out.dtype == torch.bfloat16
    assert torch.isfinite(G).all() and torch.isfinite(W).all()
    # the resolve's weights are those of the stand-alone solve on its Gram
    w_mgda, _ = gpu_lib.solve(G, "mgda", max_iter=20)
    assert torch.allclose(W, w_mgda, rtol=0, atol=1e-6)
    # and its update is the stand-alone combine with those weights
    assert torch.equal(gpu_lib.combine(grads, offsets, W).view(torch.int16), out.view(torch.int16))
