"""The Python example of README.md runs as written on the GPU, and its results agree with the oracle."""
import os
import re

import numpy as np
import pytest
import torch

import oracle
from parity import bits

pytestmark = pytest.mark.gpu

README = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "README.md")


def test_readme_example():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    blocks = re.findall(r"```python\n(.*?)```", open(README).read(), re.S)
    assert blocks, "README has no python example"
    env = {}
    torch.manual_seed(0)
    code = blocks[0]
    # keep a copy of the inputs of the first compress call to check it against the oracle
    code = code.replace("residual = torch.zeros_like(grad)\n",
                        "residual = torch.zeros_like(grad)\n_g0, _r0 = grad.cpu().numpy().copy(), residual.cpu().numpy().copy()\n", 1)
    code = code.replace("idx, val = out.idx[:out.k], out.val[:out.k]",
                        "idx, val = out.idx[:out.k], out.val[:out.k]\n_res1 = residual.cpu().numpy().copy()", 1)
    exec(compile(code, "README.md", "exec"), env)
    torch.cuda.synchronize()
    o = oracle.compress(env["_g0"], env["_r0"], env["offsets"], 0.99, per_tensor=True)
    assert np.array_equal(env["idx"].cpu().numpy().view(np.uint32), o.idx)
    assert np.array_equal(bits(env["val"].cpu().numpy()), bits(o.val))
    assert np.array_equal(bits(env["_res1"]), bits(o.residual))
