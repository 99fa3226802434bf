"""The Python example in README.md runs as printed and gives the results
its comment states (which the oracle confirms)."""
import ast
import os
import re

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_readme_example():
    text = open(os.path.join(ROOT, "README.md")).read()
    code = re.search(r"```python\n(.*?)```", text, flags=re.S).group(1)
    ns = {}
    exec(compile(code, "README.md", "exec"), ns)
    torch.cuda.synchronize()
    got = ns["out"].cpu().numpy()
    stated = re.search(r"snapshot-local: (\[\[.*\]\])", code).group(1)
    assert got.tolist() == ast.literal_eval(stated)
    u64 = lambda t: t.cpu().numpy().view(np.uint64)
    want = oracle.window_search(u64(ns["size"]), u64(ns["cost"]), ns["kind"].cpu().numpy(),
                                u64(ns["seg_offsets"]), u64(ns["req_sizes"]),
                                u64(ns["req_offsets"]))
    assert np.array_equal(got.view(np.uint64), want)
