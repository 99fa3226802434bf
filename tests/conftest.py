import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")
INF = np.uint64(0xFFFFFFFFFFFFFFFF)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def parse_golden(path):
    """Parses tests/golden/window_examples.txt into a list of
    (name, size, cost, kind, [(S, expected (start, end, cost) or None)])."""
    kinds = {"F": 0, "E": 1, "P": 2}
    examples, cur, unit = [], None, 1

    def val(tok):
        return int(tok[:-1]) * unit if tok.endswith("u") else int(tok)

    with open(path) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "example":
                cur = {"name": tok[1], "size": [], "cost": [], "kind": [], "req": []}
                examples.append(cur)
                unit = 1
            elif tok[0] == "unit":
                unit = int(tok[1])
            elif tok[0] == "block":
                cur["kind"].append(kinds[tok[1]])
                cur["size"].append(val(tok[2]))
                cur["cost"].append(int(tok[3]))
            elif tok[0] == "S":
                assert tok[2] == "->"
                exp = None if tok[3] == "infeasible" else tuple(int(t) for t in tok[3:6])
                cur["req"].append((val(tok[1]), exp))
            else:
                raise ValueError(f"bad golden line: {raw!r}")
    return examples


@pytest.fixture(scope="session")
def golden_examples():
    return parse_golden(os.path.join(GOLDEN, "window_examples.txt"))


def parse_greedy_golden(path):
    """Parses tests/golden/greedy_examples.txt into a list of cases
    {"name", "pool": [(kind, bytes, id, cost)], "steps": [{"op", "expect",
    "after": [(kind, bytes, id)]}]}; sizes in the file are MiB."""
    kinds, mib = {"F": 0, "E": 1, "P": 2}, 1 << 20
    cases, cur, step = [], None, None
    with open(path) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "case":
                cur = {"name": tok[1], "pool": [], "steps": []}
                cases.append(cur)
            elif tok[0] == "pool":
                cur["pool"].append((kinds[tok[1]], int(tok[2]) * mib, int(tok[3]), int(tok[4])))
            elif tok[0] == "op":
                step = {"op": tok[1:]}
                cur["steps"].append(step)
            elif tok[0] == "expect":
                step["expect"] = tok[1:]
            elif tok[0] == "after":
                step["after"] = [(kinds[k], int(s) * mib, int(i)) for k, s, i in
                                 (p.split() for p in line[len("after"):].split("|"))]
    return cases


def parse_real_golden(path):
    """Parses tests/golden/real_examples.txt into a list of
    {"name", "blocks": [(kind, bytes, h)], "reqs": [(S, (start, end, hi, lo)
    or None)]}; h may be a decimal, a hex float or C/S (the binary64
    quotient)."""
    kinds, mib = {"F": 0, "E": 1, "P": 2}, 1 << 20

    def real(tok):
        if "/" in tok:
            c, s = tok.split("/")
            return int(c) / int(s)
        return float.fromhex(tok) if tok.startswith("0x") else float(tok)

    out, cur = [], None
    with open(path) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "example":
                cur = {"name": tok[1], "blocks": [], "reqs": []}
                out.append(cur)
            elif tok[0] == "block":
                cur["blocks"].append((kinds[tok[1]], int(tok[2]) * mib, real(tok[3])))
            elif tok[0] == "req":
                want = None if tok[3] == "infeasible" else tuple(int(x) for x in tok[3:7])
                cur["reqs"].append((int(tok[1]) * mib, want))
    return out
