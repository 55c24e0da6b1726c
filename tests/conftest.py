import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")


def read_golden(name):
    """Lines of a golden fixture with comments and blanks removed."""
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                out.append(line.split())
    return out


@pytest.fixture(scope="session")
def fig1():
    """The Fig. 1 layout and hand-derived token cases."""
    import numpy as np
    kv = {}
    ranks = {}
    for f in read_golden("fig1_layout.txt"):
        if f[0] == "rank":
            ranks[int(f[1])] = [int(v) for v in f[2:]]
        else:
            kv[f[0]] = [int(v) for v in f[1:]]
    N, g, E, S = kv["N"][0], kv["g"][0], kv["E"][0], kv["S"][0]
    table = np.full((N * g, S), -1, np.int32)
    for r, es in ranks.items():
        table[r, : len(es)] = es
    toks = {"tokens": [], "coact": [], "pos": None}
    for f in read_golden("fig1_tokens.txt"):
        if f[0] == "token":
            toks["tokens"].append([int(v) for v in f[1:]])
        elif f[0] == "coact":
            toks["coact"].append([int(v) for v in f[1:]])
        else:
            toks[f[0]] = [int(v) for v in f[1:]]
    return dict(N=N, g=g, E=E, S=S, table=table, owner=np.array(kv["owner"], np.int32),
                replicas=kv["replicas"], **toks)
