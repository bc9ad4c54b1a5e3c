"""Values the paper prints for worked examples (fixtures in tests/golden/,
each citing its passage), checked against the host-side planning code.  No
GPU: host-only contexts plan without device memory.

* Eq. 1's example: sharing 1 GB among models that need 1.5 GB gives each
  model 66.7% of its demand when the memory term alone decides, i.e. when
  the performance scores are proportional to the demands.
* The block count n = ceil(m s / b): a 170 MB model under a 136 MB budget
  runs as three blocks.  The planner accepts three equal blocks at that
  budget without splitting them (Eq. 3's pair constraint holds), needs
  more slabs once the pair constraint fails, and its balanced re-cut uses
  the printed n rounded up to an even count (consecutive slabs alternate
  between the two ends of the arena).
"""
import math
import os

import numpy as np
import pytest

from paper_2401_16757_amd import swapnet as S
from paper_2401_16757_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_fixture(name):
    vals = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].strip()
        if line:
            k, v = (t.strip() for t in line.split("=", 1))
            vals[k] = float(v)
    return vals


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(S.LIB_PATH):
        from paper_2401_16757_amd import build
        build.build()
    S.load_library()


def test_eq1_worked_example():
    g = read_fixture("eq1_budget_split.txt")
    unit = 1 << 30
    total = int(g["total_demand"] * unit)
    # three models sharing the printed total demand; scores PS = latency /
    # memory made proportional to demand (latency ~ demand^2), so both terms
    # of Eq. 1 split in proportion to demand
    need = [total // 5, total // 3, total - total // 5 - total // 3]
    lat = [(n / unit) ** 2 for n in need]
    out = S.split_budget(need, lat, [1.0, 1.0, 1.0], int(g["available"] * unit))
    for o, n in zip(out, need):
        assert round(100.0 * o / n, 1) == g["share_of_demand_percent"], (o, n)


def uniform_net(n_layers, width=256):
    """n_layers linear layers of identical size (weights + bias)."""
    layers = [W.LayerSpec(name="fc%d" % i, op="linear", src=i, dst=i + 1, c_in=width, c_out=width)
              for i in range(n_layers)]
    return W.Network("uniform", 77, layers, [[0, n_layers]], (width, 1, 1), n_layers)


def test_block_count_worked_example():
    g = read_fixture("block_count.txt")
    s_units, b_units, m = int(g["model_bytes"]), int(g["budget"]), int(g["parallel_blocks"])
    # the printed count follows from the rule
    assert math.ceil(m * s_units / b_units) == g["blocks"]
    # one layer per MB of the model: the size ratio s / b is kept exactly
    net = uniform_net(s_units)
    wts = W.make_weights(net)
    with S.build_engine(net, wts, budget=1 << 30, host_only=True) as eng:
        image = eng.stats()["image_bytes"]
    assert image % s_units == 0
    per_layer = image // s_units   # one layer's tensors in the image, aligned
    budget = b_units * per_layer
    n = int(g["blocks"])
    cuts = [round(i * s_units / n) for i in range(n + 1)]
    blocks = [[cuts[i], cuts[i + 1]] for i in range(n)]
    with S.build_engine(net, wts, budget=budget, blocks=blocks, host_only=True) as eng:
        st = eng.stats()
        assert st["n_slabs"] == n and not st["resident"], st
        sl = eng.slabs()
        assert all(a["bytes"] + b["bytes"] <= budget for a, b in zip(sl, sl[1:]))
    # below the pair constraint of three equal blocks the planner must split
    tight = int(0.9 * (2 * s_units / n) * per_layer)
    with S.build_engine(net, wts, budget=tight, blocks=blocks, host_only=True) as eng:
        assert eng.stats()["n_slabs"] > n
    # balanced re-cut: ceil(2 s / b) slabs, rounded up to an even count
    with S.build_engine(net, wts, budget=budget, host_only=True, partition=1) as eng:
        want = math.ceil(m * s_units / b_units)
        assert eng.stats()["n_slabs"] == want + (want & 1)
