"""The acceptance model of the draft-depth sweep (bench.py --workload ksweep):
depth d accepted with the paper's conditional rate a_d given depths < d.
Pinned against the tau values the paper prints in its decoding-efficiency
table (tests/golden/speculative_efficiency_table.json)."""
import json
import os

import pytest

import bench

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "speculative_efficiency_table.json")


def test_distribution_is_a_distribution():
    for mode, a in bench.PAPER_A_D.items():
        for K in range(4):
            p = bench.m_distribution(a, K)
            assert len(p) == K + 1
            assert all(x >= 0 for x in p)
            assert sum(p) == pytest.approx(1.0, abs=1e-12)


def test_rates_are_the_printed_ones():
    g = json.load(open(GOLDEN))
    assert tuple(g["conditional_acceptance"]["eager"]) == bench.PAPER_A_D["eager"]
    assert tuple(g["conditional_acceptance"]["graph"]) == bench.PAPER_A_D["hipgraph"]


@pytest.mark.parametrize("mode,key", [("eager", "eager"), ("hipgraph", "graph")])
def test_tau_reproduces_the_table(mode, key):
    g = json.load(open(GOLDEN))
    for row in g["rows"]:
        if row["mode"] != key or row["k"] == 0:
            continue
        p = bench.m_distribution(bench.PAPER_A_D[mode], row["k"])
        tau = sum((j + 1) * x for j, x in enumerate(p))
        assert tau == pytest.approx(row["tau"], abs=0.011)
