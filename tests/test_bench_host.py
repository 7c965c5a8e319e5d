"""Host-side rules of the benchmark (no GPU): how many decode steps one HIP
graph holds."""
import importlib.util
import math
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_module", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("periods", [(6, 8), (2, 8), (15, 8), (10, 8), (40, 8), (18, 8), (1, 1), (64,), (33,)])
def test_graph_steps_whole_rotations_of_at_least_32(bench, periods):
    lcm = 1
    for p in periods:
        lcm = lcm * p // math.gcd(lcm, p)
    k = bench.graph_steps(*periods)
    assert k <= 64
    if lcm <= 64:
        # a whole number of rotations, the smallest one of at least 32 steps
        assert k % lcm == 0 and k >= min(bench.GRAPH_MIN_STEPS, 64)
        assert k - lcm < bench.GRAPH_MIN_STEPS
    else:
        assert k == 64


def test_graph_steps_of_the_128k_rotation(bench):
    # 6 layer copies and 8 query sets: two rotations of 24
    assert bench.graph_steps(6, 8) == 48
