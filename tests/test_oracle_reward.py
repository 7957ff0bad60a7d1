"""Pins of the oracle's performance (Eq. 3) and reward (Eq. 4) against what
Sec. 4.2.2, Sec. 4.3 and Sec. 5 state about them."""
import math

import numpy as np


def test_performance_is_the_reciprocal_latency(oracle):
    # Eq. (3) and the RScore of Sec. 5: a 2 ms kernel scores 0.5, a 0.25 ms kernel 4
    assert oracle.performance(2.0) == 0.5
    assert oracle.performance(0.25) == 4.0
    lat = np.random.default_rng(3).uniform(1e-3, 1e3, 1000)
    for t in lat:
        assert oracle.performance(float(t)) == 1.0 / float(t)


def test_failing_compilation_is_penalised(oracle):
    # Sec. 4.3: a kernel that does not compile receives a penalty, whatever else is known about it
    for v in (0, 1):
        for p in (0.0, 1.0, 123.0, math.inf, math.nan):
            assert oracle.reward(0, v, p) == -1.0


def test_compiled_but_wrong_gets_nothing_from_performance(oracle):
    # fail-fast (Sec. 4.2.2): a kernel failing the functional check is not profiled, so speed cannot help it
    for p in (0.0, 1.0, 1e9, math.inf, math.nan):
        assert oracle.reward(1, 0, p) == 0.0
    assert oracle.reward(1, 0, 0.0) > oracle.reward(0, 0, 0.0)


def test_correct_kernels_are_ranked_by_performance(oracle):
    # Sec. 4.3: compiled and correct -> the performance decides, higher is better
    ps = np.sort(np.random.default_rng(4).uniform(0.0, 100.0, 200))
    rs = [oracle.reward(1, 1, float(p)) for p in ps]
    assert all(b > a for a, b in zip(rs, rs[1:]))
    for p in ps:
        assert oracle.reward(1, 1, float(p)) == float(p)
    assert oracle.reward(1, 1, oracle.performance(2.0)) == 0.5
    assert oracle.reward(1, 1, 0.0) == 0.0 and oracle.reward(1, 1, 1e-12) > oracle.reward(1, 0, 1e9)


def test_performance_of_a_failing_stage_may_be_anything(oracle):
    assert math.isnan(oracle.reward(1, 1, math.nan))
    assert math.isnan(oracle.reward(1, 1, -1.0))
