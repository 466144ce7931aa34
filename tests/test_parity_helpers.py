"""The ranking check agrees with a brute-force pair count."""
import numpy as np

from tests.parity import ranking_violations, tolerance


def _brute(g, o, tol):
    n = 0
    for i in range(len(o)):
        for j in range(len(o)):
            if o[j] - tol[j] > o[i] + tol[i] and not g[j] > g[i]:
                n += 1
    return n


def test_ranking_violations_brute_force():
    rng = np.random.default_rng(0)
    for trial in range(30):
        o = rng.standard_normal(40)
        tol = tolerance(o, "bf16") * rng.uniform(0.5, 20)
        g = o + rng.standard_normal(40) * rng.uniform(0, 0.3)
        if trial % 3 == 0:
            g[rng.integers(0, 40, 5)] = g[rng.integers(0, 40, 5)]  # ties
        assert ranking_violations(g, o, tol) == _brute(g, o, tol)
