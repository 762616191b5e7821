"""Pins of the diagnostics oracle (section 5 improvement score and relative
compute, Appendix B correlations) against independent implementations,
closed forms and hand-counted examples; and the library's host functions
against the oracle."""
import itertools
import json
import os

import numpy as np
import pytest
from scipy import stats

from oracle import diagnostics as dg

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_pearson_matches_scipy_and_numpy():
    rng = np.random.default_rng(0)
    for n in (2, 3, 17, 500):
        x = rng.normal(size=n)
        y = 0.3 * x + rng.normal(size=n)
        want = stats.pearsonr(x, y)[0]
        assert abs(dg.pearson(x, y) - want) < 1e-12
        assert abs(dg.pearson(x, y) - np.corrcoef(x, y)[0, 1]) < 1e-12


def test_pearson_closed_forms():
    x = np.arange(10.0)
    assert abs(dg.pearson(x, 3 * x + 2) - 1.0) < 1e-15
    assert abs(dg.pearson(x, -0.5 * x + 7) + 1.0) < 1e-15
    rng = np.random.default_rng(1)
    a, b = rng.normal(size=(2, 40))
    r = dg.pearson(a, b)
    assert abs(dg.pearson(5 * a + 1, 0.1 * b - 3) - r) < 1e-12       # positive affine maps
    assert abs(dg.pearson(-a, b) + r) < 1e-12                         # a sign flip
    assert np.isnan(dg.pearson(np.ones(5), np.arange(5.0)))


def test_kendall_hand_counted_examples():
    with open(os.path.join(GOLDEN, "kendall_examples.json")) as f:
        for c in json.load(f)["cases"]:
            n = len(c["x"])
            assert abs(dg.kendall(c["x"], c["y"]) - c["kendall"]) < 1e-15
            assert abs(c["kendall"] - 2 * c["concordant_minus_discordant"] / (n * (n - 1))) < 1e-15


def test_kendall_permutations_closed_form():
    """For a permutation, the coefficient is 1 - 4 inv / (n (n - 1)) with inv
    its number of inversions; averaged over all permutations it is 0."""
    n = 6
    base = np.arange(n)
    total = 0.0
    for perm in itertools.permutations(range(n)):
        inv = sum(1 for i in range(n) for j in range(i + 1, n) if perm[i] > perm[j])
        k = dg.kendall(base, perm)
        assert abs(k - (1 - 4 * inv / (n * (n - 1)))) < 1e-12
        total += k
    assert abs(total) < 1e-9


def test_kendall_matches_scipy_tau_b_with_and_without_ties():
    """Without ties it equals scipy's tau-b; with ties tau-b divides the same
    pair sum by sqrt((n0 - n1)(n0 - n2)) instead of n0 (n0 pairs, n1 and n2
    pairs tied in x and in y)."""
    rng = np.random.default_rng(2)
    x, y = rng.normal(size=(2, 60))
    assert abs(dg.kendall(x, y) - stats.kendalltau(x, y).statistic) < 1e-12
    xi = rng.integers(0, 5, size=80).astype(float)
    yi = rng.integers(0, 7, size=80).astype(float)
    n = len(xi)
    n0 = n * (n - 1) / 2
    ties = lambda v: sum(t * (t - 1) / 2 for t in np.unique(v, return_counts=True)[1])
    tau_b = stats.kendalltau(xi, yi).statistic
    assert abs(dg.kendall(xi, yi) - tau_b * np.sqrt((n0 - ties(xi)) * (n0 - ties(yi))) / n0) < 1e-12


def test_improvement_score_and_compute_ratios():
    z = [1.0, 4.0, 3.0, -2.0]
    assert dg.improvement_score(z, 4.0) == 100.0
    assert dg.improvement_score(z, -2.0) == 0.0
    assert abs(dg.improvement_score(z, 1.0) - 50.0) < 1e-12
    assert np.isnan(dg.improvement_score([2.0, 2.0], 2.0))
    # the worked example of section 4.1: Speculative Rejection returns y1,
    # the better of the two full responses
    with open(os.path.join(GOLDEN, "paper_example_sec41.json")) as f:
        ex = json.load(f)
    assert dg.improvement_score(ex["final_scores"], ex["final_scores"][ex["returned"]]) == 100.0
    assert dg.relative_gpu_compute(3.0, 12.0) == 0.25 and dg.speedup(3.0, 12.0) == 4.0


# ---- the library's host functions against the oracle (no GPU needed)

@pytest.fixture(scope="module")
def sr():
    import paper_2410_20290_amd as sr
    if not os.path.exists(sr.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return sr


@pytest.mark.parametrize("n,ties", [(2, False), (3, False), (64, False), (512, False), (200, True), (4096, True)])
def test_library_correlation_matches_oracle(sr, n, ties):
    rng = np.random.default_rng(n)
    if ties:
        x = rng.integers(-4, 5, size=n).astype(np.float32)
        y = (x + rng.integers(-2, 3, size=n)).astype(np.float32)
    else:
        x = rng.normal(size=n).astype(np.float32)
        y = (0.5 * x + rng.normal(size=n)).astype(np.float32)
    p, k = sr.correlation(x, y)
    assert abs(p - dg.pearson(x, y)) < 1e-12
    want_k = dg.kendall(x, y)
    assert abs(k - want_k) < 1e-12   # the same integer pair sum over the same divisor


def test_library_improvement_score_matches_oracle(sr):
    rng = np.random.default_rng(7)
    z = rng.normal(size=300).astype(np.float32)
    for r in (z.max(), z.min(), z[17], np.float32(0.25)):
        assert abs(sr.improvement_score(z, r) - dg.improvement_score(z, r)) < 1e-9
    assert np.isnan(sr.improvement_score(np.ones(4, np.float32), 1.0))


def test_library_diagnostics_reject_bad_input(sr):
    with pytest.raises(RuntimeError):
        sr.correlation([1.0], [2.0])
    with pytest.raises(RuntimeError):
        sr.correlation([1.0, float("nan")], [2.0, 3.0])
    with pytest.raises(RuntimeError):
        sr.improvement_score([], 1.0)
    with pytest.raises(RuntimeError):
        sr.improvement_score([1.0, 2.0], float("inf"))
    assert np.isnan(sr.correlation(np.ones(3), np.arange(3.0))[0])
