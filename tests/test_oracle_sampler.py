"""The oracle's sampler: exp_sr accuracy, exact inverse-CDF invariants and the
sampling distribution (eq. auto-regressive, section 3)."""
import numpy as np
import pytest
from scipy import stats

from oracle import sampler
from oracle.philox import philox4x32_10


def test_exp_sr_accuracy_and_shape():
    z = np.linspace(-24.0, 0.0, 2_000_001).astype(np.float32)
    e = sampler.exp_sr(z)
    ref = np.exp(z.astype(np.float64))
    rel = np.abs(e.astype(np.float64) - ref) / ref
    assert rel.max() < 2.0 * 2.0**-23          # within two float32 ulps
    assert sampler.exp_sr(np.float32(0.0)) == np.float32(1.0)
    assert np.all(np.diff(e) >= 0)              # monotone on the grid
    assert sampler.exp_sr(np.float32(-24.5)) == 0.0
    assert sampler.exp_sr(np.float32(-np.inf)) == 0.0


def test_exp_sr_at_powers_of_two():
    # e^(-k ln 2) = 2^-k: the range reduction must land exactly on n = -k.
    # z is the float32 nearest -k ln 2, so compare against e^z in float64.
    for k in range(0, 30):
        z = np.float32(-k * np.log(2.0))
        assert abs(float(sampler.exp_sr(z)) / np.exp(np.float64(z)) - 1.0) < 2.5e-7


def test_draw_threshold_is_exact():
    rng = np.random.default_rng(1)
    for _ in range(1000):
        x = int(rng.integers(0, 2**32))
        w = int(rng.integers(1, 2**50))
        assert sampler.draw_threshold(x, w) == (x * w) >> 32


def test_two_equal_logits_closed_form():
    # w = [2^32, 2^32], W = 2^33, t = 2x: token 0 iff x < 2^31.
    for cand in range(40):
        x = sampler.uniform_word(42, cand, 3)
        tok = sampler.sample(np.zeros(2, np.float32), 1.0, 42, cand, 3)
        assert tok == (0 if x < 2**31 else 1)


def test_uniform_word_is_philox_word0():
    seed = (7 << 32) | 99
    assert sampler.uniform_word(seed, 5, 11) == philox4x32_10((11, 5, 0, 0), (99, 7))[0]


def test_zero_weight_never_drawn_and_threshold_below_total():
    logits = np.array([0.0, -30.0, -1.0, -100.0, -2.0], np.float32)
    w = sampler.weights(logits, 1.0)
    assert w[1] == 0 and w[3] == 0
    W = int(w.sum())
    for cand in range(2000):
        x = sampler.uniform_word(3, cand, 0)
        assert sampler.draw_threshold(x, W) < W
        assert sampler.sample(logits, 1.0, 3, cand, 0) not in (1, 3)


def test_inverse_cdf_at_exact_boundaries():
    # token = min{i : w_0 + ... + w_i > t}: a threshold equal to a cumulative
    # weight belongs to the next token (strict inequality), and zero weights
    # are skipped.  Hand-counted: cumulative weights 5, 8, 15.
    w = np.array([5, 3, 7], np.uint64)
    for t, tok in [(0, 0), (4, 0), (5, 1), (7, 1), (8, 2), (14, 2)]:
        assert sampler.inverse_cdf(w, t) == tok, t
    # cumulative weights 0, 4, 4, 4, 10
    w = np.array([0, 4, 0, 0, 6], np.uint64)
    for t, tok in [(0, 1), (3, 1), (4, 4), (9, 4)]:
        assert sampler.inverse_cdf(w, t) == tok, t
    # weights near 2^32 (a token of probability close to 1): exact in uint64
    big = 2**32
    w = np.array([big - 1, 1, big], np.uint64)
    assert sampler.inverse_cdf(w, big - 2) == 0
    assert sampler.inverse_cdf(w, big - 1) == 1
    assert sampler.inverse_cdf(w, big) == 2
    assert sampler.inverse_cdf(w, 2 * big - 1) == 2


def test_greedy_is_first_argmax():
    logits = np.array([0.5, 2.0, -1.0, 2.0], np.float32)
    assert sampler.sample(logits, 0.0, 1, 2, 3) == 1


def test_chi_square_against_softmax():
    rng = np.random.default_rng(5)
    V = 16
    logits = rng.normal(0, 1.5, V).astype(np.float32)
    p = np.exp(logits.astype(np.float64) - logits.max())
    p /= p.sum()
    n = 40000
    w = sampler.weights(logits, 1.0)
    cum = np.cumsum(w)
    W = int(w.sum())
    counts = np.zeros(V, np.int64)
    for i in range(n):
        x = sampler.uniform_word(1234, i % 997, i // 997)
        counts[np.searchsorted(cum, sampler.draw_threshold(x, W), side="right")] += 1
    chi2 = ((counts - n * p) ** 2 / (n * p)).sum()
    assert chi2 < stats.chi2.ppf(0.999, V - 1)
    # temperature 2 flattens the distribution accordingly
    p2 = np.exp((logits.astype(np.float64) - logits.max()) / 2.0)
    p2 /= p2.sum()
    w2 = sampler.weights(logits, 2.0).astype(np.float64)
    assert np.allclose(w2 / w2.sum(), p2, rtol=1e-5, atol=1e-9)
