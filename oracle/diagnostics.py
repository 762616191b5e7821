"""Evaluation diagnostics of section 5 and Appendix B, written out as the
paper defines them (float64, pure numpy).

TEST INFRASTRUCTURE ONLY (see the package header).

* ``improvement_score`` -- section 5, eq. (subopt.experiment): the reward
  of the Speculative Rejection answer, placed on the range of the rewards of
  the Best-of-N responses z_1..z_N and scaled to 100:
  (1 - (max_k s(z_k) - s(y_SR)) / (max_k s(z_k) - min_k s(z_k))) * 100.
* ``relative_gpu_compute`` and ``speedup`` -- the same equation: T / T_BoN
  and T_BoN / T for wall-clock times.
* ``pearson`` and ``kendall`` -- Appendix B: the empirical Pearson
  correlation of n pairs, and Kendall's coefficient
  2 / (n (n - 1)) * sum_{i<j} sgn(x_i - x_j) sgn(y_i - y_j) (no correction
  for ties: tied pairs count zero), applied to the partial and final rewards
  of the candidates of one prompt.
"""
import numpy as np


def improvement_score(bon_rewards, sr_reward):
    """Section 5, eq. (subopt.experiment).  NaN when the Best-of-N rewards are
    all equal (the range is zero)."""
    z = np.asarray(bon_rewards, dtype=np.float64)
    hi, lo = z.max(), z.min()
    if hi == lo:
        return float("nan")
    return (1.0 - (hi - float(sr_reward)) / (hi - lo)) * 100.0


def relative_gpu_compute(t, t_bon):
    """Section 5, eq. (subopt.experiment): T / T_BoN."""
    return float(t) / float(t_bon)


def speedup(t, t_bon):
    """Section 5, eq. (subopt.experiment): T_BoN / T."""
    return float(t_bon) / float(t)


def pearson(x, y):
    """Appendix B: sum (x_i - xbar)(y_i - ybar) / sqrt(sum (x_i - xbar)^2 *
    sum (y_i - ybar)^2).  NaN when either sample is constant."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    dx, dy = x - x.mean(), y - y.mean()
    den = np.sqrt((dx * dx).sum() * (dy * dy).sum())
    if den == 0.0:
        return float("nan")
    return float((dx * dy).sum() / den)


def kendall(x, y):
    """Appendix B: 2 / (n (n-1)) * sum over pairs i < j of
    sgn(x_i - x_j) * sgn(y_i - y_j)."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    n = len(x)
    total = 0
    for i in range(n):
        total += int((np.sign(x[i] - x[i + 1:]) * np.sign(y[i] - y[i + 1:])).sum())
    return 2.0 * total / (n * (n - 1))
