"""Pins of oracle/tis.py (token-level TIS weights, Eq. (2)-(3), and the mismatch KL)
against closed forms and an independent library KL."""
import math

import numpy as np
import scipy.stats

from oracle import tis


def test_kl_estimators_reproduce_the_library_kl_of_two_categoricals():
    """Tokens drawn from the rollout policy p in exact proportions (outcome i appears
    N p_i times): the mean of either per-token term is KL(p || q) as scipy computes
    it from p and q, up to the fp32 rounding of the log-probabilities."""
    p = np.array([0.5, 0.25, 0.125, 0.0625, 0.03125, 0.03125])
    q = np.array([0.3, 0.3, 0.2, 0.1, 0.05, 0.05])
    n = 1 << 14
    counts = (p * n).astype(int)
    outcome = np.repeat(np.arange(p.size), counts)
    lr = np.log(p)[outcome].astype(np.float32)
    lt = np.log(q)[outcome].astype(np.float32)
    w, stats = tis.tis_weights_kl(lt, lr)
    kl = scipy.stats.entropy(p, q)
    assert stats[2] == n
    assert abs(stats[0] / n - kl) < 1e-6
    assert abs(stats[1] / n - kl) < 1e-6
    # and the weights average to sum(q) = 1 before truncation (none of q/p exceeds 2 here)
    assert stats[3] == 0
    assert abs(w.astype(np.float64).mean() - 1.0) < 1e-6


def test_truncation_closed_forms_and_mask():
    d = np.array([0.0, math.log(3.0), -math.log(4.0), -200.0, 1.0, 0.5], dtype=np.float64)
    lr = np.array([-1.0, -2.0, -0.5, -3.0, -7.0, -1.0], dtype=np.float32)
    lt = (lr.astype(np.float64) + d).astype(np.float32)
    mask = np.array([1, 1, 1, 1, 0, 1], dtype=np.uint8)
    w, stats = tis.tis_weights_kl(lt, lr, mask, clip_c=2.0)
    dd = lt.astype(np.float64) - lr.astype(np.float64)
    assert w[0] == 1.0 and w[1] == 2.0 and w[4] == 0.0
    assert w[2] == np.float32(math.exp(dd[2])) and abs(w[2] - 0.25) < 1e-6
    assert w[3] == 0.0                                   # e^-200 underflows fp32
    assert w[5] == np.float32(math.exp(dd[5]))
    assert stats[2] == 5 and stats[3] == 1
    assert stats[0] == -(dd[[0, 1, 2, 3, 5]]).sum()


def test_k3_is_nonnegative_and_second_order():
    rng = np.random.default_rng(3)
    lr = rng.uniform(-12, 0, 5000).astype(np.float32)
    lt = (lr + rng.normal(0, 1e-3, 5000)).astype(np.float32)
    _, stats = tis.tis_weights_kl(lt, lr)
    d = lt.astype(np.float64) - lr.astype(np.float64)
    assert stats[1] >= 0
    assert abs(stats[1] - (d * d / 2).sum()) <= 1e-3 * stats[1]
    # k3 for a single token equals (w - 1) - log w evaluated directly where that is accurate
    big = np.array([0.7, -1.3, 2.5])
    for x in big:
        _, s = tis.tis_weights_kl(np.array([x], np.float32), np.array([0.0], np.float32))
        dx = float(np.float32(x))
        assert abs(s[1] - ((math.exp(dx) - 1.0) - dx)) < 1e-15


def test_weights_stay_in_range_and_count_truncations():
    rng = np.random.default_rng(4)
    lr = rng.uniform(-20, 0, 20000).astype(np.float32)
    lt = (lr + rng.normal(0, 1.5, 20000)).astype(np.float32)
    mask = (rng.uniform(0, 1, 20000) < 0.9).astype(np.uint8)
    w, stats = tis.tis_weights_kl(lt, lr, mask, clip_c=2.0)
    assert np.all((w >= 0) & (w <= 2.0))
    assert np.all(w[mask == 0] == 0)
    d = lt.astype(np.float64) - lr.astype(np.float64)
    assert stats[3] == ((d > math.log(2.0)) & (mask == 1)).sum()
    assert stats[2] == mask.sum()
