"""Pins of the oracle's confidence monitor and budget rule (Sec. 6.1, Alg. 2).

Token confidence against its closed forms and against scipy's logsumexp plus a full sort;
the trace-level threshold against numpy.percentile (linear interpolation) and the slope
against numpy.polyfit; hand-worked windows; the budget growth sequence of the paper's
settings (start 512, x1.75, cap 30K).
"""
import numpy as np
import pytest
from scipy.special import logsumexp

import oracle


def test_uniform_distribution_has_confidence_log_v():
    for V in (7, 1000, 151936):
        T = oracle.token_confidence(np.full((1, V), 3.25, np.float32), k=20)
        assert abs(T[0] - np.log(V)) < 1e-12 * np.log(V)


def test_two_level_distribution_closed_form():
    # m tokens at logit a, the rest at 0, k <= m: every top-k log-prob is a - LSE
    V, m, a, k = 5000, 40, 6.5, 20
    x = np.zeros((1, V), np.float32)
    x[0, :m] = a
    lse = np.log(m * np.exp(a) + (V - m))
    assert abs(oracle.token_confidence(x, k)[0] - (lse - a)) < 1e-12


@pytest.mark.parametrize("k", [1, 20, 64])
def test_token_confidence_matches_logsumexp_and_sort(k):
    rng = np.random.default_rng(k)
    x = (rng.standard_normal((6, 30000)) * rng.uniform(0.5, 8, size=(6, 1))).astype(np.float32)
    x[2, 17] = 40.0   # one very peaked row
    ref = logsumexp(x.astype(np.float64), axis=1) - np.sort(x.astype(np.float64), axis=1)[:, -k:].mean(axis=1)
    np.testing.assert_allclose(oracle.token_confidence(x, k), ref, rtol=1e-12, atol=1e-12)


def test_k_beyond_the_vocabulary_takes_the_whole_row():
    x = np.array([[1.0, 2.0, 3.0]], np.float32)
    ref = logsumexp([1.0, 2.0, 3.0]) - 2.0
    assert abs(oracle.token_confidence(x, 50)[0] - ref) < 1e-14


def test_one_dominant_token_closed_form():
    # one token at logit a, the rest at 0: T = log(e^a + V - 1) - a / k, far above the
    # uniform log V once a is large (a peaked distribution reads as confident)
    V, k = 151936, 20
    for a in (10.0, 30.0):
        x = np.zeros((1, V), np.float32)
        x[0, 123] = a
        ref = np.log(np.exp(a) + V - 1) - a / k
        assert abs(oracle.token_confidence(x, k)[0] - ref) < 1e-11 * ref
    assert oracle.token_confidence(x, k)[0] > np.log(V) + 10


def test_hand_worked_windows_and_percentile():
    # w = 2, s = 1: R' = [3, 3, 1, 1]; b = 50: pos 1.5 between sorted 1 and 3 -> Q = 2;
    # retained m = 2, 3 (both 1): slope 0, budget unchanged
    out = oracle.budget_update([np.array([5, 3, 4, 1, 2], np.float32)], [512], window=2,
                               stride=1, bottom_pct=50.0)
    assert out["thresholds"][0] == 2.0 and out["retained"][0] == 2
    assert out["slopes"][0] == 0.0 and out["budgets"][0] == 512
    # w = 2, s = 2, b = 100: R' = [5, 3, 1], all retained, slope -2: the budget grows
    out = oracle.budget_update([np.array([6, 5, 4, 3, 2, 1], np.float32)], [512], window=2,
                               stride=2, bottom_pct=100.0)
    assert out["thresholds"][0] == 5.0 and out["retained"][0] == 3
    assert out["slopes"][0] == -2.0 and out["budgets"][0] == 896


@pytest.mark.parametrize("seed", range(4))
def test_threshold_and_slope_against_numpy(seed):
    rng = np.random.default_rng(seed)
    n, w, s, b = int(rng.integers(200, 5000)), 64, 8, 10.0
    t = (rng.standard_normal(n) * 0.3 + np.linspace(9, 8 + seed, n)).astype(np.float32)
    out = oracle.budget_update([t], [1000], window=w, stride=s, bottom_pct=b)
    M = (n - w) // s + 1
    rp = np.array([t[m * s:m * s + w].min() for m in range(M)], np.float64)
    q = np.percentile(rp, b)   # numpy's default: linear interpolation
    assert abs(out["thresholds"][0] - q) <= 1e-12 * abs(q)
    keep = rp <= out["thresholds"][0]
    assert out["retained"][0] == keep.sum()
    if keep.sum() >= 2:
        ref = np.polyfit(np.nonzero(keep)[0].astype(np.float64), rp[keep], 1)[0]
        assert abs(out["slopes"][0] - ref) <= 1e-9 * max(1.0, abs(ref))


def test_budget_growth_sequence_and_cap():
    down = np.linspace(10, 5, 400).astype(np.float32)   # confidence falling: slope < 0
    b, seq = 512, [512]
    for _ in range(9):
        b = int(oracle.budget_update([down], [b])["budgets"][0])
        seq.append(b)
    assert seq == [512, 896, 1568, 2744, 4802, 8403, 14705, 25733, 30000, 30000]
    up = np.linspace(5, 10, 400).astype(np.float32)
    assert oracle.budget_update([up], [2744])["budgets"][0] == 2744   # never shrinks


def test_short_traces_keep_their_budget():
    out = oracle.budget_update([np.arange(63, dtype=np.float32)[::-1],
                                np.arange(64, dtype=np.float32)[::-1], np.zeros(0, np.float32)],
                               [700, 700, 700])
    assert out["budgets"].tolist() == [700, 700, 700]   # < w tokens; one window; empty
    assert out["retained"].tolist() == [0, 1, 0]
    assert np.isnan(out["thresholds"][0]) and out["thresholds"][1] == 0.0
