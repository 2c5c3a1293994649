"""Pins for the oracle's drift statistics and Theorem 3.1 (CPU)."""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import drift, loss, step

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_worked_example():
    with open(os.path.join(GOLDEN, "drift_worked.json")) as f:
        ex = json.load(f)
    r = drift.drift_stats(np.array(ex["x"], float), np.array(ex["master"], float))
    for key, val in ex["expected"].items():
        assert r[key] == float(Fraction(val)), key


def test_identical_replicas_have_zero_drift():
    x = np.repeat(np.random.default_rng(0).standard_normal((1, 300)), 5, 0)
    r = drift.drift_stats(x, x[0])
    assert r["max_abs"] == 0 and r["mean_sq"] == 0 and r["mean_abs_to_master"] == 0


def test_pair_sum_equals_variance_identity_and_brute_force_max():
    # sum_{i<k} (x_i - x_k)^2 = N^2 * population variance (a different
    # formula, evaluated with numpy's var); max_abs against all pairs.
    rng = np.random.default_rng(1)
    for n in (2, 3, 7, 16):
        x = rng.standard_normal((n, 200))
        r = drift.drift_stats(x)
        assert math.isclose(r["pair_sum"], float(np.sum(n * n * np.var(x, axis=0))),
                            rel_tol=1e-12)
        brute = max(abs(x[i, e] - x[k, e]) for i, k in itertools.combinations(range(n), 2)
                    for e in range(200))
        assert r["max_abs"] == brute
        assert r["pairs"] == n * (n - 1) // 2


def test_single_replica_and_empty():
    r = drift.drift_stats(np.ones((1, 10)))
    assert r["mean_sq"] == 0 and r["max_abs"] == 0
    r = drift.drift_stats(np.ones((4, 0)))
    assert r["mean_sq"] == 0 and r["max_abs"] == 0


@pytest.mark.parametrize("p", [0.1, 0.3])
def test_long_run_drift_is_bounded_at_the_geometric_age_constant(p):
    # Theorem 3.1 setting: the owner's shard takes independent zero-mean
    # increments of variance sigma^2 per step; every replica keeps its stale
    # value when the broadcast is lost (i.i.d. Bernoulli, step (4)).  A
    # replica's age is geometric, so the stationary E[D^2] between two
    # replicas is sigma^2 * E|a_i - a_k| = 2p / (1 - p^2) * sigma^2.  The
    # paper prints 2p / (1 + p) (its proof drops the other replica's
    # staleness); the bound stays O(1) either way.
    n, e, steps, burn = 8, 4096, 260, 60
    sigma = 1e-3
    rng = np.random.default_rng(11)
    theta = np.zeros(e)
    reps = np.zeros((n, e))
    series = []
    for t in range(steps):
        theta = theta + sigma * rng.standard_normal(e)
        R = loss.bernoulli_arrivals(0, t, loss.BCAST, n, np.arange(e), p)  # 1-elem packets
        reps = step.broadcast(reps, theta[None, :], R)
        series.append(drift.drift_stats(reps, theta)["mean_sq"])
    s = np.array(series[burn:]) / sigma**2
    corrected = 2 * p / (1 - p * p)
    paper = 2 * p / (1 + p)
    # Stationary mean within 5% (there are e * n(n-1)/2 pairs per step).
    assert abs(s.mean() - corrected) < 0.05 * corrected, (s.mean(), corrected, paper)
    # Bounded: no trend between the two halves of the stationary window.
    half = len(s) // 2
    assert abs(s[:half].mean() - s[half:].mean()) < 0.05 * corrected
    if p >= 0.3:
        assert abs(s.mean() - paper) > 0.1 * paper  # distinguishes the constants
