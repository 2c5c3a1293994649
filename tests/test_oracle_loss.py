"""Pins for the oracle's loss processes (CPU only)."""
import math

import numpy as np
import pytest

from oracle import loss


def _np_word(seed, k, i, t, direction):
    """w0, w1 of the draw for (k, i, t, dir) from numpy's independent Philox."""
    ctr = k | (i << 64) | (t << 128) | (direction << 192)
    c = (ctr - 1) % (1 << 256)
    words = np.array([(c >> (64 * j)) & ((1 << 64) - 1) for j in range(4)], dtype=np.uint64)
    bg = np.random.Philox(counter=words, key=np.array([seed, 0], dtype=np.uint64))
    w = bg.random_raw(4)
    return int(w[0]), int(w[1])


def test_threshold_closed_forms():
    assert loss.threshold(0.0) == 0
    assert loss.threshold(1.0) == 2**32
    assert loss.threshold(0.5) == 2**31
    assert loss.threshold(0.1) == 429496730  # ceil(429496729.6)
    with pytest.raises(ValueError):
        loss.threshold(1.5)


def test_uniform_less_than_p_is_the_drop_rule():
    # Algorithm 1 drops when Uniform(0,1) < p; u = hi32(w0) / 2**32 exactly.
    rng = np.random.default_rng(0)
    for _ in range(2000):
        p = float(rng.random())
        x = int(rng.integers(0, 2**32))
        assert (x < loss.threshold(p)) == (x / 2**32 < p)
    for x in (0, 1, 2**31 - 1, 2**31, 2**32 - 1):
        assert (x < loss.threshold(0.5)) == (x / 2**32 < 0.5)


def test_bernoulli_matches_independent_philox_draws():
    seed, t, n = 3, 17, 5
    packets = [0, 1, 2, 999, 25695]
    for direction in (loss.GRAD, loss.BCAST):
        a = loss.bernoulli_arrivals(seed, t, direction, n, packets, 0.37)
        for i in range(n):
            for j, k in enumerate(packets):
                w0, _ = _np_word(seed, k, i, t, direction)
                assert a[i, j] == (0 if (w0 >> 32) / 2**32 < 0.37 else 1)


def test_bernoulli_p0_p1():
    pk = np.arange(4096)
    assert loss.bernoulli_arrivals(0, 0, 0, 8, pk, 0.0).min() == 1
    assert loss.bernoulli_arrivals(0, 0, 0, 8, pk, 1.0).max() == 0


@pytest.mark.parametrize("p", [0.01, 0.1, 0.3])
def test_bernoulli_rate_binomial_interval(p):
    n, P = 64, 25696
    a = loss.bernoulli_arrivals(0, 0, loss.GRAD, n, np.arange(P), p)
    trials = n * P
    lost = trials - int(a.sum())
    q = loss.threshold(p) / 2**32
    sigma = math.sqrt(trials * q * (1 - q))
    assert abs(lost - trials * q) < 5 * sigma


def test_bernoulli_independence_between_directions_steps_workers():
    n, P, p = 16, 20000, 0.3
    pk = np.arange(P)
    a = loss.bernoulli_arrivals(0, 0, 0, n, pk, p).astype(float)
    b = loss.bernoulli_arrivals(0, 0, 1, n, pk, p).astype(float)
    c = loss.bernoulli_arrivals(0, 1, 0, n, pk, p).astype(float)
    m = n * P
    bound = 5 / math.sqrt(m)
    for x, y in ((a, b), (a, c), (a[:-1], a[1:])):
        r = np.corrcoef(x.ravel(), y.ravel())[0, 1]
        assert abs(r) < bound


def _ge(p_gb, p_bg, lg, lb, n=1, P=3, t=0, seed=0, state=None):
    state = np.zeros(n, np.uint8) if state is None else state
    return loss.ge_arrivals(seed, t, 0, n, P, p_gb, p_bg, lg, lb, state)


def test_ge_equal_loss_in_both_states_is_bernoulli_on_w1():
    a, _ = _ge(0.3, 0.2, 0.25, 0.25, n=4, P=300, t=5, seed=9)
    for i in range(4):
        for k in range(0, 300, 7):
            _, w1 = _np_word(9, k, i, 5, 0)
            assert a[i, k] == (0 if (w1 >> 32) / 2**32 < 0.25 else 1)


def test_ge_never_leaving_good_never_loses():
    a, s = _ge(0.0, 0.5, 0.0, 1.0, n=8, P=5000)
    assert a.min() == 1 and s.max() == 0


def test_ge_absorbing_bad_is_bernoulli_loss_bad():
    a, s = _ge(1.0, 0.0, 0.0, 0.5, n=8, P=20000)
    assert s.min() == 1
    lost = a.size - int(a.sum())
    sigma = math.sqrt(a.size * 0.25)
    assert abs(lost - a.size * 0.5) < 5 * sigma


def _path_probabilities(P, p_gb, p_bg, lg, lb):
    """Exact probability of each arrival pattern of a chain of P packets,
    started in Good, by summing over all state paths (transition, then emit)."""
    T = np.array([[1 - p_gb, p_gb], [p_bg, 1 - p_bg]])
    L = np.array([lg, lb])
    probs = {}
    for states in np.ndindex(*(2,) * P):
        ps, prev = 1.0, 0
        for s in states:
            ps *= T[prev, s]
            prev = s
        for pattern in np.ndindex(*(2,) * P):  # 1 = arrived
            pe = ps
            for s, arr in zip(states, pattern):
                pe *= (1 - L[s]) if arr else L[s]
            probs[pattern] = probs.get(pattern, 0.0) + pe
    return probs


def test_ge_pattern_distribution_brute_force():
    # Many independent chains (one per worker row) of 3 packets, compared with
    # the exact path-sum distribution.
    p_gb, p_bg, lg, lb = 0.3, 0.4, 0.1, 0.6
    n = 40000
    a, _ = loss.ge_arrivals(11, 0, 0, n, 3, p_gb, p_bg, lg, lb, np.zeros(n, np.uint8))
    exact = _path_probabilities(3, p_gb, p_bg, lg, lb)
    assert abs(sum(exact.values()) - 1) < 1e-12
    codes = a[:, 0] * 4 + a[:, 1] * 2 + a[:, 2]
    counts = np.bincount(codes, minlength=8)
    for pattern, pr in exact.items():
        code = pattern[0] * 4 + pattern[1] * 2 + pattern[2]
        sigma = math.sqrt(n * pr * (1 - pr))
        assert abs(counts[code] - n * pr) < 5 * sigma + 1


def test_ge_state_carries_across_steps():
    # Steps chain: the end state of step t starts step t+1.  With p_bg = 0 and
    # p_gb = 1 a chain is Bad after its first packet; carrying that into the
    # next step with p_gb = 0 keeps it Bad (lossy), starting fresh does not.
    _, s0 = _ge(1.0, 0.0, 0.0, 1.0, n=4, P=1)
    assert s0.tolist() == [1, 1, 1, 1]
    a_carry, s1 = loss.ge_arrivals(0, 1, 0, 4, 50, 0.0, 0.0, 0.0, 1.0, s0)
    a_fresh, _ = loss.ge_arrivals(0, 1, 0, 4, 50, 0.0, 0.0, 0.0, 1.0, np.zeros(4, np.uint8))
    assert a_carry.max() == 0 and a_fresh.min() == 1 and s1.tolist() == [1, 1, 1, 1]


def test_ge_stationary_loss_and_burst_length():
    # The Gilbert-Elliott workload: p_gb = 0.01, p_bg = 0.2, loss 0.5 in Bad.
    p_gb, p_bg, lb = 0.01, 0.2, 0.5
    n, P = 16, 65536
    state = np.zeros(n, np.uint8)
    lost = total = 0
    for t in range(3):
        a, state = loss.ge_arrivals(0, t, 0, n, P, p_gb, p_bg, 0.0, lb, state)
        lost += a.size - int(a.sum())
        total += a.size
    pi_b = p_gb / (p_gb + p_bg)
    want = pi_b * lb  # 0.0238
    rate = lost / total
    # Autocorrelated chain: inflate the binomial sigma by the correlation time.
    lam = 1 - p_gb - p_bg
    sigma = math.sqrt(want * (1 - want) / total * (1 + lam) / (1 - lam)) * 3
    assert abs(rate - want) < 6 * sigma, (rate, want)

    # Mean Bad sojourn: count Bad runs via loss_bad = 1 (every Bad packet is
    # lost, every Good one arrives), so runs of losses are Bad sojourns.
    a, _ = loss.ge_arrivals(0, 0, 0, n, P, p_gb, p_bg, 0.0, 1.0, np.zeros(n, np.uint8))
    runs = []
    for row in (1 - a.astype(int)):
        edges = np.diff(np.concatenate([[0], row, [0]]))
        starts, ends = np.where(edges == 1)[0], np.where(edges == -1)[0]
        runs.extend((ends - starts).tolist())
    mean_run = float(np.mean(runs))
    se = math.sqrt((1 - p_bg) / p_bg**2 / len(runs))
    assert abs(mean_run - 1 / p_bg) < 5 * se, mean_run


@pytest.mark.parametrize("p_gb,p_bg,lg,lb", [(0.01, 0.2, 0.0, 0.5), (0.6, 0.7, 0.1, 0.9),
                                            (0.0, 0.3, 0.05, 0.5), (1.0, 1.0, 0.0, 1.0)])
def test_ge_marginal_arrival_by_forward_recursion(p_gb, p_bg, lg, lb):
    # Propagate the state distribution packet by packet with the transition
    # matrix (no closed form) and compare the marginal arrival probabilities.
    P = 7
    T = np.array([[1 - p_gb, p_gb], [p_bg, 1 - p_bg]])
    dist = np.array([1.0, 0.0])
    for t in range(3):
        want = []
        for k in range(P):
            dist = dist @ T
            want.append(1.0 - (dist[0] * lg + dist[1] * lb))
        got = loss.ge_arrival_probability(t, np.arange(P), P, p_gb, p_bg, lg, lb)
        assert np.allclose(got, want, atol=1e-14), (t, got, want)


def test_ge_marginal_matches_the_drawn_chains():
    # Empirical arrival rate of the Philox-drawn chains, per packet position,
    # over many workers: within 5 sigma of the marginal.
    n, P, p_gb, p_bg, lg, lb = 4000, 12, 0.05, 0.3, 0.0, 0.6
    a, _ = loss.ge_arrivals(3, 0, loss.GRAD, n, P, p_gb, p_bg, lg, lb, np.zeros(n, np.uint8))
    q = loss.ge_arrival_probability(0, np.arange(P), P, p_gb, p_bg, lg, lb)
    rate = a.mean(axis=0)
    sigma = np.sqrt(q * (1 - q) / n)
    assert (np.abs(rate - q) < 5 * sigma + 1e-12).all(), (rate, q)
