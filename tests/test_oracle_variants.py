"""Pins for the oracle's estimator and delivery variants (CPU only):
Horvitz-Thompson and stale-fill aggregates, owner / reliable-packet
overrides and broadcast ages."""
import itertools

import numpy as np
import pytest

from oracle import drift, loss, step


def _enumerate(n, q):
    """All masks of n independent Bernoulli(q_i) arrivals with probabilities."""
    q = np.broadcast_to(np.asarray(q, dtype=np.float64), (n,))
    for bits in itertools.product((0, 1), repeat=n):
        s = np.array(bits)
        yield s, float(np.prod(np.where(s == 1, q, 1 - q)))


def test_horvitz_thompson_worked_example():
    g = np.array([[1.0], [2.0], [3.0], [4.0]])
    S = np.array([[1], [0], [1], [1]])
    q = np.full((4, 1), 0.5)
    g_hat, scale = step.aggregate_horvitz_thompson(g, S, q)
    assert g_hat.tolist() == [4.0]  # (1 + 3 + 4) / 0.5 / 4
    assert scale.tolist() == [4.0]


@pytest.mark.parametrize("n,qv,owner", [(3, 0.9, -1), (5, 0.6, -1), (6, 0.3, 2), (1, 0.5, -1)])
def test_horvitz_thompson_unbiased_and_variance_by_enumeration(n, qv, owner):
    rng = np.random.default_rng(n)
    e = 4
    g = rng.standard_normal((n, e))
    q = np.full(n, qv)
    if owner >= 0:
        q[owner] = 1.0  # the owner's own contribution cannot be lost
    Q = np.repeat(q[:, None], e, axis=1)
    mean = np.zeros(e)
    second = np.zeros(e)
    for s, pr in _enumerate(n, q):
        gh, _ = step.aggregate_horvitz_thompson(g, np.repeat(s[:, None], e, 1), Q)
        mean += pr * gh
        second += pr * gh * gh
    assert np.allclose(mean, g.mean(axis=0), atol=1e-12)  # no conditioning
    var = second - mean**2
    want = (g**2 * ((1 - q) / q)[:, None]).sum(axis=0) / n**2
    assert np.allclose(var, want, atol=1e-12)


def test_horvitz_thompson_without_loss_is_the_mean():
    g = np.random.default_rng(0).standard_normal((7, 50))
    gh, _ = step.aggregate_horvitz_thompson(g, np.ones_like(g), np.ones_like(g))
    assert np.allclose(gh, g.mean(axis=0), atol=1e-15)


def test_stale_fill_worked_example():
    g = np.array([[1.0, 10.0], [2.0, 20.0], [3.0, 30.0]])
    prev = np.array([[-1.0, -10.0], [-2.0, -20.0], [-3.0, -30.0]])
    S = np.array([[1, 0], [0, 0], [1, 1]])
    gh, new_prev, _ = step.aggregate_stale_fill(g, S, prev)
    assert gh.tolist() == [(1 - 2 + 3) / 3, (-10 - 20 + 30) / 3]
    assert new_prev.tolist() == [[1.0, -10.0], [-2.0, -20.0], [3.0, 30.0]]


def test_stale_fill_no_loss_and_total_loss():
    rng = np.random.default_rng(1)
    g = rng.standard_normal((5, 30))
    prev = rng.standard_normal((5, 30))
    gh, new_prev, _ = step.aggregate_stale_fill(g, np.ones_like(g), prev)
    assert np.allclose(gh, g.mean(axis=0), atol=1e-15) and np.array_equal(new_prev, g)
    gh, new_prev, _ = step.aggregate_stale_fill(g, np.zeros_like(g), prev)
    assert np.allclose(gh, prev.mean(axis=0), atol=1e-15) and np.array_equal(new_prev, prev)


@pytest.mark.parametrize("n,p", [(3, 0.2), (5, 0.5)])
def test_stale_fill_expectation_by_enumeration(n, p):
    # One step: E[g_hat] = (1 - p) mean(g) + p mean(g_prev), i.e. biased
    # toward the stale values unless the gradients do not change.
    rng = np.random.default_rng(n)
    g = rng.standard_normal((n, 3))
    prev = rng.standard_normal((n, 3))
    mean = np.zeros(3)
    for s, pr in _enumerate(n, 1 - p):
        gh, _, _ = step.aggregate_stale_fill(g, np.repeat(s[:, None], 3, 1), prev)
        mean += pr * gh
    assert np.allclose(mean, (1 - p) * g.mean(axis=0) + p * prev.mean(axis=0), atol=1e-12)


def test_stale_fill_constant_gradients_recover_the_mean():
    # Fixed gradients: once every row has arrived once, g_hat is the mean.
    n, P = 6, 40
    g = np.random.default_rng(2).standard_normal((n, P))
    prev = np.zeros_like(g)
    seen = np.zeros_like(g, dtype=bool)
    for t in range(60):
        S = loss.bernoulli_arrivals(0, t, loss.GRAD, n, np.arange(P), 0.4)
        gh, prev, _ = step.aggregate_stale_fill(g, S, prev)
        seen |= S.astype(bool)
    assert seen.all()
    assert np.allclose(gh, g.mean(axis=0), atol=1e-14)


def test_overrides():
    rng = np.random.default_rng(3)
    a = (rng.random((5, 12)) < 0.5).astype(np.uint8)
    rel = np.zeros(12, np.uint8)
    rel[[0, 7]] = 1
    out = loss.apply_overrides(a, owner=2, reliable=rel)
    assert (out[2] == 1).all() and (out[:, [0, 7]] == 1).all()
    keep = np.ones_like(a, dtype=bool)
    keep[2] = False
    keep[:, [0, 7]] = False
    assert np.array_equal(out[keep], a[keep])
    assert np.array_equal(loss.apply_overrides(a), a)
    # with the owner's row always present no packet is ever empty
    a0 = np.zeros((4, 9), np.uint8)
    assert loss.apply_overrides(a0, owner=0).sum(axis=0).min() == 1


def test_ages_sequence_and_saturation():
    ages = np.zeros((2, 3), np.uint16)
    R = [np.array([[1, 0, 0], [0, 0, 1]]), np.array([[0, 0, 1], [1, 0, 0]])]
    ages = step.update_ages(ages, R[0])
    assert ages.tolist() == [[0, 1, 1], [1, 1, 0]]
    ages = step.update_ages(ages, R[1])
    assert ages.tolist() == [[1, 2, 0], [0, 2, 1]]
    big = np.full((1, 2), 65535, np.uint16)
    assert step.update_ages(big, np.array([[0, 1]])).tolist() == [[65535, 0]]


@pytest.mark.parametrize("owner", [-1, 0])
def test_replicas_are_the_master_of_their_age_and_drift_matches_ages(owner):
    # Broadcast a random-walk master; every replica element equals the
    # master of `age` steps earlier, bit for bit.  The stationary squared
    # gap between replicas i and k is sigma^2 E|a_i - a_k| (2p / (1 - p^2)
    # for two lossy rows); between the owner (age 0) and a lossy replica it
    # is sigma^2 E[a] = sigma^2 p / (1 - p).
    n, e, steps, burn, p, sigma = 6, 3000, 220, 60, 0.3, 1e-3
    rng = np.random.default_rng(7)
    theta = np.zeros(e)
    history = [theta.copy()]
    reps = np.zeros((n, e))
    ages = np.zeros((n, e), np.uint16)
    ratio_pairs, ratio_owner = [], []
    for t in range(steps):
        theta = theta + sigma * rng.standard_normal(e)
        history.append(theta.copy())
        R = loss.apply_overrides(loss.bernoulli_arrivals(0, t, loss.BCAST, n, np.arange(e), p),
                                 owner=owner)
        reps = step.broadcast(reps, theta[None, :], R)
        ages = step.update_ages(ages, R)
        if t < burn:
            continue
        hist = np.array(history)  # [t+2][e]; history[-1] is the newest master
        for i in range(n):
            assert np.array_equal(reps[i], hist[len(hist) - 1 - ages[i].astype(int), np.arange(e)])
        r = drift.drift_stats(reps)
        gap = np.abs(ages[:, None, :].astype(int) - ages[None, :, :].astype(int))
        iu = np.triu_indices(n, 1)
        ratio_pairs.append(r["mean_sq"] / sigma**2 / gap[iu].mean())
        if owner >= 0:
            others = [i for i in range(n) if i != owner]
            d2 = ((reps[others] - reps[owner]) ** 2).mean()
            ratio_owner.append(d2 / sigma**2)
    # E[D^2] / (sigma^2 E|a_i - a_k|) -> 1 (the gap is measured, not modelled)
    assert abs(np.mean(ratio_pairs) - 1) < 0.05
    if owner >= 0:
        assert abs(np.mean(ratio_owner) - p / (1 - p)) < 0.05 * p / (1 - p)


def test_parity_recovery_worked_example():
    a = np.array([[1, 0, 1, 1, 0, 0, 1],
                  [0, 1, 1, 1, 1, 1, 0]], np.uint8)
    par = np.array([[1, 1], [0, 1]], np.uint8)  # group 4: packets 0-3, 4-6
    out = loss.parity_recover(a, 4, par)
    # row 0: group 0 lost one (k=1) and parity arrived -> rebuilt; group 1
    # lost two -> nothing.  row 1: group 0 parity lost -> nothing; group 1
    # lost one (k=6) and parity arrived -> rebuilt.
    assert out.tolist() == [[1, 1, 1, 1, 0, 0, 1], [0, 1, 1, 1, 1, 1, 1]]


@pytest.mark.parametrize("group,p", [(4, 0.1), (8, 0.2), (3, 0.4)])
def test_parity_residual_loss_rate(group, p):
    # A packet stays lost iff it was lost and not (every other packet of its
    # group and the parity packet arrived): rate p (1 - (1 - p)^group).
    n, P = 64, 4096 - 4096 % group
    a = loss.bernoulli_arrivals(1, 0, loss.GRAD, n, np.arange(P), p)
    par = loss.parity_arrivals(1, 0, loss.GRAD, n, np.arange(P // group), p)
    out = loss.parity_recover(a, group, par)
    q = 1 - loss.threshold(p) / 2**32
    want = (1 - q) * (1 - q**group)
    lost = out.size - int(out.sum())
    sigma = np.sqrt(out.size * want * (1 - want) * 2)  # packets of a group are dependent
    assert abs(lost - out.size * want) < 5 * sigma, (lost / out.size, want)
    assert (out >= a).all()  # recovery only adds arrivals


def test_parity_enumeration_single_group():
    # Exact: over all loss patterns of one group plus its parity packet, the
    # expected number of packets still lost is G p (1 - q^G).
    G, p = 3, 0.3
    q = 1 - p
    expect = 0.0
    for bits in itertools.product((0, 1), repeat=G + 1):
        s = np.array(bits[:G], np.uint8)[None, :]
        par = np.array([[bits[G]]], np.uint8)
        pr = np.prod([q if b else p for b in bits])
        out = loss.parity_recover(s, G, par)
        expect += pr * (G - int(out.sum()))
    assert abs(expect - G * p * (1 - q**G)) < 1e-12


@pytest.mark.parametrize("G,q", [(1, 0.5), (3, 0.7), (5, 0.9)])
def test_parity_marginal_arrival_by_enumeration(G, q):
    # Every packet's marginal arrival probability over all 2^(G+1) patterns.
    marg = np.zeros(G)
    for bits in itertools.product((0, 1), repeat=G + 1):
        pr = np.prod([q if b else 1 - q for b in bits])
        out = loss.parity_recover(np.array(bits[:G], np.uint8)[None, :], G,
                                  np.array([[bits[G]]], np.uint8))
        marg += pr * out[0]
    assert np.allclose(marg, loss.parity_arrival_probability(q, G), atol=1e-14)
    # G = 1 is a duplicate send: lost only if both copies are lost.
    if G == 1:
        assert abs(marg[0] - (1 - (1 - q) ** 2)) < 1e-14


def test_parity_respects_overrides_and_ragged_tail():
    # Reliable packets count as present inside a group; the owner row never
    # needs recovery; the last group of 7 packets under G = 3 holds one.
    a = np.array([[0, 1, 1, 0, 0, 1, 0],
                  [0, 0, 0, 0, 0, 0, 0]], np.uint8)
    rel = np.array([0, 0, 0, 0, 1, 0, 0], np.uint8)
    s = loss.apply_overrides(a, owner=1, reliable=rel)
    par = np.ones((2, 3), np.uint8)
    out = loss.parity_recover(s, 3, par)
    # row 0: group 0 (k 0-2) one lost -> rebuilt; group 1 (k 3-5) k=4 is
    # reliable, one lost (k=3) -> rebuilt; group 2 (k=6) lost -> rebuilt.
    assert out.tolist() == [[1] * 7, [1] * 7]
    par[0, 2] = 0
    assert loss.parity_recover(s, 3, par)[0, 6] == 0


@pytest.mark.parametrize("G,P,rel", [(3, 7, [0, 1, 0, 0, 0, 1, 0]), (4, 4, None), (2, 5, [1, 0, 0, 0, 1])])
def test_parity_marginals_with_reliable_and_ragged_groups_by_enumeration(G, P, rel):
    # Exact marginals over every loss pattern of the lossy packets and every
    # group's parity packet (reliable packets never lost).
    q = 0.6
    relf = np.zeros(P, np.uint8) if rel is None else np.array(rel, np.uint8)
    lossy = [k for k in range(P) if not relf[k]]
    ngroups = (P + G - 1) // G
    marg = np.zeros(P)
    for bits in itertools.product((0, 1), repeat=len(lossy) + ngroups):
        a = np.ones((1, P), np.uint8)
        for b, k in zip(bits[: len(lossy)], lossy):
            a[0, k] = b
        par = np.array([bits[len(lossy):]], np.uint8)
        pr = np.prod([q if b else 1 - q for b in bits])
        marg += pr * loss.parity_recover(loss.apply_overrides(a, reliable=relf), G, par)[0]
    want = loss.parity_arrival_probabilities(q, G, P, None if rel is None else relf)
    assert np.allclose(marg, want, atol=1e-14)
    if rel is None and P % G == 0:
        assert np.allclose(want, loss.parity_arrival_probability(q, G), atol=1e-15)
