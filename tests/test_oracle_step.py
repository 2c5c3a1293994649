"""Pins for the oracle's aggregate, optimizers, broadcast and step (CPU)."""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import bf16, loss, step

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_aggregate_worked_example():
    with open(os.path.join(GOLDEN, "aggregate_worked.json")) as f:
        ex = json.load(f)
    d, L = ex["d"], ex["packet"]
    packets = list(range(math.ceil(d / L)))
    lens = step.packet_lengths(d, L, packets)
    assert lens.tolist() == [3, 3, 2]
    S = np.repeat(np.array(ex["arrived"], dtype=np.uint8), lens, axis=1)
    g = np.array(ex["grads"], dtype=np.float64)
    g_hat, K, _ = step.aggregate(g, S, 0.0, np.array(ex["theta"], dtype=np.float64))
    want = np.array([float(Fraction(v)) for v in ex["expected_g_hat"]])
    assert np.array_equal(g_hat, want)
    counts = np.array(ex["arrived"]).sum(axis=0)
    assert counts.tolist() == ex["expected_counts"]


def test_no_loss_is_the_exact_mean():
    # With nothing lost the aggregate is the reduce-scatter mean (Appendix A:
    # all-reduce = reduce-scatter then all-gather, SUM / N).
    rng = np.random.default_rng(1)
    g = rng.standard_normal((7, 1000))
    S = np.ones_like(g, dtype=np.uint8)
    g_hat, K, _ = step.aggregate(g, S, 0.0, np.zeros(1000))
    assert np.allclose(g_hat, np.mean(g, axis=0), rtol=0, atol=1e-15)
    assert (K == 7).all()


def test_single_arrival_copies_and_identical_contributions():
    rng = np.random.default_rng(2)
    g = rng.standard_normal((5, 64))
    for i in range(5):
        S = np.zeros_like(g, dtype=np.uint8)
        S[i] = 1
        g_hat, _, _ = step.aggregate(g, S, 0.0, np.zeros(64))
        assert np.array_equal(g_hat, g[i])
    # Identical contributions with few significant bits (bf16 values): the sum
    # K*x and the division by K are then exact.
    x = bf16.to_f64(bf16.from_f32(g[0].astype(np.float32)))
    same = np.repeat(x[None], 5, axis=0)
    S = (rng.random((5, 64)) < 0.6).astype(np.uint8)
    S[0] = 1
    g_hat, _, _ = step.aggregate(same, S, 0.0, np.zeros(64))
    assert np.array_equal(g_hat, x)


def test_fallback_when_nothing_arrives():
    theta = np.linspace(-1, 1, 10)
    g = np.ones((3, 10))
    S = np.zeros((3, 10), dtype=np.uint8)
    g0, K, _ = step.aggregate(g, S, 0.0, theta)
    assert (g0 == 0).all() and (K == 0).all()
    g1, _, _ = step.aggregate(g, S, 0.25, theta)
    assert np.array_equal(g1, 0.25 * theta)


@pytest.mark.parametrize("n,p,lam", [(1, 0.3, 0.0), (3, 0.1, 0.0), (6, 0.4, 0.5),
                                     (10, 0.25, 0.0)])
def test_brute_force_expectation_over_all_masks(n, p, lam):
    # Corollary 3.2: E[g_hat | some arrived] = the mean gradient.  Enumerate
    # every mask with its Bernoulli(1-p) probability; unconditionally the
    # empty mask contributes p^n * lam * theta.
    rng = np.random.default_rng(n)
    e = 3
    g = rng.standard_normal((n, e))
    theta = rng.standard_normal(e)
    mean = g.mean(axis=0)
    total = np.zeros(e)
    cond = np.zeros(e)
    for bits in itertools.product((0, 1), repeat=n):
        s = np.array(bits, dtype=np.uint8)
        k = int(s.sum())
        pr = (1 - p) ** k * p ** (n - k)
        S = np.repeat(s[:, None], e, axis=1)
        gh, _, _ = step.aggregate(g, S, lam, theta)
        total += pr * gh
        if k > 0:
            cond += pr * gh
    assert np.allclose(total, (1 - p**n) * mean + p**n * lam * theta, atol=1e-12)
    assert np.allclose(cond / (1 - p**n), mean, atol=1e-12)


@pytest.mark.parametrize("kind", ["bernoulli", "gilbert_elliott"])
def test_monte_carlo_unbiased_with_seeded_masks(kind):
    # Masks from the oracle's own loss processes over many steps; the sample
    # mean of g_hat over steps with K > 0 converges to the mean gradient (the
    # masks are exchangeable across workers, so this holds for bursty loss
    # too, although the paper's argument assumes independence).
    n, P, steps = 8, 64, 400
    rng = np.random.default_rng(3)
    g = rng.standard_normal((n, P))  # one element per packet
    state = np.zeros(n, np.uint8)
    acc = np.zeros(P)
    acc2 = np.zeros(P)
    cnt = np.zeros(P)
    for t in range(steps):
        if kind == "bernoulli":
            a = loss.bernoulli_arrivals(0, t, loss.GRAD, n, np.arange(P), 0.3)
        else:
            a, state = loss.ge_arrivals(0, t, loss.GRAD, n, P, 0.2, 0.3, 0.05, 0.7, state)
        gh, K, _ = step.aggregate(g, a, 0.0, np.zeros(P))
        ok = K > 0
        acc[ok] += gh[ok]
        acc2[ok] += gh[ok] ** 2
        cnt[ok] += 1
    m = acc / cnt
    var = acc2 / cnt - m**2
    z = (m - g.mean(axis=0)) / np.sqrt(var / cnt)
    # 64 independent z-scores: all within 5 sigma, and their spread near 1.
    assert np.max(np.abs(z)) < 5
    assert 0.6 < np.std(z) < 1.4


def _torch_opt_run(kind, grads, theta0, **hp):
    p = torch.nn.Parameter(torch.tensor(theta0, dtype=torch.float64))
    if kind == "sgd":
        opt = torch.optim.SGD([p], lr=hp["lr"])
    elif kind == "momentum":
        opt = torch.optim.SGD([p], lr=hp["lr"], momentum=hp["momentum"])
    else:
        opt = torch.optim.Adam([p], lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]),
                               eps=hp["eps"], foreach=False)
    for gv in grads:
        p.grad = torch.tensor(gv, dtype=torch.float64)
        opt.step()
    return p.detach().numpy()


@pytest.mark.parametrize("kind", ["sgd", "momentum", "adam"])
def test_optimizers_match_torch_optim(kind):
    rng = np.random.default_rng(4)
    theta0 = rng.standard_normal(500) * 0.02
    grads = [rng.standard_normal(500) * 1e-3 for _ in range(6)]
    grads[2][:10] = 0.0  # exact zero gradients
    hp = dict(lr=3e-4, momentum=0.9, beta1=0.9, beta2=0.95, eps=1e-8)
    th = theta0.copy()
    m = np.zeros(500)
    v = np.zeros(500)
    for t, gv in enumerate(grads):
        if kind == "sgd":
            th = step.sgd(th, gv, hp["lr"])
        elif kind == "momentum":
            th, m = step.sgd_momentum(th, m, gv, hp["lr"], hp["momentum"])
        else:
            th, m, v = step.adam(th, m, v, gv, t + 1, hp["lr"], hp["beta1"],
                                 hp["beta2"], hp["eps"])
    want = _torch_opt_run(kind, grads, theta0, **hp)
    assert np.allclose(th, want, rtol=1e-13, atol=1e-17)


def test_broadcast_no_loss_is_all_gather_and_full_loss_is_identity():
    rng = np.random.default_rng(5)
    old = rng.standard_normal((4, 50))
    new = rng.standard_normal(50)
    R1 = np.ones((4, 50), dtype=np.uint8)
    assert np.array_equal(step.broadcast(old, new[None, :], R1), np.repeat(new[None], 4, 0))
    R0 = np.zeros((4, 50), dtype=np.uint8)
    assert np.array_equal(step.broadcast(old, new[None, :], R0), old)
    R = (rng.random((4, 50)) < 0.5).astype(np.uint8)
    out = step.broadcast(old, new[None, :], R)
    for i in range(4):
        for e in range(50):
            assert out[i, e] == (new[e] if R[i, e] else old[i, e])


def _small_case(n=4, d=10, L=4, gdtype="f32"):
    rng = np.random.default_rng(6)
    g = rng.standard_normal((n, d)).astype(np.float32)
    theta = (rng.standard_normal(d) * 0.02).astype(np.float32)
    if gdtype == "bf16":
        g = bf16.from_f32(g)
        reps = np.repeat(bf16.from_f32(theta)[None], n, 0)
    else:
        reps = np.repeat(theta[None], n, 0)
    return g, theta, reps


@pytest.mark.parametrize("gdtype", ["f32", "bf16"])
def test_step_without_loss_is_sgd_on_the_mean(gdtype):
    n, d, L = 4, 10, 4
    g, theta, reps = _small_case(n, d, L, gdtype)
    P = 3
    ones = np.ones((n, P), dtype=np.uint8)
    out = step.lossy_step(d=d, packet=L, packets=range(P), gdtype=gdtype, grads=g,
                          theta=theta, m=None, v=None, replicas=reps, arrived_g=ones,
                          arrived_b=ones, opt=dict(kind="sgd", lr=0.01), t=0)
    g64 = step.widen(g, gdtype)
    want = (theta.astype(np.float64) - 0.01 * np.mean(g64, axis=0).astype(np.float32)
            .astype(np.float64)).astype(np.float32)
    assert np.array_equal(out["theta"], want)
    cast = bf16.from_f32(want) if gdtype == "bf16" else want
    assert np.array_equal(out["replicas"], np.repeat(cast[None], n, 0))
    assert out["counts"].tolist() == [n] * P


def test_step_with_total_loss_keeps_everything():
    n, d, L = 3, 9, 4
    g, theta, reps = _small_case(n, d, L)
    reps = reps + np.float32(1.0)  # stale replicas differ from the master
    zeros = np.zeros((n, 3), dtype=np.uint8)
    out = step.lossy_step(d=d, packet=L, packets=range(3), gdtype="f32", grads=g,
                          theta=theta, m=None, v=None, replicas=reps, arrived_g=zeros,
                          arrived_b=zeros, opt=dict(kind="sgd", lr=0.01), t=0)
    assert np.array_equal(out["theta"], theta)
    assert np.array_equal(out["replicas"], reps)
    assert (out["g_hat"] == 0).all() and out["counts"].tolist() == [0, 0, 0]
