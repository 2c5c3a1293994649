"""The GPU parity norms (tests/parity.py) are as tight as the arithmetic: on the
CPU, an fp32 emulation of the library's order of operations passes them, and
an update that differs from the oracle's by a 5% learning-rate error, or a
missing update, fails them, on the shapes and value ranges of the workloads
(the 200-step fp32 SGD drift workload above all, whose per-step update is
smaller than 1e-5 of its parameters)."""
import numpy as np
import pytest

import workloads as wl
from oracle import loss as oloss
from oracle import step as ostep

import parity

F = np.float32


def _emulate(g_rows: np.ndarray, S: np.ndarray, theta, m, v, opt: dict, t: int):
    """fp32 in the library's order: arrived rows summed in ascending worker
    order, divided by their count; the update's operations one rounding each."""
    acc = np.zeros(g_rows.shape[1], F)
    for i in range(g_rows.shape[0]):
        acc = np.where(S[i], acc + g_rows[i], acc).astype(F)
    K = S.sum(axis=0)
    g = np.where(K > 0, acc / np.maximum(K, 1).astype(F), F(0)).astype(F)
    lr = F(opt["lr"])
    if opt["kind"] == "sgd":
        return g, theta - lr * g, None, None
    if opt["kind"] == "momentum":
        m1 = F(opt["momentum"]) * m + g
        return g, theta - lr * m1, m1, None
    b1, b2, eps = F(opt["beta1"]), F(opt["beta2"]), F(opt["eps"])
    a1, a2 = F(1) - b1, F(1) - b2
    bc1 = F(1.0 - float(b1) ** (t + 1))
    bc2 = F(1.0 - float(b2) ** (t + 1))
    m1 = b1 * m + a1 * g
    v1 = b2 * v + a2 * (g * g)
    th1 = theta - lr * ((m1 / bc1) / (np.sqrt(v1 / bc2) + eps))
    return g, th1, m1, v1


CASES = {
    # workload, packets sampled, steps run before the checked one
    "n64_d48m_f32_sgd_drift": (48, 0),
    "n16_d256m_f32_ge_momentum": (6, 2),
    "n64_llama7b_shard_bf16_adam": (12, 2),
    "n8_d16m_bf16_adam": (24, 0),
    "n4_d1m_f32_sgd": (64, 0),
}


def _setup(name):
    w = wl.WORKLOADS[name]
    n_packets, warm = CASES[name]
    rng = np.random.default_rng(11)
    packets = list(range(n_packets))
    lens = ostep.packet_lengths(w.d, w.packet, packets)
    E = int(lens.sum())
    opt = parity.opt_as_given(w.opt)
    theta = (rng.standard_normal(E) * w.theta_std).astype(F)
    m = np.zeros(E, F) if opt["kind"] in ("momentum", "adam") else None
    v = np.zeros(E, F) if opt["kind"] == "adam" else None
    reps = ostep.store(theta.astype(np.float64), w.gdtype)[None, :].repeat(w.n, axis=0)
    p = w.loss.get("p", 0.05)
    scale = w.grad[-1]

    def grads():
        x = rng.standard_normal((w.n, E)) if w.grad[0] == "normal" else rng.standard_t(3, (w.n, E))
        return ostep.store(x * scale, w.gdtype)

    def masks(t, direction):
        return oloss.bernoulli_arrivals(w.seed, t, direction, w.n, packets, p)

    for t in range(warm):
        out = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype,
                               grads=grads(), theta=theta, m=m, v=v, replicas=reps,
                               arrived_g=masks(t, 0), arrived_b=masks(t, 1), opt=opt, t=t)
        theta, m, v, reps = out["theta"], out["m"], out["v"], out["replicas"]
    t = warm
    g = grads()
    mg = masks(t, 0)
    return w, opt, t, packets, lens, g, mg, masks(t, 1), theta, m, v, reps


@pytest.mark.parametrize("name", list(CASES))
def test_norms_accept_fp32_and_reject_a_mis_scaled_update(name):
    w, opt, t, packets, lens, g, mg, mb, theta, m, v, reps = _setup(name)
    orc = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype, grads=g,
                           theta=theta, m=m, v=v, replicas=reps, arrived_g=mg, arrived_b=mb,
                           opt=opt, t=t)
    prev = dict(theta=theta, m=m, v=v)
    S = np.repeat(mg, lens, axis=1).astype(bool)
    g32 = ostep.widen(g, w.gdtype).astype(F)
    g_em, th_em, m_em, v_em = _emulate(g32, S, theta, m, v, opt, t)
    K_elem = np.repeat(orc["counts"], lens)
    parity.check_ghat(g_em, orc["g_hat"], orc["mean_abs"], K_elem)
    b = parity.state_bounds(opt, t, orc, prev, K_elem)
    parity.check_close(th_em, orc["theta"], b["theta"], "theta")
    if m is not None:
        parity.check_close(m_em, orc["m"], b["m"], "m")
    if v is not None:
        parity.check_close(v_em, orc["v"], b["v"], "v")

    # the rounding part is what resolves the update: how much of it is left
    step = np.abs(orc["theta"].astype(np.float64) - theta.astype(np.float64))
    assert float(np.median(b["theta"] / np.maximum(step, 1e-300))) < 0.05

    bad = dict(opt, lr=opt["lr"] * 1.05)
    wrong = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype, grads=g,
                             theta=theta, m=m, v=v, replicas=reps, arrived_g=mg, arrived_b=mb,
                             opt=bad, t=t)
    with pytest.raises(AssertionError):
        parity.check_close(wrong["theta"], orc["theta"], b["theta"], "theta, lr x 1.05")
    with pytest.raises(AssertionError):
        parity.check_close(theta, orc["theta"], b["theta"], "theta, no update")


def test_ghat_norm_holds_at_1e5_for_a_thousand_workers():
    # 1024 rows of either sign summed in fp32 in ascending order: the realised
    # error stays well inside 1e-5 of the mean magnitude, without the K u
    # worst case.
    rng = np.random.default_rng(3)
    n, E = 1024, 20_000
    g = (rng.standard_normal((n, E)) * 1e-3).astype(F)
    S = rng.random((n, E)) > 0.1
    g_em = _emulate(g, S, np.zeros(E, F), None, None, dict(kind="sgd", lr=0.0), 0)[0]
    want, K, mean_abs = ostep.aggregate(g.astype(np.float64), S, 0.0, np.zeros(E))
    parity.check_ghat(g_em, want.astype(F), mean_abs, K)
    err = np.abs(g_em.astype(np.float64) - want) / mean_abs
    assert float(err.max()) < 2e-6
