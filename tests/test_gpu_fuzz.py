"""Seeded random configurations of the fused step against the oracle: worker
counts across mask-word boundaries, packet sizes from 8 elements up, ragged
shards, both row types, every optimizer, loss process, estimator and
delivery override, two steps each.  Every packet is compared, masks and
counts bit-exact, and drift against the oracle's drift of the same
replicas."""
import numpy as np
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl
from oracle import drift as odrift
from oracle import loss as oloss
from oracle import step as ostep

import parity

pytestmark = pytest.mark.gpu
DEV = "cuda"

OPTS = {
    "sgd": dict(kind=wl.SGD, lr=0.01, momentum=0.0, beta1=0.0, beta2=0.0, eps=0.0),
    "momentum": dict(kind=wl.MOMENTUM, lr=0.01, momentum=0.9, beta1=0.0, beta2=0.0, eps=0.0),
    "adam": dict(wl.ADAM_DEFAULT),
}


def _cases(count=96, seed=2026):
    rng = np.random.default_rng(seed)
    out = []
    for c in range(count):
        n = int(rng.choice([1, 2, 3, 7, 8, 33, 63, 64, 65, 130]))
        packet = int(rng.choice([8, 16, 24, 1000, 1024, 2048, 4104, 8192]))
        d = int(rng.integers(1, 40_000))
        gdtype = str(rng.choice([wl.F32, wl.BF16]))
        opt = str(rng.choice(list(OPTS)))
        if rng.random() < 0.2:
            loss = dict(kind=wl.GILBERT_ELLIOTT, p_gb=float(rng.choice([0.05, 0.3])),
                        p_bg=float(rng.choice([0.2, 0.6])), loss_good=0.0,
                        loss_bad=float(rng.choice([0.5, 1.0])))
        else:
            loss = dict(kind=wl.BERNOULLI, p=float(rng.choice([0.0, 0.05, 0.5, 0.95, 1.0])))
        bern = loss["kind"] == wl.BERNOULLI
        est = str(rng.choice(["arrived_mean", "arrived_mean", "horvitz_thompson", "stale_fill"]))
        if est == "horvitz_thompson" and bern and loss["p"] == 1.0:
            est = "arrived_mean"
        owner = int(rng.integers(0, n)) if rng.random() < 0.3 else -1
        reliable = bool(rng.random() < 0.3)
        parity_g = int(rng.choice([1, 2, 5, 16])) if (bern and rng.random() < 0.3) else 0
        lam = 0.1 if (est == "arrived_mean" and rng.random() < 0.3) else 0.0
        out.append(dict(case=c, n=n, packet=packet, d=d, gdtype=gdtype, opt=opt, loss=loss,
                        est=est, owner=owner, reliable=reliable, parity=parity_g, lam=lam))
    return out


CASES = _cases()
# the largest worker count, on every path of the kernel that depends on it
CASES += [
    dict(case=1000, n=1024, packet=512, d=3000, gdtype=wl.BF16, opt="adam",
         loss=dict(kind=wl.BERNOULLI, p=0.3), est="horvitz_thompson", owner=1023,
         reliable=True, parity=3, lam=0.0),
    dict(case=1001, n=1024, packet=1000, d=2500, gdtype=wl.F32, opt="momentum",
         loss=dict(kind=wl.GILBERT_ELLIOTT, p_gb=0.3, p_bg=0.2, loss_good=0.0, loss_bad=1.0),
         est="stale_fill", owner=-1, reliable=False, parity=0, lam=0.0),
    dict(case=1002, n=1024, packet=8, d=77, gdtype=wl.BF16, opt="sgd",
         loss=dict(kind=wl.BERNOULLI, p=0.95), est="arrived_mean", owner=-1,
         reliable=False, parity=1, lam=0.1),
]
# Horvitz-Thompson with each packet's probability derived from the chain
CASES += [
    dict(case=1003, n=16, packet=1024, d=30_000, gdtype=wl.F32, opt="momentum",
         loss=dict(kind=wl.GILBERT_ELLIOTT, p_gb=0.05, p_bg=0.3, loss_good=0.02, loss_bad=0.6),
         est="horvitz_thompson", owner=3, reliable=True, parity=0, lam=0.0),
    dict(case=1004, n=65, packet=24, d=5_000, gdtype=wl.BF16, opt="adam",
         loss=dict(kind=wl.GILBERT_ELLIOTT, p_gb=0.7, p_bg=0.6, loss_good=0.1, loss_bad=0.9),
         est="horvitz_thompson", owner=-1, reliable=False, parity=0, lam=0.0),
]


def _masks(w, t, direction, state, owner, relf, G):
    l = w.loss
    P = w.num_packets
    if l["kind"] == wl.BERNOULLI:
        a = oloss.bernoulli_arrivals(w.seed, t, direction, w.n, np.arange(P), l["p"])
    else:
        a, state[direction] = oloss.ge_arrivals(w.seed, t, direction, w.n, P, l["p_gb"],
                                                l["p_bg"], l["loss_good"], l["loss_bad"],
                                                state[direction])
    a = oloss.apply_overrides(a, owner, relf)
    if G:
        par = oloss.parity_arrivals(w.seed, t, direction, w.n, np.arange((P + G - 1) // G), l["p"])
        a = oloss.parity_recover(a, G, par)
    return a


@pytest.mark.parametrize("cfg", CASES, ids=lambda c: f"case{c['case']}")
def test_random_configuration(cfg):
    base = wl.WORKLOADS["n8_d16m_bf16_adam"]
    w = wl.scaled(base, n=cfg["n"], d=cfg["d"], packet=cfg["packet"], steps=2,
                  gdtype=cfg["gdtype"], loss=cfg["loss"], opt=OPTS[cfg["opt"]])
    print(f"fuzz {cfg}", flush=True)
    P = w.num_packets
    dev = parity.DeviceState(w, pad=8 * (cfg["case"] % 3))
    relf = None
    if cfg["reliable"]:
        relf = np.zeros(P, np.uint8)
        relf[cfg["case"] % 3::4] = 1
    est, owner, G = cfg["est"], cfg["owner"], cfg["parity"]
    l = w.loss
    if l["kind"] == wl.BERNOULLI:
        q_lossy = 1.0 - l["p"]
    else:
        pi_bad = l["p_gb"] / (l["p_gb"] + l["p_bg"])
        q_lossy = 1 - pi_bad * l["loss_bad"] - (1 - pi_bad) * l["loss_good"]
    prev = torch.zeros_like(dev.grads) if est == "stale_fill" else None
    # The fused step derives q per packet: Bernoulli 1 - p (per packet under
    # parity packets), Gilbert-Elliott the chain's marginal at that packet;
    # a chain state that loses everything needs q given (the stationary one).
    ge_given = l["kind"] != wl.BERNOULLI and not (l["loss_good"] < 1 and l["loss_bad"] < 1)
    e = ll.ext(estimator=est, owner=owner,
               reliable=None if relf is None else torch.from_numpy(relf).to(DEV),
               g_prev=prev,
               arrival_prob=q_lossy if (est == "horvitz_thompson" and ge_given) else 0.0,
               parity_group=G)

    def q_of(t):
        if l["kind"] == wl.BERNOULLI and G:
            q = np.tile(oloss.parity_arrival_probabilities(q_lossy, G, P, relf), (w.n, 1))
        elif l["kind"] == wl.BERNOULLI or ge_given:
            q = np.full((w.n, P), q_lossy)
        else:
            q = np.tile(oloss.ge_arrival_probability(t, np.arange(P), P, l["p_gb"], l["p_bg"],
                                                     l["loss_good"], l["loss_bad"]), (w.n, 1))
        if owner >= 0:
            q[owner] = 1.0
        if relf is not None:
            q[:, relf.astype(bool)] = 1.0
        return q
    packets = list(range(P))
    so = parity.SampledOracle(w, packets, dev)
    prev_o = np.zeros((w.n, w.d), np.uint16 if w.gdtype == wl.BF16 else np.float32)
    state = {0: np.zeros(w.n, np.uint8), 1: np.zeros(w.n, np.uint8)}
    for t in range(w.steps):
        if t > 0:
            wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(t, lam=cfg["lam"], ext=e)
        mg = _masks(w, t, 0, state, owner, relf, G)
        mb = _masks(w, t, 1, state, owner, relf, G)
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg), f"step {t} gradient masks"
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb), f"step {t} broadcast masks"
        assert np.array_equal(dev.counts.cpu().numpy(), mg.sum(axis=0)), f"step {t} counts"
        orc = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype,
                               grads=g_host, theta=so.theta, m=so.m, v=so.v,
                               replicas=so.replicas, arrived_g=mg, arrived_b=mb, opt=parity.opt_as_given(w.opt), t=t,
                               lam=cfg["lam"], estimator=est, q=q_of(t), g_prev=prev_o)
        so.advance(orc)
        parity.compare_step(w, t, dev, so, orc, mb, f"case {cfg['case']} step {t}")
        # drift of the device's own replicas, recomputed by the oracle
        reps = parity.host_rows(dev.replicas, so.idx, w.gdtype)
        th = parity.host_vec(dev.theta, so.idx)
        ref = odrift.drift_stats(ostep.widen(reps, w.gdtype),
                                 ostep.widen(parity.cast_bits(th, w.gdtype), w.gdtype), mb)
        r = ll.read_drift(dev.drift)
        assert r["max_abs"] == ref["max_abs"], (t, r, ref)
        assert abs(r["mean_sq"] - ref["mean_sq"]) <= 1e-9 * ref["mean_sq"] + 1e-300, (t, r, ref)
        assert abs(r["mean_abs_to_master"] - ref["mean_abs_to_master"]) <= \
            1e-9 * ref["mean_abs_to_master"] + 1e-300, (t, r, ref)
        assert r["stale_packets"] == ref["stale_packets"]
        assert r["empty_packets"] == int((mg.sum(axis=0) == 0).sum())
        if est == "stale_fill":
            prev_o = orc["g_prev"]
        so.upload(dev)
