"""The fused step: bit-identical to the stage-by-stage chain, parity with the
oracle on scaled-down workloads (several tiles and a ragged tail), edge
cases, determinism and exact resume."""

import numpy as np
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl
from oracle import drift as odrift
from oracle import step as ostep

import parity

pytestmark = pytest.mark.gpu
DEV = "cuda"

SMALL = {
    # the five workloads at sizes the oracle finishes in seconds, with tails
    "n4_d1m_f32_sgd": dict(d=1_048_576 - 1000),
    "n8_d16m_bf16_adam": dict(d=300_003, steps=4),
    "n64_llama7b_shard_bf16_adam": dict(d=105_250_000 // 400 + 5),
    "n16_d256m_f32_ge_momentum": dict(d=4096 * 300 + 2056, steps=3),
    "n64_d48m_f32_sgd_drift": dict(d=2048 * 97 + 1000, steps=3),
}


def _small(name):
    return wl.scaled(wl.WORKLOADS[name], **SMALL[name])


def _stagewise(dev: parity.DeviceState, step: int):
    """The same step through the one-stage entry points."""
    w = dev.w
    spec = parity.loss_spec(w)
    P = w.num_packets
    g_hat = torch.empty(w.d, dtype=torch.float32, device=DEV)
    ll.ll_masks(w.n, P, step, ll.LL_DIR_GRAD, spec, dev.arrived_g, ge_state=dev.ge_g,
                workspace=dev.workspace)
    ll.lossy_aggregate(dev.grads, dev.arrived_g, d=w.d, packet=w.packet, g_hat=g_hat,
                       counts=dev.counts, theta=dev.theta)
    ll.shard_step(parity.opt_spec(w), step, dev.theta, g_hat, m=dev.m, v=dev.v)
    ll.ll_masks(w.n, P, step, ll.LL_DIR_BCAST, spec, dev.arrived_b, ge_state=dev.ge_b,
                workspace=dev.workspace)
    ll.lossy_broadcast(dev.theta, dev.replicas, dev.arrived_b, d=w.d, packet=w.packet)
    ll.drift_stats(dev.replicas, d=w.d, packet=w.packet, workspace=dev.workspace,
                   out=dev.drift, theta=dev.theta, arrived_bc=dev.arrived_b)


def _snapshot(dev: parity.DeviceState):
    out = {k: getattr(dev, k).clone() for k in ("theta", "replicas", "arrived_g", "arrived_b",
                                                "counts", "ge_g", "ge_b")}
    for k in ("m", "v"):
        if getattr(dev, k) is not None:
            out[k] = getattr(dev, k).clone()
    out["drift"] = ll.read_drift(dev.drift)
    return out


def _bit_equal(a: torch.Tensor, b: torch.Tensor) -> bool:
    if a.dtype in (torch.float32, torch.bfloat16, torch.float64):
        a = a.view(torch.int32 if a.dtype == torch.float32 else
                   torch.int16 if a.dtype == torch.bfloat16 else torch.int64)
        b = b.view(a.dtype)
    return torch.equal(a, b)


@pytest.mark.parametrize("name", list(SMALL))
def test_fused_is_bit_identical_to_stagewise(name):
    w = _small(name)
    print(f"fused vs stagewise {name} d={w.d}", flush=True)
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    for t in range(2):
        wl.draw_grads(w, t, device=DEV, ld=a.ld, out=a.grads)
        b.grads.copy_(a.grads)
        a.fused(t)
        _stagewise(b, t)
        sa, sb = _snapshot(a), _snapshot(b)
        stale = sa["drift"]["stale_packets"]
        # the empty-packet count is only produced by the fused step
        sa["drift"]["empty_packets"] = sb["drift"]["empty_packets"] = 0
        assert sa["drift"] == sb["drift"], (sa["drift"], sb["drift"])
        for k in sa:
            if k != "drift":
                assert _bit_equal(sa[k], sb[k]), f"{name} step {t}: {k} differs"
        assert stale == int((sa["arrived_b"] == 0).sum())


@pytest.mark.parametrize("name,rdtype", [("n8_d16m_bf16_adam", torch.float32),
                                         ("n64_d48m_f32_sgd_drift", torch.bfloat16),
                                         ("n16_d256m_f32_ge_momentum", torch.bfloat16)])
def test_mixed_row_dtypes_fused_bit_identical_to_stagewise(name, rdtype):
    # Gradient and replica rows of different types (the other two of the four
    # type pairs the library compiles): the fused step against the chain of
    # one-stage calls, each of which is compared with the oracle per type.
    w = _small(name)
    print(f"mixed dtypes {name}: grads {w.gdtype}, replicas {rdtype}", flush=True)
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    for dev in (a, b):
        dev.replicas = torch.zeros((w.n, dev.ld), dtype=rdtype, device=DEV)
        dev.replicas[:, : w.d] = dev.theta.to(rdtype)[None, :]
    for t in range(2):
        wl.draw_grads(w, t, device=DEV, ld=a.ld, out=a.grads)
        b.grads.copy_(a.grads)
        a.fused(t)
        _stagewise(b, t)
        sa, sb = _snapshot(a), _snapshot(b)
        sa["drift"]["empty_packets"] = sb["drift"]["empty_packets"] = 0
        assert sa["drift"] == sb["drift"], (sa["drift"], sb["drift"])
        for k in sa:
            if k != "drift":
                assert _bit_equal(sa[k], sb[k]), f"{name} step {t}: {k} differs"
        R = a.arrived_b.repeat_interleave(w.packet, dim=1)[:, : w.d].bool()
        own = a.theta.to(rdtype)[None, :].expand(w.n, -1)
        assert _bit_equal(a.replicas[:, : w.d][R], own[R]), "arrived replica != rounded master"


@pytest.mark.parametrize("name", list(SMALL))
def test_fused_parity_with_oracle(name):
    w = _small(name)
    dev = parity.DeviceState(w, pad=8)
    packets = list(range(w.num_packets))
    so = parity.SampledOracle(w, packets, dev)
    om = parity.OracleMasks(w)
    for t in range(w.steps):
        print(f"fused parity {name} d={w.d} step {t}", flush=True)
        if t > 0:
            wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(t)
        mg, mb = om.masks(t, 0), om.masks(t, 1)
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg), "gradient masks"
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb), "broadcast masks"
        assert np.array_equal(dev.counts.cpu().numpy(), mg.sum(axis=0)), "counts"
        if w.loss["kind"] == wl.GILBERT_ELLIOTT:
            assert np.array_equal(dev.ge_g.cpu().numpy(), om.state[0])
            assert np.array_equal(dev.ge_b.cpu().numpy(), om.state[1])
        orc = so.step(t, g_host, mg, mb)
        parity.compare_step(w, t, dev, so, orc, mb, f"{name} step {t}")
        # drift of the oracle's replicas vs the device's, bounded by the
        # replica tolerance propagated through the pair sum
        got = ll.read_drift(dev.drift)
        x = ostep.widen(orc["replicas"], w.gdtype)
        want = odrift.drift_stats(x, ostep.widen(ostep.store(orc["theta"], w.gdtype), w.gdtype), mb)
        assert got["stale_packets"] == want["stale_packets"]
        assert got["empty_packets"] == int((mg.sum(axis=0) == 0).sum())
        lens = ostep.packet_lengths(w.d, w.packet, packets)
        K_elem = np.repeat(orc["counts"], lens)
        tol_th = parity.state_bounds(parity.opt_as_given(w.opt), t, orc, so.prev, K_elem)["theta"]
        tol = np.where(np.repeat(mb, lens, axis=1).astype(bool),
                       (parity.BF16_REL * np.abs(x) if w.gdtype == wl.BF16 else 0) + tol_th, 0.0)
        dev_pair = 0.0
        for i in range(w.n - 1):
            diff = np.abs(x[i + 1:] - x[i][None, :])
            tt = tol[i + 1:] + tol[i][None, :]
            dev_pair += float(np.sum(2 * diff * tt + tt * tt))
        pairs = w.n * (w.n - 1) / 2
        assert abs(got["mean_sq"] - want["mean_sq"]) <= dev_pair / (w.d * pairs) + 1e-12 * want["mean_sq"]
        assert abs(got["max_abs"] - want["max_abs"]) <= 2 * float(tol.max(initial=0.0)) + 1e-300
        # the next step starts both sides from the oracle's state
        so.upload(dev)


def test_no_loss_is_allreduce_mean_and_allgather():
    # p = 0: the aggregate is the mean (reduce-scatter SUM / N), the broadcast
    # is an all-gather (every replica = the new master), drift is zero.
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], d=50_000, loss=dict(kind=wl.BERNOULLI, p=0.0),
                  opt=dict(kind=wl.SGD, lr=0.01, momentum=0, beta1=0, beta2=0, eps=0))
    dev = parity.DeviceState(w)
    # gradients k * 2^-12 with |k| < 128: exact in bf16, and any sum of 8 of
    # them is exact in fp32, so the mean below is the exact mean.
    q = torch.randint(-127, 128, (w.n, w.d), device=DEV, generator=torch.Generator(DEV).manual_seed(1))
    dev.grads[:, : w.d] = (q.float() * 2.0**-12).to(torch.bfloat16)
    th0 = dev.theta.clone()
    mean = dev.grads[:, : w.d].double().sum(0).div(w.n).float()
    dev.fused(0)
    want = th0 - 0.01 * mean
    assert torch.equal(dev.theta, want)
    assert torch.equal(dev.replicas[:, : w.d], want.to(torch.bfloat16).unsqueeze(0).expand(w.n, -1))
    r = ll.read_drift(dev.drift)
    assert r["max_abs"] == 0 and r["mean_sq"] == 0 and r["stale_packets"] == 0
    assert r["mean_abs_to_master"] == 0 and r["empty_packets"] == 0


@pytest.mark.parametrize("lam", [0.0, 0.5])
def test_total_loss_falls_back_and_keeps_replicas(lam):
    w = wl.scaled(wl.WORKLOADS["n4_d1m_f32_sgd"], d=20_000, loss=dict(kind=wl.BERNOULLI, p=1.0))
    dev = parity.DeviceState(w)
    th0 = dev.theta.clone()
    rep0 = dev.replicas.clone()
    dev.fused(0, lam=lam)
    want = th0 - w.opt["lr"] * (lam * th0) if lam else th0
    assert torch.equal(dev.theta, want)
    assert torch.equal(dev.replicas, rep0)
    r = ll.read_drift(dev.drift)
    assert r["empty_packets"] == w.num_packets
    assert r["stale_packets"] == w.n * w.num_packets
    assert int(dev.counts.sum()) == 0


def test_empty_shard_and_one_worker():
    w = wl.scaled(wl.WORKLOADS["n4_d1m_f32_sgd"], d=0)
    dev = parity.DeviceState(w)
    dev.drift.fill_(7.0)
    dev.fused(0)
    r = ll.read_drift(dev.drift)
    assert r == dict(max_abs=0.0, mean_sq=0.0, rms=0.0, mean_abs_to_master=0.0,
                     stale_packets=0, empty_packets=0)
    w1 = wl.scaled(wl.WORKLOADS["n4_d1m_f32_sgd"], n=1, d=5000)
    dev1 = parity.DeviceState(w1)
    dev1.fused(0)
    assert ll.read_drift(dev1.drift)["mean_sq"] == 0.0


def test_deterministic_rerun():
    w = _small("n64_llama7b_shard_bf16_adam")
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    a.fused(0)
    b.fused(0)
    sa, sb = _snapshot(a), _snapshot(b)
    assert sa["drift"] == sb["drift"]
    for k in sa:
        if k != "drift":
            assert _bit_equal(sa[k], sb[k]), k


@pytest.mark.parametrize("name", ["n16_d256m_f32_ge_momentum", "n8_d16m_bf16_adam"])
def test_resume_is_exact(name):
    # Ten steps straight equal five steps, a copy of the whole state (master,
    # moments, replicas, GE chain state) into fresh buffers, and five more.
    w = wl.scaled(_small(name), steps=10)
    a = parity.DeviceState(w)
    for t in range(10):
        wl.draw_grads(w, t, device=DEV, ld=a.ld, out=a.grads)
        a.fused(t)
    b = parity.DeviceState(w)
    for t in range(5):
        wl.draw_grads(w, t, device=DEV, ld=b.ld, out=b.grads)
        b.fused(t)
    c = parity.DeviceState(w)
    for k in ("theta", "m", "v", "replicas", "ge_g", "ge_b"):
        if getattr(b, k) is not None:
            getattr(c, k).copy_(getattr(b, k))
    del b
    for t in range(5, 10):
        wl.draw_grads(w, t, device=DEV, ld=c.ld, out=c.grads)
        c.fused(t)
    sa, sc = _snapshot(a), _snapshot(c)
    for k in sa:
        if k != "drift":
            assert _bit_equal(sa[k], sc[k]), k
    assert sa["drift"] == sc["drift"]


def test_logged_masks_replay_the_step():
    # The exported masks are a per-(worker, packet) routing log: feeding them
    # to the stage-by-stage path reproduces the step bit-for-bit.
    w = _small("n8_d16m_bf16_adam")
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    a.fused(3)
    P = w.num_packets
    g_hat = torch.empty(w.d, dtype=torch.float32, device=DEV)
    ll.lossy_aggregate(b.grads, a.arrived_g, d=w.d, packet=w.packet, g_hat=g_hat)
    ll.shard_step(parity.opt_spec(w), 3, b.theta, g_hat, m=b.m, v=b.v)
    ll.lossy_broadcast(b.theta, b.replicas, a.arrived_b, d=w.d, packet=w.packet)
    assert P > 0
    for k in ("theta", "m", "v", "replicas"):
        assert _bit_equal(getattr(a, k), getattr(b, k)), k
