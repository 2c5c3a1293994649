"""The five workloads at full size, in the launch configuration the benchmark
times (fused step with drift): masks and counts bit-exact over every packet,
sampled packets compared with the oracle step by step, the whole shard's
drift figures against plain torch fp64 arithmetic, and the long-run drift of
Theorem 3.1 on the 200-step N=64 workload."""
import gc
import math

import numpy as np
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl

import parity

pytestmark = pytest.mark.gpu
DEV = "cuda"

FULL_STEPS = {
    "n4_d1m_f32_sgd": 1,
    "n8_d16m_bf16_adam": 10,
    "n64_llama7b_shard_bf16_adam": 1,
    "n16_d256m_f32_ge_momentum": 5,
    "n64_d48m_f32_sgd_drift": 3,
}


def _free():
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", list(FULL_STEPS))
def test_full_size_sampled_parity(name):
    w = wl.WORKLOADS[name]
    print(f"full-size parity {name}: n={w.n} d={w.d} P={w.num_packets}", flush=True)
    dev = parity.DeviceState(w)
    packets = wl.packet_sample(w, 24)
    assert w.num_packets - 1 in packets
    so = parity.SampledOracle(w, packets, dev)
    om = parity.OracleMasks(w)
    try:
        for t in range(FULL_STEPS[name]):
            if t > 0:
                wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
            g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
            dev.fused(t)
            mg, mb = om.masks(t, 0), om.masks(t, 1)
            assert np.array_equal(dev.arrived_g.cpu().numpy(), mg), f"step {t} gradient masks"
            assert np.array_equal(dev.arrived_b.cpu().numpy(), mb), f"step {t} broadcast masks"
            K = mg.sum(axis=0)
            assert np.array_equal(dev.counts.cpu().numpy(), K), f"step {t} counts"
            r = ll.read_drift(dev.drift)
            assert r["stale_packets"] == int((mb == 0).sum())
            assert r["empty_packets"] == int((K == 0).sum())
            assert math.isfinite(r["mean_sq"]) and r["mean_sq"] >= 0
            # the whole shard's drift figures, recomputed by plain torch fp64
            parity.check_drift_close(r, parity.torch_drift(dev.replicas, dev.theta, w.d),
                                     f"{name} step {t} drift")
            orc = so.step(t, g_host, mg, mb)
            parity.compare_step(w, t, dev, so, orc, mb[:, packets], f"{name} step {t}")
            so.upload(dev)
            print(f"  step {t} ok: drift rms={r['rms']:.3e} max={r['max_abs']:.3e}", flush=True)
    finally:
        del dev
        _free()


def test_long_run_drift_is_bounded():
    # Theorem 3.1 as corrected for both replicas' staleness: with independent
    # per-step master increments of variance sigma^2 and i.i.d. broadcast
    # loss p, the stationary mean squared inter-replica discrepancy is
    # 2p / (1 - p^2) * sigma^2 (the paper prints 2p / (1 + p)).
    w = wl.WORKLOADS["n64_d48m_f32_sgd_drift"]
    p = w.loss["p"]
    dev = parity.DeviceState(w)
    prev = dev.theta.clone()
    ms, sig = [], []
    try:
        for t in range(w.steps):
            if t > 0:
                wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
            dev.fused(t)
            r = ll.read_drift(dev.drift)
            step = (dev.theta - prev).double()
            sig.append(float(step.square().mean()))
            prev.copy_(dev.theta)
            ms.append(r["mean_sq"])
            if t % 50 == 0:
                print(f"  step {t}: mean_sq={r['mean_sq']:.4e} sigma2={sig[-1]:.4e}", flush=True)
    finally:
        del dev
        _free()
    burn = 50
    ms = np.array(ms[burn:])
    s2 = float(np.mean(sig[burn:]))
    corrected = 2 * p / (1 - p * p)
    paper = 2 * p / (1 + p)
    ratio = float(ms.mean()) / s2
    print(f"stationary E[D^2]/sigma^2 = {ratio:.4f}; 2p/(1-p^2) = {corrected:.4f}; "
          f"paper's 2p/(1+p) = {paper:.4f}", flush=True)
    assert abs(ratio - corrected) < 0.03 * corrected
    half = len(ms) // 2
    assert abs(ms[:half].mean() - ms[half:].mean()) < 0.03 * ms.mean()  # no growth


def test_drift_workload_all_steps_on_a_packet_slice():
    # Every one of the 200 steps of the N=64 drift workload at full size on
    # the GPU; the oracle follows a slice of four packets (restarted from the
    # device's state each step, so fp32 rounding order cannot accumulate),
    # and drift_stats on the slice's sub-view is compared with the oracle's
    # drift of the same replicas.
    from oracle import drift as odrift
    from oracle import loss as oloss
    w = wl.WORKLOADS["n64_d48m_f32_sgd_drift"]
    assert w.loss["kind"] == wl.BERNOULLI and w.gdtype == wl.F32
    packets = [0, 1, 2, 3]
    e1 = len(packets) * w.packet
    dev = parity.DeviceState(w)
    so = parity.SampledOracle(w, packets, dev)
    out = ll.drift_buffer()
    try:
        for t in range(w.steps):
            if t > 0:
                wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
            g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
            dev.fused(t)
            mg = oloss.bernoulli_arrivals(w.seed, t, 0, w.n, packets, w.loss["p"])
            mb = oloss.bernoulli_arrivals(w.seed, t, 1, w.n, packets, w.loss["p"])
            assert np.array_equal(dev.arrived_g[:, packets].cpu().numpy(), mg), f"step {t}"
            assert np.array_equal(dev.arrived_b[:, packets].cpu().numpy(), mb), f"step {t}"
            orc = so.step(t, g_host, mg, mb)
            parity.compare_step(w, t, dev, so, orc, mb, f"slice step {t}")
            ll.drift_stats(dev.replicas[:, :e1], d=e1, packet=w.packet, workspace=dev.workspace,
                           out=out, theta=dev.theta[:e1])
            r = ll.read_drift(out)
            x = parity.host_rows(dev.replicas, so.idx, w.gdtype).astype(np.float64)
            ref = odrift.drift_stats(x, master=parity.host_vec(dev.theta, so.idx).astype(np.float64))
            assert r["max_abs"] == ref["max_abs"], f"step {t} max_abs"
            for k in ("mean_sq", "mean_abs_to_master"):
                assert abs(r[k] - ref[k]) <= 1e-9 * abs(ref[k]) + 1e-300, (t, k, r[k], ref[k])
            so.upload(dev)
            if t % 50 == 0:
                print(f"  step {t}: slice rms drift {r['rms']:.3e}", flush=True)
    finally:
        del dev
        _free()


def test_drift_stays_bounded_over_two_thousand_steps():
    # Theorem 3.1's claim over a long horizon: 2000 steps of N = 64 replicas
    # (a 409,600-element slice of the drift workload's shape).  The mean
    # squared discrepancy per unit of master movement is the same in each
    # 500-step window and equals 2p / (1 - p^2).
    w = wl.scaled(wl.WORKLOADS["n64_d48m_f32_sgd_drift"], d=2048 * 200, steps=2000)
    p = w.loss["p"]
    dev = parity.DeviceState(w)
    prev = dev.theta.clone()
    ratio = []
    try:
        for t in range(w.steps):
            if t > 0:
                wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
            dev.fused(t)
            step = (dev.theta - prev).double().square().mean()
            prev.copy_(dev.theta)
            ratio.append((ll.read_drift(dev.drift)["mean_sq"], float(step)))
            if t % 500 == 0:
                print(f"  step {t}: mean_sq {ratio[-1][0]:.3e}", flush=True)
    finally:
        del dev
        _free()
    ms = np.array([r[0] for r in ratio])
    s2 = np.array([r[1] for r in ratio])
    corrected = 2 * p / (1 - p * p)
    windows = [float(ms[a:a + 500].mean() / s2[a:a + 500].mean()) for a in range(0, 2000, 500)]
    print(f"E[D^2]/sigma^2 per 500-step window: {windows}; 2p/(1-p^2) = {corrected:.4f}", flush=True)
    for r in windows[1:]:   # the first window includes the burn-in from identical replicas
        assert abs(r - corrected) < 0.04 * corrected
    assert max(windows[1:]) - min(windows[1:]) < 0.04 * corrected


def test_full_size_variants_on_the_7b_shard():
    # The 7B-shard workload at full size with every delivery variant at once:
    # owner row, every 10th packet reliable, parity packets in groups of 7
    # (the last group ragged: 25,696 = 7 * 3670 + 6), Horvitz-Thompson with
    # each packet's weight derived in the kernel, broadcast ages.
    from oracle import loss as oloss
    from oracle import step as ostep
    w = wl.WORKLOADS["n64_llama7b_shard_bf16_adam"]
    P, G, owner, p = w.num_packets, 7, 5, w.loss["p"]
    assert P % G != 0
    relf = np.zeros(P, np.uint8)
    relf[::10] = 1
    dev = parity.DeviceState(w)
    ages = torch.zeros((w.n, P), dtype=torch.int16, device=DEV)
    e = ll.ext(estimator="horvitz_thompson", owner=owner,
               reliable=torch.from_numpy(relf).to(DEV), ages=ages, parity_group=G)
    packets = sorted(set(wl.packet_sample(w, 20)) | {P - 6, P - 1, 10, 11})
    so = parity.SampledOracle(w, packets, dev)
    try:
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(0, ext=e)

        def masks(direction):
            a = oloss.apply_overrides(
                oloss.bernoulli_arrivals(w.seed, 0, direction, w.n, np.arange(P), p), owner, relf)
            par = oloss.parity_arrivals(w.seed, 0, direction, w.n, np.arange((P + G - 1) // G), p)
            return oloss.parity_recover(a, G, par)
        mg, mb = masks(0), masks(1)
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg)
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb)
        assert np.array_equal(ages.cpu().numpy().view(np.uint16), np.where(mb == 1, 0, 1))
        q = np.tile(oloss.parity_arrival_probabilities(1 - p, G, P, relf), (w.n, 1))
        q[owner] = 1.0
        orc = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype,
                               grads=g_host, theta=so.theta, m=so.m, v=so.v,
                               replicas=so.replicas, arrived_g=mg[:, packets],
                               arrived_b=mb[:, packets], opt=parity.opt_as_given(w.opt), t=0,
                               estimator="horvitz_thompson", q=q[:, packets])
        so.advance(orc)
        parity.compare_step(w, 0, dev, so, orc, mb[:, packets], "7B shard, all variants")
    finally:
        del dev
        _free()
