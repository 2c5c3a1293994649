"""A shard past 2^31 elements: every element offset, row offset and packet
index of the path needs 64 bits there.  Two workers, D = 2^31 + 5000 bf16
elements (about 26 GB of device buffers), one fused step compared with the
oracle on packets at the start, on both sides of element 2^31 and at the
ragged end, and the fused drift against the standalone drift pass.  Then the
drift fold at more partials than any workload makes, against the oracle."""
import gc

import numpy as np
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl
from oracle import loss as oloss

import parity

pytestmark = pytest.mark.gpu
DEV = "cuda"


def test_fused_step_past_two_to_the_31_elements():
    d = 2**31 + 5000
    w = wl.scaled(wl.WORKLOADS["n64_d48m_f32_sgd_drift"], n=2, d=d, packet=4096, steps=1,
                  gdtype=wl.BF16, loss=dict(kind=wl.BERNOULLI, p=0.3))
    P = w.num_packets
    assert (P - 2) * w.packet == 2**31  # packet P - 2 starts at element 2^31
    packets = [0, 1, P // 2, P - 3, P - 2, P - 1]
    print(f"large shard: n={w.n} d={d} P={P}, sampled packets {packets}", flush=True)
    dev = parity.DeviceState(w)
    try:
        so = parity.SampledOracle(w, packets, dev)
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(0)
        mg = oloss.bernoulli_arrivals(w.seed, 0, 0, w.n, np.arange(P), w.loss["p"])
        mb = oloss.bernoulli_arrivals(w.seed, 0, 1, w.n, np.arange(P), w.loss["p"])
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg)
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb)
        assert np.array_equal(dev.counts.cpu().numpy(), mg.sum(axis=0))
        orc = so.step(0, g_host, mg, mb)
        parity.compare_step(w, 0, dev, so, orc, mb[:, packets], "large shard")
        fused = ll.read_drift(dev.drift)
        out = ll.drift_buffer()
        ll.drift_stats(dev.replicas, d=d, packet=w.packet, workspace=dev.workspace, out=out,
                       theta=dev.theta, arrived_bc=dev.arrived_b)
        alone = ll.read_drift(out)
        assert fused["empty_packets"] == int((mg.sum(axis=0) == 0).sum())
        fused["empty_packets"] = alone["empty_packets"] = 0
        assert fused == alone
        print(f"  ok: drift rms {fused['rms']:.3e}, stale {fused['stale_packets']}", flush=True)
    finally:
        del dev
        gc.collect()
        torch.cuda.empty_cache()


def test_drift_fold_over_four_hundred_thousand_partials():
    # 400,000 packets of 8 fp32 elements, one workgroup each: the second
    # level of the drift fold then takes 1563 partials per group and runs its
    # four-at-a-time loop before the remainder.  Fused and standalone drift
    # are each compared with the oracle's definition on the device's own
    # replicas.
    from oracle import drift as odrift
    n, L, P = 4, 8, 400_000
    w = wl.scaled(wl.WORKLOADS["n64_d48m_f32_sgd_drift"], n=n, d=P * L, packet=L, steps=1,
                  loss=dict(kind=wl.BERNOULLI, p=0.3))
    print(f"drift fold: n={n} d={w.d} L={L} partials={P}", flush=True)
    dev = parity.DeviceState(w)
    try:
        dev.fused(0)
        reps = dev.replicas[:, : w.d].cpu().numpy().astype(np.float64)
        master = dev.theta.cpu().numpy().astype(np.float64)
        mb = dev.arrived_b.cpu().numpy()
        assert np.array_equal(mb, oloss.bernoulli_arrivals(w.seed, 0, 1, n, np.arange(P), 0.3))
        ref = odrift.drift_stats(reps, master, mb)
        out = ll.drift_buffer()
        ll.drift_stats(dev.replicas, d=w.d, packet=L, workspace=dev.workspace, out=out,
                       theta=dev.theta, arrived_bc=dev.arrived_b)
        for label, r in (("fused", ll.read_drift(dev.drift)), ("standalone", ll.read_drift(out))):
            assert r["max_abs"] == ref["max_abs"], (label, r, ref)
            assert abs(r["mean_sq"] - ref["mean_sq"]) <= 1e-9 * ref["mean_sq"], (label, r, ref)
            assert abs(r["mean_abs_to_master"] - ref["mean_abs_to_master"]) <= \
                1e-9 * ref["mean_abs_to_master"], (label, r, ref)
            assert r["stale_packets"] == ref["stale_packets"] == int((mb == 0).sum())
        assert ref["mean_sq"] > 0
    finally:
        del dev
        gc.collect()
        torch.cuda.empty_cache()
