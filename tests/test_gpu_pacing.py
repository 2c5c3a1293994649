"""Pacing and access forms never change a result.

* The paced fused step (rounds of adjacent tiles whose row accesses wait for
  clock slots, Bernoulli masks drawn beforehand by the mask kernel when there
  is memory for them) is bit-identical to the unpaced step: every output,
  mask, count and drift figure, for both row types, with and without drift,
  mask outputs or a workspace, under schedules that are kept and schedules
  laid out far too fast to keep, with a workgroup per tile or one round of
  workgroups looping over the rounds.
* Packets whose length is not a multiple of 8 elements, and fp32 rows whose
  stride is 4 (mod 8) elements, take the element-by-element access form;
  they match the oracle and the stage-by-stage chain.
"""

import numpy as np
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl

import parity
from test_gpu_fused import _bit_equal, _snapshot, _stagewise

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture
def restore_pacing():
    before = ll.ll_get_pacing()
    yield
    ll.ll_set_pacing(**before)


def _step(dev: parity.DeviceState, t: int, *, masks_out: bool, drift: bool, workspace: bool):
    w = dev.w
    spec = parity.loss_spec(w)
    ll.lossy_step_fused(
        d=w.d, packet=w.packet, step=t, loss_g=spec, loss_b=spec, grads=dev.grads,
        opt=parity.opt_spec(w), theta=dev.theta, replicas=dev.replicas, m=dev.m, v=dev.v,
        ge_state_g=dev.ge_g, ge_state_b=dev.ge_b,
        arrived_g=dev.arrived_g if masks_out else None,
        arrived_b=dev.arrived_b if masks_out else None,
        counts=dev.counts, workspace=dev.workspace if workspace else None,
        drift=dev.drift if drift else None)


PACED = {
    # workloads scaled so that the step spans several rounds of resident
    # workgroups at the default layout, with ragged tails; the last two have
    # several mask words per packet, the last one ragged
    "n64_llama7b_shard_bf16_adam": ("n64_llama7b_shard_bf16_adam", dict(d=4096 * 2100 + 3280)),
    "n64_d48m_f32_sgd_drift": ("n64_d48m_f32_sgd_drift", dict(d=2048 * 4000 + 1000)),
    "n8_d16m_bf16_adam": ("n8_d16m_bf16_adam", dict(d=2048 * 9000 + 77)),
    "n16_d256m_f32_ge_momentum": ("n16_d256m_f32_ge_momentum", dict(d=4096 * 3000 + 2056)),
    "n200_bf16_adam": ("n64_llama7b_shard_bf16_adam", dict(n=200, d=4096 * 1500 + 1000)),
    "n130_f32_sgd_drift": ("n64_d48m_f32_sgd_drift", dict(n=130, d=2048 * 1200 + 500)),
}

SCHEDULES = [
    dict(overlap=1, resident=1, bytes_per_s=6.3e12),   # the default: one round at a time
    dict(overlap=2, resident=2, bytes_per_s=6.0e12),   # two rounds streaming at once
    dict(overlap=2, resident=3, bytes_per_s=5.0e14),   # far too fast to keep
    # one round of workgroups looping over the rounds (steps in the plain
    # configuration with whole tiles; the others fall back to a tile per
    # workgroup), kept and far too fast to keep
    dict(overlap=1, resident=1, bytes_per_s=6.3e12, persistent=1),
    dict(overlap=1, resident=1, bytes_per_s=5.0e14, persistent=1),
]


@pytest.mark.parametrize("name", list(PACED))
@pytest.mark.parametrize("sched", range(len(SCHEDULES)))
@pytest.mark.parametrize("masks_out,drift,workspace", [(True, True, True), (False, True, True),
                                                       (False, False, False)])
def test_paced_step_is_bit_identical_to_unpaced(name, sched, masks_out, drift, workspace,
                                                restore_pacing):
    base, sizes = PACED[name]
    w = wl.scaled(wl.WORKLOADS[base], **sizes)
    if w.loss["kind"] == wl.GILBERT_ELLIOTT:
        workspace = True  # the chain scan needs it
    cfg = SCHEDULES[sched]
    print(f"paced vs unpaced {name} d={w.d} {cfg} masks_out={masks_out} drift={drift} "
          f"workspace={workspace}", flush=True)
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    for t in range(2):
        wl.draw_grads(w, t, device=DEV, ld=a.ld, out=a.grads)
        b.grads.copy_(a.grads)
        # the schedule's rate for either row type
        ll.ll_set_pacing("always", gap_us=2.0, lead_us=4.0, headroom=0.9,
                         bytes_per_s_f32=cfg["bytes_per_s"], **cfg)
        _step(a, t, masks_out=masks_out, drift=drift, workspace=workspace)
        ll.ll_set_pacing("never")
        _step(b, t, masks_out=masks_out, drift=drift, workspace=workspace)
        sa, sb = _snapshot(a), _snapshot(b)
        if drift:
            assert sa["drift"] == sb["drift"], (sa["drift"], sb["drift"])
        for k in sa:
            if k == "drift" or (k.startswith("arrived") and not masks_out):
                continue
            assert _bit_equal(sa[k], sb[k]), f"{name} step {t}: {k} differs"


# ---------------------------------------------------------------------------
# Element-by-element access: packets not a multiple of 8, fp32 rows at 4 mod 8
# ---------------------------------------------------------------------------
ODD = [
    # (workload, d, packet, pad): pad makes the row stride d rounded to 256 + pad
    ("n4_d1m_f32_sgd", 3001, 1, 0),
    ("n8_d16m_bf16_adam", 20_003, 3, 0),
    ("n64_d48m_f32_sgd_drift", 30_007, 100, 4),
    ("n64_llama7b_shard_bf16_adam", 50_001, 4097, 8),
    ("n16_d256m_f32_ge_momentum", 41_000, 4097, 4),
    ("n4_d1m_f32_sgd", 50_000, 1024, 4),   # whole packets, fp32 stride 4 mod 8
]


@pytest.mark.parametrize("name,d,L,pad", ODD)
def test_odd_packets_and_strides_match_the_oracle(name, d, L, pad):
    w = wl.scaled(wl.WORKLOADS[name], d=d, packet=L, steps=2)
    dev = parity.DeviceState(w, pad=pad)
    print(f"odd shapes {name} d={d} L={L} ld={dev.ld}", flush=True)
    assert dev.ld % 8 == pad % 8
    packets = list(range(w.num_packets))
    so = parity.SampledOracle(w, packets, dev)
    om = parity.OracleMasks(w)
    for t in range(w.steps):
        if t > 0:
            wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(t)
        mg, mb = om.masks(t, 0), om.masks(t, 1)
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg), "gradient masks"
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb), "broadcast masks"
        orc = so.step(t, g_host, mg, mb)
        parity.compare_step(w, t, dev, so, orc, mb, f"{name} L={L} step {t}")
        so.upload(dev)


@pytest.mark.parametrize("name,d,L,pad", ODD)
def test_odd_packets_and_strides_fused_equals_stagewise(name, d, L, pad):
    w = wl.scaled(wl.WORKLOADS[name], d=d, packet=L)
    a = parity.DeviceState(w, pad=pad)
    b = parity.DeviceState(w, pad=pad)
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
                assert _bit_equal(sa[k], sb[k]), f"{name} L={L} step {t}: {k} differs"
