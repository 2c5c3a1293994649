"""The fused step is graph-capturable: it only enqueues kernels (no
allocation, no memset, no host synchronisation), so a captured step replays
like the eager call, unpaced and paced (the paced step's schedule anchor is
written by a kernel of its own, so every replay lays out a fresh schedule).
Each replay is checked against the eager result, with eager work and
synchronisation between replays."""
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl

import parity

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _state(dev):
    out = [dev.theta, dev.replicas, dev.arrived_g, dev.arrived_b, dev.counts, dev.ge_g, dev.ge_b]
    out += [x for x in (dev.m, dev.v) if x is not None]
    return [x.clone() for x in out] + [ll.read_drift(dev.drift)]


def _same(a, b):
    for x, y in zip(a[:-1], b[:-1]):
        if x.dtype in (torch.float32, torch.bfloat16):
            x, y = x.view(torch.int16 if x.dtype == torch.bfloat16 else torch.int32), \
                y.view(torch.int16 if y.dtype == torch.bfloat16 else torch.int32)
        if not torch.equal(x, y):
            return False
    return a[-1] == b[-1]


@pytest.fixture
def restore_pacing():
    before = ll.ll_get_pacing()
    yield
    ll.ll_set_pacing(**before)


# (workload, parity group, pacing, d, mask outputs): the paced cases span
# several rounds, so the graph holds the mask launch, the schedule anchor and
# the paced step; the persistent form takes steps without mask outputs
CASES = [
    ("n8_d16m_bf16_adam", 0, None, 4096 * 33 + 72, True),
    ("n16_d256m_f32_ge_momentum", 0, None, 4096 * 33 + 72, True),
    ("n8_d16m_bf16_adam", 4, None, 4096 * 33 + 72, True),
    ("n64_llama7b_shard_bf16_adam", 0, dict(mode="always"), 4096 * 2100 + 3280, True),
    ("n64_llama7b_shard_bf16_adam", 0, dict(mode="always", persistent=1), 4096 * 2100 + 3280,
     False),
    ("n64_d48m_f32_sgd_drift", 0, dict(mode="always"), 2048 * 4000 + 1000, False),
]


@pytest.mark.parametrize("name,G,pace,d,masks_out", CASES)
def test_captured_step_replays_like_eager(name, G, pace, d, masks_out, restore_pacing):
    w = wl.scaled(wl.WORKLOADS[name], d=d)
    print(f"graph capture {name} parity={G} pacing={pace} masks_out={masks_out}", flush=True)
    # the setting is read when the step is enqueued: eager calls and the
    # capture take the same launches
    ll.ll_set_pacing(**(pace or dict(mode="never")))
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    e = ll.ext(parity_group=G) if G else None
    t = 3
    # warm-up on a side stream, as capture requires, then restore b's state
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    snap = _state(b)
    with torch.cuda.stream(side):
        b.fused(t, ext=e, masks_out=masks_out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for x, y in zip([b.theta, b.replicas, b.arrived_g, b.arrived_b, b.counts, b.ge_g, b.ge_b]
                    + [x for x in (b.m, b.v) if x is not None], snap[:-1]):
        x.copy_(y)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        b.fused(t, ext=e, masks_out=masks_out)
    torch.cuda.synchronize()
    for rep in range(3):
        a.fused(t, ext=e, masks_out=masks_out)  # eager reference
        _ = (a.theta * 2).sum()  # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert _same(_state(a), _state(b)), f"replay {rep} differs from the eager step"
