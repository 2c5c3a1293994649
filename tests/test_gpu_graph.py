"""The fused step is graph-capturable: it only enqueues kernels (no
allocation, no memset, no host synchronisation), so a captured step replays
like the eager call.  Each replay is checked against the eager result, with
eager work and synchronisation between replays."""
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


@pytest.mark.parametrize("name,G", [("n8_d16m_bf16_adam", 0), ("n16_d256m_f32_ge_momentum", 0),
                                    ("n8_d16m_bf16_adam", 4)])
def test_captured_step_replays_like_eager(name, G):
    w = wl.scaled(wl.WORKLOADS[name], d=4096 * 33 + 72)
    print(f"graph capture {name} parity={G}", flush=True)
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    e = ll.ext(parity_group=G) if G else None
    t = 3
    # warm-up on a side stream, as capture requires, then restore b's state
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    snap = _state(b)
    with torch.cuda.stream(side):
        b.fused(t, ext=e)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for x, y in zip([b.theta, b.replicas, b.arrived_g, b.arrived_b, b.counts, b.ge_g, b.ge_b]
                    + [x for x in (b.m, b.v) if x is not None], snap[:-1]):
        x.copy_(y)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        b.fused(t, ext=e)
    torch.cuda.synchronize()
    for rep in range(3):
        a.fused(t, ext=e)            # eager reference
        _ = (a.theta * 2).sum()      # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert _same(_state(a), _state(b)), f"replay {rep} differs from the eager step"
