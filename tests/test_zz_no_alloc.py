"""lossy_step_fused_noalloc: the fused step on the library's static device
scratch gives bit for bit what lossy_step_fused gives with a workspace, on two
calls in a row, the second on a smaller input (the scratch keeps the first
call's contents), and refuses sizes whose workspace exceeds the scratch."""

import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl

import parity
from test_gpu_fused import _bit_equal, _snapshot

pytestmark = pytest.mark.gpu


def _run(dev: parity.DeviceState, t: int, noalloc: bool):
    w = dev.w
    spec = parity.loss_spec(w)
    kw = dict(d=w.d, packet=w.packet, step=t, loss_g=spec, loss_b=spec, grads=dev.grads,
              opt=parity.opt_spec(w), theta=dev.theta, replicas=dev.replicas, m=dev.m, v=dev.v,
              ge_state_g=dev.ge_g, ge_state_b=dev.ge_b, arrived_g=dev.arrived_g,
              arrived_b=dev.arrived_b, counts=dev.counts, drift=dev.drift)
    if noalloc:
        ll.lossy_step_fused_noalloc(**kw)
    else:
        ll.lossy_step_fused(workspace=dev.workspace, **kw)


@pytest.fixture
def restore_pacing():
    before = ll.ll_get_pacing()
    yield
    ll.ll_set_pacing(**before)


def test_noalloc_matches_the_workspace_entry_point_twice(restore_pacing):
    # call 1: the 7B-shard workload scaled to 2100 packets plus a ragged one,
    # paced (masks drawn beforehand into the scratch); call 2: the
    # Gilbert-Elliott workload at a smaller size (chain scan scratch), unpaced.
    cases = [
        (wl.scaled(wl.WORKLOADS["n64_llama7b_shard_bf16_adam"], d=4096 * 2100 + 3280), "always"),
        (wl.scaled(wl.WORKLOADS["n16_d256m_f32_ge_momentum"], d=4096 * 300 + 2056), "never"),
    ]
    sizes = [ll.ll_workspace_bytes(w.n, w.d, w.packet) for w, _ in cases]
    assert sizes[1] < sizes[0] <= ll.LL_NOALLOC_SCRATCH_BYTES
    for j, (w, mode) in enumerate(cases):
        print(f"noalloc call {j}: n={w.n} d={w.d} packet={w.packet} pacing={mode}", flush=True)
        ll.ll_set_pacing(mode=mode)
        ref = parity.DeviceState(w)
        got = parity.DeviceState(w)
        for t in range(2):
            _run(ref, t, noalloc=False)
            _run(got, t, noalloc=True)
            torch.cuda.synchronize()
            a, b = _snapshot(ref), _snapshot(got)
            for k in a:
                if k == "drift":
                    assert a[k] == b[k], f"call {j} step {t}: drift {a[k]} != {b[k]}"
                else:
                    assert _bit_equal(a[k], b[k]), f"call {j} step {t}: {k} differs"
            assert a["drift"]["stale_packets"] > 0
        del ref, got


def test_noalloc_refuses_sizes_beyond_its_scratch():
    w = wl.scaled(wl.WORKLOADS["n64_llama7b_shard_bf16_adam"], d=4096 * 64 + 8)
    dev = parity.DeviceState(w)
    spec = parity.loss_spec(w)
    # a shard 64x longer than the scratch allows: refused before any device work
    d_big = 400_000_000 * 8
    assert ll.ll_workspace_bytes(w.n, d_big, 8) > ll.LL_NOALLOC_SCRATCH_BYTES
    theta0 = dev.theta.clone()
    # the binding's own size checks would refuse first: call the C entry point
    lib = ll._load()
    with pytest.raises(ll.LossyError) as e:
        code = lib.lossy_step_fused_noalloc(
            w.n, d_big, 8, 0, ll.ctypes.byref(spec), ll.ctypes.byref(spec), None, None,
            ll.LL_BF16, dev.grads.data_ptr(), d_big, ll.ctypes.byref(parity.opt_spec(w)),
            dev.theta.data_ptr(), dev.m.data_ptr(), dev.v.data_ptr(), ll.LL_BF16,
            dev.replicas.data_ptr(), d_big, None, None, None, dev.drift.data_ptr(), None,
            torch.cuda.current_stream().cuda_stream)
        ll._check("lossy_step_fused_noalloc", code)
    assert e.value.code == -1 and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.equal(dev.theta, theta0)
