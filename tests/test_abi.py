"""The C ABI library loads and exports every declared entry point; argument
validation rejects bad input before any device work (CPU only: no call
here reaches a kernel launch)."""
import ctypes
import os
import re

import pytest

import paper_2507_07114_amd as ll

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lossy.h")


def _declared():
    text = open(HEADER).read()
    return re.findall(r"^LL_API\s+[\w\s\*]*?\b(\w+)\s*\(", text, flags=re.M)


def test_header_declares_the_boundary():
    names = set(_declared())
    assert names == {"ll_masks", "lossy_aggregate", "shard_step", "lossy_broadcast",
                     "drift_stats", "lossy_step_fused", "lossy_step_fused_noalloc",
                     "ll_workspace_bytes",
                     "ll_masks_workspace_bytes", "ll_ages_update", "ll_last_error",
                     "ll_set_pacing", "ll_get_pacing"}


def test_library_exports_every_declared_symbol():
    assert os.path.exists(ll.library_path()), "run `python -m paper_2507_07114_amd.build`"
    lib = ctypes.CDLL(ll.library_path())
    for name in _declared():
        assert hasattr(lib, name), name
    # and the binding wraps each of them under the same name
    for name in _declared():
        assert callable(getattr(ll, name)), name


def test_struct_layouts():
    assert ctypes.sizeof(ll.LossSpec) == 56
    assert ctypes.sizeof(ll.OptSpec) == 28
    assert ctypes.sizeof(ll.Ext) == 48
    assert ll.Ext.parity_group.offset == 40


def test_workspace_bytes_host_logic():
    # partials: 32 B per workgroup of the smallest geometry (P * ceil(L / 1024))
    # and 256 second-level
    # ones of 40 B, then two n*P mask areas and the Gilbert-Elliott scan scratch of
    # both directions, each region rounded up to 256 B.
    def r256(x):
        return (x + 255) // 256 * 256
    def ge(n, P):  # per direction: run maps, segment maps, state copy
        S = (P + 4095) // 4096
        return r256(n * S * 256) + r256(n * S) + r256(n)
    n, d, L = 64, 105_250_000, 4096
    P = (d + L - 1) // L
    groups = r256(256 * 40 + 16)  # second-level drift partials and their counter
    assert ll.ll_workspace_bytes(n, d, L) == (r256(P * 4 * 32) + groups + 2 * r256(n * P)
                                              + 2 * ge(n, P))
    assert ll.ll_workspace_bytes(4, 10, 8) == 256 + groups + 2 * 256 + 2 * ge(4, 2)
    assert ll.ll_masks_workspace_bytes(16, 65536) == ge(16, 65536)
    assert ll.ll_masks_workspace_bytes(0, 5) == 0
    assert ll.ll_workspace_bytes(0, 10, 8) == 0      # invalid n
    assert ll.ll_workspace_bytes(4, 10, 0) == 0      # packet < 1
    # any packet length >= 1: P = ceil(d / L), one partial per chunk of 1024
    assert ll.ll_workspace_bytes(4, 10, 3) == r256(4 * 32) + groups + 2 * 256 + 2 * ge(4, 4)
    assert ll.ll_workspace_bytes(4, 10, 12) == 256 + groups + 2 * 256 + 2 * ge(4, 1)
    assert ll.ll_workspace_bytes(4, -1, 8) == 0


def _raw():
    return ctypes.CDLL(ll.library_path())


@pytest.mark.parametrize("args,code,frag", [
    ((0, 16, 8, 0, 16, 16, 0, 0.0, 0, 16, 0, 0), -1, "n=0"),
    ((2000, 16, 8, 0, 16, 16, 0, 0.0, 0, 16, 0, 0), -1, "n=2000"),
    ((2, -5, 8, 0, 16, 16, 16, 0.0, 0, 16, 0, 0), -1, "negative"),
    ((2, 16, 0, 0, 16, 16, 16, 0.0, 0, 16, 0, 0), -1, "packet=0 must be at least 1"),
    ((2, 16, -3, 0, 16, 16, 16, 0.0, 0, 16, 0, 0), -1, "at least 1"),
    ((2, 16, 8, 7, 16, 16, 16, 0.0, 0, 16, 0, 0), -1, "dtype"),
    ((2, 16, 8, 0, 0, 16, 16, 0.0, 0, 16, 0, 0), -1, "grads is NULL"),
    ((2, 16, 8, 0, 16, 8, 16, 0.0, 0, 16, 0, 0), -1, "ld=8 < d=16"),
    # fp32 rows need ld a multiple of 4 elements, bf16 rows a multiple of 8
    ((2, 16, 8, 0, 16, 18, 16, 0.0, 0, 16, 0, 0), -2, "not a multiple of 16 bytes"),
    ((2, 16, 8, 1, 16, 20, 16, 0.0, 0, 16, 0, 0), -2, "ld=20 elements of 2 bytes"),
    ((2, 16, 8, 0, 18, 16, 16, 0.0, 0, 16, 0, 0), -2, "aligned"),
    ((2, 16, 8, 0, 16, 16, 0, 0.0, 0, 16, 0, 0), -1, "arrived is NULL"),
    ((2, 16, 8, 0, 16, 16, 16, 0.5, 0, 16, 0, 0), -1, "theta is NULL"),
])
def test_aggregate_rejects_bad_arguments(args, code, frag):
    lib = _raw()
    f = lib.lossy_aggregate
    f.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                  ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    assert f(*args[:11], None, args[11]) == code
    lib.ll_last_error.restype = ctypes.c_char_p
    assert frag in lib.ll_last_error().decode()


def test_masks_and_opt_validation():
    lib = _raw()
    lib.ll_last_error.restype = ctypes.c_char_p
    bad_p = ll.bernoulli(1.5)
    fm = lib.ll_masks
    fm.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int32,
                   ctypes.POINTER(ll.LossSpec), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                   ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    assert fm(4, 10, 0, 0, ctypes.byref(bad_p), None, 16, None, 0, None, None) == -1
    assert "p outside" in lib.ll_last_error().decode()
    ge = ll.gilbert_elliott(0.1, 0.2, 0.0, 0.5)
    assert fm(4, 10, 0, 0, ctypes.byref(ge), None, 16, None, 0, None, None) == -1
    assert "ge_state" in lib.ll_last_error().decode()
    assert fm(4, 10, 0, 0, ctypes.byref(ge), 16, 16, None, 0, None, None) == -1
    assert "workspace" in lib.ll_last_error().decode()
    assert fm(4, 10, 0, 3, ctypes.byref(ll.bernoulli(0.1)), None, 16, None, 0, None, None) == -1
    # Zero packets is a valid no-op that touches no device.
    assert fm(4, 0, 0, 0, ctypes.byref(ll.bernoulli(0.1)), None, 16, None, 0, None, None) == 0

    fs = lib.shard_step
    fs.argtypes = [ctypes.POINTER(ll.OptSpec), ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    adam = ll.adam(1e-3, 0.9, 0.95, 1e-8)
    assert fs(ctypes.byref(adam), 16, 0, 16, 16, None, 16, None) == -1
    assert "v is NULL" in lib.ll_last_error().decode()
    mom = ll.sgd_momentum(1e-2, 0.9)
    assert fs(ctypes.byref(mom), 16, 0, 16, None, None, 16, None) == -1
    bad = ll.OptSpec(9, 0.1, 0, 0, 0, 0, 0)
    assert fs(ctypes.byref(bad), 16, 0, 16, None, None, 16, None) == -1
    assert "unknown optimizer" in lib.ll_last_error().decode()
    # d = 0 returns before touching the device.
    assert fs(ctypes.byref(ll.sgd(0.1)), 0, 0, 16, None, None, 16, None) == 0


def test_ext_validation():
    lib = _raw()
    lib.ll_last_error.restype = ctypes.c_char_p
    f = lib.lossy_aggregate
    f.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                  ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ll.Ext), ctypes.c_void_p]
    base = (4, 16, 8, 0, 16, 16, 16, 0.0, None, 16, None)
    cases = [(ll.Ext(7, -1, None, None, None, 0.0), "unknown estimator"),
             (ll.Ext(0, 4, None, None, None, 0.0), "owner=4"),
             (ll.Ext(0, -2, None, None, None, 0.0), "owner=-2"),
             (ll.Ext(1, -1, None, None, None, 0.0), "arrival probability"),
             (ll.Ext(1, -1, None, None, None, 1.5), "arrival_prob"),
             (ll.Ext(2, -1, None, None, None, 0.0), "g_prev is NULL"),
             (ll.Ext(0, -1, None, None, None, 0.0, -1), "parity_group=-1"),
             (ll.Ext(0, -1, None, None, None, 0.0, 257), "parity_group=257")]
    for e, frag in cases:
        assert f(*base, ctypes.byref(e), None) == -1
        assert frag in lib.ll_last_error().decode(), (frag, lib.ll_last_error())
    fa = lib.ll_ages_update
    fa.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    assert fa(4, 10, None, 16, None) == -1
    assert fa(4, 0, None, None, None) == 0


def test_parity_validation():
    lib = _raw()
    lib.ll_last_error.restype = ctypes.c_char_p
    fm = lib.ll_masks
    fm.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int32,
                   ctypes.POINTER(ll.LossSpec), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                   ctypes.c_size_t, ctypes.POINTER(ll.Ext), ctypes.c_void_p]
    ge = ll.gilbert_elliott(0.1, 0.2, 0.0, 0.5)
    e = ll.Ext(0, -1, None, None, None, 0.0, 4)
    assert fm(4, 10, 0, 0, ctypes.byref(ge), 16, 16, 16, 1 << 20, ctypes.byref(e), None) == -1
    assert "Bernoulli" in lib.ll_last_error().decode()
    # Zero packets stays a no-op with parity on.
    assert fm(4, 0, 0, 0, ctypes.byref(ll.bernoulli(0.1)), None, 16, None, 0,
              ctypes.byref(e), None) == 0

    ff = lib.lossy_step_fused
    ff.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_uint64,
                   ctypes.POINTER(ll.LossSpec), ctypes.POINTER(ll.LossSpec), ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.POINTER(ll.OptSpec), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                   ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                   ctypes.c_void_p, ctypes.POINTER(ll.Ext), ctypes.c_void_p]
    b = ll.bernoulli(0.2)
    sgd = ll.sgd(0.1)

    def call(e, lb=b, d=64, packet=8):
        return ff(4, d, packet, 0, ctypes.byref(b), ctypes.byref(lb), 16, 16, 0, 16, d,
                  ctypes.byref(sgd), 16, None, None, 0, 16, d, None, None, None, None, 0,
                  None, ctypes.byref(e), None)

    assert call(ll.Ext(0, -1, None, None, None, 0.0, 4), lb=ge) == -1
    assert "Bernoulli" in lib.ll_last_error().decode()
    # Horvitz-Thompson with a derived q under parity packets is accepted for
    # ragged groups (P = 8 packets, G = 3) and reliable packets (the kernel
    # derives each packet's probability); with everything else valid the
    # call stops at the missing workspace, as parity masks go through memory.
    for e in (ll.Ext(1, -1, None, None, None, 0.0, 3), ll.Ext(1, -1, 16, None, None, 0.0, 4),
              ll.Ext(1, -1, None, None, None, 0.0, 4)):
        assert call(e) == -1
        assert "workspace" in lib.ll_last_error().decode()


def test_binding_rejects_host_and_misshapen_tensors():
    # The binding refuses what the C ABI cannot take before any call: host
    # tensors, wrong dtypes, non-2-D rows, rows with a non-unit column stride.
    import pytest
    import torch
    rows = torch.zeros((4, 16), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensor"):
        ll.lossy_broadcast(torch.zeros(16), rows, torch.zeros((4, 2), dtype=torch.uint8),
                           d=16, packet=8)
    with pytest.raises(ValueError, match="2-D"):
        ll.lossy_aggregate(torch.zeros(16, dtype=torch.bfloat16), torch.zeros((4, 2), dtype=torch.uint8),
                           d=16, packet=8, g_hat=torch.zeros(16))
    with pytest.raises(ValueError, match="unit column stride"):
        ll.lossy_aggregate(torch.zeros((16, 4), dtype=torch.bfloat16).t(),
                           torch.zeros((4, 2), dtype=torch.uint8), d=16, packet=8,
                           g_hat=torch.zeros(16))
    with pytest.raises(ValueError, match="float32 or bfloat16"):
        ll.lossy_aggregate(torch.zeros((4, 16), dtype=torch.float16),
                           torch.zeros((4, 2), dtype=torch.uint8), d=16, packet=8,
                           g_hat=torch.zeros(16))
    with pytest.raises(ValueError, match="unknown estimator"):
        ll.ext(estimator="median")


def test_missing_library_fails_loudly(monkeypatch):
    # No fallback: without liblossy.so every entry point raises.
    import pytest
    monkeypatch.setattr(ll, "_lib", None)
    monkeypatch.setattr(ll, "library_path", lambda: "/nonexistent/liblossy.so")
    with pytest.raises(RuntimeError, match="not built"):
        ll.ll_workspace_bytes(4, 100, 8)
    with pytest.raises(RuntimeError, match="not built"):
        ll.ll_last_error()


def test_pacing_setting_round_trips_and_rejects_bad_values():
    before = ll.ll_get_pacing()
    try:
        want = dict(mode="never", bytes_per_s=5.0e12, gap_us=1.5, lead_us=3.0, overlap=1,
                    resident=2, headroom=0.75, tail_us=1.25, persistent=0,
                    bytes_per_s_f32=4.5e12)
        ll.ll_set_pacing(**want)
        assert ll.ll_get_pacing() == want
        for bad in ((0.0, 1.0, 1.0, 2, 3), (-1.0, 1.0, 1.0, 2, 3), (2e15, 1.0, 1.0, 2, 3),
                    (6e12, -1.0, 1.0, 2, 3), (6e12, 2e4, 1.0, 2, 3), (6e12, 1.0, -1.0, 2, 3),
                    (6e12, 1.0, 1.0, 0, 3), (6e12, 1.0, 1.0, 3, 3), (6e12, 1.0, 1.0, 2, 1),
                    (6e12, 1.0, 1.0, 1, 5), (6e12, 1.0, 1.0, 1, 1, 0.0), (6e12, 1.0, 1.0, 1, 1, 1.5),
                    (6e12, 1.0, 1.0, 1, 1, 1.0, -1.0), (6e12, 1.0, 1.0, 1, 1, 1.0, 2e4),
                    (6e12, 1.0, 1.0, 1, 1, 1.0, 1.0, 2), (6e12, 1.0, 1.0, 1, 1, 1.0, 1.0, -1),
                    (6e12, 1.0, 1.0, 2, 2, 1.0, 1.0, 1), (6e12, 1.0, 1.0, 1, 2, 1.0, 1.0, 1),
                    (6e12, 1.0, 1.0, 1, 1, 1.0, 1.0, 0, 0.0),
                    (6e12, 1.0, 1.0, 1, 1, 1.0, 1.0, 0, 2e15)):
            with pytest.raises(ll.LossyError):
                ll.ll_set_pacing("auto", *bad)
        lib = _raw()
        lib.ll_set_pacing.argtypes = [ctypes.c_void_p]
        lib.ll_last_error.restype = ctypes.c_char_p
        cfg = ll.Pacing(7, 6e12, 2.0, 2.5, 2, 2, 0.9, 2.5, 0, 6e12)
        assert lib.ll_set_pacing(ctypes.byref(cfg)) == -1
        assert "unknown pacing mode 7" in lib.ll_last_error().decode()
        assert lib.ll_set_pacing(None) == -1
        # a rejected setting leaves the previous one in place
        assert ll.ll_get_pacing() == want
    finally:
        ll.ll_set_pacing(**before)


PROBE_HEADER = os.path.join(ROOT, "include", "hbm_probe.h")


def test_probe_library_exports_its_header_and_rejects_bad_arguments():
    from paper_2507_07114_amd import probe
    names = re.findall(r"^HBM_PROBE_API\s+[\w\s\*]*?\b(\w+)\s*\(", open(PROBE_HEADER).read(),
                       flags=re.M)
    assert set(names) == {"hbm_probe_copy", "hbm_probe_read", "hbm_probe_write",
                          "hbm_probe_rows"}
    lib = probe._load()
    for name in names:
        assert hasattr(lib, name), name
        assert callable(getattr(probe, name)), name
    # host-side checks only: none of these reaches a launch
    assert lib.hbm_probe_copy(16, 32, 15, None) == -1          # size not a multiple of 16
    assert lib.hbm_probe_copy(8, 32, 16, None) == -1           # misaligned source
    assert lib.hbm_probe_copy(None, 32, 16, None) == -1
    assert lib.hbm_probe_read(16, 16, None, None) == -1        # no sink
    assert lib.hbm_probe_write(24, 16, None) == -1
    assert lib.hbm_probe_rows(16, 0, 32, 0, 16, 16, 64, None) == -1    # nothing to move
    assert lib.hbm_probe_rows(16, 2, 32, 2, 32, 16, 64, None) == -1    # ld < row
    assert lib.hbm_probe_rows(16, 2, None, 1, 32, 32, 64, None) == -1  # missing dst
    assert lib.hbm_probe_copy(16, 32, 0, None) == 0                    # nothing to copy


def test_binding_checks_every_buffer_against_the_sizes():
    # Each mismatch between a buffer and (n, d, P) is refused by the binding
    # before any device pointer is taken (CPU tensors suffice to show it).
    import pytest
    import torch
    n, d, L = 4, 40, 8
    P = 5
    bf, f32, u8 = torch.bfloat16, torch.float32, torch.uint8

    def args(**over):
        a = dict(d=d, packet=L, step=0, loss_g=ll.bernoulli(0.1), loss_b=ll.bernoulli(0.1),
                 grads=torch.zeros((n, 48), dtype=bf), opt=ll.adam(3e-4, 0.9, 0.95, 1e-8),
                 theta=torch.zeros(d), replicas=torch.zeros((n, 48), dtype=bf),
                 m=torch.zeros(d), v=torch.zeros(d), arrived_g=torch.zeros((n, P), dtype=u8),
                 arrived_b=torch.zeros((n, P), dtype=u8),
                 counts=torch.zeros(P, dtype=torch.int32), drift=torch.zeros(6, dtype=torch.float64))
        a.update(over)
        return a

    cases = [
        (dict(theta=torch.zeros(d - 1)), "theta has 39 elements"),
        (dict(m=torch.zeros(d - 8)), "m has 32 elements"),
        (dict(v=torch.zeros(d, dtype=torch.float64)), "v must have dtype"),
        (dict(arrived_g=torch.zeros((n, P - 1), dtype=u8)), "arrived_g must have shape"),
        (dict(arrived_b=torch.zeros((n + 1, P), dtype=u8)), "arrived_b must have shape"),
        (dict(arrived_g=torch.zeros((n, P), dtype=torch.int8)), "arrived_g must have dtype"),
        (dict(counts=torch.zeros(P - 1, dtype=torch.int32)), "counts has 4 elements"),
        (dict(drift=torch.zeros(5, dtype=torch.float64)), "drift has 5 elements"),
        (dict(replicas=torch.zeros((n - 1, 48), dtype=bf)), "same number of rows"),
        (dict(grads=torch.zeros((n, d - 1), dtype=bf)), "fewer than d"),
        (dict(ge_state_g=torch.zeros(n - 1, dtype=u8)), "ge_state_g has 3 elements"),
        (dict(ext=ll.ext(ages=torch.zeros((n, P + 1), dtype=torch.int16))), "ages must have shape"),
        (dict(ext=ll.ext(reliable=torch.zeros(P - 1, dtype=u8))), "reliable has 4 elements"),
        # g_prev must match grads in shape, row stride and dtype
        (dict(ext=ll.ext(estimator="stale_fill", g_prev=torch.zeros((n, d), dtype=bf))),
         "g_prev must match grads"),
        (dict(ext=ll.ext(estimator="stale_fill", g_prev=torch.zeros((n, 48), dtype=f32))),
         "g_prev must match grads"),
        (dict(ext=ll.ext(estimator="stale_fill",
                         g_prev=torch.zeros((n, 64), dtype=bf)[:, :48])), "g_prev must match grads"),
    ]
    for over, msg in cases:
        with pytest.raises(ValueError, match=msg):
            ll.lossy_step_fused(**args(**over))
    # the aggregate and the other stages check their own buffers too
    with pytest.raises(ValueError, match="g_hat has 39 elements"):
        ll.lossy_aggregate(torch.zeros((n, 48), dtype=bf), torch.zeros((n, P), dtype=u8), d=d,
                           packet=L, g_hat=torch.zeros(d - 1))
    with pytest.raises(ValueError, match="counts has 4 elements"):
        ll.lossy_aggregate(torch.zeros((n, 48), dtype=bf), torch.zeros((n, P), dtype=u8), d=d,
                           packet=L, g_hat=torch.zeros(d), counts=torch.zeros(P - 1, dtype=torch.int32))
    with pytest.raises(ValueError, match="g_prev must match grads"):
        ll.lossy_aggregate(torch.zeros((n, 48), dtype=bf), torch.zeros((n, P), dtype=u8), d=d,
                           packet=L, g_hat=torch.zeros(d),
                           ext=ll.ext(estimator="stale_fill", g_prev=torch.zeros((n, 40), dtype=bf)))
    with pytest.raises(ValueError, match="arrived_bc must have shape"):
        ll.lossy_broadcast(torch.zeros(d), torch.zeros((n, 48), dtype=bf),
                           torch.zeros((n, P + 1), dtype=u8), d=d, packet=L)
    with pytest.raises(ValueError, match="ages must have shape"):
        ll.ll_ages_update(torch.zeros((n, P), dtype=u8), torch.zeros((n, P - 1), dtype=torch.int16))
