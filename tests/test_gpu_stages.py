"""Stage-by-stage parity of the HIP entry points with the oracle, on identical
seeded inputs (masks bit-exact, floats within the stated norms)."""
import math

import numpy as np
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl
from oracle import bf16 as obf16
from oracle import drift as odrift
from oracle import loss as oloss
from oracle import step as ostep

import parity

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _to_dev_u8(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(DEV)


def _rows_to_dev(a: np.ndarray, gdtype: str, ld: int) -> torch.Tensor:
    n, d = a.shape
    if gdtype == wl.BF16:
        t = torch.from_numpy(a.astype(np.int32).astype(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    out = torch.zeros((n, ld), dtype=t.dtype, device=DEV)
    out[:, :d] = t.to(DEV)
    return out


def _rows_to_host(t: torch.Tensor, d: int, gdtype: str) -> np.ndarray:
    x = t[:, :d].cpu()
    if gdtype == wl.BF16:
        return wl.bf16_bits(x).numpy().astype(np.uint16)
    return x.numpy()


def _seeded_rows(rng, n, d, gdtype, scale=1.0):
    x = (rng.standard_normal((n, d)) * scale).astype(np.float32)
    return obf16.from_f32(x) if gdtype == wl.BF16 else x


# --------------------------------------------------------------------- masks
@pytest.mark.parametrize("n,P", [(1, 1), (4, 1024), (65, 333), (64, 25696), (1024, 100)])
@pytest.mark.parametrize("p", [0.0, 0.1, 1.0])
def test_bernoulli_masks_bit_exact(n, P, p):
    for step, direction, seed in ((0, 0, 0), (7, 1, 12345), (2**40 + 3, 0, 2**63 + 5)):
        print(f"masks n={n} P={P} p={p} step={step} dir={direction}", flush=True)
        out = torch.full((n, P), 7, dtype=torch.uint8, device=DEV)
        ll.ll_masks(n, P, step, direction, ll.bernoulli(p, seed=seed), out)
        want = oloss.bernoulli_arrivals(seed, step, direction, n, np.arange(P), p)
        assert np.array_equal(out.cpu().numpy(), want)


@pytest.mark.parametrize("n,P,steps", [(3, 5, 3), (7, 1500, 2), (16, 65536, 3), (2, 1024, 2),
                                        (5, 4096 * 3 + 17, 2),    # ragged last segment
                                        (1, 1_100_000, 1)])       # > 256 segments per chain
def test_gilbert_elliott_masks_and_state_bit_exact(n, P, steps):
    p_gb, p_bg, lg, lb = 0.01, 0.2, 0.0, 0.5
    if P < 2000:  # make short chains switch often
        p_gb, p_bg, lg, lb = 0.3, 0.4, 0.1, 0.6
    spec = ll.gilbert_elliott(p_gb, p_bg, lg, lb, seed=3)
    st_dev = torch.zeros(n, dtype=torch.uint8, device=DEV)
    ws = torch.zeros(ll.ll_masks_workspace_bytes(n, P), dtype=torch.uint8, device=DEV)
    st_orc = np.zeros(n, np.uint8)
    out = torch.zeros((n, P), dtype=torch.uint8, device=DEV)
    for t in range(steps):
        print(f"GE masks n={n} P={P} step={t}", flush=True)
        ll.ll_masks(n, P, t, 1, spec, out, ge_state=st_dev, workspace=ws)
        want, st_orc = oloss.ge_arrivals(3, t, 1, n, P, p_gb, p_bg, lg, lb, st_orc)
        assert np.array_equal(out.cpu().numpy(), want)
        assert np.array_equal(st_dev.cpu().numpy(), st_orc)


# ----------------------------------------------------------------- aggregate
AGG_CASES = [
    # n, d, packet, dtype, p, lam
    (4, 10_000, 1024, wl.F32, 0.1, 0.0),
    (8, 50_003, 2048, wl.BF16, 0.3, 0.0),      # ragged tail, d not a multiple of 8
    (65, 20_000, 4104, wl.F32, 0.5, 0.25),     # 3 chunks per packet, 2 mask words
    (3, 4096, 8, wl.BF16, 0.7, 0.5),           # minimal packets, many empty
    (1024, 4096, 512, wl.F32, 0.1, 0.0),       # maximum worker count
    (1, 777, 16, wl.F32, 0.0, 0.0),            # one worker, no loss
    (64, 8192, 4096, wl.BF16, 0.0, 0.0),       # no loss: the exact mean
]


@pytest.mark.parametrize("n,d,L,gdtype,p,lam", AGG_CASES)
def test_aggregate_parity(n, d, L, gdtype, p, lam):
    print(f"aggregate n={n} d={d} L={L} {gdtype} p={p} lam={lam}", flush=True)
    rng = np.random.default_rng(n * 7 + d)
    P = math.ceil(d / L)
    g = _seeded_rows(rng, n, d, gdtype, 1e-3)
    theta = (rng.standard_normal(d) * 0.02).astype(np.float32)
    mask = oloss.bernoulli_arrivals(5, 1, 0, n, np.arange(P), p)
    ld = (d + 7) // 8 * 8 + 8
    g_dev = _rows_to_dev(g, gdtype, ld)
    g_hat = torch.full((d,), float("nan"), dtype=torch.float32, device=DEV)
    counts = torch.full((P,), -1, dtype=torch.int32, device=DEV)
    ll.lossy_aggregate(g_dev, _to_dev_u8(mask), d=d, packet=L, g_hat=g_hat,
                       fallback_lambda=lam, theta=torch.from_numpy(theta).to(DEV), counts=counts)
    lens = ostep.packet_lengths(d, L, range(P))
    S = np.repeat(mask, lens, axis=1)
    want, K, mean_abs = ostep.aggregate(ostep.widen(g, gdtype), S, lam, theta.astype(np.float64))
    assert np.array_equal(counts.cpu().numpy(), mask.sum(axis=0))
    parity.check_ghat(g_hat.cpu().numpy(), want.astype(np.float32), mean_abs, K)
    if p == 0.0 and gdtype == wl.BF16:
        pass  # covered by the norm; sums of bf16 values are exact below 2^16 terms
    if (K == 1).any():  # a single arrival is copied exactly
        one = K == 1
        assert np.array_equal(g_hat.cpu().numpy()[one], want.astype(np.float32)[one])


def test_aggregate_never_reads_lost_rows():
    # Lost rows hold NaN; the aggregate must not touch them.
    n, d, L = 8, 8192, 1024
    P = d // L
    rng = np.random.default_rng(0)
    g = rng.standard_normal((n, d)).astype(np.float32)
    mask = oloss.bernoulli_arrivals(1, 0, 0, n, np.arange(P), 0.4)
    S = np.repeat(mask, L, axis=1).astype(bool)
    g_poison = np.where(S, g, np.float32(np.nan))
    g_hat = torch.zeros(d, dtype=torch.float32, device=DEV)
    ll.lossy_aggregate(_rows_to_dev(g_poison, wl.F32, d), _to_dev_u8(mask), d=d, packet=L,
                       g_hat=g_hat)
    assert torch.isfinite(g_hat).all()


# ---------------------------------------------------------------- shard step
@pytest.mark.parametrize("kind", ["sgd", "momentum", "adam"])
def test_shard_step_parity(kind):
    d = 100_003
    rng = np.random.default_rng(1)
    opt = parity.opt_as_given(dict(kind=kind, lr=3e-4 if kind == "adam" else 0.01,
                                   momentum=0.9, beta1=0.9, beta2=0.95, eps=1e-8))
    spec = {"sgd": ll.sgd(opt["lr"]), "momentum": ll.sgd_momentum(opt["lr"], 0.9),
            "adam": ll.adam(opt["lr"], 0.9, 0.95, 1e-8)}[kind]
    th = (rng.standard_normal(d) * 0.02).astype(np.float32)
    m = np.zeros(d, np.float32)
    v = np.zeros(d, np.float32)
    for t in range(3):
        print(f"shard_step {kind} t={t}", flush=True)
        g = (rng.standard_normal(d) * 1e-3).astype(np.float32)
        g[:50] = 0.0
        d_th = torch.from_numpy(th).to(DEV)
        d_m = torch.from_numpy(m).to(DEV) if kind != "sgd" else None
        d_v = torch.from_numpy(v).to(DEV) if kind == "adam" else None
        ll.shard_step(spec, t, d_th, torch.from_numpy(g).to(DEV), m=d_m, v=d_v)
        G = g.astype(np.float64)
        if kind == "sgd":
            th1, m1, v1 = ostep.sgd(th.astype(np.float64), G, opt["lr"]), None, None
        elif kind == "momentum":
            th1, m1 = ostep.sgd_momentum(th.astype(np.float64), m.astype(np.float64), G,
                                         opt["lr"], opt["momentum"])
            v1 = None
        else:
            th1, m1, v1 = ostep.adam(th.astype(np.float64), m.astype(np.float64),
                                     v.astype(np.float64), G, t + 1, opt["lr"], opt["beta1"],
                                     opt["beta2"], opt["eps"])
        # identical inputs: the update's own roundings, no propagated term
        orc = dict(g_hat=g, mean_abs=np.zeros(d), theta=th1.astype(np.float32),
                   m=None if m1 is None else m1.astype(np.float32),
                   v=None if v1 is None else v1.astype(np.float32))
        b = parity.state_bounds(opt, t, orc, dict(theta=th, m=m, v=v))
        parity.check_close(d_th.cpu().numpy(), orc["theta"], b["theta"], "theta")
        if m1 is not None:
            parity.check_close(d_m.cpu().numpy(), orc["m"], b["m"], "m")
        if v1 is not None:
            parity.check_close(d_v.cpu().numpy(), orc["v"], b["v"], "v")
        th, m, v = orc["theta"], orc["m"] if m1 is not None else m, orc["v"] if v1 is not None else v


# ----------------------------------------------------------------- broadcast
@pytest.mark.parametrize("n,d,L,rdtype,p", [(4, 10_000, 1024, wl.F32, 0.1),
                                            (64, 50_003, 4096, wl.BF16, 0.1),
                                            (65, 9000, 8, wl.BF16, 0.5),
                                            (3, 5000, 2048, wl.F32, 1.0),
                                            (8, 5000, 2048, wl.BF16, 0.0)])
def test_broadcast_bit_exact(n, d, L, rdtype, p):
    print(f"broadcast n={n} d={d} L={L} {rdtype} p={p}", flush=True)
    rng = np.random.default_rng(2)
    P = math.ceil(d / L)
    theta = (rng.standard_normal(d) * 0.02).astype(np.float32)
    old = _seeded_rows(rng, n, d, rdtype, 0.02)
    mask = oloss.bernoulli_arrivals(9, 4, 1, n, np.arange(P), p)
    ld = (d + 7) // 8 * 8 + 16
    reps = _rows_to_dev(old, rdtype, ld)
    pad_before = reps[:, d:].clone()
    ll.lossy_broadcast(torch.from_numpy(theta).to(DEV), reps, _to_dev_u8(mask), d=d, packet=L)
    lens = ostep.packet_lengths(d, L, range(P))
    R = np.repeat(mask, lens, axis=1)
    want = ostep.broadcast(old, ostep.store(theta.astype(np.float64), rdtype)[None, :], R)
    got = _rows_to_host(reps, d, rdtype)
    if rdtype == wl.F32:
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    else:
        assert np.array_equal(got, want)
    assert torch.equal(reps[:, d:], pad_before)  # row padding untouched


# --------------------------------------------------------------------- drift
@pytest.mark.parametrize("n,d,L,rdtype", [(4, 10_000, 1024, wl.F32), (64, 50_003, 4096, wl.BF16),
                                          (65, 9000, 8, wl.F32), (1, 100, 8, wl.F32),
                                          (2, 4096, 4096, wl.BF16)])
@pytest.mark.parametrize("with_master", [True, False])
def test_drift_stats_parity(n, d, L, rdtype, with_master):
    print(f"drift n={n} d={d} L={L} {rdtype} master={with_master}", flush=True)
    rng = np.random.default_rng(3)
    P = math.ceil(d / L)
    theta = (rng.standard_normal(d) * 0.02).astype(np.float32)
    base = ostep.store(theta.astype(np.float64), rdtype)
    mask = oloss.bernoulli_arrivals(2, 0, 1, n, np.arange(P), 0.3)
    lens = ostep.packet_lengths(d, L, range(P))
    R = np.repeat(mask, lens, axis=1).astype(bool)
    stale = _seeded_rows(rng, n, d, rdtype, 0.02)
    reps = np.where(R, base[None, :], stale)
    ld = (d + 7) // 8 * 8
    ws = torch.zeros(ll.ll_workspace_bytes(n, d, L), dtype=torch.uint8, device=DEV)
    out = ll.drift_buffer()
    ll.drift_stats(_rows_to_dev(reps, rdtype, ld), d=d, packet=L, workspace=ws, out=out,
                   theta=torch.from_numpy(theta).to(DEV) if with_master else None,
                   arrived_bc=_to_dev_u8(mask))
    got = ll.read_drift(out)
    x = ostep.widen(reps, rdtype)
    want = odrift.drift_stats(x, ostep.widen(base, rdtype) if with_master else None, mask)
    assert got["max_abs"] == want["max_abs"]
    assert got["stale_packets"] == want["stale_packets"]
    assert got["empty_packets"] == 0
    assert math.isclose(got["mean_sq"], want["mean_sq"], rel_tol=1e-9, abs_tol=1e-300)
    assert math.isclose(got["rms"], want["rms"], rel_tol=1e-9, abs_tol=1e-300)
    if with_master:
        assert math.isclose(got["mean_abs_to_master"], want["mean_abs_to_master"], rel_tol=1e-9)
    else:
        assert math.isnan(got["mean_abs_to_master"])


def test_drift_identical_replicas_is_zero_and_empty_shard():
    n, d, L = 16, 10_000, 1024
    theta = torch.randn(d, device=DEV) * 0.02
    reps = theta.to(torch.bfloat16).unsqueeze(0).repeat(n, 1).contiguous()
    reps = torch.nn.functional.pad(reps, (0, 8 - d % 8 if d % 8 else 0))
    ws = torch.zeros(ll.ll_workspace_bytes(n, d, L), dtype=torch.uint8, device=DEV)
    out = ll.drift_buffer()
    ll.drift_stats(reps, d=d, packet=L, workspace=ws, out=out, theta=theta)
    r = ll.read_drift(out)
    assert r["max_abs"] == 0 and r["mean_sq"] == 0 and r["mean_abs_to_master"] == 0
    out2 = torch.full((6,), 5.0, dtype=torch.float64, device=DEV)
    ll.drift_stats(reps, d=0, packet=L, workspace=ws, out=out2)
    r = ll.read_drift(out2)
    assert r["max_abs"] == 0 and r["mean_sq"] == 0 and r["stale_packets"] == 0
