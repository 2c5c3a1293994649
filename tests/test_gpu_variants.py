"""GPU parity of the step variants: owner / reliable-packet overrides,
Horvitz-Thompson and stale-fill estimators, broadcast ages."""
import numpy as np
import pytest
import torch

import paper_2507_07114_amd as ll
import workloads as wl
from oracle import loss as oloss
from oracle import step as ostep

import parity

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _u8(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(DEV)


def _reliable(P, every=5, offset=2):
    r = np.zeros(P, np.uint8)
    r[offset::every] = 1
    return r


def _ages_host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("kind", ["bernoulli", "gilbert_elliott"])
@pytest.mark.parametrize("owner,rel", [(-1, False), (3, False), (-1, True), (0, True)])
def test_mask_overrides_bit_exact(kind, owner, rel):
    n, P = 9, 5000
    relf = _reliable(P) if rel else None
    e = ll.ext(owner=owner, reliable=None if relf is None else _u8(relf))
    out = torch.zeros((n, P), dtype=torch.uint8, device=DEV)
    st = torch.zeros(n, dtype=torch.uint8, device=DEV)
    ws = torch.zeros(ll.ll_masks_workspace_bytes(n, P), dtype=torch.uint8, device=DEV)
    st_orc = np.zeros(n, np.uint8)
    for t in range(2):
        print(f"overrides {kind} owner={owner} rel={rel} step {t}", flush=True)
        if kind == "bernoulli":
            ll.ll_masks(n, P, t, 0, ll.bernoulli(0.4, seed=5), out, ext=e)
            want = oloss.bernoulli_arrivals(5, t, 0, n, np.arange(P), 0.4)
        else:
            ll.ll_masks(n, P, t, 1, ll.gilbert_elliott(0.2, 0.3, 0.1, 0.6, seed=5), out,
                        ge_state=st, workspace=ws, ext=e)
            want, st_orc = oloss.ge_arrivals(5, t, 1, n, P, 0.2, 0.3, 0.1, 0.6, st_orc)
            assert np.array_equal(st.cpu().numpy(), st_orc)
        want = oloss.apply_overrides(want, owner=owner, reliable=relf)
        assert np.array_equal(out.cpu().numpy(), want)


AGG_VARIANTS = [
    # n, d, packet, dtype, p, estimator, owner, reliable
    (8, 20_003, 2048, wl.BF16, 0.3, "horvitz_thompson", -1, False),
    (8, 20_003, 2048, wl.F32, 0.3, "horvitz_thompson", 2, True),
    (65, 9_000, 512, wl.F32, 0.5, "horvitz_thompson", 64, False),
    (8, 20_003, 2048, wl.BF16, 0.3, "stale_fill", -1, False),
    (16, 10_000, 1024, wl.F32, 0.6, "stale_fill", 5, True),
]


@pytest.mark.parametrize("n,d,L,gdtype,p,est,owner,rel", AGG_VARIANTS)
def test_aggregate_variants_parity(n, d, L, gdtype, p, est, owner, rel):
    print(f"aggregate {est} n={n} d={d} L={L} {gdtype} owner={owner} rel={rel}", flush=True)
    rng = np.random.default_rng(n + d)
    P = (d + L - 1) // L
    ld = (d + 7) // 8 * 8
    x = (rng.standard_normal((n, d)) * 1e-3).astype(np.float32)
    xp = (rng.standard_normal((n, d)) * 1e-3).astype(np.float32)
    g = ostep.store(x.astype(np.float64), gdtype)
    gp = ostep.store(xp.astype(np.float64), gdtype)
    relf = _reliable(P) if rel else None
    mask = oloss.apply_overrides(oloss.bernoulli_arrivals(3, 0, 0, n, np.arange(P), p), owner, relf)
    grads = parity_rows(g, gdtype, ld)
    prev = parity_rows(gp, gdtype, ld)
    e = ll.ext(estimator=est, owner=owner, reliable=None if relf is None else _u8(relf),
               g_prev=prev if est == "stale_fill" else None, arrival_prob=1 - p)
    g_hat = torch.full((d,), float("nan"), dtype=torch.float32, device=DEV)
    ll.lossy_aggregate(grads, _u8(mask), d=d, packet=L, g_hat=g_hat, ext=e)
    lens = ostep.packet_lengths(d, L, range(P))
    S = np.repeat(mask, lens, axis=1)
    if est == "horvitz_thompson":
        q = np.full((n, P), 1 - p)
        if owner >= 0:
            q[owner] = 1.0
        if relf is not None:
            q[:, relf.astype(bool)] = 1.0
        want, scale = ostep.aggregate_horvitz_thompson(ostep.widen(g, gdtype), S,
                                                       np.repeat(q, lens, axis=1))
        K = np.full(d, n)
    else:
        want, new_prev, scale = ostep.aggregate_stale_fill(ostep.widen(g, gdtype), S,
                                                           ostep.widen(gp, gdtype))
        K = np.full(d, n)
        got_prev = parity.host_rows(prev, np.arange(d), gdtype)
        want_prev = np.where(S.astype(bool), g, gp)
        assert np.array_equal(got_prev.view(np.uint32) if gdtype == wl.F32 else got_prev,
                              want_prev.view(np.uint32) if gdtype == wl.F32 else want_prev)
    parity.check_ghat(g_hat.cpu().numpy(), want.astype(np.float32), scale, K)


def parity_rows(a, gdtype, ld):
    n, d = a.shape
    if gdtype == wl.BF16:
        t = torch.from_numpy(a.astype(np.int32).astype(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    out = torch.zeros((n, ld), dtype=t.dtype, device=DEV)
    out[:, :d] = t.to(DEV)
    return out


VARIANTS = [
    ("horvitz_thompson", -1, False),
    ("horvitz_thompson", 1, True),
    ("stale_fill", -1, False),
    ("stale_fill", 0, True),
    ("arrived_mean", 2, True),
]


def _variant_setup(w, est, owner, rel, dev):
    relf = _reliable(w.num_packets) if rel else None
    relt = None if relf is None else _u8(relf)
    prev = torch.zeros_like(dev.grads) if est == "stale_fill" else None
    ages = torch.zeros((w.n, w.num_packets), dtype=torch.int16, device=DEV)
    return relf, relt, prev, ages


@pytest.mark.parametrize("name", ["n8_d16m_bf16_adam", "n16_d256m_f32_ge_momentum"])
@pytest.mark.parametrize("est,owner,rel", VARIANTS)
def test_fused_variants_bit_identical_to_stagewise(name, est, owner, rel):
    _fused_vs_stagewise(wl.WORKLOADS[name], est, owner, rel, 0)


@pytest.mark.parametrize("est,owner,rel,G", [
    ("arrived_mean", -1, False, 4), ("stale_fill", 1, True, 3), ("arrived_mean", 0, True, 1),
])
def test_fused_parity_bit_identical_to_stagewise(est, owner, rel, G):
    _fused_vs_stagewise(wl.WORKLOADS["n8_d16m_bf16_adam"], est, owner, rel, G)


def _fused_vs_stagewise(w0, est, owner, rel, G):
    w = wl.scaled(w0, d=4096 * 40 + 1000)
    print(f"fused vs stagewise {w0.name} {est} owner={owner} rel={rel} parity={G}", flush=True)
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    _, rel_a, prev_a, ages_a = _variant_setup(w, est, owner, rel, a)
    _, rel_b, prev_b, ages_b = _variant_setup(w, est, owner, rel, b)
    l = w.loss
    if l["kind"] == wl.BERNOULLI:
        q = 1 - l["p"]
    else:  # stationary arrival probability of the Gilbert-Elliott chain
        pi_bad = l["p_gb"] / (l["p_gb"] + l["p_bg"])
        q = 1 - pi_bad * l["loss_bad"] - (1 - pi_bad) * l["loss_good"]
    # the fused side derives q itself for Bernoulli loss; GE needs it given
    qa = q if l["kind"] != wl.BERNOULLI else 0.0
    ea = ll.ext(estimator=est, owner=owner, reliable=rel_a, g_prev=prev_a, ages=ages_a,
                arrival_prob=qa, parity_group=G)
    eb = ll.ext(estimator=est, owner=owner, reliable=rel_b, g_prev=prev_b, arrival_prob=q,
                parity_group=G)
    spec = parity.loss_spec(w)
    P = w.num_packets
    for t in range(3):
        wl.draw_grads(w, t, device=DEV, ld=a.ld, out=a.grads)
        b.grads.copy_(a.grads)
        a.fused(t, ext=ea)
        g_hat = torch.empty(w.d, dtype=torch.float32, device=DEV)
        ll.ll_masks(w.n, P, t, 0, spec, b.arrived_g, ge_state=b.ge_g, workspace=b.workspace, ext=eb)
        ll.lossy_aggregate(b.grads, b.arrived_g, d=w.d, packet=w.packet, g_hat=g_hat,
                           counts=b.counts, theta=b.theta, ext=eb)
        ll.shard_step(parity.opt_spec(w), t, b.theta, g_hat, m=b.m, v=b.v)
        ll.ll_masks(w.n, P, t, 1, spec, b.arrived_b, ge_state=b.ge_b, workspace=b.workspace, ext=eb)
        ll.lossy_broadcast(b.theta, b.replicas, b.arrived_b, d=w.d, packet=w.packet)
        ll.ll_ages_update(b.arrived_b, ages_b)
        ll.drift_stats(b.replicas, d=w.d, packet=w.packet, workspace=b.workspace, out=b.drift,
                       theta=b.theta, arrived_bc=b.arrived_b)
        for k in ("theta", "m", "v", "replicas", "arrived_g", "arrived_b", "counts", "ge_g", "ge_b"):
            x, y = getattr(a, k), getattr(b, k)
            if x is not None:
                assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), f"step {t}: {k}"
        assert torch.equal(ages_a, ages_b), f"step {t}: ages"
        if prev_a is not None:
            assert torch.equal(prev_a.view(torch.uint8), prev_b.view(torch.uint8)), f"step {t}: g_prev"
        da, db = ll.read_drift(a.drift), ll.read_drift(b.drift)
        da["empty_packets"] = db["empty_packets"] = 0
        assert da == db


@pytest.mark.parametrize("est,owner,rel", VARIANTS)
def test_fused_variants_parity_with_oracle(est, owner, rel):
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], d=2048 * 60 + 24, steps=4,
                  loss=dict(kind=wl.BERNOULLI, p=0.3))
    print(f"fused parity {est} owner={owner} rel={rel}", flush=True)
    dev = parity.DeviceState(w, pad=8)
    relf, relt, prev, ages = _variant_setup(w, est, owner, rel, dev)
    e = ll.ext(estimator=est, owner=owner, reliable=relt, g_prev=prev, ages=ages)
    packets = list(range(w.num_packets))
    so = parity.SampledOracle(w, packets, dev)
    prev_o = np.zeros((w.n, w.d), np.uint16)
    ages_o = np.zeros((w.n, w.num_packets), np.uint16)
    p = w.loss["p"]
    q = np.full((w.n, w.num_packets), 1 - p)
    if owner >= 0:
        q[owner] = 1.0
    if relf is not None:
        q[:, relf.astype(bool)] = 1.0
    for t in range(w.steps):
        if t > 0:
            wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(t, ext=e)
        mg = oloss.apply_overrides(oloss.bernoulli_arrivals(w.seed, t, 0, w.n, packets, p), owner, relf)
        mb = oloss.apply_overrides(oloss.bernoulli_arrivals(w.seed, t, 1, w.n, packets, p), owner, relf)
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg)
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb)
        orc = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype,
                               grads=g_host, theta=so.theta, m=so.m, v=so.v,
                               replicas=so.replicas, arrived_g=mg, arrived_b=mb, opt=parity.opt_as_given(w.opt), t=t,
                               estimator=est, q=q, g_prev=prev_o)
        so.advance(orc)
        parity.compare_step(w, t, dev, so, orc, mb, f"{est} step {t}")
        ages_o = ostep.update_ages(ages_o, mb)
        assert np.array_equal(_ages_host(ages), ages_o), f"step {t}: ages"
        if est == "stale_fill":
            prev_o = orc["g_prev"]
            assert np.array_equal(parity.host_rows(prev, so.idx, w.gdtype), prev_o), f"step {t}: g_prev"
        so.upload(dev)


def test_replicas_hold_the_master_of_their_age():
    # GPU-internal bookkeeping check over 25 steps: every replica element
    # equals the device's own master of `age` steps earlier, bit for bit.
    w = wl.scaled(wl.WORKLOADS["n64_d48m_f32_sgd_drift"], n=6, d=2048 * 30 + 8,
                  loss=dict(kind=wl.BERNOULLI, p=0.4))
    dev = parity.DeviceState(w)
    ages = torch.zeros((w.n, w.num_packets), dtype=torch.int16, device=DEV)
    e = ll.ext(owner=2, ages=ages)
    history = [dev.theta.clone()]
    lens = ostep.packet_lengths(w.d, w.packet, range(w.num_packets))
    for t in range(25):
        wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
        dev.fused(t, ext=e)
        history.append(dev.theta.clone())
    hist = torch.stack(history).cpu().numpy()  # [steps + 1][d]
    a = np.repeat(_ages_host(ages).astype(np.int64), lens, axis=1)  # [n][d]
    reps = dev.replicas[:, : w.d].cpu().numpy()
    idx = len(history) - 1 - np.minimum(a, len(history) - 1)
    want = hist[idx, np.arange(w.d)[None, :]]
    never = a >= len(history) - 1  # not refreshed since the start: initial copy
    assert np.array_equal(reps[~never].view(np.uint32), want[~never].view(np.uint32))
    assert (a[2] == 0).all()  # the owner's own replica is always current


def _parity_masks(seed, t, direction, n, P, p, G, owner=-1, relf=None):
    a = oloss.apply_overrides(oloss.bernoulli_arrivals(seed, t, direction, n, np.arange(P), p),
                              owner, relf)
    par = oloss.parity_arrivals(seed, t, direction, n, np.arange((P + G - 1) // G), p)
    return oloss.parity_recover(a, G, par)


@pytest.mark.parametrize("G,n,P,owner,rel", [
    (1, 5, 3000, -1, False), (3, 9, 5003, 2, True), (8, 64, 4096, -1, False),
    (8, 65, 2001, 64, True), (256, 4, 1000, -1, False), (256, 3, 200, 0, False),
])
def test_parity_masks_bit_exact(G, n, P, owner, rel):
    print(f"parity masks G={G} n={n} P={P} owner={owner} rel={rel}", flush=True)
    relf = _reliable(P) if rel else None
    e = ll.ext(owner=owner, reliable=None if relf is None else _u8(relf), parity_group=G)
    out = torch.full((n, P), 7, dtype=torch.uint8, device=DEV)
    for t, direction in ((0, 0), (1, 1), (4, 0)):
        ll.ll_masks(n, P, t, direction, ll.bernoulli(0.3, seed=11), out, ext=e)
        want = _parity_masks(11, t, direction, n, P, 0.3, G, owner, relf)
        assert np.array_equal(out.cpu().numpy(), want), (t, direction)


@pytest.mark.parametrize("est,G,owner,rel", [
    ("arrived_mean", 4, -1, False), ("arrived_mean", 3, 1, True),
    ("horvitz_thompson", 6, -1, False), ("horvitz_thompson", 4, 2, True),
    ("stale_fill", 2, 0, False),
])
def test_fused_parity_with_oracle(est, G, owner, rel):
    # 2048 * 60 + 24 elements in packets of 2048: 61 packets, the last ragged
    # (G = 6 with Horvitz-Thompson runs on 60 full-group packets; G = 4 with
    # reliable packets and the ragged tail takes each packet's own q).
    d = 2048 * 60 + (0 if (est, G) == ("horvitz_thompson", 6) else 24)
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], d=d, steps=3,
                  loss=dict(kind=wl.BERNOULLI, p=0.3))
    print(f"fused parity {est} G={G} owner={owner} rel={rel}", flush=True)
    dev = parity.DeviceState(w, pad=8)
    relf, relt, prev, ages = _variant_setup(w, est, owner, rel, dev)
    e = ll.ext(estimator=est, owner=owner, reliable=relt, g_prev=prev, ages=ages, parity_group=G)
    packets = list(range(w.num_packets))
    so = parity.SampledOracle(w, packets, dev)
    prev_o = np.zeros((w.n, w.d), np.uint16)
    p = w.loss["p"]
    q = np.tile(oloss.parity_arrival_probabilities(1 - p, G, w.num_packets, relf), (w.n, 1))
    if owner >= 0:
        q[owner] = 1.0
    for t in range(w.steps):
        if t > 0:
            wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(t, ext=e)
        mg = _parity_masks(w.seed, t, 0, w.n, w.num_packets, p, G, owner, relf)
        mb = _parity_masks(w.seed, t, 1, w.n, w.num_packets, p, G, owner, relf)
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg)
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb)
        orc = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype,
                               grads=g_host, theta=so.theta, m=so.m, v=so.v,
                               replicas=so.replicas, arrived_g=mg, arrived_b=mb, opt=parity.opt_as_given(w.opt), t=t,
                               estimator=est, q=q, g_prev=prev_o)
        so.advance(orc)
        parity.compare_step(w, t, dev, so, orc, mb, f"{est} parity step {t}")
        if est == "stale_fill":
            prev_o = orc["g_prev"]
        so.upload(dev)


def test_fused_parity_masks_in_workspace_match_masks_out():
    # With no mask outputs the parity masks live in the workspace; the step's
    # results are the same bytes.
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], d=2048 * 33 + 40, steps=2,
                  loss=dict(kind=wl.BERNOULLI, p=0.4))
    a = parity.DeviceState(w)
    b = parity.DeviceState(w)
    for t in range(2):
        wl.draw_grads(w, t, device=DEV, ld=a.ld, out=a.grads)
        b.grads.copy_(a.grads)
        a.fused(t, ext=ll.ext(parity_group=5))
        b.fused(t, masks_out=False, ext=ll.ext(parity_group=5))
        for k in ("theta", "m", "v", "replicas"):
            assert torch.equal(getattr(a, k).view(torch.uint8), getattr(b, k).view(torch.uint8)), k
        assert ll.read_drift(a.drift) == ll.read_drift(b.drift)


@pytest.mark.parametrize("est", ["horvitz_thompson", "stale_fill"])
def test_all_variants_at_once_with_oracle(est):
    # Owner row, reliable packets, parity packets, ages and an estimator
    # variant together.  Horvitz-Thompson takes an explicit q here (with
    # reliable packets inside the groups no single q is exact); the oracle
    # is given the same weights, so the comparison is of the arithmetic.
    G, owner = 3, 2
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], d=2048 * 45 + 40, steps=3,
                  loss=dict(kind=wl.BERNOULLI, p=0.35))
    print(f"all variants {est}", flush=True)
    dev = parity.DeviceState(w, pad=8)
    relf, relt, prev, ages = _variant_setup(w, est, owner, True, dev)
    p = w.loss["p"]
    q_hat = oloss.parity_arrival_probability(1 - p, G)
    e = ll.ext(estimator=est, owner=owner, reliable=relt, g_prev=prev, ages=ages,
               arrival_prob=q_hat if est == "horvitz_thompson" else 0.0, parity_group=G)
    packets = list(range(w.num_packets))
    so = parity.SampledOracle(w, packets, dev)
    prev_o = np.zeros((w.n, w.d), np.uint16)
    ages_o = np.zeros((w.n, w.num_packets), np.uint16)
    q = np.full((w.n, w.num_packets), q_hat)
    q[owner] = 1.0
    q[:, relf.astype(bool)] = 1.0
    for t in range(w.steps):
        if t > 0:
            wl.draw_grads(w, t, device=DEV, ld=dev.ld, out=dev.grads)
        g_host = parity.host_rows(dev.grads, so.idx, w.gdtype)
        dev.fused(t, ext=e)
        mg = _parity_masks(w.seed, t, 0, w.n, w.num_packets, p, G, owner, relf)
        mb = _parity_masks(w.seed, t, 1, w.n, w.num_packets, p, G, owner, relf)
        assert np.array_equal(dev.arrived_g.cpu().numpy(), mg), f"step {t}"
        assert np.array_equal(dev.arrived_b.cpu().numpy(), mb), f"step {t}"
        orc = ostep.lossy_step(d=w.d, packet=w.packet, packets=packets, gdtype=w.gdtype,
                               grads=g_host, theta=so.theta, m=so.m, v=so.v,
                               replicas=so.replicas, arrived_g=mg, arrived_b=mb, opt=parity.opt_as_given(w.opt), t=t,
                               estimator=est, q=q, g_prev=prev_o)
        so.advance(orc)
        parity.compare_step(w, t, dev, so, orc, mb, f"all variants {est} step {t}")
        ages_o = ostep.update_ages(ages_o, mb)
        assert np.array_equal(_ages_host(ages), ages_o), f"step {t}: ages"
        if est == "stale_fill":
            prev_o = orc["g_prev"]
            assert np.array_equal(parity.host_rows(prev, so.idx, w.gdtype), prev_o)
        so.upload(dev)
