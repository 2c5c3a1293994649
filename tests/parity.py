"""Shared helpers of the GPU parity tests: host copies of sampled packets and
the comparison norms.

Norms, each with the floating-point reasoning behind it (u = 2^-24, the unit
roundoff of fp32; every bound is per element):
  * masks, counts, packet bookkeeping, GE state: bit-exact.
  * g_hat: |gpu - orc| <= 1e-5 * A_e, A_e = mean |arrived contribution| (for
    an empty packet A_e = |lam * theta|), for every worker count.  (The
    worst case of a sequential fp32 sum of K terms is K u A_e, above 1e-5
    for K > 167; the realised error of a sum of K terms of either sign grows
    like sqrt(K) u A_e and stays far below.)
  * theta, m, v after one step from the same state: the roundings the
    update performs, plus the g_hat tolerance carried through the update:
      bound = min(R, 1e-5 * max(|orc|, rms(orc))) + |d x / d g_hat| dg
    where R counts the fp32 roundings of the library's update against the
    oracle's fp64 value rounded once: one ulp of the stored result (2u |x|,
    two different roundings), one rounding per fp32 operation on the
    intermediate terms (products, the moment sums, the bias-corrected
    ratios, the square root) carried to the result, and dg is the g_hat
    tolerance.  The 1e-5 relative cap is the outer limit on the rounding
    part; the carried g_hat part is the update's own conditioning (Adam
    where g_hat is within its rounding of eps).  The oracle is given the
    hyper-parameters as the library receives them (ll_opt holds fp32).
  * replicas: equal bit-for-bit to the GPU's own rounding of its theta, and
    within 2e-2 relative (plus the theta bound) of the oracle's.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import step as ostep

import workloads as wl

GHAT_REL = 1e-5
STATE_REL = 1e-5
BF16_REL = 2e-2
U = 2.0 ** -24


def opt_as_given(opt: dict) -> dict:
    """Hyper-parameters as the library receives them (ll_opt fields are fp32)."""
    return {k: (v if k == "kind" else float(np.float32(v))) for k, v in opt.items()}


def elements_of(w: wl.Workload, packets) -> np.ndarray:
    return ostep.packet_elements(w.d, w.packet, packets)


def host_rows(t: torch.Tensor, idx: np.ndarray, gdtype: str) -> np.ndarray:
    """Columns idx of a [n][ld] device tensor -> numpy storage (fp32 or bf16 bits)."""
    sel = t.index_select(1, torch.as_tensor(idx, device=t.device)).cpu()
    if gdtype == wl.BF16:
        return wl.bf16_bits(sel).numpy().astype(np.uint16)
    return sel.numpy().astype(np.float32)


def host_vec(t: torch.Tensor, idx: np.ndarray) -> np.ndarray:
    return t.index_select(0, torch.as_tensor(idx, device=t.device)).cpu().numpy()


def rms(x: np.ndarray) -> float:
    x = np.asarray(x, dtype=np.float64)
    return float(np.sqrt(np.mean(x * x))) if x.size else 0.0


def ghat_bound(mean_abs: np.ndarray, k_elem=None) -> np.ndarray:
    """Tolerance of g_hat: 1e-5 of the mean arrived magnitude, for every K
    (k_elem is accepted for call compatibility and not used)."""
    return GHAT_REL * np.asarray(mean_abs, np.float64) + 1e-30


def check_ghat(gpu: np.ndarray, orc: np.ndarray, mean_abs: np.ndarray, k_elem=None,
               what="g_hat"):
    err = np.abs(gpu.astype(np.float64) - orc.astype(np.float64))
    bound = ghat_bound(mean_abs, k_elem)
    bad = np.where(~(err <= bound))[0]
    assert bad.size == 0, (f"{what}: {bad.size} elements out of tolerance; first {bad[:5]} "
                           f"gpu={gpu[bad[:5]]} orc={orc[bad[:5]]} bound={bound[bad[:5]]}")


def _f64(x):
    return None if x is None else np.asarray(x, np.float32).astype(np.float64)


def _sensitivities(opt: dict, t: int, g: np.ndarray, m1, v1):
    """|d theta'/d g|, |d m'/d g|, |d v'/d g| of one update, at the oracle's point."""
    kind = opt["kind"]
    if kind == "sgd":
        return np.full_like(g, opt["lr"]), None, None
    if kind == "momentum":
        return np.full_like(g, opt["lr"]), np.ones_like(g), None
    b1, b2, eps, lr = opt["beta1"], opt["beta2"], opt["eps"], opt["lr"]
    bc1, bc2 = 1 - b1 ** (t + 1), 1 - b2 ** (t + 1)
    m1 = m1.astype(np.float64)
    v1 = v1.astype(np.float64)
    s = np.sqrt(v1 / bc2)
    ds = np.where(s > 0, (1 - b2) * np.abs(g) / (bc2 * np.maximum(s, 1e-300)),
                  np.sqrt((1 - b2) / bc2))
    dth = lr * ((1 - b1) / (bc1 * (s + eps)) + np.abs(m1) / (bc1 * (s + eps) ** 2) * ds)
    return dth, np.full_like(g, 1 - b1), 2 * (1 - b2) * np.abs(g)


def rounding_bounds(opt: dict, t: int, orc: dict, prev: dict) -> dict:
    """Rounding part R of the theta/m/v tolerances (see the module docstring):
    the library's fp32 update of the same inputs against the oracle's fp64
    update rounded once.  prev holds the inputs (theta, m, v)."""
    kind = opt["kind"]
    G = np.asarray(orc["g_hat"], np.float32).astype(np.float64)
    th0, th1 = _f64(prev["theta"]), _f64(orc["theta"])
    step = np.abs(th1 - th0)
    lr = opt["lr"]
    out = {}
    if kind == "sgd":
        # fl(lr g) then fl(theta - .): two roundings of the step, one ulp of theta
        out["theta"] = 2 * U * np.abs(th1) + 4 * U * step
    elif kind == "momentum":
        mu = opt["momentum"]
        b0, b1 = _f64(prev["m"]), _f64(orc["m"])
        eb = 2 * U * np.abs(b1) + 2 * U * mu * np.abs(b0)      # fl(mu b) + g, stored
        out["m"] = eb
        out["theta"] = 2 * U * np.abs(th1) + 4 * U * step + lr * eb
    else:
        b1, b2, eps = opt["beta1"], opt["beta2"], opt["eps"]
        a1, a2 = 1.0 - b1, 1.0 - b2
        m0, m1 = _f64(prev["m"]), _f64(orc["m"])
        v0, v1 = _f64(prev["v"]), _f64(orc["v"])
        em = 2 * U * np.abs(m1) + 2 * U * (b1 * np.abs(m0) + a1 * np.abs(G))
        ev = 2 * U * np.abs(v1) + 3 * U * (b2 * np.abs(v0) + a2 * G * G)
        out["m"], out["v"] = em, ev
        bc1, bc2 = 1.0 - b1 ** (t + 1), 1.0 - b2 ** (t + 1)
        s = np.sqrt(np.maximum(v1, 0.0) / bc2)
        den = s + eps
        # the step lr m^/(sqrt(v^) + eps) carries the m and v roundings, and
        # rounds bc1, bc2, m/bc1, v/bc2, sqrt, + eps, /, lr * once each
        from_m = lr * em / (bc1 * den)
        from_v = np.where(s > 0, step * ev / (2.0 * np.maximum(s, 1e-300) * bc2 * den), 0.0)
        out["theta"] = 2 * U * np.abs(th1) + 10 * U * step + from_m + from_v
    return out


def state_bounds(opt: dict, t: int, orc: dict, prev: dict, k_elem=None):
    """Per-element tolerances for theta, m, v after one step from the same
    state prev (the inputs theta, m, v) on both sides."""
    g = orc["g_hat"].astype(np.float64)
    dg = ghat_bound(orc["mean_abs"], k_elem)
    dth, dm, dv = _sensitivities(opt, t, g, orc["m"], orc["v"])
    rnd = rounding_bounds(opt, t, orc, prev)

    def capped(name, x, carried):
        x = x.astype(np.float64)
        cap = STATE_REL * np.maximum(np.abs(x), rms(x))
        return np.minimum(rnd[name], cap) + carried + 1e-45

    out = {"theta": capped("theta", orc["theta"], 2 * dth * dg)}
    if orc["m"] is not None:
        out["m"] = capped("m", orc["m"], 2 * dm * dg)
    if orc["v"] is not None:
        out["v"] = capped("v", orc["v"], 2 * dv * dg)
    return out


def check_close(gpu, orc, bound, what):
    err = np.abs(np.asarray(gpu, np.float64) - np.asarray(orc, np.float64))
    bad = np.where(~(err <= bound))[0]
    assert bad.size == 0, (f"{what}: {bad.size}/{err.size} out of tolerance; first {bad[:5]} "
                           f"gpu={np.asarray(gpu)[bad[:5]]} orc={np.asarray(orc)[bad[:5]]} "
                           f"bound={np.asarray(bound)[bad[:5]]}")


def rep_values(rep: np.ndarray, gdtype: str) -> np.ndarray:
    return ostep.widen(rep, gdtype)


def cast_bits(theta32: np.ndarray, gdtype: str) -> np.ndarray:
    """Storage form of fp32 values in the replica dtype, by torch's conversion
    (used on GPU outputs, so the oracle is not involved)."""
    if gdtype == wl.BF16:
        t = torch.from_numpy(np.ascontiguousarray(theta32, dtype=np.float32)).to(torch.bfloat16)
        return wl.bf16_bits(t).numpy().astype(np.uint16)
    return np.asarray(theta32, np.float32)


def check_replicas(gpu_rep, gpu_theta, orc_rep, old_rep, R_elem, theta_bound, gdtype, what="replicas"):
    """Arrived elements: exactly the GPU's own rounding of its theta, close to the
    oracle's; lost elements: bit-identical to their previous contents."""
    gpu_rep = np.asarray(gpu_rep)
    R = R_elem.astype(bool)
    own = np.broadcast_to(cast_bits(gpu_theta, gdtype)[None, :], gpu_rep.shape)
    as_bits = (lambda a: a.view(np.uint32)) if gdtype == wl.F32 else (lambda a: a)
    assert np.array_equal(as_bits(gpu_rep)[R], as_bits(np.ascontiguousarray(own))[R]), \
        f"{what}: arrived packets differ from the rounding of the GPU master"
    assert np.array_equal(as_bits(gpu_rep)[~R], as_bits(np.asarray(old_rep))[~R]), \
        f"{what}: a lost packet was modified"
    gv = rep_values(gpu_rep, gdtype)
    ov = rep_values(orc_rep, gdtype)
    bound = BF16_REL * np.abs(ov) + np.broadcast_to(theta_bound[None, :], ov.shape) + 1e-30
    if gdtype == wl.F32:
        bound = np.broadcast_to(theta_bound[None, :], ov.shape) + 1e-30
    check_close(gv[R], ov[R], bound[R], what)


def torch_drift(replicas: torch.Tensor, theta: torch.Tensor, d: int, chunk: int = 1 << 22) -> dict:
    """Drift figures of [n][>= d] device replicas by plain torch fp64
    arithmetic, column chunk by column chunk: an independent check of the
    library's figures at full size, where the CPU oracle cannot take the
    whole shard.  Per element, with r = the replica rounding of theta and
    x_i - r exact in fp64: range max_i x - min_i x, pair sum
    N sum (x_i - r)^2 - (sum (x_i - r))^2 (clamped at 0), sum |x_i - r|."""
    n = replicas.shape[0]
    mx, pair, absum = 0.0, 0.0, 0.0
    for c0 in range(0, d, chunk):
        c1 = min(d, c0 + chunk)
        x = replicas[:, c0:c1].double()
        r = theta[c0:c1].to(replicas.dtype).double()
        mx = max(mx, float((x.max(0).values - x.min(0).values).max()))
        x -= r[None, :]
        s1 = x.sum(0)
        s2 = (x * x).sum(0)
        pair += float((n * s2 - s1 * s1).clamp_min(0.0).sum())
        absum += float(x.abs().sum())
        del x, r, s1, s2
    pairs = n * (n - 1) / 2
    return dict(max_abs=mx, mean_sq=pair / (d * pairs) if pairs else 0.0,
                mean_abs_to_master=absum / (n * d))


def check_drift_close(got: dict, ref: dict, what: str):
    """max_abs exactly; mean_sq and mean_abs_to_master to 1e-9 relative
    (fp64 sums of the same terms in another order)."""
    assert got["max_abs"] == ref["max_abs"], (what, got, ref)
    for k in ("mean_sq", "mean_abs_to_master"):
        assert abs(got[k] - ref[k]) <= 1e-9 * abs(ref[k]) + 1e-300, (what, k, got, ref)


# ---------------------------------------------------------------------------
# Device state of a workload and the oracle's view of sampled packets
# ---------------------------------------------------------------------------
import paper_2507_07114_amd as ll  # noqa: E402,F401
from workloads.device import DeviceState, loss_spec, opt_spec  # noqa: E402,F401

from oracle import loss as oloss  # noqa: E402


class OracleMasks:
    """The oracle's masks of a workload, all packets, carrying GE state."""

    def __init__(self, w: wl.Workload):
        self.w = w
        self.state = {0: np.zeros(w.n, np.uint8), 1: np.zeros(w.n, np.uint8)}

    def masks(self, t: int, direction: int) -> np.ndarray:
        w, l = self.w, self.w.loss
        if l["kind"] == wl.BERNOULLI:
            return oloss.bernoulli_arrivals(w.seed, t, direction, w.n,
                                            np.arange(w.num_packets), l["p"])
        a, self.state[direction] = oloss.ge_arrivals(
            w.seed, t, direction, w.n, w.num_packets, l["p_gb"], l["p_bg"],
            l["loss_good"], l["loss_bad"], self.state[direction])
        return a


class SampledOracle:
    """Oracle state restricted to the elements of a packet sample."""

    def __init__(self, w: wl.Workload, packets, dev: DeviceState):
        self.w = w
        self.packets = list(packets)
        self.idx = elements_of(w, self.packets)
        self.theta = host_vec(dev.theta, self.idx).astype(np.float32)
        self.m = None if dev.m is None else host_vec(dev.m, self.idx).astype(np.float32)
        self.v = None if dev.v is None else host_vec(dev.v, self.idx).astype(np.float32)
        self.replicas = host_rows(dev.replicas, self.idx, w.gdtype)

    def run(self, t: int, grads_host, mg: np.ndarray, mb: np.ndarray, **kw) -> dict:
        """One oracle step of the sampled elements from the current state
        (mg, mb: masks of the sampled packets); the state is not advanced."""
        w = self.w
        return ostep.lossy_step(d=w.d, packet=w.packet, packets=self.packets, gdtype=w.gdtype,
                                grads=grads_host, theta=self.theta, m=self.m, v=self.v,
                                replicas=self.replicas, arrived_g=mg, arrived_b=mb,
                                opt=opt_as_given(w.opt), t=t, **kw)

    def advance(self, out: dict):
        """Take an oracle step's outputs as the new state, keeping the inputs
        (compare_step bounds the update from them)."""
        self.prev = dict(theta=self.theta, m=self.m, v=self.v)
        self.prev_replicas = self.replicas
        self.theta, self.m, self.v, self.replicas = out["theta"], out["m"], out["v"], out["replicas"]

    def step(self, t: int, grads_host, mg: np.ndarray, mb: np.ndarray, lam: float = 0.0):
        """run() on the sample's columns of full-width masks, then advance()."""
        out = self.run(t, grads_host, mg[:, self.packets], mb[:, self.packets], lam=lam)
        self.advance(out)
        return out

    def upload(self, dev: DeviceState):
        """Put the oracle's state of the sampled elements into the device buffers."""
        ix = torch.as_tensor(self.idx, device=dev.theta.device)
        dev.theta.index_copy_(0, ix, torch.from_numpy(self.theta).to(dev.theta.device))
        if self.m is not None:
            dev.m.index_copy_(0, ix, torch.from_numpy(self.m).to(dev.theta.device))
        if self.v is not None:
            dev.v.index_copy_(0, ix, torch.from_numpy(self.v).to(dev.theta.device))
        if self.w.gdtype == wl.BF16:
            rep = torch.from_numpy(self.replicas.astype(np.int32).astype(np.int16)).view(torch.bfloat16)
        else:
            rep = torch.from_numpy(self.replicas)
        dev.replicas.index_copy_(1, ix, rep.to(dev.replicas.device))


def compare_step(w: wl.Workload, t: int, dev: DeviceState, so: SampledOracle, orc: dict,
                 mb_sample: np.ndarray, label: str):
    """Compare the device state on the sampled elements with one oracle step."""
    lens = ostep.packet_lengths(w.d, w.packet, so.packets)
    K_elem = np.repeat(orc["counts"], lens)
    g_theta = host_vec(dev.theta, so.idx)
    bounds = state_bounds(opt_as_given(w.opt), t, orc, so.prev, K_elem)
    check_close(g_theta, orc["theta"], bounds["theta"], f"{label} theta")
    if dev.m is not None:
        check_close(host_vec(dev.m, so.idx), orc["m"], bounds["m"], f"{label} m")
    if dev.v is not None:
        check_close(host_vec(dev.v, so.idx), orc["v"], bounds["v"], f"{label} v")
    R_elem = np.repeat(mb_sample, lens, axis=1)
    check_replicas(host_rows(dev.replicas, so.idx, w.gdtype), g_theta, orc["replicas"],
                   so.prev_replicas, R_elem, bounds["theta"], w.gdtype, f"{label} replicas")
