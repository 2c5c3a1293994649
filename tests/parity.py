"""Shared helpers of the GPU parity tests: host copies of sampled packets and
the comparison norms.

Norms, each with the floating-point reasoning behind it:
  * masks, counts, packet bookkeeping, GE state: bit-exact.
  * g_hat: |gpu - orc| <= max(1e-5, K 2^-24) * A_e, A_e = mean |arrived
    contribution| (for an empty packet A_e = |lam * theta|).  A sequential
    fp32 sum of K terms is within (K-1) 2^-24 sum|g| of the exact sum, and
    the division adds one rounding, so the error is at most K 2^-24 A_e:
    below 1e-5 A_e up to K = 167 workers, the worst-case bound above that.
  * theta, m, v: 1e-5 * max(|orc|, rms(orc)) plus the first-order effect of
    the g_hat tolerance propagated through the update (|d theta / d g_hat|
    times the g_hat bound, doubled for slack).  This matters only for Adam
    where g_hat is within its own rounding of zero.
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
    rel = GHAT_REL
    if k_elem is not None:
        rel = np.maximum(GHAT_REL, np.asarray(k_elem, np.float64) * 2.0**-24)
    return rel * mean_abs + 1e-30


def check_ghat(gpu: np.ndarray, orc: np.ndarray, mean_abs: np.ndarray, k_elem=None,
               what="g_hat"):
    err = np.abs(gpu.astype(np.float64) - orc.astype(np.float64))
    bound = ghat_bound(mean_abs, k_elem)
    bad = np.where(~(err <= bound))[0]
    assert bad.size == 0, (f"{what}: {bad.size} elements out of tolerance; first {bad[:5]} "
                           f"gpu={gpu[bad[:5]]} orc={orc[bad[:5]]} bound={bound[bad[:5]]}")


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


def state_bounds(opt: dict, t: int, orc: dict, k_elem=None):
    """Per-element tolerances for theta, m, v after one step from identical state."""
    g = orc["g_hat"].astype(np.float64)
    dg = ghat_bound(orc["mean_abs"], k_elem)
    dth, dm, dv = _sensitivities(opt, t, g, orc["m"], orc["v"])
    th = orc["theta"].astype(np.float64)
    out = {"theta": STATE_REL * np.maximum(np.abs(th), rms(th)) + 2 * dth * dg}
    if orc["m"] is not None:
        mm = orc["m"].astype(np.float64)
        out["m"] = STATE_REL * np.maximum(np.abs(mm), rms(mm)) + 2 * dm * dg + 1e-30
    if orc["v"] is not None:
        vv = orc["v"].astype(np.float64)
        out["v"] = STATE_REL * np.maximum(np.abs(vv), rms(vv)) + 2 * dv * dg + 1e-30
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

    def step(self, t: int, grads_host, mg: np.ndarray, mb: np.ndarray, lam: float = 0.0):
        w = self.w
        out = ostep.lossy_step(d=w.d, packet=w.packet, packets=self.packets, gdtype=w.gdtype,
                               grads=grads_host, theta=self.theta, m=self.m, v=self.v,
                               replicas=self.replicas, arrived_g=mg[:, self.packets],
                               arrived_b=mb[:, self.packets], opt=w.opt, t=t, lam=lam)
        self.prev_replicas = self.replicas
        self.theta, self.m, self.v, self.replicas = out["theta"], out["m"], out["v"], out["replicas"]
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
    bounds = state_bounds(w.opt, t, orc, K_elem)
    check_close(g_theta, orc["theta"], bounds["theta"], f"{label} theta")
    if dev.m is not None:
        check_close(host_vec(dev.m, so.idx), orc["m"], bounds["m"], f"{label} m")
    if dev.v is not None:
        check_close(host_vec(dev.v, so.idx), orc["v"], bounds["v"], f"{label} v")
    R_elem = np.repeat(mb_sample, lens, axis=1)
    check_replicas(host_rows(dev.replicas, so.idx, w.gdtype), g_theta, orc["replicas"],
                   so.prev_replicas, R_elem, bounds["theta"], w.gdtype, f"{label} replicas")
