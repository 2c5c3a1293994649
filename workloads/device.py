"""Device buffers of a workload and the call of the fused step on them.

Allocation and argument conversion only: the step itself runs in the HIP
library through its Python binding.
"""
from __future__ import annotations

import torch

import paper_2507_07114_amd as ll

from . import (ADAM, BERNOULLI, MOMENTUM, SGD, Workload, draw_grads, draw_theta0,
               initial_replicas, torch_dtype)

def loss_spec(w: Workload) -> "ll.LossSpec":
    l = w.loss
    if l["kind"] == BERNOULLI:
        return ll.bernoulli(l["p"], seed=w.seed)
    return ll.gilbert_elliott(l["p_gb"], l["p_bg"], l["loss_good"], l["loss_bad"], seed=w.seed)


def opt_spec(w: Workload, lam: float = 0.0) -> "ll.OptSpec":
    o = w.opt
    if o["kind"] == SGD:
        return ll.sgd(o["lr"], lam)
    if o["kind"] == MOMENTUM:
        return ll.sgd_momentum(o["lr"], o["momentum"], lam)
    return ll.adam(o["lr"], o["beta1"], o["beta2"], o["eps"], lam)


class DeviceState:
    """All device buffers of one workload (rows padded to `ld`)."""

    def __init__(self, w: Workload, device="cuda", pad: int = 0, draw_grads_now=True):
        self.w = w
        self.ld = w.ld(pad)
        self.theta = draw_theta0(w, device)
        self.m = torch.zeros(w.d, dtype=torch.float32, device=device) \
            if w.opt["kind"] in (MOMENTUM, ADAM) else None
        self.v = torch.zeros(w.d, dtype=torch.float32, device=device) \
            if w.opt["kind"] == ADAM else None
        self.replicas = initial_replicas(self.theta, w, ld=self.ld)
        self.grads = torch.zeros((w.n, self.ld), dtype=torch_dtype(w.gdtype), device=device)
        if draw_grads_now:
            draw_grads(w, 0, device=device, ld=self.ld, out=self.grads)
        P = w.num_packets
        self.arrived_g = torch.zeros((w.n, P), dtype=torch.uint8, device=device)
        self.arrived_b = torch.zeros((w.n, P), dtype=torch.uint8, device=device)
        self.counts = torch.zeros(P, dtype=torch.int32, device=device)
        self.ge_g = torch.zeros(w.n, dtype=torch.uint8, device=device)
        self.ge_b = torch.zeros(w.n, dtype=torch.uint8, device=device)
        self.workspace = torch.zeros(max(ll.ll_workspace_bytes(w.n, w.d, w.packet), 256),
                                     dtype=torch.uint8, device=device)
        self.drift = ll.drift_buffer(device)

    def fused(self, step: int, drift=True, lam: float = 0.0, masks_out=True, ext=None):
        w = self.w
        spec = loss_spec(w)
        ll.lossy_step_fused(
            d=w.d, packet=w.packet, step=step, loss_g=spec, loss_b=spec, grads=self.grads,
            opt=opt_spec(w, lam), theta=self.theta, replicas=self.replicas, m=self.m, v=self.v,
            ge_state_g=self.ge_g, ge_state_b=self.ge_b,
            arrived_g=self.arrived_g if masks_out else None,
            arrived_b=self.arrived_b if masks_out else None,
            counts=self.counts if masks_out else None, workspace=self.workspace,
            drift=self.drift if drift else None, ext=ext)
