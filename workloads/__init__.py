"""Seeded synthetic workloads for the lossy data-parallel step.

This module only draws inputs: gradient rows, the initial fp32 master shard
and the replica buffers.  It holds none of the method's arithmetic (no masks,
no aggregation, no optimizer, no broadcast); both the HIP path and the CPU
oracle receive what it produces.

The paper trains LLaMA-2 7B on 64 accelerators (Section 4, Table 1); its
gradients, weights and corpus are not available, so these seeded
distributions stand in for them at the paper's shard shape (a 6.74e9-element
model split 64 ways, Section 3 "Model Formulation").
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

F32 = "f32"
BF16 = "bf16"

SGD = "sgd"
MOMENTUM = "momentum"
ADAM = "adam"

BERNOULLI = "bernoulli"
GILBERT_ELLIOTT = "gilbert_elliott"


@dataclasses.dataclass(frozen=True)
class Workload:
    """One configuration of the lossy step.

    n       worker count N (Section 3, shards owned by W_1..W_N)
    d       elements of the owned shard
    packet  elements per packet L; P = ceil(d / L), the last may be short
    gdtype  gradient row dtype; the replica dtype is the same
    grad    gradient distribution: ("normal", std) or ("student_t", dof, scale)
    loss    loss-process parameters (kind, p or Gilbert-Elliott rates)
    opt     optimizer kind and hyper-parameters
    steps   number of steps the configuration runs
    """
    name: str
    n: int
    d: int
    packet: int
    gdtype: str
    grad: tuple
    loss: dict
    opt: dict
    steps: int
    theta_std: float = 0.02
    drift_every_step: bool = False
    seed: int = 0

    @property
    def num_packets(self) -> int:
        return (self.d + self.packet - 1) // self.packet

    @property
    def elem_bytes(self) -> int:
        return 2 if self.gdtype == BF16 else 4

    def ld(self, pad: int = 0) -> int:
        """Row stride in elements: d rounded up to 256 elements, plus `pad`."""
        return ((self.d + 255) // 256) * 256 + pad


ADAM_DEFAULT = dict(kind=ADAM, lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, momentum=0.0)

WORKLOADS = {
    # N=4 workers, 1 Mi fp32 elements, SGD, one step.
    "n4_d1m_f32_sgd": Workload(
        name="n4_d1m_f32_sgd", n=4, d=1_048_576, packet=1024, gdtype=F32,
        grad=("normal", 1.0),
        loss=dict(kind=BERNOULLI, p=0.1),
        opt=dict(kind=SGD, lr=0.01, momentum=0.0, beta1=0.0, beta2=0.0, eps=0.0),
        steps=1),
    # N=8 workers, 16 Mi bf16 elements, Adam, ten steps with fresh gradients.
    "n8_d16m_bf16_adam": Workload(
        name="n8_d16m_bf16_adam", n=8, d=16_777_216, packet=2048, gdtype=BF16,
        grad=("normal", 1e-3),
        loss=dict(kind=BERNOULLI, p=0.01),
        opt=dict(ADAM_DEFAULT), steps=10),
    # N=64: one worker's ZeRO-2 shard of a 6.74e9-element model, bf16, Adam.
    "n64_llama7b_shard_bf16_adam": Workload(
        name="n64_llama7b_shard_bf16_adam", n=64, d=105_250_000, packet=4096,
        gdtype=BF16, grad=("normal", 1e-3),
        loss=dict(kind=BERNOULLI, p=0.1),
        opt=dict(ADAM_DEFAULT), steps=1),
    # N=16, 256 Mi fp32 heavy-tailed gradients, bursty Gilbert-Elliott loss.
    "n16_d256m_f32_ge_momentum": Workload(
        name="n16_d256m_f32_ge_momentum", n=16, d=268_435_456, packet=4096,
        gdtype=F32, grad=("student_t", 3, 1e-3),
        loss=dict(kind=GILBERT_ELLIOTT, p_gb=0.01, p_bg=0.2,
                  loss_good=0.0, loss_bad=0.5),
        opt=dict(kind=MOMENTUM, lr=0.01, momentum=0.9, beta1=0.0, beta2=0.0,
                 eps=0.0),
        steps=5),
    # N=64 replicas, 48 Mi fp32 elements, SGD, 200 steps with drift each step.
    "n64_d48m_f32_sgd_drift": Workload(
        name="n64_d48m_f32_sgd_drift", n=64, d=50_331_648, packet=2048,
        gdtype=F32, grad=("normal", 1e-3),
        loss=dict(kind=BERNOULLI, p=0.1),
        opt=dict(kind=SGD, lr=1e-3, momentum=0.0, beta1=0.0, beta2=0.0, eps=0.0),
        steps=200, drift_every_step=True),
}

METRIC_WORKLOAD = "n64_llama7b_shard_bf16_adam"


def scaled(w: Workload, *, n: Optional[int] = None, d: Optional[int] = None,
           packet: Optional[int] = None, steps: Optional[int] = None,
           **kw) -> Workload:
    """A copy of `w` with some sizes replaced (for small parity cases)."""
    rep = {}
    if n is not None:
        rep["n"] = n
    if d is not None:
        rep["d"] = d
    if packet is not None:
        rep["packet"] = packet
    if steps is not None:
        rep["steps"] = steps
    rep.update(kw)
    return dataclasses.replace(w, **rep)


def torch_dtype(gdtype: str) -> torch.dtype:
    return torch.bfloat16 if gdtype == BF16 else torch.float32


def _gen(device, seed: int, stream: int) -> torch.Generator:
    g = torch.Generator(device=device)
    # Distinct, fixed sub-seeds per purpose: (seed, stream) -> one 63-bit seed.
    g.manual_seed((seed * 1_000_003 + stream * 7_919 + 12345) & ((1 << 63) - 1))
    return g


def draw_theta0(w: Workload, device="cpu") -> torch.Tensor:
    """Initial fp32 master shard, N(0, theta_std^2) (std convention)."""
    g = _gen(device, w.seed, 1)
    return torch.randn(w.d, generator=g, device=device, dtype=torch.float32) * w.theta_std


def _fill_grad_row(out_row: torch.Tensor, w: Workload, g: torch.Generator):
    kind = w.grad[0]
    d = out_row.numel()
    if kind == "normal":
        std = float(w.grad[1])
        tmp = torch.randn(d, generator=g, device=out_row.device, dtype=torch.float32)
        out_row.copy_(tmp.mul_(std))
    elif kind == "student_t":
        dof, scale = int(w.grad[1]), float(w.grad[2])
        # t_nu = Z / sqrt(chi2_nu / nu), chi2_nu = sum of nu squared normals.
        z = torch.randn(d, generator=g, device=out_row.device, dtype=torch.float32)
        chi = torch.zeros(d, device=out_row.device, dtype=torch.float32)
        for _ in range(dof):
            y = torch.randn(d, generator=g, device=out_row.device, dtype=torch.float32)
            chi.addcmul_(y, y)
        out_row.copy_(z.div_(chi.div_(dof).sqrt_()).mul_(scale))
    else:
        raise ValueError(f"unknown gradient distribution {kind!r}")


def draw_grads(w: Workload, step: int, device="cpu", ld: Optional[int] = None,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Gradient rows [N][ld] for step `step` (fresh per step), dtype per workload.

    Columns d..ld-1 (row padding) are left zero.
    """
    ld = w.ld() if ld is None else ld
    dt = torch_dtype(w.gdtype)
    if out is None:
        out = torch.zeros((w.n, ld), dtype=dt, device=device)
    g = _gen(device, w.seed, 1000 + step)
    for i in range(w.n):
        _fill_grad_row(out[i, : w.d], w, g)
    return out


def initial_replicas(theta0: torch.Tensor, w: Workload, ld: Optional[int] = None,
                     out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Replica rows [N][ld]: every worker starts from the same copy of theta0
    stored in the replica dtype (torch's own conversion)."""
    ld = w.ld() if ld is None else ld
    dt = torch_dtype(w.gdtype)
    if out is None:
        out = torch.zeros((w.n, ld), dtype=dt, device=theta0.device)
    out[:, : w.d].copy_(theta0.to(dt).unsqueeze(0).expand(w.n, -1))
    return out


def packet_sample(w: Workload, count: int, seed: int = 7) -> list:
    """A fixed sample of packet indices: first, last (possibly ragged) and
    `count - 2` others spread by a seeded draw."""
    P = w.num_packets
    if P <= count:
        return list(range(P))
    g = torch.Generator(device="cpu").manual_seed(seed)
    mid = torch.randperm(P - 2, generator=g)[: count - 2] + 1
    return sorted({0, P - 1, *mid.tolist()})


def bf16_bits(x: torch.Tensor) -> torch.Tensor:
    """bf16 tensor -> its bit patterns as uint16-valued int32 (for numpy)."""
    return x.contiguous().view(torch.int16).to(torch.int32) & 0xFFFF


def describe(w: Workload) -> dict:
    return dict(workload=w.name, n=w.n, d=w.d, packet=w.packet,
                packets=w.num_packets, gdtype=w.gdtype, loss=w.loss,
                opt=w.opt["kind"], steps=w.steps)


__all__ = [
    "Workload", "WORKLOADS", "METRIC_WORKLOAD", "scaled", "draw_theta0",
    "draw_grads", "initial_replicas", "packet_sample", "torch_dtype",
    "bf16_bits", "describe", "F32", "BF16", "SGD", "MOMENTUM", "ADAM",
    "BERNOULLI", "GILBERT_ELLIOTT",
]
