"""The seeded input recipes (CPU only): shapes, padding, determinism and the
value distributions the five workloads state."""
import numpy as np
import pytest
import torch

import workloads as wl


def test_workload_table():
    w = wl.WORKLOADS
    assert (w["n64_llama7b_shard_bf16_adam"].n, w["n64_llama7b_shard_bf16_adam"].d) == (64, 105_250_000)
    assert w["n64_llama7b_shard_bf16_adam"].num_packets == 25_696
    assert w["n16_d256m_f32_ge_momentum"].num_packets == 65_536
    assert w["n64_d48m_f32_sgd_drift"].num_packets == 24_576
    assert wl.METRIC_WORKLOAD == "n64_llama7b_shard_bf16_adam"
    for x in w.values():
        assert x.ld() % 256 == 0 and x.ld() >= x.d


def test_grads_deterministic_fresh_per_step_and_padded():
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], d=1000)
    a = wl.draw_grads(w, 3, ld=1024)
    b = wl.draw_grads(w, 3, ld=1024)
    c = wl.draw_grads(w, 4, ld=1024)
    assert a.dtype == torch.bfloat16 and a.shape == (8, 1024)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert not torch.equal(a, c)
    assert (a[:, 1000:] == 0).all()
    assert not torch.equal(a[0], a[1])   # rows are different workers


@pytest.mark.parametrize("name,std", [("n8_d16m_bf16_adam", 1e-3), ("n4_d1m_f32_sgd", 1.0)])
def test_normal_gradient_moments(name, std):
    w = wl.scaled(wl.WORKLOADS[name], n=2, d=200_000)
    g = wl.draw_grads(w, 0).float()[:, : w.d].double().numpy()
    se = std / np.sqrt(g.size)
    assert abs(g.mean()) < 5 * se
    assert abs(g.std() / std - 1) < 0.01


def test_student_t_gradient_recipe():
    # 1e-3 * t_3: variance 3 (dof / (dof - 2)) times 1e-6; heavy tails.
    w = wl.scaled(wl.WORKLOADS["n16_d256m_f32_ge_momentum"], n=2, d=400_000)
    g = wl.draw_grads(w, 0)[:, : w.d].double().numpy() / 1e-3
    assert abs(np.median(g)) < 0.01
    # P(|t_3| > 3.182) = 0.05 (two-sided 95% point of t with 3 dof)
    assert abs(np.mean(np.abs(g) > 3.182) - 0.05) < 0.003
    # heavy tail, closed form of the t_3 survival function:
    # S(x) = 1/2 - (atan(x / sqrt 3) + (x / sqrt 3) / (1 + x^2 / 3)) / pi
    u = 10 / np.sqrt(3)
    tail = 2 * (0.5 - (np.arctan(u) + u / (1 + u * u)) / np.pi)
    assert abs(np.mean(np.abs(g) > 10) / tail - 1) < 0.15


def test_theta0_and_replicas():
    w = wl.scaled(wl.WORKLOADS["n8_d16m_bf16_adam"], d=100_000)
    th = wl.draw_theta0(w)
    assert th.dtype == torch.float32 and abs(th.std().item() / 0.02 - 1) < 0.02
    r = wl.initial_replicas(th, w)
    assert r.shape == (8, w.ld())
    own = th.to(torch.bfloat16)
    assert all(torch.equal(r[i, : w.d].view(torch.int16), own.view(torch.int16)) for i in range(8))


def test_packet_sample_has_first_and_last():
    w = wl.WORKLOADS["n64_llama7b_shard_bf16_adam"]
    s = wl.packet_sample(w, 24)
    assert s[0] == 0 and s[-1] == w.num_packets - 1 and len(s) == 24 and s == sorted(set(s))
