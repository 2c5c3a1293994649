"""One lossy step on the owner's shard: aggregate, update, broadcast.

Test infrastructure (see the package docstring).  All arithmetic is float64;
values are rounded only where the product stores them (fp32 g_hat, fp32
master and optimizer state, replicas in their storage dtype).

The shard is cut into packets of L elements (the last may be short); every
function here works on the elements of a chosen list of packets, so large
shards can be checked on a sample.
"""
from __future__ import annotations

import numpy as np

from . import bf16

F32 = "f32"
BF16 = "bf16"


def packet_lengths(d: int, packet: int, packets) -> np.ndarray:
    k = np.asarray(packets, dtype=np.int64)
    return np.minimum((k + 1) * packet, d) - k * packet


def packet_elements(d: int, packet: int, packets) -> np.ndarray:
    """Element indices of the chosen packets, in packet order."""
    parts = [np.arange(k * packet, min((k + 1) * packet, d), dtype=np.int64)
             for k in packets]
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)


def widen(values, dtype: str) -> np.ndarray:
    """Stored values (fp32 numbers, or bf16 bit patterns) -> float64."""
    if dtype == BF16:
        return bf16.to_f64(values)
    return np.asarray(values, dtype=np.float32).astype(np.float64)


def store(values64, dtype: str) -> np.ndarray:
    """float64 -> storage: fp32 values, or bf16 bit patterns of the fp32 value."""
    f32 = np.asarray(values64, dtype=np.float64).astype(np.float32)
    return bf16.from_f32(f32) if dtype == BF16 else f32


def aggregate(g: np.ndarray, S: np.ndarray, lam: float, theta: np.ndarray):
    """Unbiased aggregate of Section 3 step (2), restated in "Unbiased Gradient
    Aggregation": per element, the sum of the contributions that arrived
    divided by how many arrived.  For a packet with no arrival the paper
    leaves the substitute value open (some small regularising term); the
    reading here is lam * theta.

    g: [n][E] float64, S: [n][E] in {0,1}, theta: [E] float64.
    Returns (g_hat [E], K [E], mean |contribution| [E]).
    """
    S = S.astype(np.float64)
    K = S.sum(axis=0)
    total = (S * g).sum(axis=0)
    mag = (S * np.abs(g)).sum(axis=0)
    safe = np.maximum(K, 1.0)
    g_hat = np.where(K > 0, total / safe, lam * theta)
    mean_abs = np.where(K > 0, mag / safe, np.abs(lam * theta))
    return g_hat, K.astype(np.int64), mean_abs


def aggregate_horvitz_thompson(g: np.ndarray, S: np.ndarray, q: np.ndarray):
    """Horvitz-Thompson form of the aggregate (one of the estimator variants
    for unreliable delivery): every arrived contribution is weighted by the
    inverse of its arrival probability q and the sum is divided by N, so
    E[g_hat] = mean over all N rows with no conditioning and no fallback.

    g, S, q: [n][E] (q = 1 for rows or packets that cannot be lost).
    Returns (g_hat [E], scale [E]) with scale = sum_i S |g| / q / N.
    """
    n = g.shape[0]
    S = S.astype(np.float64)
    g_hat = (S * g / q).sum(axis=0) / n
    scale = (S * np.abs(g) / q).sum(axis=0) / n
    return g_hat, scale


def aggregate_stale_fill(g: np.ndarray, S: np.ndarray, g_prev: np.ndarray):
    """Algorithm 1's gradient half, per contribution: a lost contribution is
    replaced by the last one that arrived from that worker for the same
    element (g_prev, zero before the first arrival), an arrived one is used
    and remembered; the N values are then averaged.

    Returns (g_hat [E], new g_prev [n][E], scale [E] = mean |value|).
    """
    n = g.shape[0]
    A = S.astype(bool)
    vals = np.where(A, g, g_prev)
    return vals.sum(axis=0) / n, np.where(A, g, g_prev), np.abs(vals).sum(axis=0) / n


def update_ages(ages: np.ndarray, R: np.ndarray, cap: int = 65535) -> np.ndarray:
    """Steps since each (replica, packet) last received the broadcast:
    0 where it arrived this step, previous age + 1 (saturating) otherwise."""
    a = np.asarray(ages, dtype=np.int64)
    return np.where(np.asarray(R).astype(bool), 0, np.minimum(a + 1, cap)).astype(np.uint16)


def sgd(theta, g_hat, lr):
    """Section 3 step (3): theta_{t+1} = theta_t - eta * g_hat."""
    return theta - lr * g_hat


def sgd_momentum(theta, buf, g_hat, lr, mu):
    """Heavy-ball momentum (buffer starts at zero, no dampening):
    b = mu b + g_hat;  theta = theta - eta b."""
    buf = mu * buf + g_hat
    return theta - lr * buf, buf


def adam(theta, m, v, g_hat, t, lr, beta1, beta2, eps):
    """Adam (Kingma & Ba) with bias correction, eps added after the square
    root, no weight decay; t is the 1-based step count."""
    m = beta1 * m + (1.0 - beta1) * g_hat
    v = beta2 * v + (1.0 - beta2) * g_hat * g_hat
    m_hat = m / (1.0 - beta1 ** t)
    v_hat = v / (1.0 - beta2 ** t)
    return theta - lr * m_hat / (np.sqrt(v_hat) + eps), m, v


def broadcast(old, new, R):
    """Section 3 step (4): a replica takes the owner's new value where the
    broadcast arrived (R = 1) and keeps its stale value otherwise."""
    return np.where(R.astype(bool), new, old)


def lossy_step(*, d: int, packet: int, packets, gdtype: str, grads, theta, m, v,
               replicas, arrived_g, arrived_b, opt: dict, t: int,
               lam: float = 0.0, estimator: str = "arrived_mean", q=None,
               g_prev=None):
    """One step over the chosen packets.

    grads, replicas: [n][E] storage values for the packets' elements
    (fp32, or bf16 bit patterns); theta, m, v: [E] fp32 (m, v may be None);
    arrived_g, arrived_b: uint8 [n][len(packets)]; t: 0-based step index.
    estimator: "arrived_mean" (Section 3 step (2)), "horvitz_thompson" (needs
    q: arrival probabilities [n][len(packets)]) or "stale_fill" (Algorithm 1;
    needs g_prev, storage values [n][E], returned updated).
    Returns a dict with g_hat (fp32), counts (per packet), mean_abs (per
    element: the scale of the terms summed), theta, m, v (fp32), replicas
    (storage dtype) and g_prev (stale_fill only).
    """
    lens = packet_lengths(d, packet, packets)
    S = np.repeat(np.asarray(arrived_g), lens, axis=1)
    R = np.repeat(np.asarray(arrived_b), lens, axis=1)
    g = widen(grads, gdtype)
    th = np.asarray(theta, dtype=np.float32).astype(np.float64)

    new_prev = None
    if estimator == "arrived_mean":
        g_hat64, _, mean_abs = aggregate(g, S, lam, th)
    elif estimator == "horvitz_thompson":
        Q = np.repeat(np.asarray(q, dtype=np.float64), lens, axis=1)
        g_hat64, mean_abs = aggregate_horvitz_thompson(g, S, Q)
    elif estimator == "stale_fill":
        g_hat64, prev64, mean_abs = aggregate_stale_fill(g, S, widen(g_prev, gdtype))
        new_prev = np.where(S.astype(bool), np.asarray(grads), np.asarray(g_prev))
    else:
        raise ValueError(f"unknown estimator {estimator!r}")
    g_hat32 = g_hat64.astype(np.float32)
    G = g_hat32.astype(np.float64)

    kind = opt["kind"]
    m1 = v1 = None
    if kind == "sgd":
        th1 = sgd(th, G, opt["lr"])
    elif kind == "momentum":
        th1, m1 = sgd_momentum(th, np.asarray(m, np.float32).astype(np.float64), G,
                               opt["lr"], opt["momentum"])
    elif kind == "adam":
        th1, m1, v1 = adam(th, np.asarray(m, np.float32).astype(np.float64),
                           np.asarray(v, np.float32).astype(np.float64), G, t + 1,
                           opt["lr"], opt["beta1"], opt["beta2"], opt["eps"])
    else:
        raise ValueError(f"unknown optimizer {kind!r}")

    theta32 = th1.astype(np.float32)
    new_val = store(theta32.astype(np.float64), gdtype)
    reps = broadcast(np.asarray(replicas), new_val[None, :], R)
    counts = np.asarray(arrived_g).astype(np.int64).sum(axis=0)
    return dict(
        g_hat=g_hat32, counts=counts, mean_abs=mean_abs, theta=theta32,
        m=None if m1 is None else m1.astype(np.float32),
        v=None if v1 is None else v1.astype(np.float32),
        replicas=reps, g_prev=new_prev)
