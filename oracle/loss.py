"""Loss processes: which (worker, packet) transfers arrive.

Test infrastructure (see the package docstring).

Section 3 step (2) draws s_t^(i,j) ~ Bernoulli(1-p) for the gradient transfer
from worker i to owner j, and step (4) draws r_t^(j,i) ~ Bernoulli(1-p) for
the broadcast back; Algorithm 1 tests Uniform(0,1) < p to drop.  Here the
indicator is drawn per (worker i, packet k) of the owner's shard, 1 meaning
"arrived".  The uniform variate of Algorithm 1 is the top 32 bits of a
Philox4x64-10 word divided by 2**32, so "Uniform < p" is the integer test
hi32(w0) < ceil(p * 2**32); p = 0 never drops and p = 1 always drops.

Counter of the draw for step t (0-based), worker i, packet k and direction
dir (0 = gradient, 1 = broadcast):  ctr = (k, i, t, dir), key = (seed, 0).

The bursty Gilbert-Elliott process goes beyond the paper's i.i.d. model (its
Section 5 names bursty loss as open); each (dir, worker) runs a two-state
Markov chain over the packet sequence (step-major, then packet), starting in
Good before step 0.  Per packet the state first moves (Good->Bad when
hi32(w0) < ceil(p_gb 2^32), Bad->Good when hi32(w0) < ceil(p_bg 2^32)), then
the packet is lost when hi32(w1) < ceil(loss_state 2^32).

Parity packets (erasure coding, proposed in Section 5 for shards whose loss
hurts most): per row and group of G consecutive packets, one XOR parity
packet travels under the same Bernoulli p, drawn with counter (group, i, t,
dir + 2).  A group that lost exactly one packet, with its parity packet
arrived, rebuilds that packet bit for bit, so recovery changes only the
arrival indicators.
"""
from __future__ import annotations

import math

import numpy as np

from .philox import philox4x64

GRAD = 0
BCAST = 1
GOOD = 0
BAD = 1


def threshold(p: float) -> int:
    """ceil(p * 2**32) for p in [0, 1]: hi32(w) < threshold  <=>  hi32(w)/2**32 < p."""
    if not (0.0 <= p <= 1.0):
        raise ValueError("probability outside [0, 1]")
    return int(math.ceil(float(p) * 4294967296.0))


def draw_words(seed: int, t: int, direction: int, workers, packets):
    """Philox words (w0, w1) for every (worker, packet) pair: arrays [n][k]."""
    i = np.asarray(workers, dtype=np.uint64)[:, None]
    k = np.asarray(packets, dtype=np.uint64)[None, :]
    w0, w1, _, _ = philox4x64(k, i, np.uint64(t), np.uint64(direction), seed, 0)
    return w0, w1


def hi32(w: np.ndarray) -> np.ndarray:
    return (w >> np.uint64(32)).astype(np.int64)


def bernoulli_arrivals(seed: int, t: int, direction: int, n: int, packets, p: float):
    """uint8 [n][len(packets)], 1 = arrived, for i.i.d. loss probability p."""
    w0, _ = draw_words(seed, t, direction, np.arange(n), packets)
    lost = hi32(w0) < threshold(p)
    return (~lost).astype(np.uint8)


def ge_arrivals(seed: int, t: int, direction: int, n: int, num_packets: int,
                p_gb: float, p_bg: float, loss_good: float, loss_bad: float,
                state_in):
    """Gilbert-Elliott arrivals for all packets of step t.

    state_in: [n] states (0 Good, 1 Bad) at the end of step t-1 (all Good
    before step 0).  Returns (uint8 [n][num_packets], state_out [n]).
    The chain is walked packet by packet, all workers at once.
    """
    w0, w1 = draw_words(seed, t, direction, np.arange(n), np.arange(num_packets))
    u_move = hi32(w0)
    u_loss = hi32(w1)
    t_gb, t_bg = threshold(p_gb), threshold(p_bg)
    t_loss = np.array([threshold(loss_good), threshold(loss_bad)], dtype=np.int64)
    state = np.array(state_in, dtype=np.int64).copy()
    arrived = np.empty((n, num_packets), dtype=np.uint8)
    for k in range(num_packets):
        to_bad = (state == GOOD) & (u_move[:, k] < t_gb)
        to_good = (state == BAD) & (u_move[:, k] < t_bg)
        state = np.where(to_bad, BAD, np.where(to_good, GOOD, state))
        lost = u_loss[:, k] < t_loss[state]
        arrived[:, k] = np.where(lost, 0, 1)
    return arrived, state.astype(np.uint8)


def apply_overrides(arrived: np.ndarray, owner: int = -1, reliable=None) -> np.ndarray:
    """Transfers that never cross the lossy network.

    owner >= 0: the owner's own row always arrives (its own gradient piece
    and its own replica stay local; Section 3 step (4) broadcasts to the
    other workers).  reliable: per-packet flags (1 = sent over a reliable
    channel, the hybrid transport the paper's Section 5 proposes); a flagged
    packet arrives at every row.  arrived: uint8 [n][len(reliable)].
    """
    out = np.array(arrived, dtype=np.uint8, copy=True)
    if owner >= 0:
        out[owner, :] = 1
    if reliable is not None:
        out[:, np.asarray(reliable).astype(bool)] = 1
    return out


def parity_arrivals(seed: int, t: int, direction: int, n: int, groups, p: float):
    """Arrival of each worker's parity packet for the given packet groups:
    the same Bernoulli rule, drawn on direction dir + 2 (2 = gradient
    parity, 3 = broadcast parity) with the group index in the packet slot."""
    return bernoulli_arrivals(seed, t, direction + 2, n, groups, p)


def parity_recover(arrived: np.ndarray, group: int, parity_arrived: np.ndarray) -> np.ndarray:
    """Erasure coding over groups of `group` consecutive packets (the parity
    packets the paper's Section 5 proposes): a worker that sends an XOR
    parity packet per group lets the receiver rebuild exactly one lost packet
    of that group, bit for bit, when the parity packet itself arrived.

    arrived: uint8 [n][P] (after overrides); parity_arrived: uint8
    [n][ceil(P / group)].  Returns the arrivals after recovery.
    """
    n, P = arrived.shape
    out = np.array(arrived, dtype=np.uint8, copy=True)
    for gi in range((P + group - 1) // group):
        lo, hi = gi * group, min((gi + 1) * group, P)
        for i in range(n):
            lost = [k for k in range(lo, hi) if out[i, k] == 0]
            if len(lost) == 1 and parity_arrived[i, gi]:
                out[i, lost[0]] = 1
    return out


def parity_arrival_probability(q: float, group: int) -> float:
    """Marginal arrival probability of a packet in a full group of `group`
    i.i.d. packets plus parity, each arriving with probability q: it arrives,
    or it alone was lost and the other group - 1 packets and the parity
    packet arrived."""
    return q + (1.0 - q) * q**group


def parity_arrival_probabilities(q: float, group: int, num_packets: int, reliable=None):
    """Marginal arrival probability of every packet of a row under parity
    packets, float64 [num_packets].  A reliable packet always arrives (1).  A
    lossy packet k in a group of size g_k (the last group may be shorter)
    with r_k reliable other members arrives, or was lost while the other
    g_k - 1 - r_k lossy members and the parity packet arrived:
    q + (1 - q) q^(g_k - r_k)."""
    rel = np.zeros(num_packets, bool) if reliable is None else np.asarray(reliable).astype(bool)
    out = np.empty(num_packets)
    for k in range(num_packets):
        if rel[k]:
            out[k] = 1.0
            continue
        lo = (k // group) * group
        hi = min(lo + group, num_packets)
        r = int(rel[lo:hi].sum())  # k itself is not reliable
        out[k] = q + (1.0 - q) * q ** (hi - lo - r)
    return out


def ge_arrival_probability(t: int, k, num_packets: int, p_gb: float, p_bg: float,
                           loss_good: float, loss_bad: float):
    """Marginal arrival probability of packet k (array-like) of step t under
    the Gilbert-Elliott process above: the chain starts in Good before step 0
    and moves once before each packet, so packet k of step t follows
    n = t * num_packets + k + 1 moves.  For a two-state chain started in Good,
    P(Bad after n moves) = pi_B (1 - (1 - p_gb - p_bg)^n) with
    pi_B = p_gb / (p_gb + p_bg) (0 when the chain never moves)."""
    k = np.asarray(k, dtype=np.float64)
    n = float(t) * num_packets + k + 1.0
    s = p_gb + p_bg
    if s == 0.0:
        bad = np.zeros_like(n)
    else:
        lam = 1.0 - s
        bad = (p_gb / s) * (1.0 - np.power(lam, n))
    return 1.0 - (bad * loss_bad + (1.0 - bad) * loss_good)
