"""Inter-replica drift statistics.

Test infrastructure (see the package docstring).  Theorem 3.1 studies the
discrepancy D = theta^(i,j) - theta^(k,j) between two workers' copies of the
same shard.  Over N replicas x_1..x_N of every element e this module reports

  max_abs            max over e of the largest pairwise |x_i - x_k|
                     (= max_i x_i - min_i x_i);
  mean_sq            mean over elements and unordered pairs i < k of
                     (x_i - x_k)^2, the quantity the theorem bounds;
  rms                sqrt(mean_sq);
  mean_abs_to_master mean over i and e of |x_i - c(theta_e)|, c the
                     replica storage rounding of the owner's master value;
  stale_packets      number of (replica, packet) broadcasts that were lost.

Everything is float64; the pairwise sum is the plain double loop over pairs.
"""
from __future__ import annotations

import math

import numpy as np


def drift_stats(x: np.ndarray, master=None, arrived_b=None) -> dict:
    """x: [n][E] float64 replica values; master: [E] float64 or None;
    arrived_b: broadcast arrivals uint8 [n][packets] or None."""
    x = np.asarray(x, dtype=np.float64)
    n, e = x.shape
    if e == 0:
        max_abs = 0.0
    else:
        max_abs = float(np.max(np.max(x, axis=0) - np.min(x, axis=0)))
    pair_sum = 0.0
    for i in range(n - 1):
        diff = x[i + 1:, :] - x[i, :][None, :]
        pair_sum += float(np.sum(diff * diff))
    pairs = n * (n - 1) // 2
    mean_sq = pair_sum / (e * pairs) if e * pairs > 0 else 0.0
    if master is None:
        mean_abs_to_master = math.nan
    else:
        mean_abs_to_master = (float(np.sum(np.abs(x - np.asarray(master)[None, :])))
                              / (n * e) if n * e > 0 else 0.0)
    stale = 0 if arrived_b is None else int(np.sum(np.asarray(arrived_b) == 0))
    return dict(max_abs=max_abs, mean_sq=mean_sq, rms=math.sqrt(mean_sq),
                mean_abs_to_master=mean_abs_to_master, stale_packets=stale,
                pair_sum=pair_sum, elements=e, pairs=pairs)
