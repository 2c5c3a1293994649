"""CPU oracle for the packet-loss-tolerant data-parallel step.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 restatement of
what the paper "Distributed Training under Packet Loss" (Weintraub, Banner,
Orda, 2025) defines for one owner's shard:

  * Section 3 step (2): per-(worker, packet) Bernoulli arrival indicators and
    the rescaled aggregate  g_hat = sum_i s_i g_i / sum_i s_i;
  * Section 3 "Unbiased Gradient Aggregation": the same estimator, with a
    fallback when nothing arrives;
  * Section 3 step (3): the owner's local update (plus momentum and Adam);
  * Section 3 step (4): the lossy broadcast that keeps stale values;
  * Theorem 3.1: the inter-replica discrepancy D = theta^(i,j) - theta^(k,j);
  * Algorithm 1's gradient half: a lost contribution replaced by the last one
    that arrived, averaged over N (stale fill);
  * Section 5 directions: transfers that cannot be lost (the owner's own row,
    reliable packets), XOR parity packets over groups of packets, and the
    per-replica record of broadcast ages (the routing log);
  * beyond the paper: a Horvitz-Thompson form of the aggregate and bursty
    Gilbert-Elliott loss (Section 5 names bursty loss as open).

It shares no code with the HIP library and never imports it.  Only the test
suite, the smoke entry point and the benchmark's CPU-baseline leg may import
anything from here; the product path never does.

Parity pins: every function here is checked by `tests/test_oracle_*.py`
against values the paper or mathematics fixes (closed forms, special cases,
brute-force enumeration, Monte Carlo, third-party library routines).
"""
from . import bf16, drift, loss, philox, step  # noqa: F401

__all__ = ["bf16", "drift", "loss", "philox", "step"]
