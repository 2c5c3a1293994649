#!/usr/bin/env python3
"""Benchmark of the lossy data-parallel step on one MI355X.

One step = the whole hot path over one owner's shard: gradient and broadcast
masks, per-packet unbiased aggregate, Adam update of the fp32 master, lossy
broadcast into N bf16 replicas and drift statistics, i.e. one
lossy_step_fused call (the fused kernel plus its small drift reduction).

Default workload: N = 64 workers, one worker's ZeRO-2 shard of a
6.74e9-element model (D = 105,250,000 bf16 gradients per worker), packets of
4096 elements, i.i.d. loss p = 0.1 both ways, Adam, 64 bf16 replicas.

Throughput is algorithmic HBM bytes per second: arrived gradient packets
read, master + moments read and written, arrived replica packets written
and, for drift, stale replica packets read (lost gradient packets are never
needed, so never counted).  Prints one JSON line on stdout.  Workloads
smaller than 1 GiB get a 1 GiB scratch read between timed steps so that
they are not served from the 256 MB memory-side cache; their throughput is
then taken over the per-step events.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

HBM_PEAK_GBS = 8000.0
METRIC = "aggregate+step+broadcast GB/s and % of HBM peak; N=64 7B-shard step"
PMC_PROFILE = os.path.join(HERE, "profiles", "k_step_paced_n64_llama7b_shard_pmc.txt")
KERNEL_SOURCES = ["paper_2507_07114_amd/csrc/kernels.hip",
                  "paper_2507_07114_amd/csrc/lossy_device.h",
                  "paper_2507_07114_amd/csrc/kernels.h"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the kernel sources with comments and whitespace removed, so a
    stored counter profile stays valid across edits that change no code."""
    import re
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(HERE, rel)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def algorithmic_bytes(w, mg, mb, lens, drift: bool, estimator: str = "arrived_mean",
                      ages: bool = False, reliable: bool = False) -> dict:
    """Bytes the step must move given realised masks (numpy [n][P] arrays).
    The stale-fill estimator also reads the last arrived value of every lost
    contribution and stores every arrived one; ages are read and written
    once per (replica, packet); reliable flags are read once per packet."""
    import numpy as np
    eb = w.elem_bytes
    K = mg.sum(axis=0).astype(np.int64)
    R = mb.sum(axis=0).astype(np.int64)
    lens = lens.astype(np.int64)
    nstate = {"sgd": 1, "momentum": 2, "adam": 3}[w.opt["kind"]]
    d = int(lens.sum())
    out = dict(
        grads_read=int((K * lens).sum()) * eb,
        state_rw=2 * 4 * nstate * d,
        replicas_written=int((R * lens).sum()) * eb,
        stale_read=int(((w.n - R) * lens).sum()) * eb if drift else 0,
    )
    if estimator == "stale_fill":
        out["g_prev_read"] = int(((w.n - K) * lens).sum()) * eb
        out["g_prev_written"] = int((K * lens).sum()) * eb
    if ages:
        out["ages_rw"] = 2 * 2 * w.n * len(lens)
    if reliable:
        out["reliable_read"] = len(lens)
    out["total"] = sum(out.values())
    return out


def read_pmc_traffic(expect_hash: str, workload: str):
    """HBM bytes per dispatch from the committed rocprofv3 counter summary, or
    None when it is absent, was taken on different kernel sources or on
    another workload."""
    if not os.path.exists(PMC_PROFILE):
        return None
    vals = {}
    with open(PMC_PROFILE) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256") != expect_hash or vals.get("workload") != workload:
        return None
    try:
        return float(vals["hbm_bytes_per_dispatch"])
    except (KeyError, ValueError):
        return None


def _median_gbs(launch, reps: int = 3, batch: int = 5) -> float:
    """Median rate of `launch()` (which enqueues one kernel on torch's current
    stream and returns its bytes) over `reps` event-timed batches of `batch`
    back-to-back calls, after one untimed call."""
    import numpy as np
    import torch
    launch()
    torch.cuda.synchronize()
    rates = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        nbytes = sum(launch() for _ in range(batch))
        b.record()
        torch.cuda.synchronize()
        rates.append(nbytes / (a.elapsed_time(b) * 1e-3) / 1e9)
    return float(np.median(rates))


def hbm_copy_probe(nbytes: int = 2 << 30, reps: int = 3) -> float:
    """Device-to-device copy of a known size by the runtime (torch's copy
    kernel), as context beside the hand-written probes."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)

    def launch():
        dst.copy_(src)
        return 2 * nbytes
    gbs = _median_gbs(launch, reps)
    del src, dst
    torch.cuda.empty_cache()
    return gbs


def hbm_probes(rows_src=None, rows_dst=None, row_bytes: int = 0, nbytes: int = 2 << 30) -> dict:
    """Achievable HBM rates (GB/s) from the hand-written probes of
    libhbmprobe.so: a contiguous 16-byte copy, read-only and write-only
    streams of 2 GiB, and, given the step's own row buffers, the step's
    many-row shape (every row of the gradient buffer read, then every row of
    the replica buffer written, 4 KiB of each row per workgroup)."""
    import torch
    from paper_2507_07114_amd import probe
    sink = torch.zeros(probe.SINK_BYTES, dtype=torch.uint8, device="cuda")
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    out = {
        "copy_16B": _median_gbs(lambda: probe.hbm_probe_copy(a, b)),
        "read_16B": _median_gbs(lambda: probe.hbm_probe_read(a, sink)),
        "write_16B_nontemporal": _median_gbs(lambda: probe.hbm_probe_write(b)),
    }
    del a, b
    torch.cuda.empty_cache()
    if rows_src is not None and rows_dst is not None:
        n = rows_src.shape[0]
        out[f"rows_{n}r_{n}w"] = _median_gbs(
            lambda: probe.hbm_probe_rows(rows_src, n, rows_dst, n, row_bytes, sink))
        out[f"rows_{n}r"] = _median_gbs(
            lambda: probe.hbm_probe_rows(rows_src, n, None, 0, row_bytes, sink))
    return {k: round(v, 1) for k, v in out.items()}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_baseline(w, dev, packets_sample: int):
    """The oracle, as it stands, on a bounded sample of packets of the same
    workload (inputs copied from the device before any step runs)."""
    import numpy as np
    from oracle import drift as odrift
    from oracle import loss as oloss
    from oracle import step as ostep
    P = w.num_packets
    sample = list(range(0, P, max(1, P // packets_sample)))[:packets_sample]
    idx = ostep.packet_elements(w.d, w.packet, sample)
    import torch
    ix = torch.as_tensor(idx, device=dev.theta.device)

    def rows(t):
        x = t.index_select(1, ix).cpu()
        if w.gdtype == "bf16":
            return (x.view(torch.int16).to(torch.int32) & 0xFFFF).numpy().astype(np.uint16)
        return x.numpy()

    g = rows(dev.grads)
    reps = rows(dev.replicas)
    th = dev.theta.index_select(0, ix).cpu().numpy()
    m = None if dev.m is None else dev.m.index_select(0, ix).cpu().numpy()
    v = None if dev.v is None else dev.v.index_select(0, ix).cpu().numpy()
    t0 = time.perf_counter()
    c0 = time.process_time()
    if w.loss["kind"] == "bernoulli":
        p = w.loss["p"]
        mg = oloss.bernoulli_arrivals(w.seed, 0, oloss.GRAD, w.n, sample, p)
        mb = oloss.bernoulli_arrivals(w.seed, 0, oloss.BCAST, w.n, sample, p)
    else:  # the chain runs over every packet; only the sample's columns are used
        l = w.loss
        zero = np.zeros(w.n, np.uint8)
        mg = oloss.ge_arrivals(w.seed, 0, oloss.GRAD, w.n, P, l["p_gb"], l["p_bg"],
                               l["loss_good"], l["loss_bad"], zero)[0][:, sample]
        mb = oloss.ge_arrivals(w.seed, 0, oloss.BCAST, w.n, P, l["p_gb"], l["p_bg"],
                               l["loss_good"], l["loss_bad"], zero)[0][:, sample]
    out = ostep.lossy_step(d=w.d, packet=w.packet, packets=sample, gdtype=w.gdtype, grads=g,
                           theta=th, m=m, v=v, replicas=reps, arrived_g=mg, arrived_b=mb,
                           opt=w.opt, t=0)
    odrift.drift_stats(ostep.widen(out["replicas"], w.gdtype),
                       ostep.widen(ostep.store(out["theta"], w.gdtype), w.gdtype), mb)
    wall = time.perf_counter() - t0
    cpu = time.process_time() - c0
    lens = ostep.packet_lengths(w.d, w.packet, sample)
    b = algorithmic_bytes(w, mg, mb, lens, True)["total"]
    return dict(value=round(b / wall / 1e9, 4), unit="GB/s",
                cores=max(1, int(round(cpu / wall))), kind="oracle",
                sample=f"{len(sample)} of {P} packets (one in every {max(1, P // packets_sample)}), "
                       f"one step incl. masks and drift, {wall:.1f} s wall; "
                       f"{len(os.sched_getaffinity(0))} host cores available ({cpu_model()})")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    help="one of the workloads in workloads/__init__.py (default: the N=64 "
                         "7B-shard step)")
    ap.add_argument("--cpu-packets", type=int, default=768,
                    help="packets of the workload the CPU oracle baseline runs on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--estimator", default="arrived_mean",
                    choices=["arrived_mean", "horvitz_thompson", "stale_fill"])
    ap.add_argument("--owner", type=int, default=-1,
                    help="row whose gradient and replica never cross the network")
    ap.add_argument("--reliable-every", type=int, default=0,
                    help="flag every k-th packet as sent over a reliable channel")
    ap.add_argument("--ages", action="store_true", help="track broadcast ages")
    ap.add_argument("--parity-group", type=int, default=0,
                    help="packets per XOR parity packet (0: no parity packets)")
    ap.add_argument("--mall-flush", choices=("read", "write"), default="read",
                    help="how a 1 GiB buffer evicts small workloads from the memory-side "
                         "cache between timed steps")
    ap.add_argument("--stagewise", action="store_true",
                    help="time the chain of one-stage entry points (ll_masks, lossy_aggregate, "
                         "shard_step, lossy_broadcast, drift_stats) instead of the fused step")
    args = ap.parse_args()
    if args.stagewise and (args.estimator != "arrived_mean" or args.owner >= 0
                           or args.reliable_every > 0 or args.ages or args.parity_group > 0):
        ap.error("--stagewise times the default step only")
    variant = (args.estimator != "arrived_mean" or args.owner >= 0 or args.reliable_every > 0
               or args.ages or args.parity_group > 0)

    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library simulates the N workers of one "
              f"owner's shard on a single device and has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2507_07114_amd as ll
    import workloads as wl
    from workloads.device import DeviceState, loss_spec

    if not torch.cuda.is_available():
        log("no GPU visible")
        sys.exit(1)
    name = args.workload or wl.METRIC_WORKLOAD
    w = wl.WORKLOADS[name]
    copy_gbs = hbm_copy_probe()
    log(f"runtime 2 GiB device copy: {copy_gbs:.0f} GB/s")
    log(f"workload {name}: n={w.n} d={w.d} packet={w.packet} P={w.num_packets}")
    dev = DeviceState(w)
    ext = None
    rel_np = None
    if variant:
        rel_t = None
        if args.reliable_every > 0:
            rel_np = np.zeros(w.num_packets, np.uint8)
            rel_np[:: args.reliable_every] = 1
            rel_t = torch.from_numpy(rel_np).cuda()
        # Horvitz-Thompson weights are derived per packet by the library
        # (arrival_prob 0), except for a chain with a state that loses every
        # packet, where the stationary arrival probability is given.
        q = 0.0
        l = w.loss
        if (args.estimator == "horvitz_thompson" and l["kind"] != wl.BERNOULLI
                and not (l["loss_good"] < 1 and l["loss_bad"] < 1)):
            pi_bad = l["p_gb"] / (l["p_gb"] + l["p_bg"])
            q = 1 - pi_bad * l["loss_bad"] - (1 - pi_bad) * l["loss_good"]
        ext = ll.ext(estimator=args.estimator, owner=args.owner, reliable=rel_t,
                     g_prev=torch.zeros_like(dev.grads) if args.estimator == "stale_fill" else None,
                     ages=(torch.zeros((w.n, w.num_packets), dtype=torch.int16, device="cuda")
                           if args.ages else None), arrival_prob=q,
                     parity_group=args.parity_group)
    torch.cuda.synchronize()

    cpu = None
    if not args.no_cpu_baseline and not variant:
        log(f"timing the CPU oracle on {args.cpu_packets} packets ...")
        cpu = cpu_baseline(w, dev, args.cpu_packets)
        log(f"cpu oracle: {cpu}")

    # Realised masks of the timed steps, for the algorithmic byte count.
    P = w.num_packets
    spec = loss_spec(w)
    lens = np.minimum((np.arange(P) + 1) * w.packet, w.d) - np.arange(P) * w.packet
    mg_dev = torch.empty((w.n, P), dtype=torch.uint8, device="cuda")
    mb_dev = torch.empty((w.n, P), dtype=torch.uint8, device="cuda")
    ge_g = torch.zeros(w.n, dtype=torch.uint8, device="cuda")  # chain state (GE only)
    ge_b = torch.zeros(w.n, dtype=torch.uint8, device="cuda")
    ge_ws = torch.zeros(max(ll.ll_masks_workspace_bytes(w.n, P), 256), dtype=torch.uint8,
                        device="cuda")
    per_step_bytes = []
    mext = None if ext is None else ll.ext(owner=args.owner, reliable=ext.reliable,
                                           parity_group=args.parity_group)
    for t in range(args.warmup + args.steps):
        ll.ll_masks(w.n, P, t, ll.LL_DIR_GRAD, spec, mg_dev, ge_state=ge_g, workspace=ge_ws,
                    ext=mext)
        ll.ll_masks(w.n, P, t, ll.LL_DIR_BCAST, spec, mb_dev, ge_state=ge_b, workspace=ge_ws,
                    ext=mext)
        if t >= args.warmup:
            per_step_bytes.append(algorithmic_bytes(
                w, mg_dev.cpu().numpy(), mb_dev.cpu().numpy(), lens, True,
                estimator=args.estimator, ages=args.ages, reliable=rel_np is not None))

    step_fn = (lambda t: dev.fused(t, masks_out=False, ext=ext))
    if args.stagewise:
        from workloads.device import opt_spec
        g_hat = torch.empty(w.d, dtype=torch.float32, device="cuda")

        def step_fn(t):
            ll.ll_masks(w.n, P, t, ll.LL_DIR_GRAD, spec, dev.arrived_g, ge_state=dev.ge_g,
                        workspace=dev.workspace)
            ll.lossy_aggregate(dev.grads, dev.arrived_g, d=w.d, packet=w.packet, g_hat=g_hat,
                               counts=dev.counts, theta=dev.theta)
            ll.shard_step(opt_spec(w), t, dev.theta, g_hat, m=dev.m, v=dev.v)
            ll.ll_masks(w.n, P, t, ll.LL_DIR_BCAST, spec, dev.arrived_b, ge_state=dev.ge_b,
                        workspace=dev.workspace)
            ll.lossy_broadcast(dev.theta, dev.replicas, dev.arrived_b, d=w.d, packet=w.packet)
            ll.drift_stats(dev.replicas, d=w.d, packet=w.packet, workspace=dev.workspace,
                           out=dev.drift, theta=dev.theta, arrived_bc=dev.arrived_b)

    for t in range(args.warmup):
        step_fn(t)
    torch.cuda.synchronize()

    # A workload smaller than the 256 MB memory-side cache (MALL) would be
    # served from it on every step after the first: for footprints under
    # 1 GiB a 1 GiB scratch buffer streams through the cache between steps,
    # outside the timed events, and the throughput is taken over the events
    # alone.  By default the buffer is read (the hand-written read probe), so
    # the cache is left holding clean lines; written ("write"), it is left
    # holding dirty lines that the timed step then has to write back.
    footprint = sum(t.numel() * t.element_size()
                    for t in (dev.grads, dev.replicas, dev.theta, dev.m, dev.v) if t is not None)
    mall_flush = footprint < (1 << 30)
    scratch = torch.zeros(1 << 28, dtype=torch.float32, device="cuda") if mall_flush else None
    if mall_flush and args.mall_flush == "read":
        from paper_2507_07114_amd import probe
        sink = torch.zeros(probe.SINK_BYTES, dtype=torch.uint8, device="cuda")
        flush = lambda j: probe.hbm_probe_read(scratch, sink)
    else:
        flush = lambda j: scratch.fill_(float(j))

    stream = torch.cuda.current_stream()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for j in range(args.steps):
        if mall_flush:
            flush(j)
        starts[j].record(stream)
        step_fn(args.warmup + j)
        ends[j].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    if mall_flush:
        wall = sum(ms) / 1e3
    drift = ll.read_drift(dev.drift)

    # Bandwidth probes after the timed steps (the row probe overwrites the
    # replicas): plain streams and the step's own row shape.
    row_bytes = (w.d * w.elem_bytes) // 16 * 16
    probes = hbm_probes(dev.grads, dev.replicas, row_bytes)
    log(f"hbm probes (GB/s): {probes}")

    total_bytes = sum(b["total"] for b in per_step_bytes)
    ms_per_step = wall * 1e3 / args.steps
    value = total_bytes / wall / 1e9
    mean_bytes = total_bytes / args.steps
    launch_ms = float(np.mean(ms))
    achieved = mean_bytes / (launch_ms * 1e-3) / 1e9
    khash = kernel_source_hash()
    # the counters were taken on the plain fused step of one workload
    traffic = None if (args.stagewise or variant) else read_pmc_traffic(khash, w.name)
    mean_b = {k: int(np.mean([b[k] for b in per_step_bytes])) for k in per_step_bytes[0]}
    log(f"per-launch event times (ms): min {min(ms):.3f} median {float(np.median(ms)):.3f} "
        f"max {max(ms):.3f}; algorithmic bytes/step {mean_b}")
    log(f"drift after last step: {drift}")
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": name, "n": w.n, "d": w.d, "packet": w.packet,
                   "packets": P, "loss": w.loss, "optimizer": w.opt["kind"],
                   "grad_dtype": w.gdtype, "replica_dtype": w.gdtype,
                   "drift": True, "parallelism": "single-gpu simulation of n workers",
                   "estimator": args.estimator, "owner": args.owner,
                   "reliable_every": args.reliable_every, "ages": args.ages,
                   "parity_group": args.parity_group, "stagewise": args.stagewise,
                   "footprint_bytes": footprint,
                   "mall_flush_between_steps": (args.mall_flush if mall_flush else False)},
        "pct_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "elements_per_s": round(w.n * w.d / (ms_per_step * 1e-3), 1),
        "shard_elements_per_s": round(w.d / (ms_per_step * 1e-3), 1),
        "algorithmic_bytes_per_step": mean_b,
        # every gradient row read and every replica row written, as a
        # loss-oblivious pass would move them (context for the count above)
        "dense_equivalent_bytes_per_step": 2 * w.n * w.d * w.elem_bytes + mean_b["state_rw"],
        "hbm_copy_probe_gbs": round(copy_gbs, 1),
        "hbm_probes_gbs": probes,
        "frac_of_best_copy_probe": round(value / probes["copy_16B"], 4),
        # per-step event times: a paced step either keeps its schedule (the
        # minimum) or slips; `value` is over all of them
        "step_ms": {"min": round(min(ms), 4), "median": round(float(np.median(ms)), 4),
                    "max": round(max(ms), 4)},
        "roofline": {
            "bound": "hbm",
            "kernel": ("stage chain: masks x2, k_aggregate, k_shard_step, k_broadcast, k_drift "
                       "(+ reductions)") if args.stagewise else
                      "lossy_step_fused: k_step_paced or k_step_fused (+ mask, anchor and "
                      "drift-fold launches)",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else round(traffic),
            "launch_ms": round(launch_ms, 4),
            "kernel_source_sha256": khash,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
