#!/usr/bin/env python3
"""Throughput of batched embedding get + put_grad on one MI355X.

One step = mlkv_get(keys) then mlkv_put_grad(keys, grads) on one batch of
the DLRM-shaped workload (26 features, 10M rows of dim 64 prefilled,
8192 samples x 26 features = 212,992 lookups, per-feature Zipf(1.1),
row-wise Adagrad lr 0.01 eps 1e-8). All inputs are generated on the host
from fixed seeds and copied to HBM before the timed region.

With --config kv-uniform or kv-zipf a step is instead the paper's key-value
mix: gets of half a batch of 2^20 record keys, then puts (upserts of new
16-byte values) of the other half, over 10M prefilled records.

Prints one JSON line. `value` is get+put keys per second; the line also
carries effective HBM GB/s from algorithmic bytes, the roofline of the
dominant kernel (per-launch durations from HIP events recorded by the
library around every launch, beside the kernel's rocprofv3 duration from the
committed profile when that was taken on the same kernel sources) and the
CPU oracle timed on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
METRIC = "embedding get+put keys/sec and achieved HBM GB/s (% of peak), 1 MI355X"
METRIC_KV = "key-value operations/sec, 50% get / 50% put, 1 MI355X"
KERNELS = ("get_probe_gather", "assign_new", "put_probe", "put_reduce")


def kernel_bytes(n, U, M, D):
    """Algorithmic bytes each kernel must move for one batch: n lookups, U
    distinct keys of which M are new, rows of D fp32."""
    return {
        # keys in, one index entry (8 B tag + 4 B row) per distinct key,
        # distinct existing rows read, output rows written
        "get_probe_gather": 8 * n + 12 * U + 4 * D * (U - M) + 4 * D * n,
        # new rows, their accumulators, index tag + row id
        "assign_new": (4 * D + 16) * M,
        # keys in, one index entry per distinct key
        "put_probe": 8 * n + 12 * U,
        # gradient rows in, distinct rows read and written, accumulators read
        # and written
        "put_reduce": 4 * D * n + 8 * D * U + 8 * U,
    }


def kernel_bytes_kv(nr, Ur, nw, Uw, D):
    """The same for one step of the key-value mix: nr gets over Ur distinct
    existing keys, then a put of nw values over Uw distinct existing keys
    (the last value of each key is written)."""
    return {
        "get_probe_gather": 8 * nr + 12 * Ur + 4 * D * Ur + 4 * D * nr,
        "assign_new": 0,
        "put_probe": 8 * nw + 12 * Uw,
        # the winning value of each key in, its row written
        "put_reduce": 8 * D * Uw,
    }


def source_digest():
    h = hashlib.sha256()
    for f in ("mlkv_device.h", "mlkv_kernels.h", "mlkv_kernels.hip"):
        with open(os.path.join(ROOT, "paper_2504_01506_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_profile(kernel, digest, field):
    """A per-launch figure of `kernel` from the committed rocprofv3 runs on the
    DLRM-shaped workload (HBM bytes from the counter runs, average duration
    from the kernel trace), if they were taken on the current kernel sources."""
    p = os.path.join(ROOT, "profiles", "traffic_dlrm.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        t = json.load(f)
    if t.get("source_digest") != digest:
        return None
    return t.get("kernels", {}).get(kernel, {}).get(field)


def load_traffic(kernel, digest):
    return load_profile(kernel, digest, "hbm_bytes_per_launch")


def cpu_baseline(wl, seconds, kv=False):
    from oracle import oracle as O

    t = O.OracleTable(wl.dim, wl.capacity)
    pre = wl.prefill_keys()
    if pre.size:
        assert t.prefill_sorted(pre) == O.OK
    steps, elapsed = 0, 0.0
    while steps == 0 or elapsed < seconds:
        keys = wl.keys(steps)
        if kv:
            h = wl.n // 2
            vals = wl.values(steps)
            t0 = time.perf_counter()
            rc, _ = t.get(keys[:h])
            rc2 = t.put(keys[h:], vals)
        else:
            grads = wl.grads(steps)
            t0 = time.perf_counter()
            rc, _ = t.get(keys)
            rc2 = t.put_grad(keys, grads, wl.lr, wl.eps)
        elapsed += time.perf_counter() - t0
        assert rc == O.OK and rc2 == O.OK
        steps += 1
    t.close()
    unit = "ops/s" if kv else "keys/s"
    return {"value": wl.n * steps / elapsed, "unit": unit, "cores": 1, "kind": "oracle",
            "sample": f"first {steps} steps of the same workload ({wl.n} keys each) after the "
                      f"same prefill, single-threaded C++ oracle, {elapsed:.1f} s",
            "host_cpus": os.cpu_count(), "host_affinity": len(os.sched_getaffinity(0)),
            "cpu_model": host_cpu_model()}


def host_cpu_model():
    """The host CPU's model name, as /proc/cpuinfo states it."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="dlrm",
                    choices=["tiny", "dlrm", "kg", "gnn", "large", "kv-uniform", "kv-zipf"])
    ap.add_argument("--scale", type=float, default=1.0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--staleness-bound", type=int, default=None,
                    help="open the table with this staleness bound (gets then report blocked keys)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path is single-GPU by design)", file=sys.stderr)
        sys.exit(2)

    if args.staleness_bound is not None and args.config.startswith("kv-"):
        print("--staleness-bound applies to the training-step workloads (get then put_grad of the same keys)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2504_01506_amd import mlkv
    from paper_2504_01506_amd import workloads as W

    log = lambda *a: print("[bench]", *a, file=sys.stderr, flush=True)  # noqa: E731
    torch.cuda.set_device(0)
    mlkv.load()
    wl = W.make(args.config, scale=args.scale)
    D, n = wl.dim, wl.n
    kv = args.config.startswith("kv-")  # half gets, half puts of values
    h = n // 2
    total_steps = args.warmup + 2 * args.steps

    # ---- inputs (host, seeded) -> HBM ------------------------------------
    t0 = time.perf_counter()
    pre = wl.prefill_keys()
    known = np.sort(pre)
    keys_h, grads_d, keys_d, UM = [], [], [], []
    for s in range(total_steps):
        k = wl.keys(s)
        keys_d.append(torch.from_numpy(k.view(np.int64)).cuda())
        if kv:  # every key is a prefilled record
            UM.append((np.unique(k[:h]).size, np.unique(k[h:]).size))
            grads_d.append(torch.from_numpy(wl.values(s)).cuda())
            continue
        u = np.unique(k)
        if known.size:
            pos = np.minimum(np.searchsorted(known, u), known.size - 1)
            new = u[known[pos] != u]
        else:
            new = u
        if new.size:
            known = np.union1d(known, new)
        UM.append((u.size, new.size))
        grads_d.append(torch.from_numpy(wl.grads(s)).cuda())
        if (s + 1) % 20 == 0:
            log(f"inputs: {s + 1} of {total_steps} batches")
    out = torch.empty((n, D), dtype=torch.float32, device="cuda")
    log(f"inputs ready in {time.perf_counter() - t0:.1f}s: {total_steps} batches of {n} keys")

    bounded = args.staleness_bound is not None
    t = mlkv.Table(D, wl.capacity, staleness_bound=args.staleness_bound)
    blocked = torch.empty(n, dtype=torch.uint8, device="cuda")
    t0 = time.perf_counter()
    chunk = 1 << 16
    zero_rows = torch.zeros((chunk, D), dtype=torch.float32, device="cuda") if bounded else None
    for s in range(0, pre.size, chunk):
        kc = torch.from_numpy(pre[s:s + chunk].view(np.int64)).cuda()
        if bounded:
            # insert, then complete the inserting get with a put that changes no row
            t.get_bounded(kc, None, blocked[:kc.numel()])
            t.put_grad_sgd(kc, zero_rows[:kc.numel()], 0.0)
        else:
            t.get(kc, None)
    assert t.sync() == mlkv.MLKV_OK
    log(f"prefill {pre.size} keys in {time.perf_counter() - t0:.2f}s, size={t.size}")

    def get(k, o):
        if bounded:
            t.get_bounded(k, o, blocked[:k.numel()])
        else:
            t.get(k, o)

    def step(s):
        if kv:
            get(keys_d[s][:h], out[:h])
            t.put(keys_d[s][h:], grads_d[s])
        else:
            get(keys_d[s], out)
            t.put_grad(keys_d[s], grads_d[s], wl.lr, wl.eps)

    # warm-up; the first step after the prefill is timed on its own (the cold
    # step: first touch of the scratch, and the most inserts on a table that
    # starts empty)
    first_ms = None
    for s in range(args.warmup):
        if s == 0:
            e_a, e_b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e_a.record()
            step(s)
            e_b.record()
            torch.cuda.synchronize()
            first_ms = e_a.elapsed_time(e_b)
        else:
            step(s)
    torch.cuda.synchronize()
    assert t.sync() == mlkv.MLKV_OK

    # ---- timed region: K steps, nothing else on the stream ---------------
    first = args.warmup
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record()
    for s in range(first, first + args.steps):
        step(s)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = ev0.elapsed_time(ev1)
    assert t.sync() == mlkv.MLKV_OK
    if bounded:  # each step's put completes its get, so no get is ever blocked
        assert int(blocked.sum()) == 0, "a get was blocked"

    ms_step = ms / args.steps
    keys_per_s = n * args.steps / (ms * 1e-3)
    if kv:
        bytes_steps = [kernel_bytes_kv(h, Ur, n - h, Uw, D) for (Ur, Uw) in UM]
    else:
        bytes_steps = [kernel_bytes(n, U, M, D) for (U, M) in UM]
    alg_bytes = sum(sum(b.values()) for b in bytes_steps[first:first + args.steps])
    gbps = alg_bytes / (ms * 1e-3) / 1e9
    log(f"timed {args.steps} steps: {ms_step * 1e3:.2f} us/step (wall {wall * 1e3 / args.steps:.2f}), "
        f"{keys_per_s / 1e9:.3f} G keys/s, {gbps:.0f} GB/s effective")

    # ---- per-kernel durations: the next K steps with events around every launch
    second = first + args.steps
    mlkv.mlkv_profile_enable(t.h, True)
    ev2, ev3 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev2.record()
    for s in range(second, second + args.steps):
        step(s)
    ev3.record()
    torch.cuda.synchronize()
    prof = mlkv.mlkv_profile_read(t.h)
    mlkv.mlkv_profile_enable(t.h, False)
    ms_prof = ev2.elapsed_time(ev3) / args.steps
    assert t.sync() == mlkv.MLKV_OK
    kinfo = {}
    for kname in KERNELS:
        tot_ms, cnt = prof[kname]
        b = sum(bs[kname] for bs in bytes_steps[second:second + args.steps])
        if cnt == 0:
            continue
        avg_us = tot_ms * 1e3 / cnt
        kinfo[kname] = {"avg_us": round(avg_us, 3), "launches": cnt,
                        "alg_bytes_per_launch": int(b / cnt),
                        "gbps": round(b / cnt / (avg_us * 1e-6) / 1e9, 1)}
    dom = max(kinfo, key=lambda k: kinfo[k]["avg_us"] * kinfo[k]["launches"])
    digest = source_digest()
    # the committed counters were taken on the full-size DLRM-shaped workload
    same_workload = args.config == "dlrm" and args.scale == 1.0 and not bounded
    traffic = load_traffic(dom, digest) if same_workload else None
    # the kernel's rocprofv3 duration, for comparison with the event-timed one
    # (an event pair around every launch adds about 2 us to each)
    traced_us = load_profile(dom, digest, "avg_us") if same_workload else None
    roof = {"kernel": dom, "bound": "hbm", "achieved": kinfo[dom]["gbps"], "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": round(kinfo[dom]["gbps"] / PEAK_HBM_GBPS, 4), "traffic": traffic,
            "alg_bytes_per_launch": kinfo[dom]["alg_bytes_per_launch"],
            "avg_launch_us": kinfo[dom]["avg_us"], "rocprofv3_avg_us": traced_us}
    log(f"kernels (events around every launch, {ms_prof * 1e3:.2f} us/step): {kinfo}")

    if args.copy_mib:
        a = torch.empty(args.copy_mib << 18, dtype=torch.float32, device="cuda").fill_(1.0)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        log(f"copy of {args.copy_mib} MiB done")

    t.close()
    del keys_d, grads_d, out
    torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline: oracle on the host")
        cpu = cpu_baseline(wl, args.cpu_seconds, kv)
        log(f"cpu baseline: {cpu['value'] / 1e6:.3f} M {cpu['unit']}")

    U_avg = float(np.mean([a + b if kv else a for a, b in UM[first:first + args.steps]]))
    if kv:
        workload = (f"{wl.name} key-value mix: {wl.capacity} records of dim {D} fp32 (16-byte values), "
                    f"{h} gets then {n - h} puts per step")
    else:
        workload = (f"{wl.name}-shaped embedding table: {wl.capacity} rows x dim {D} fp32, "
                    f"{n} lookups per step (get + row-wise Adagrad put_grad)")
    res = {
        "metric": METRIC_KV if kv else METRIC,
        "value": keys_per_s,
        "unit": "ops/s" if kv else "keys/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": workload,
            "rows": wl.capacity, "dim": D, "lookups_per_step": n, "prefill": int(pre.size),
            "unique_keys_per_step": round(U_avg, 1), "scale": args.scale,
            **({"staleness_bound": args.staleness_bound} if bounded else {}),
        },
        "gbps_effective": round(gbps, 1),
        "pct_of_peak_hbm": round(100.0 * gbps / PEAK_HBM_GBPS, 2),
        "alg_bytes_per_step": int(alg_bytes / args.steps),
        "ms_per_step_with_kernel_events": ms_prof,
        "ms_first_step": first_ms,
        "roofline": roof,
        "kernels": kinfo,
        "cpu_baseline": cpu,
        "kernel_source_digest": digest,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
