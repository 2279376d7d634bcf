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
carries the mean and median step time, get-only and put-only rates (events
between the calls), effective HBM GB/s from algorithmic bytes, the roofline
of the dominant kernel (per-launch durations from HIP events recorded by the
library around every launch, beside the kernel's rocprofv3 duration from the
committed profile when that was taken on the same kernel sources), a plain
device copy timed as the achievable ceiling, a parity pass of the first steps
against the CPU oracle (outside the timed region), and the oracle timed on
this host.
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
KERNELS = ("get_probe_gather", "assign_new", "put_probe", "put_reduce", "rsort_count", "rsort_scatter",
           "rsort_reduce")


def kernel_bytes(n, U, M, D, dedup="hash"):
    """Algorithmic bytes each kernel must move for one batch: n lookups, U
    distinct keys of which M are new, rows of D fp32. With radix dedup the
    reduce's bytes are rsort_reduce's; the sort passes move scratch only."""
    b = {
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
    return radix_bytes(b) if dedup == "radix" else b


def radix_bytes(b):
    return {**b, "rsort_count": 0, "rsort_scatter": 0, "rsort_reduce": b["put_reduce"], "put_reduce": 0}


def kernel_bytes_kv(nr, Ur, nw, Uw, D, dedup="hash"):
    """The same for one step of the key-value mix: nr gets over Ur distinct
    existing keys, then a put of nw values over Uw distinct existing keys
    (the last value of each key is written)."""
    b = {
        "get_probe_gather": 8 * nr + 12 * Ur + 4 * D * Ur + 4 * D * nr,
        "assign_new": 0,
        "put_probe": 8 * nw + 12 * Uw,
        # the winning value of each key in, its row written
        "put_reduce": 8 * D * Uw,
    }
    return radix_bytes(b) if dedup == "radix" else b


def source_digest():
    h = hashlib.sha256()
    for f in ("mlkv_device.h", "mlkv_kernels.h", "mlkv_kernels.hip", "mlkv_tier.hip"):
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


def row_scaled_err(a, b):
    """|a - b| / max(|b|, max |b| over the row) element by element; non-finite
    elements count 0 when both sides agree in kind (same infinity, or NaN)."""
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    nonfin = ~np.isfinite(a64) | ~np.isfinite(b64)
    fb = np.where(np.isfinite(b64), np.abs(b64), 0.0)
    scale = np.maximum(fb, fb.max(axis=-1, keepdims=True))
    scale = np.where(scale == 0, 1.0, scale)
    with np.errstate(invalid="ignore"):
        err = np.where(nonfin, 0.0, np.abs(a64 - b64) / scale)
    same = (np.isnan(a64) & np.isnan(b64)) | (a64 == b64)
    return np.where(nonfin & ~same, np.inf, err)


def max_ulp(a, b):
    fin = np.isfinite(a) & np.isfinite(b)
    ia = a[fin].astype(np.float32).view(np.int32).astype(np.int64)
    ib = b[fin].astype(np.float32).view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, -(ia & 0x7FFFFFFF), ia)
    ib = np.where(ib < 0, -(ib & 0x7FFFFFFF), ib)
    return int(np.abs(ia - ib).max()) if ia.size else 0


def parity_and_cpu_baseline(wl, args, kv, bounded, log):
    """Runs the first parity_steps steps of the workload on a fresh GPU table
    and on the CPU oracle, compares them (get outputs: bit-exact for rows no
    put has changed, row-scaled error otherwise; then key -> row, rows and
    accumulators of the last batch's keys), and keeps running the oracle alone
    for about cpu_seconds of step time, which gives the CPU baseline. Returns
    (parity record, cpu baseline record)."""
    import torch
    from oracle import oracle as O
    from paper_2504_01506_amd import mlkv

    D, n, h = wl.dim, wl.n, wl.n // 2
    bound = args.staleness_bound
    ora = O.OracleTable(D, wl.capacity, staleness_bound=bound)
    pre = wl.prefill_keys()
    if pre.size:
        assert ora.prefill_sorted(pre) == O.OK
    P = 0 if args.no_parity else args.parity_steps
    if P and args.pipelined:
        P = max(P, 2)  # the first put comes with the second get
    rec = None
    if P:
        cache = max(1, int(wl.capacity * args.cache_frac)) if args.cache_frac else None
        gpu = mlkv.Table(D, wl.capacity, staleness_bound=bound, cache_rows=cache, dedup=args.dedup)
        gpu.reserve(n)
        blocked = torch.empty(n, dtype=torch.uint8, device="cuda")
        zero = torch.zeros((1 << 16, D), device="cuda") if bounded else None
        for s0 in range(0, pre.size, 1 << 16):
            kc = torch.from_numpy(pre[s0:s0 + (1 << 16)].view(np.int64)).cuda()
            if bounded:
                gpu.get_bounded(kc, None, blocked[:kc.numel()])
                gpu.put_grad_sgd(kc, zero[:kc.numel()], 0.0)
            else:
                gpu.get(kc, None)
        assert gpu.sync() == mlkv.MLKV_OK and gpu.size == ora.size
        updated = np.zeros(wl.capacity, dtype=bool)
        rec = {"steps": P, "max_row_scaled_err": 0.0, "max_ulp": 0, "get_rows_compared": 0,
               "unupdated_rows_bit_exact": True}
    # with --pipelined, step s is the get of batch s then the put of batch s - 1
    # (on the GPU one mlkv_get_put_grad call), as in the timed steps
    ov = args.pipelined
    cpu_s, steps = 0.0, 0
    prev = None  # the previous step's put keys and gradients (pipelined steps)
    while steps < P or cpu_s < args.cpu_seconds:
        keys = wl.keys(steps)
        kg = keys[:h] if kv else keys
        kp = keys[h:] if kv else keys
        src = wl.values(steps) if kv else wl.grads(steps)
        t0 = time.perf_counter()
        if bounded:
            rc, want, _ = ora.get_bounded(kg)
        else:
            rc, want = ora.get(kg)
        if not ov:
            rc2 = ora.put(kp, src) if kv else ora.put_grad(kp, src, wl.lr, wl.eps)
        else:
            rc2 = ora.put_grad(prev[0], prev[1], wl.lr, wl.eps) if prev is not None else O.OK
        cpu_s += time.perf_counter() - t0
        assert rc == O.OK and rc2 == O.OK
        if steps < P:
            k_d = torch.from_numpy(kg.view(np.int64)).cuda()
            if args.cache_frac:
                gpu.lookahead(k_d)
            out = torch.empty((kg.size, D), device="cuda")
            kp_d = torch.from_numpy(kp.view(np.int64)).cuda()
            src_d = torch.from_numpy(src).cuda()
            if ov and prev is not None:
                gpu.get_put_grad(k_d, out, prev[2], prev[3], wl.lr, wl.eps,
                                 blocked=blocked[:kg.size] if bounded else None)
            elif bounded:
                gpu.get_bounded(k_d, out, blocked[:kg.size])
            else:
                gpu.get(k_d, out)
            if kv:
                gpu.put(kp_d, src_d)
            elif not ov:
                gpu.put_grad(kp_d, src_d, wl.lr, wl.eps)
            assert gpu.sync() == mlkv.MLKV_OK
            got = out.cpu().numpy()
            rows_g = ora.lookup_rows(kg)
            fresh = ~updated[rows_g]
            if fresh.any() and not np.array_equal(got[fresh].view(np.uint32), want[fresh].view(np.uint32)):
                rec["unupdated_rows_bit_exact"] = False
            if (~fresh).any():
                rec["max_row_scaled_err"] = max(rec["max_row_scaled_err"],
                                                float(row_scaled_err(got[~fresh], want[~fresh]).max()))
                rec["max_ulp"] = max(rec["max_ulp"], max_ulp(got[~fresh], want[~fresh]))
            rec["get_rows_compared"] += int(kg.size)
            if ov:  # this step's put is the previous batch's
                kp, kp_d = (prev[0], prev[2]) if prev is not None else (kp[:0], kp_d[:0])
            rows_p = ora.lookup_rows(kp)
            updated[rows_p] = True
            if steps == P - 1:  # the last batch: key -> row, rows and accumulators
                rows_d = gpu.lookup_rows(kp_d).cpu().numpy()
                rec["key_to_row_bit_exact"] = bool(np.array_equal(rows_d, rows_p))
                ur = np.unique(rows_p)
                w_d, st_d = gpu.read_rows(torch.from_numpy(ur).cuda())
                w_o, st_o = ora.read_rows(ur)
                w_d, st_d = w_d.cpu().numpy(), st_d.cpu().numpy()
                rec["rows_compared"] = int(ur.size)
                rec["max_row_scaled_err"] = max(rec["max_row_scaled_err"], float(row_scaled_err(w_d, w_o).max()))
                rec["max_ulp"] = max(rec["max_ulp"], max_ulp(w_d, w_o))
                with np.errstate(invalid="ignore", divide="ignore"):
                    st_err = np.where(st_d == st_o, 0.0, np.abs(st_d - st_o.astype(np.float64)) / np.abs(st_o))
                rec["max_state_rel_err"] = float(np.nanmax(st_err)) if st_err.size else 0.0
                rec["within_1e-5"] = bool(rec["max_row_scaled_err"] <= 1e-5 and rec["max_state_rel_err"] <= 1e-5)
                gpu.close()
                log(f"parity over {P} steps: {rec}")
        if ov:
            prev = (keys, src) + ((torch.from_numpy(keys.view(np.int64)).cuda(), torch.from_numpy(src).cuda())
                                  if steps < P - 1 else (None, None))
        steps += 1
    ora.close()
    unit = "ops/s" if kv else "keys/s"
    cpu = {"value": wl.n * steps / cpu_s, "unit": unit, "cores": 1, "kind": "oracle",
           "sample": f"the first {steps} steps of the same workload ({wl.n} keys each) after the "
                     f"same prefill, single-threaded C++ oracle, {cpu_s:.1f} s of step time",
           "host_cpus": os.cpu_count(), "host_affinity": len(os.sched_getaffinity(0)),
           "cpu_model": host_cpu_model()}
    return rec, cpu


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
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (CPU baseline and parity pass)")
    ap.add_argument("--no-parity", action="store_true", help="skip the parity pass against the oracle")
    ap.add_argument("--parity-steps", type=int, default=3)
    ap.add_argument("--staleness-bound", type=int, default=None,
                    help="open the table with this staleness bound (gets then report blocked keys)")
    ap.add_argument("--cache-frac", type=float, default=None,
                    help="tiered table: rows in pinned host memory, this fraction of them cached in HBM; "
                         "each step is lookahead(keys), get(keys), put_grad(keys)")
    ap.add_argument("--dedup", choices=("hash", "radix"), default="hash",
                    help="how puts find equal keys: hash partition + LDS grouping, or radix sort + run-length "
                         "encoding (same results)")
    ap.add_argument("--pipelined", action="store_true",
                    help="each step is one mlkv_get_put_grad call: the get of batch s, then the put_grad of "
                         "batch s - 1 (asynchronous training; with a staleness bound, from bound 1)")
    ap.add_argument("--copy-mib", type=int, default=1024,
                    help="size of the plain device copy timed as the achievable ceiling (and used to "
                         "calibrate rocprofv3 counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path is single-GPU by design)", file=sys.stderr)
        sys.exit(2)

    if args.cache_frac is not None and (args.config.startswith("kv-") or args.staleness_bound is not None
                                        or not 0.0 < args.cache_frac <= 1.0):
        print("--cache-frac (0 < f <= 1) applies to the training-step workloads without a staleness bound",
              file=sys.stderr)
        sys.exit(2)
    if args.pipelined and (args.config.startswith("kv-") or args.staleness_bound == 0):
        print("--pipelined applies to the training-step workloads, without a staleness bound or with a bound of "
              "at least 1 (at bound 0 the get blocks every key the pending put updates)", file=sys.stderr)
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
    total_steps = args.warmup + args.steps  # the later passes reuse the timed batches

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
    tiered = args.cache_frac is not None
    cache_rows = max(1, int(wl.capacity * args.cache_frac)) if tiered else None
    t = mlkv.Table(D, wl.capacity, staleness_bound=args.staleness_bound, cache_rows=cache_rows, dedup=args.dedup)
    t.reserve(n)  # scratch for the batch: no allocation inside the steps
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
    if tiered:  # warm the cache with a slice of the table
        warm = np.random.default_rng(5).choice(pre, size=min(cache_rows, pre.size), replace=False)
        t.lookahead(torch.from_numpy(warm.view(np.int64)).cuda())
        assert t.sync() == mlkv.MLKV_OK
        log(f"cache of {cache_rows} rows warmed: {t.cache_stats()}")

    def get(s):
        k, o = (keys_d[s][:h], out[:h]) if kv else (keys_d[s], out)
        if bounded:
            t.get_bounded(k, o, blocked[:k.numel()])
        else:
            t.get(k, o)

    def put(s):
        if kv:
            t.put(keys_d[s][h:], grads_d[s])
        else:
            t.put_grad(keys_d[s], grads_d[s], wl.lr, wl.eps)

    ov = args.pipelined

    def step(s):
        if tiered:
            t.lookahead(keys_d[s])
        if ov and s > 0:  # the get of batch s, then the put of batch s - 1
            t.get_put_grad(keys_d[s], out, keys_d[s - 1], grads_d[s - 1], wl.lr, wl.eps,
                           blocked=blocked if bounded else None)
            return
        get(s)
        if not ov:
            put(s)

    Ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    # warm-up; the first step after the prefill is timed on its own (the cold
    # step: the most inserts on a table that starts empty)
    first_ms = None
    for s in range(args.warmup):
        if s == 0:
            e_a, e_b = Ev(), Ev()
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

    # ---- timed region: K steps, nothing else on the stream
    first = args.warmup
    timed = range(first, first + args.steps)
    ev0, ev1 = Ev(), Ev()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record()
    for s in timed:
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
        bytes_steps = [kernel_bytes_kv(h, Ur, n - h, Uw, D, args.dedup) for (Ur, Uw) in UM]
    else:
        bytes_steps = [kernel_bytes(n, U, M, D, args.dedup) for (U, M) in UM]
    alg_bytes = sum(sum(bytes_steps[s].values()) for s in timed)
    gbps = alg_bytes / (ms * 1e-3) / 1e9
    log(f"timed {args.steps} steps: {ms_step * 1e3:.2f} us/step (wall {wall * 1e3 / args.steps:.2f}), "
        f"{keys_per_s / 1e9:.3f} G keys/s, {gbps:.0f} GB/s effective")

    # ---- the same batches again, events between the get and the put calls
    # (per-step times for the median, and the get and the put apart)
    ev_g = [(Ev(), Ev(), Ev()) for _ in timed]
    for (ea, eb, ec), s in zip(ev_g, timed):
        ea.record()
        if ov:  # one call per step: the get and the put are not apart
            step(s)
        else:
            get(s)
        eb.record()
        if not ov:
            put(s)
        ec.record()
    torch.cuda.synchronize()
    assert t.sync() == mlkv.MLKV_OK
    t_get = None if ov else float(np.median([ea.elapsed_time(eb) for ea, eb, _ in ev_g]))
    t_put = None if ov else float(np.median([eb.elapsed_time(ec) for _, eb, ec in ev_g]))
    per_step = [ea.elapsed_time(ec) for ea, _, ec in ev_g]
    n_get, n_put = (h, n - h) if kv else (n, n)
    if not ov:
        log(f"get {t_get * 1e3:.2f} us, put {t_put * 1e3:.2f} us (medians)")

    # ---- once more with events around every launch: per-kernel durations
    tier0 = t.cache_stats() if tiered else None
    mlkv.mlkv_profile_enable(t.h, True)
    ev2, ev3 = Ev(), Ev()
    ev2.record()
    for s in timed:
        step(s)
    ev3.record()
    torch.cuda.synchronize()
    prof = mlkv.mlkv_profile_read(t.h)
    mlkv.mlkv_profile_enable(t.h, False)
    ms_prof = ev2.elapsed_time(ev3) / args.steps
    assert t.sync() == mlkv.MLKV_OK
    kinfo = {}
    host_link = None
    for kname in KERNELS:
        tot_ms, cnt = prof[kname]
        b = sum(bytes_steps[s].get(kname, 0) for s in timed)
        if cnt == 0:
            continue
        avg_us = tot_ms * 1e3 / cnt
        kinfo[kname] = {"avg_us": round(avg_us, 3), "launches": cnt,
                        "alg_bytes_per_launch": int(b / cnt),
                        "gbps": round(b / cnt / (avg_us * 1e-6) / 1e9, 1)}
    if tiered and prof["tier_copy"][1] > 0:
        # the steps' lookahead copies: rows in over the host link, dirty rows back
        tier1 = t.cache_stats()
        for kname in ("tier_mark", "tier_plan", "tier_copy"):
            tot_ms, cnt = prof[kname]
            kinfo[kname] = {"avg_us": round(tot_ms * 1e3 / cnt, 3), "launches": cnt}
        cnt = prof["tier_copy"][1]
        kinfo["tier_copy"].update({"rows_in_per_launch": (tier1["loaded"] - tier0["loaded"]) / cnt,
                                   "rows_back_per_launch": (tier1["written_back"] - tier0["written_back"]) / cnt})
        # a bulk lookahead of rows mostly not cached: the copy is link-bound
        bulk = np.random.default_rng(6).choice(pre, size=min(cache_rows, 1 << 20), replace=False)
        bulk_d = torch.from_numpy(bulk.view(np.int64)).cuda()
        torch.cuda.synchronize()
        mlkv.mlkv_profile_enable(t.h, True)
        t.lookahead(bulk_d)
        torch.cuda.synchronize()
        bprof = mlkv.mlkv_profile_read(t.h)
        mlkv.mlkv_profile_enable(t.h, False)
        assert t.sync() == mlkv.MLKV_OK
        tier2 = t.cache_stats()
        rows_in = tier2["loaded"] - tier1["loaded"]
        rows_back = tier2["written_back"] - tier1["written_back"]
        link_bytes = 4 * D * (rows_in + rows_back)
        us = bprof["tier_copy"][0] * 1e3
        host_link = {"kernel": "tier_copy", "what": f"lookahead of {bulk.size} random rows, {rows_in} of them "
                                                    f"copied in and {rows_back} dirty ones written back",
                     "achieved_gbps": round(link_bytes / (us * 1e-6) / 1e9, 2), "bytes": int(link_bytes),
                     "launch_us": round(us, 2), "cache_rows": cache_rows, "counters": tier2}
    dom = max((k for k in kinfo if "alg_bytes_per_launch" in kinfo[k]),
              key=lambda k: kinfo[k]["avg_us"] * kinfo[k]["launches"])
    digest = source_digest()
    # the committed counters were taken on the full-size DLRM-shaped workload
    same_workload = (args.config == "dlrm" and args.scale == 1.0 and not bounded and not tiered
                     and args.dedup == "hash" and not ov)
    traffic = load_traffic(dom, digest) if same_workload else None
    # the kernel's rocprofv3 duration, for comparison with the event-timed one
    # (an event pair around every launch adds about 2 us to each)
    traced_us = load_profile(dom, digest, "avg_us") if same_workload else None
    roof = {"kernel": dom, "bound": "hbm", "achieved": kinfo[dom]["gbps"], "peak": PEAK_HBM_GBPS,
            "unit": "GB/s", "frac": round(kinfo[dom]["gbps"] / PEAK_HBM_GBPS, 4), "traffic": traffic,
            "alg_bytes_per_launch": kinfo[dom]["alg_bytes_per_launch"],
            "avg_launch_us": kinfo[dom]["avg_us"], "rocprofv3_avg_us": traced_us}
    log(f"kernels (events around every launch, {ms_prof * 1e3:.2f} us/step): {kinfo}")

    t.close()
    del keys_d, grads_d, out
    torch.cuda.empty_cache()

    # ---- the achievable ceiling on this device: a plain 1 GiB device copy
    copy_bytes = max(1, args.copy_mib) << 20
    ca = torch.empty(copy_bytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    cb = torch.empty_like(ca)
    best = None
    for _ in range(3):
        e_a, e_b = Ev(), Ev()
        e_a.record()
        cb.copy_(ca)
        e_b.record()
        torch.cuda.synchronize()
        ms_c = e_a.elapsed_time(e_b)
        best = ms_c if best is None else min(best, ms_c)
    copy_gbps = 2 * copy_bytes / (best * 1e-3) / 1e9  # bytes read + written
    del ca, cb
    torch.cuda.empty_cache()
    log(f"device copy of {copy_bytes >> 20} MiB: {copy_gbps:.0f} GB/s read+write")
    if host_link is not None:
        # the host link's ceiling: plain copies between pinned host memory and HBM
        hb = 256 << 20
        ph = torch.empty(hb // 4, dtype=torch.float32, pin_memory=True).fill_(1.0)
        dd = torch.empty(hb // 4, dtype=torch.float32, device="cuda")
        rates = {}
        for name, (dst, src) in (("h2d", (dd, ph)), ("d2h", (ph, dd))):
            best_l = None
            for _ in range(3):
                e_a, e_b = Ev(), Ev()
                e_a.record()
                dst.copy_(src, non_blocking=True)
                e_b.record()
                torch.cuda.synchronize()
                ms_l = e_a.elapsed_time(e_b)
                best_l = ms_l if best_l is None else min(best_l, ms_l)
            rates[name] = round(hb / (best_l * 1e-3) / 1e9, 2)
        del ph, dd
        host_link["link_copy_gbps"] = rates
        host_link["frac_of_h2d_copy"] = round(host_link["achieved_gbps"] / rates["h2d"], 4)
        log(f"host link: lookahead copy {host_link['achieved_gbps']} GB/s, pinned copies {rates}")

    parity, cpu = None, None
    if not args.no_cpu_baseline:
        log("parity pass and cpu baseline: the oracle on the host")
        parity, cpu = parity_and_cpu_baseline(wl, args, kv, bounded, log)
        log(f"cpu baseline: {cpu['value'] / 1e6:.3f} M {cpu['unit']}")

    U_avg = float(np.mean([UM[s][0] + UM[s][1] if kv else UM[s][0] for s in timed]))
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
        "ms_per_step_median": float(np.median(per_step)),
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
            **({"tiered_cache_rows": cache_rows, "step": "lookahead + get + put_grad"} if tiered else {}),
            **({"dedup": "radix sort + run-length encoding"} if args.dedup == "radix" else {}),
            **({"step": "get(batch s) then put_grad(batch s - 1), one mlkv_get_put_grad call"} if ov else {}),
        },
        "gbps_effective": round(gbps, 1),
        "pct_of_peak_hbm": round(100.0 * gbps / PEAK_HBM_GBPS, 2),
        "alg_bytes_per_step": int(alg_bytes / args.steps),
        "get_keys_per_s": None if ov else n_get / (t_get * 1e-3),
        "put_keys_per_s": None if ov else n_put / (t_put * 1e-3),
        "ms_get_median": t_get,
        "ms_put_median": t_put,
        "ms_per_step_with_kernel_events": ms_prof,
        "ms_first_step": first_ms,
        "copy_ceiling": {"gbps": round(copy_gbps, 1), "frac_of_peak": round(copy_gbps / PEAK_HBM_GBPS, 4),
                         "what": f"device-to-device copy of {copy_bytes >> 20} MiB, read + write bytes, best of 3"},
        "roofline": roof,
        **({"host_link": host_link} if host_link is not None else {}),
        "kernels": kinfo,
        "parity": parity,
        "cpu_baseline": cpu,
        "kernel_source_digest": digest,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
