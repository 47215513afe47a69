#!/usr/bin/env python3
"""Benchmark of forced-weight subset evaluation on one MI355X.

Default run: the streaming top-k workload (32 layers x 8 kv heads x 256 query
rows, n = 4096, d = 128, bf16, budgets 128/512/1024) timed as the headline
(attention rows per second), plus one pass of every other entry point on its
own workload as components (exhaustive subsets/s, swap pairs/s, candidate-set
subsets/s, group-vote rows/s, curve and compaction GB/s, and the tiny
exhaustive case).  Prints
ONE JSON line.

Timing: W warm-up passes, then K timed passes bracketed by device
synchronisation, with HIP events recorded on the stream the library launches
on (torch's current stream).  Inputs are resident in HBM before timing.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9  # CUs x SIMDs x lanes x clock: one VALU op per lane


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--only", default="", help="comma list: topk,exhaustive,swap,pool,poolcap,vote,curve,tiny,copy (copy: device copy and read)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--cpu-configs", action="store_true",
                    help="time the oracle on a sample of each of the five workloads (no GPU) and exit")
    return ap.parse_args()


def _time(torch, fn, steps, warmup):
    """Median milliseconds per step over `steps` timed steps after `warmup`
    untimed ones, from HIP events recorded on the stream the library launches
    on (torch's current stream) between consecutive steps; also returns the
    wall time of the timed region and the per-step list."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    ev[0].record(st)
    for i in range(steps):
        fn()
        ev[i + 1].record(st)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    mid = per[len(per) // 2] if len(per) % 2 else 0.5 * (per[len(per) // 2 - 1] + per[len(per) // 2])
    return mid, wall, per


# Frank-Wolfe steps at most per row and budget in the candidate-set search
FW_ITERS = 64


def _stat(holder, b, name):
    """One column of the candidate-set statistics for budget b, flattened."""
    from paper_2608_25230_amd import fw
    return holder["stats"][b, ..., fw.POOL_STATS.index(name)].flatten().double()


def _progress(msg):
    """One line on stderr when a piece of the run ends (the JSON result is the
    only line on stdout)."""
    print("bench: " + msg, file=sys.stderr, flush=True)


def _roofline(bound, achieved, peak, unit, traffic=None):
    return {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic}


def _traffic(name, source):
    """HBM bytes per launch from the committed counter summary
    profiles/traffic_<name>.txt (FETCH_SIZE and WRITE_SIZE, scaled by a plain
    copy of known size), or None when the kernel source has changed since the
    counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_%s.txt" % name)
    src = os.path.join(ROOT, "paper_2608_25230_amd", "csrc", source)
    if not (os.path.exists(path) and os.path.exists(src)):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                key, val = line.split(":", 1)
                kv[key.strip()] = val.strip()
    if kv.get("source_sha256") != hashlib.sha256(open(src, "rb").read()).hexdigest():
        return None
    try:
        return int(float(kv["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


# ---------------------------------------------------------------------------
# CPU baseline: the oracle, on a bounded sample, in a process pool
# ---------------------------------------------------------------------------
def _oracle_unit(args):
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import fw_oracle as O
    q, k, v, scale, bias, ks = args
    with threadpool_limits(1):
        t0 = time.perf_counter()
        Z = O.logits(q, k, scale, bias)
        for g in range(q.shape[0]):
            O.row_dense_topk(Z[g], v, ks)
        return time.perf_counter() - t0, q.shape[0]


def cpu_baseline(wl, seconds):
    import numpy as np
    from concurrent.futures import ProcessPoolExecutor
    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    rows = wl.rows
    q, k, v = rows.as_f64("q"), rows.as_f64("k"), rows.as_f64("v")
    bias = rows.bias.astype(np.float64)
    # calibrate one unit's rows, then size the sample to ~`seconds` of work
    t, nr = _oracle_unit((q[0, :8], k[0], v[0], float(rows.scale[0]), bias, tuple(wl.ks)))
    per_row = t / nr
    rows_per_unit = rows.G
    total_rows = int(seconds * cores / per_row)
    units = max(cores, min(rows.H, total_rows // rows_per_unit))
    jobs = [(q[h], k[h], v[h], float(rows.scale[h]), bias, tuple(wl.ks)) for h in range(units)]
    t0 = time.perf_counter()
    with ProcessPoolExecutor(max_workers=cores) as ex:
        res = list(ex.map(_oracle_unit, jobs))
    wall = time.perf_counter() - t0
    done = sum(r[1] for r in res)
    return {"value": round(done / wall, 2), "unit": "rows/s", "cores": cores, "kind": "oracle",
            "sample": f"{units} units x {rows_per_unit} rows of the same workload ({done} rows, "
                      f"float64 NumPy, one process per core, {wall:.1f} s)"}


# Per-workload CPU baselines (``--cpu-configs``): the oracle on a bounded
# sample of each of the five workloads, one process per core.
def _cpu_tiny(args):
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import fw_oracle as O
    q, k, v, scale, bias, kb, iters = args
    with threadpool_limits(1):
        t0 = time.perf_counter()
        for h in range(q.shape[0]):
            z = O.logits(q[h, 0], k[h], scale[h], bias)
            O.row_dense_topk(z, v[h], (kb,))
            O.row_best_subset(z, v[h], kb)
            O.swap_rule(O.weights(z), v[h], kb, iters, start=O.top_mass_set(z, kb))
        return time.perf_counter() - t0, q.shape[0]


def _cpu_exhaustive(args):
    from threadpoolctl import threadpool_limits
    from oracle import fw_oracle as O
    q, k, v, scale, kb = args
    with threadpool_limits(1):
        t0 = time.perf_counter()
        for h in range(q.shape[0]):
            O.row_best_subset(O.logits(q[h, 0], k[h], scale[h]), v[h], kb)
        return time.perf_counter() - t0, q.shape[0]


def _cpu_swap(args):
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import fw_oracle as O
    q, k, v, scale, bias, kb, iters = args
    with threadpool_limits(1):
        t0 = time.perf_counter()
        sweeps = 0
        for g in range(q.shape[0]):
            z = O.logits(q[g], k, scale, bias)
            _, _, ns = O.swap_rule(O.weights(z), v, kb, iters, start=O.top_mass_set(z, kb), method="gform")
            sweeps += ns + (1 if ns < iters else 0)
        return time.perf_counter() - t0, sweeps


def _cpu_curve(args):
    from threadpoolctl import threadpool_limits
    from oracle import fw_oracle as O
    q, k, scale = args
    with threadpool_limits(1):
        t0 = time.perf_counter()
        O.dropped_mass_curve(O.importance(q, k, scale))
        return time.perf_counter() - t0, 1


def _pool_run(fn, jobs, cores):
    from concurrent.futures import ProcessPoolExecutor
    t0 = time.perf_counter()
    with ProcessPoolExecutor(max_workers=cores) as ex:
        res = list(ex.map(fn, jobs))
    return time.perf_counter() - t0, sum(r[1] for r in res)


def cpu_configs(seconds):
    """The oracle, timed on this host's cores, on a stated sample of each of
    the five workloads (each sized to about `seconds` of work)."""
    import platform
    import numpy as np
    from paper_2608_25230_amd import workloads as W
    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    try:
        cfg = np.show_config(mode="dicts")
        blas = cfg.get("Build Dependencies", {}).get("blas", {})
        blas = f"{blas.get('name', '?')} {blas.get('version', '')}".strip()
    except Exception:  # noqa: BLE001
        blas = "unknown"
    out = {"cpu_model": model, "host_cpus": os.cpu_count(), "cores": cores, "numpy": np.__version__, "blas": blas,
           "python": platform.python_version(), "kind": "oracle", "configs": []}

    # 1. tiny exhaustive: every row (top-k, exhaustive best subset, swap rule)
    wl = W.tiny_exhaustive(seed=0)
    r = wl.rows
    q, k, v = r.as_f64("q"), r.as_f64("k"), r.as_f64("v")
    bias = r.bias.astype(np.float64)
    chunks = np.array_split(np.arange(r.H), cores)
    jobs = [(q[c], k[c], v[c], r.scale[c].astype(np.float64), bias, wl.k, 64) for c in chunks]
    wall, done = _pool_run(_cpu_tiny, jobs, cores)
    out["configs"].append({"config": 1, "workload": wl.name, "sample": f"all {done} rows", "wall_s": round(wall, 2),
                           "rows_per_s": round(done / wall, 1),
                           "subsets_per_s": round(done * math.comb(r.n, wl.k) / wall, 1)})
    _progress("cpu config %d done" % out["configs"][-1]["config"])

    # 2. streaming top-k: the headline's own leg
    wl = W.streaming_topk(seed=0)
    b = cpu_baseline(wl, seconds)
    out["configs"].append({"config": 2, "workload": wl.name, "sample": b["sample"], "rows_per_s": b["value"]})
    _progress("cpu config %d done" % out["configs"][-1]["config"])

    # 3. exhaustive: a sample of rows, sized from a calibration row
    wl = W.exhaustive_rows(seed=0, rows=cores * 64)
    r = wl.rows
    q, k, v = r.as_f64("q"), r.as_f64("k"), r.as_f64("v")
    t, _ = _cpu_exhaustive((q[:1], k[:1], v[:1], r.scale[:1].astype(np.float64), wl.k))
    nrows = int(min(r.H, max(cores, seconds * cores / t)))
    chunks = np.array_split(np.arange(nrows), cores)
    jobs = [(q[c], k[c], v[c], r.scale[c].astype(np.float64), wl.k) for c in chunks]
    wall, done = _pool_run(_cpu_exhaustive, jobs, cores)
    out["configs"].append({"config": 3, "workload": "exhaustive_R168192_n24_k6",
                           "sample": f"the first {done} of 168192 rows", "wall_s": round(wall, 2),
                           "rows_per_s": round(done / wall, 2),
                           "subsets_per_s": round(done * math.comb(r.n, wl.k) / wall, 1)})
    _progress("cpu config %d done" % out["configs"][-1]["config"])

    # 4. swap rule on long rows: a sample of rows, a bounded number of swaps
    wl = W.swap_long_rows(seed=0)
    r = wl.rows
    iters = 2
    q, k, v = r.as_f64("q"), r.as_f64("k"), r.as_f64("v")
    bias = r.bias.astype(np.float64)
    jobs = [(q[i % r.H, i // r.H: i // r.H + 1], k[i % r.H], v[i % r.H], float(r.scale[i % r.H]), bias, wl.k, iters)
            for i in range(cores)]
    wall, sweeps = _pool_run(_cpu_swap, jobs, cores)
    out["configs"].append({"config": 4, "workload": wl.name,
                           "sample": f"{cores} rows (one per core) with at most {iters} swaps each, {sweeps} sweeps",
                           "wall_s": round(wall, 2), "pairs_per_s": round(sweeps * wl.k * (r.n - wl.k) / wall, 1),
                           "sweeps_per_s": round(sweeps / wall, 3)})
    _progress("cpu config %d done" % out["configs"][-1]["config"])

    # 5. curve: a sample of cells (window importance, sort, suffix sums)
    # (cells are seeded one by one, so the first cells of a smaller call are
    # the first cells of the full 256-cell workload)
    wl = W.curve_ragged(seed=0, layers=max(1, (cores + 7) // 8))
    r = wl.rows
    ncell = min(cores, r.H)
    jobs = [(r.as_f64("q")[h], W.bf16_to_f32(r.k[h]).astype(np.float64), float(r.scale[h])) for h in range(ncell)]
    wall, done = _pool_run(_cpu_curve, jobs, cores)
    out["configs"].append({"config": 5, "workload": "curve_ragged_L32_kv8_n131072",
                           "sample": f"the first {done} of 256 cells (importance and curve)",
                           "wall_s": round(wall, 2), "cells_per_s": round(done / wall, 3)})
    _progress("cpu config %d done" % out["configs"][-1]["config"])
    return out


# ---------------------------------------------------------------------------
def main():
    a = _args()
    if a.cpu_configs:
        print(json.dumps(cpu_configs(a.cpu_seconds)))
        return
    if a.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU: the entry points take one device "
                                   "and exchange nothing across GPUs; run with --gpus 1"}))
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2608_25230_amd import fw
    from paper_2608_25230_amd import workloads as W

    fw.lib()
    torch.cuda.set_device(0)
    only = set(x for x in a.only.split(",") if x)
    want = lambda name: not only or name in only
    components = []
    head = None

    # ---- headline: streaming top-k ------------------------------------------
    if want("topk"):
        wl = W.streaming_topk(seed=0)
        r = wl.rows
        dev = fw.upload(r)
        R = r.H * r.G
        ws = [None]

        def step():
            out = fw.dense_topk(dev["q"], dev["k"], dev["v"], wl.ks, dev["scale"], dev["bias"],
                                want_idx=False, ws=ws[0])
            ws[0] = out["_ws"]

        ms, wall, per = _time(torch, step, a.steps, a.warmup)
        kv = 2 * r.H * r.n * r.d * 2
        qb = R * r.d * 2
        outb = R * r.d * 4 * (1 + len(wl.ks)) + 2 * len(wl.ks) * R * 4
        alg = kv + qb + outb
        head = dict(wl=wl, ms=ms, R=R, alg_bytes=alg, wall=wall, mean=sum(per) / len(per), lo=per[0], hi=per[-1])

        # the same step with the rank-ordered top-k indices of the largest
        # budget as a further output (int32 [rows][kmax])
        def step_idx():
            out = fw.dense_topk(dev["q"], dev["k"], dev["v"], wl.ks, dev["scale"], dev["bias"], ws=ws[0])
            ws[0] = out["_ws"]

        ms_i, _, _ = _time(torch, step_idx, a.steps, a.warmup)
        alg_i = alg + R * max(wl.ks) * 4
        components.append({"workload": wl.name + "_with_topk_idx", "metric": "attention rows/s (top-k gap)",
                           "value": round(R / (ms_i / 1e3), 1), "unit": "rows/s", "ms": round(ms_i, 4),
                           "outputs": "o, o_S, gap, dropped, topk_idx", "algorithmic_bytes": alg_i,
                           "roofline": _roofline("hbm", alg_i / (ms_i / 1e3) / 1e9, HBM_PEAK_GBS, "GB/s"),
                           "dtype": "bf16"})
        del dev, ws
        torch.cuda.empty_cache()
        _progress("%s done" % wl.name)

    # ---- exhaustive best subset ------------------------------------------------
    if want("exhaustive"):
        wl = W.exhaustive_rows(seed=0)
        r = wl.rows
        dev = fw.upload(r)
        ws = [None]

        def step():
            out = fw.best_subset(dev["q"], dev["k"], dev["v"], wl.k, dev["scale"], dev["bias"], ws=ws[0])
            ws[0] = out["_ws"]

        ms, _, _ = _time(torch, step, max(3, a.steps // 3), 1)
        subsets = r.H * r.G * math.comb(r.n, wl.k)
        sps = subsets / (ms / 1e3)
        # the walk's work per subset: two adds for the running sum, one
        # multiply-add and one add for the test value, one compare (float64
        # VALU lane-ops); peak = 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
        ops = 5 * sps
        components.append({"workload": wl.name, "metric": "subsets evaluated/s", "value": round(sps, 1),
                           "unit": "subsets/s", "ms": round(ms, 3), "subsets": subsets,
                           "dtype": "f64",
                           "roofline": dict(_roofline("alu", ops / 1e12, round(VALU_LANE_OPS / 1e12, 2),
                                                      "TOP/s"), kernel="best_subset_kernel",
                                            ops_per_subset=5),
                           # context: the direct d-dimensional update costs 3d + 6 flops
                           # per subset; the Gram form does the same search in 5 ops
                           "d_dim_equivalent_tflops": round(sps * (3 * r.d + 6) / 1e12, 1)})
        del dev, ws
        torch.cuda.empty_cache()
        _progress("%s done" % wl.name)

    # ---- swap rule --------------------------------------------------------------
    if want("swap"):
        wl = W.swap_long_rows(seed=0)
        r = wl.rows
        dev = fw.upload(r)
        holder = {}

        def step():
            out = fw.swap(dev["q"], dev["k"], dev["v"], wl.k, wl.max_iters, dev["scale"], dev["bias"],
                          ws=holder.get("ws"))
            holder["ws"] = out["_ws"]
            holder["n_swaps"] = out["n_swaps"]

        ms, _, _ = _time(torch, step, 3, 1)
        R = r.H * r.G
        ns = holder["n_swaps"]
        # sweeps run: one per accepted swap, plus the final sweep that finds no
        # improving pair on rows that stop before max_iters
        sweeps = int(ns.sum().item()) + int((ns < wl.max_iters).sum().item())
        pairs = sweeps * wl.k * (r.n - wl.k)
        # Work the pruned search is known to do per row and sweep: the dots
        # g . u_j (d multiply-adds per key) and one whole-slice bound test
        # (about three lane-ops) per kept key and 16-key slice of dropped keys.
        # The per-pair tests inside the slices that pass, and the survivors'
        # exact scores, are not counted: the fraction is a lower bound.  A
        # dense sweep would take every pair's cross term on MFMA: 2 k n d flops
        # per row and sweep (context only).
        lane_ops = sweeps * (r.n * r.d + 3 * wl.k * ((r.n - wl.k + 15) // 16))
        dense_flop = sweeps * wl.k * r.n * r.d * 2
        components.append({"workload": wl.name, "metric": "swap pairs evaluated/s",
                           "value": round(pairs / (ms / 1e3), 1), "unit": "pairs/s", "ms": round(ms, 3),
                           "rows_per_s": round(R / (ms / 1e3), 2),
                           "median_swaps": float(holder["n_swaps"].float().median().item()),
                           "dtype": "bf16",
                           "roofline": dict(_roofline("alu", lane_ops / (ms / 1e3) / 1e12, round(VALU_LANE_OPS / 1e12, 2), "TOP/s"),
                                            kernel="fw_swap (all launches: dots, bound test, survivors)",
                                            lane_ops=lane_ops, sweeps=sweeps,
                                            note="lower bound: per-pair tests in passing slices not counted"),
                           "dense_sweep_equivalent_tflops": round(dense_flop / (ms / 1e3) / 1e12, 1)})
        del dev, holder
        torch.cuda.empty_cache()
        _progress("%s done" % components[-1]["workload"])

    # ---- candidate-set search (ES_pool, pool balancing, certificate) -------------
    if want("pool"):
        wl = W.pool_rows(seed=0)
        r = wl.rows
        dev = fw.upload(r)
        holder = {}

        def step():
            o = fw.pool_subset(dev["q"], dev["k"], dev["v"], wl.meta["budgets"], wl.max_iters, dev["scale"],
                               dev["bias"], fw_iters=FW_ITERS, ws=holder.get("ws"))
            holder["ws"] = o["_ws"]
            holder["n_swaps"] = o["n_swaps"]
            holder["stats"] = o["stats"]

        ms, _, _ = _time(torch, step, max(3, a.steps // 2), 1)
        R = r.H * r.G
        subsets = R * sum(math.comb(s_ + e_, s_) for s_, e_ in wl.meta["budgets"])
        # float64 lane-ops of the method: per row the logits, the dense output
        # and the deviations (4 n d: one multiply-add per element, plus the
        # subtraction of the deviations), and per pool subset the walk's five
        # (as for the exhaustive search); peak = 256 CUs x 4 SIMDs x 16 lanes
        lane_ops = R * 4 * r.n * r.d + 5 * subsets
        components.append({"workload": wl.name, "metric": "pool subsets evaluated/s",
                           "value": round(subsets / (ms / 1e3), 1), "unit": "subsets/s", "ms": round(ms, 3),
                           "rows_per_s": round(R / (ms / 1e3), 1), "subsets": subsets,
                           "roofline": dict(_roofline("alu", lane_ops / (ms / 1e3) / 1e12,
                                                      round(VALU_LANE_OPS / 1e12, 2), "TOP/s"),
                                            kernel="pool_row_kernel + pool_enum_kernel", lane_ops=lane_ops),
                           "budgets": [list(b) for b in wl.meta["budgets"]],
                           "median_swaps": {str(s_): float(holder["n_swaps"][b].float().median().item())
                                            for b, (s_, _) in enumerate(wl.meta["budgets"])},
                           "fw_iters": FW_ITERS,
                           "median_fw_steps": {str(s_): float(_stat(holder, b, "fw_steps").median().item())
                                               for b, (s_, _) in enumerate(wl.meta["budgets"])},
                           "median_pi_hat": {str(s_): float(_stat(holder, b, "pi_hat").median().item())
                                             for b, (s_, _) in enumerate(wl.meta["budgets"])},
                           "median_geo_over_top": {
                               str(s_): float((_stat(holder, b, "es_geo") / _stat(holder, b, "es_top")).median().item())
                               for b, (s_, _) in enumerate(wl.meta["budgets"])},
                           "dtype": "f64"})
        del dev, holder
        torch.cuda.empty_cache()
        _progress("%s done" % components[-1]["workload"])

    # ---- candidate-set search with the widened enumeration cap ---------------------
    if want("poolcap"):
        wl = W.pool_rows(seed=0)
        r = wl.rows
        budgets = [(32, 5), (32, 6)]
        dev = fw.upload(r)
        holder = {}

        def step():
            o = fw.pool_subset(dev["q"], dev["k"], dev["v"], budgets, wl.max_iters, dev["scale"], dev["bias"],
                               fw_iters=FW_ITERS, want_cells=False, ws=holder.get("ws"))
            holder["ws"] = o["_ws"]

        ms, _, _ = _time(torch, step, 3, 1)
        R = r.H * r.G
        subsets = R * sum(math.comb(s_ + e_, s_) for s_, e_ in budgets)
        lane_ops = R * 4 * r.n * r.d + 5 * subsets
        components.append({"workload": wl.name + "_cap", "metric": "pool subsets evaluated/s",
                           "value": round(subsets / (ms / 1e3), 1), "unit": "subsets/s", "ms": round(ms, 3),
                           "subsets": subsets, "budgets": [list(b) for b in budgets],
                           "subsets_per_row": [math.comb(s_ + e_, s_) for s_, e_ in budgets],
                           "roofline": dict(_roofline("alu", lane_ops / (ms / 1e3) / 1e12,
                                                      round(VALU_LANE_OPS / 1e12, 2), "TOP/s"),
                                            kernel="pool_row_kernel + pool_enum_kernel", lane_ops=lane_ops),
                           "dtype": "f64"})
        del dev, holder
        torch.cuda.empty_cache()
        _progress("%s done" % components[-1]["workload"])

    # ---- group vote ------------------------------------------------------------------
    if want("vote"):
        wl = W.pool_rows(seed=0)
        r = wl.rows
        dev = fw.upload(r)
        holder = {}
        gs, sv = 4, 8  # the 4 query heads of a key/value head, at s = 8

        def step():
            holder["out"] = fw.group_vote(dev["q"], dev["k"], dev["v"], sv, gs, dev["scale"], dev["bias"])

        ms, _, _ = _time(torch, step, max(3, a.steps // 2), 1)
        R = r.H * r.G
        o = holder["out"]
        ratio = (o["es_vote"] / o["es_top"].clamp_min(1e-30)).float().median().item()
        # float64 lane-ops of the method: per row the logits and the dense
        # output (one multiply-add per element each)
        lane_ops = R * 2 * r.n * r.d
        components.append({"workload": wl.name + "_vote", "metric": "group-vote rows/s",
                           "value": round(R / (ms / 1e3), 1), "unit": "rows/s", "ms": round(ms, 3),
                           "group_size": gs, "s": sv, "median_es_vote_over_es_top": round(ratio, 4),
                           "roofline": dict(_roofline("alu", lane_ops / (ms / 1e3) / 1e12,
                                                      round(VALU_LANE_OPS / 1e12, 2), "TOP/s"),
                                            kernel="vote_group_kernel", lane_ops=lane_ops),
                           "dtype": "f64"})
        del dev, holder
        torch.cuda.empty_cache()
        _progress("%s done" % components[-1]["workload"])

    # ---- dropped-mass curve + ragged compaction --------------------------------
    if want("curve"):
        wl = W.curve_ragged(seed=0)
        r = wl.rows
        dev = fw.upload(r)
        holder = {}

        def step():
            c = fw.dropped_mass_curve(dev["q"], dev["k"], dev["scale"], dev["bias"], want_order=False,
                                      ws=holder.get("ws1"))
            holder["ws1"] = c["_ws"]
            o = fw.ragged_compact(dev["k"], dev["v"], c["importance"], wl.budget, wl.floor,
                                  wl.heads_per_layer, ws=holder.get("ws2"))
            holder["ws2"] = o["_ws"]

        ms, _, _ = _time(torch, step, max(3, a.steps // 3), 1)
        kb = r.H * r.n * r.d * 2
        imp = r.H * r.n * 4
        alg = kb + r.H * r.G * r.d * 2 + 3 * imp + r.H * (r.n + 1) * 4 + 2 * wl.budget * r.d * 2 * 2 \
            + wl.budget * 4
        components.append({"workload": wl.name, "metric": "cells/s", "value": round(r.H / (ms / 1e3), 2),
                           "unit": "cells/s", "ms": round(ms, 3), "algorithmic_bytes": alg,
                           "dtype": "f32",
                           "roofline": _roofline("hbm", alg / (ms / 1e3) / 1e9, HBM_PEAK_GBS, "GB/s")})
        del dev, holder
        torch.cuda.empty_cache()
        _progress("%s done" % components[-1]["workload"])

    # ---- tiny exhaustive ------------------------------------------------------------
    if want("tiny"):
        wl = W.tiny_exhaustive(seed=0)
        r = wl.rows
        dev = fw.upload(r)
        ws = [None]

        def step():
            out = fw.best_subset(dev["q"], dev["k"], dev["v"], wl.k, dev["scale"], dev["bias"], ws=ws[0])
            ws[0] = out["_ws"]

        ms, _, _ = _time(torch, step, a.steps, a.warmup)
        subsets = r.H * math.comb(r.n, wl.k)
        components.append({"workload": wl.name, "metric": "subsets evaluated/s",
                           "value": round(subsets / (ms / 1e3), 1), "unit": "subsets/s",
                           "ms": round(ms, 4), "dtype": "f64", "note": "launch-bound"})
        _progress("%s done" % wl.name)

    # ---- plain device copy (calibrates the HBM byte counters) -------------------
    if want("copy"):
        nbytes = 1 << 31
        src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").uniform_()
        dst = torch.empty_like(src)
        ms, _, _ = _time(torch, lambda: dst.copy_(src), a.steps, a.warmup)
        components.append({"workload": "device copy 2 GiB", "metric": "GB/s",
                           "value": round(2 * nbytes / (ms / 1e3) / 1e9, 1), "unit": "GB/s",
                           "ms": round(ms, 4), "bytes_read": nbytes, "bytes_written": nbytes})
        del src, dst
        _progress("copy done")
        # a plain streaming read (a library reduction over 8 GiB): the HBM read
        # rate a kernel can reach on this part, context for the HBM-bound lines
        nbytes = 8 << 30
        src = torch.ones(nbytes // 8, dtype=torch.int64, device="cuda")
        ms, _, _ = _time(torch, lambda: src.sum(), a.steps, a.warmup)
        components.append({"workload": "device read 8 GiB", "metric": "GB/s",
                           "value": round(nbytes / (ms / 1e3) / 1e9, 1), "unit": "GB/s",
                           "ms": round(ms, 4), "bytes_read": nbytes,
                           "note": "torch.sum over int64: achievable read rate, context only"})
        del src
        _progress("read done")

    if head is None:
        print(json.dumps({"components": components}))
        return
    wl = head["wl"]
    r = wl.rows
    ms = head["ms"]
    gbs = head["alg_bytes"] / (ms / 1e3) / 1e9
    line = {
        "metric": "attention rows/s (top-k gap)",
        "value": round(head["R"] / (ms / 1e3), 1),
        "unit": "rows/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded bf16 N(0,1) rows shaped like the paper's grouped-query heads)",
        "config": {"workload": wl.name, "units": r.H, "rows_per_unit": r.G, "n": r.n, "d": r.d,
                   "ks": list(wl.ks), "rows": head["R"], "outputs": "o, o_S, gap, dropped"},
        "roofline": dict(_roofline("hbm", gbs, HBM_PEAK_GBS, "GB/s", _traffic("streaming_topk_n4096",
                                                                               "k_topk_mp.hip")),
                         kernel="topk_mp_kernel (fw_dense_topk: the 128-row multi-pass kernel, with a flag "
                                "clear before it and the fallback pass after it, timed together)",
                         algorithmic_bytes=head["alg_bytes"], launches_per_step=1),
        "components": components,
    }
    if not a.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, a.cpu_seconds)
        _progress("cpu baseline done")
    print(json.dumps(line))


if __name__ == "__main__":
    main()
