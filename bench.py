"""Benchmark: candidate schedules evaluated per second on one MI355X.

One step = one taccl_eval_batch over the whole batch of the chosen workload
(route decode, send set, Step-2 keys, per-link order, contention timing,
postcondition and makespan for every candidate), inputs already resident in
HBM. Prints one JSON line (rank 0).

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
# int32 VALU issue: 256 CUs x 64 lanes x 2.4 GHz (published unit counts and
# clock), in tera lane-operations per second
INT_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
MAX_ORACLE_THREADS = 16
DEFAULT_WORKLOAD = "twonode16_ag"
# the two workloads the roofline targets are set on: the two-node 2x8-rank
# Allgather and the four-node 64-rank Alltoall
TARGETS = ("twonode16_ag", "fournode64_a2a")


# Kernel that dominates each workload's launch (the only kernel it runs).
KERNEL_OF = {"ring4_ag": "tree_rank", "cubemesh8_ag": "tree_rank",
             "twonode16_ag": "tree_rank", "switch16_a2a": "path_eval_fast",
             "fournode64_a2a": "path_eval_fast", "twonode16_ag_contig": "tree_layers",
             "fournode64_a2a_contig": "path_eval_fast", "cubemesh8_ar": "tree_layers",
             "twonode16_rs": "tree_layers", "twonode16_ar": "tree_layers",
             "cubemesh8_ag_greedy": "tree_greedy", "twonode16_ag_greedy": "tree_greedy",
             "switch16_a2a_ports": "path_eval", "fournode64_a2a_ports": "path_eval",
             "switch16_a2a_greedy": "path_greedy", "fournode64_a2a_greedy": "path_greedy_block",
             "twonode16_ag_rgreedy": "tree_greedy"}


def csrc_digest():
    """SHA-256 over the library sources; measured HBM traffic is only reported
    while the sources are the ones the counters were taken from."""
    d = os.path.join(ROOT, "paper_2111_04867_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".cpp", ".h")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated) from the
    committed counter summary of this workload's kernel, or None when that
    summary is missing or was taken from different sources."""
    path = os.path.join(ROOT, "profiles", f"{KERNEL_OF.get(workload, '?')}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    src = re.search(r"^csrc_sha256: ([0-9a-f]{64})$", text, re.M)
    val = re.search(r"^traffic_bytes_per_launch: ([0-9]+)$", text, re.M)
    if not src or not val or src.group(1) != csrc_digest():
        return None
    return int(val.group(1))


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def time_launches(plan, d_r, d_p, d_m, d_v, steps, warmup):
    """Per-launch durations (ms) from HIP events on the launch stream, plus
    the wall time of the whole timed region."""
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        plan.eval_tensors(d_r, d_p, d_m, d_v, stream=stream)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    ev[0].record(stream)
    for k in range(steps):
        plan.eval_tensors(d_r, d_p, d_m, d_v, stream=stream)
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(steps)])
    return per, wall


def time_calls(fn, steps, warmup):
    """Per-call durations (ms) of fn() from HIP events on torch's current stream."""
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record(stream)
    for k in range(steps):
        fn()
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    return np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(steps)])


def setup(name):
    import torch
    from paper_2111_04867_amd.binding import Plan
    from workloads import generate, named
    w = named(name)
    plan = Plan.from_workload(w)
    opts = plan.route_options()
    t = time.perf_counter()
    routes, prio = generate(w.seed, 0, w.n_candidates, opts, plan.prio_stride)
    log(f"[bench] {name}: generated {w.n_candidates} candidates in "
        f"{time.perf_counter() - t:.2f}s")
    d_r = torch.from_numpy(routes).cuda()
    d_p = torch.from_numpy(prio.view(np.int32)).cuda()
    d_m = torch.empty(w.n_candidates, dtype=torch.int32, device="cuda")
    d_v = torch.empty(w.n_candidates, dtype=torch.uint8, device="cuda")
    return w, plan, routes, prio, (d_r, d_p, d_m, d_v)


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_threads():
    """(hardware threads this process may run on, threads the oracle uses):
    the oracle takes every visible hardware thread, at most MAX_ORACLE_THREADS
    (a GPU machine grants one GPU's share of the host's cores)."""
    try:
        visible = len(os.sched_getaffinity(0))
    except AttributeError:
        visible = os.cpu_count() or 1
    return visible, max(1, min(visible, MAX_ORACLE_THREADS))


def time_oracle(ref, routes, prio, threads, budget_s):
    """Candidates/s of the oracle on a growing prefix of the batch: the prefix
    doubles until the last pass alone took budget_s / 2 or the batch ends.
    Returns (rate, candidates in the last pass, its seconds)."""
    n = max(1, min(threads, routes.shape[0]))
    while True:
        t = time.perf_counter()
        if threads == 1:
            ref.eval(routes[:n], prio[:n])
        else:
            ref.eval_threads(routes[:n], prio[:n], threads=threads)
        dt = time.perf_counter() - t
        if dt >= budget_s / 2 or n == routes.shape[0]:
            return n / dt, n, dt
        n = min(routes.shape[0], n * 2 if dt > 0.05 else n * 8)


def oracle_ops(ref, routes, prio, n):
    """Mean algorithmic operations per candidate over the first n candidates
    (the oracle's exact count of the op model)."""
    _, _, ops = ref.eval_ops(routes[:n], prio[:n])
    return float(ops.mean()), n


def cpu_baselines(names, setups, budget_s):
    """The oracle on the host cores, on one thread and on every visible
    thread, for each named workload: candidates/s, with the samples stated.
    `setups` maps a name to its (workload, routes, prio)."""
    from oracle import OraclePlan
    visible, T = host_threads()
    out = {}
    for name in names:
        w, routes, prio = setups[name]
        ref = OraclePlan.from_workload(w)
        r1, n1, t1 = time_oracle(ref, routes, prio, 1, budget_s)
        rT, nT, tT = time_oracle(ref, routes, prio, T, budget_s)
        ops, n_ops = oracle_ops(ref, routes, prio, min(n1, 64))
        out[name] = {"one_thread": r1, "threads": T, "all_threads": rT,
                     "sample_one_thread": f"first {n1} of {w.n_candidates} ({t1:.2f} s)",
                     "sample_all_threads": f"first {nT} of {w.n_candidates} ({tT:.2f} s)",
                     "ops_per_candidate": ops, "ops_sample": n_ops}
        log(f"[bench] oracle {name}: {r1:.3e} cand/s on 1 thread, {rT:.3e} on {T}; "
            f"{ops:.0f} ops/candidate")
    return out, visible, T


def roofline_pair(n_cand_per_s, bytes_per_cand, ops_per_cand):
    """Both bounds for one workload: achieved HBM bandwidth over algorithmic
    bytes, achieved integer issue over the oracle's op count, and the
    governing (lower) roofline in candidates/s."""
    hbm = n_cand_per_s * bytes_per_cand / 1e9
    out = {"hbm_GBs": hbm, "hbm_frac": hbm / HBM_PEAK_GBS,
           "hbm_roofline_candidates_per_s": HBM_PEAK_GBS * 1e9 / bytes_per_cand}
    if ops_per_cand:
        ti = n_cand_per_s * ops_per_cand / 1e12
        out.update({"int_Tops": ti, "int_issue_frac": ti / INT_PEAK_TOPS,
                    "int_roofline_candidates_per_s": INT_PEAK_TOPS * 1e12 / ops_per_cand})
        gov = min(out["hbm_roofline_candidates_per_s"], out["int_roofline_candidates_per_s"])
        out["governing"] = ("hbm" if gov == out["hbm_roofline_candidates_per_s"]
                            else "int_issue")
        out["governing_frac"] = n_cand_per_s / gov
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cpu-seconds", type=float, default=3.0,
                    help="oracle time budget per workload and thread count")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-all", action="store_true", help="skip the per-workload table")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run device-to-device copies of BYTES (counter calibration)")
    ap.add_argument("--calibrate-read", type=int, default=0, metavar="BYTES",
                    help="only run sums over BYTES of int32 (a second, read-only pattern)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("this evaluator runs on one GPU; candidates shard trivially across GPUs but no "
              "multi-GPU run is implemented (use --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        src = torch.empty(args.calibrate_copy, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": args.calibrate_copy, "copies": args.steps}))
        return
    if args.calibrate_read:
        src = torch.ones(args.calibrate_read // 4, dtype=torch.int32, device="cuda")
        total = 0
        for _ in range(args.steps):
            total += int(src.sum().item())
        print(json.dumps({"calibrate_read_bytes": args.calibrate_read, "sums": args.steps,
                          "checksum": total}))
        return
    from workloads import (CONTIG_ORDER, GREEDY_LARGE_ORDER, GREEDY_ORDER, ORDER, PORTS_ORDER,
                           REDUCE_ORDER)

    w, plan, routes, prio, bufs = setup(args.workload)
    per, wall = time_launches(plan, *bufs, args.steps, args.warmup)
    n = w.n_candidates
    total_s = per.sum() / 1e3
    value = n * args.steps / total_s
    bytes_launch = n * plan.bytes_per_candidate
    avg_s = per.mean() / 1e3
    achieved = bytes_launch / avg_s / 1e9
    rec = {
        "metric": "candidate schedules evaluated/sec (alpha-beta timing + postcondition)",
        "value": value,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": per.mean(),
        "ms_per_step_p10_p50_p90": [float(np.percentile(per, q)) for q in (10, 50, 90)],
        "wall_s_timed_region": wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic (seeded SplitMix64 routes and priorities)",
        "config": {"workload": w.name, "candidates": n, "ranks": w.P, "vertices": w.V,
                   "links": w.E, "chunks": plan.num_chunks,
                   "collective": ["allgather", "alltoall", "explicit", "reducescatter",
                                  "allreduce"][w.kind],
                   "chunk_bytes": w.chunk_bytes, "bytes_per_candidate":
                       plan.bytes_per_candidate, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(w.name),
                     "algorithmic_bytes_per_launch": bytes_launch,
                     "kernel": KERNEL_OF.get(w.name)},
    }
    # host inputs of the five configurations, for the oracle leg
    host = {w.name: (w, routes, prio)}
    timed = {w.name: (value, plan.bytes_per_candidate, per.mean())}
    if not args.no_all:
        table = {}
        for name in (ORDER + CONTIG_ORDER + REDUCE_ORDER + GREEDY_ORDER + GREEDY_LARGE_ORDER +
                     PORTS_ORDER):
            if name == args.workload:
                wl, pl, pr_ = w, plan, per
            else:
                wl, pl, r2, p2, b2 = setup(name)
                pr_, _ = time_launches(pl, *b2, max(10, args.steps // 2), args.warmup)
                del b2
                if name in ORDER:
                    host[name] = (wl, r2, p2)
            a_s = pr_.mean() / 1e3
            gbs = wl.n_candidates * pl.bytes_per_candidate / a_s / 1e9
            table[name] = {"candidates": wl.n_candidates, "ms_per_launch": pr_.mean(),
                           "candidates_per_s": wl.n_candidates / a_s, "achieved_GBs": gbs,
                           "hbm_roofline_frac": gbs / HBM_PEAK_GBS}
            timed[name] = (wl.n_candidates / a_s, pl.bytes_per_candidate, pr_.mean())
            log(f"[bench] {name}: {table[name]['candidates_per_s']:.3e} cand/s, "
                f"{gbs:.1f} GB/s ({100 * gbs / HBM_PEAK_GBS:.2f}% of HBM)")
        rec["all_workloads"] = table
        # switch-hyperedge connection counts (the uc-max / uc-min term)
        conn = {}
        for name in ("switch16_a2a", "fournode64_a2a"):
            wl, pl, _, _, b2 = setup(name)
            d_c = torch.empty(wl.n_candidates, dtype=torch.int32, device="cuda")
            pr_ = time_calls(lambda: pl.connections_tensors(b2[0], d_c),
                             max(10, args.steps // 2), args.warmup)
            a_s = pr_.mean() / 1e3
            conn[name] = {"candidates": wl.n_candidates, "ms_per_launch": pr_.mean(),
                          "candidates_per_s": wl.n_candidates / a_s}
            log(f"[bench] {name} connections: {conn[name]['candidates_per_s']:.3e} cand/s")
            del b2
        rec["connections"] = conn
    if not args.no_cpu:
        names = [nm for nm in ORDER if nm in host] or [w.name]
        if w.name not in names:
            names.append(w.name)
        base, visible, T = cpu_baselines(names, host, args.cpu_seconds)
        hb = base[w.name]
        rec["cpu_baseline"] = {
            "value": hb["all_threads"], "unit": "candidates/s", "cores": T, "kind": "oracle",
            "sample": f"{hb['sample_all_threads']} {w.name} candidates on {T} threads "
                      f"(contiguous ranges); one thread: {hb['sample_one_thread']}",
            "one_thread_value": hb["one_thread"], "cpu_model": cpu_model(),
            "hardware_threads_visible": visible, "per_config": base}
        ops = hb["ops_per_candidate"]
        ti = value * ops / 1e12
        rec["roofline_int_issue"] = {
            "bound": "int_issue", "achieved": ti, "peak": INT_PEAK_TOPS, "unit": "Tops/s",
            "frac": ti / INT_PEAK_TOPS, "ops_per_candidate": ops,
            "ops_sample": f"oracle op count over the first {hb['ops_sample']} candidates"}
        targets = {}
        for name in names:
            if name not in timed:
                continue
            cps, bpc, ms = timed[name]
            b = base[name]
            r = {"candidates_per_s": cps, "ms_per_launch": ms,
                 "bytes_per_candidate": bpc, "ops_per_candidate": b["ops_per_candidate"],
                 "oracle_one_thread": b["one_thread"], "oracle_all_threads": b["all_threads"],
                 "oracle_threads": b["threads"]}
            r.update(roofline_pair(cps, bpc, b["ops_per_candidate"]))
            targets[name] = r
            if "all_workloads" in rec and name in rec["all_workloads"]:
                rec["all_workloads"][name]["int_issue_frac"] = r.get("int_issue_frac")
        rec["configs"] = targets
        rec["targets"] = {nm: targets[nm] for nm in TARGETS if nm in targets}
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
