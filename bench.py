"""Throughput of the multi-signal iteration on one MI355X.

One step = one whole iteration (find winners -> resolve conflicts -> adapt -> update
edges, one gsn_iterate call: the lock-set update runs fused) over one batch of m signals,
on the genus-3 workload (200,000 units, 16,384 signals per iteration, signals drawn from a
4,000,000-point cloud).  All signal batches are resident in HBM before the timed region
starts.

Prints one JSON line:
  value            whole-iteration signal-unit distance evaluations per second (m*N/step)
  signals_per_s    m per step time
  fw_evals_per_s   m*N per find-winners call (HIP events around the call)
  phase_ms         per-call times of the steps, from phase_steps further iterations run
                   after the timed ones with every timer on (inside the timed steps only
                   the scan kernel carries an event pair)
  roofline         the find-winners scan kernel (fh_scan, the screened scan on the matrix
                   cores in split binary16): algorithmic FLOP/s (8 per evaluation) from HIP
                   events around each of its launches in the timed steps, on the library's
                   stream, against the peak of
                   the contraction's type (binary16 dense, 2.5 PFLOP/s); also the matrix
                   cores' executed rate (32 flops per pair: 32x32x16 products, K = 16) and
                   the algorithmic rate against the fp32 peak; HBM traffic per launch from
                   rocprofv3 counters when a summary for the current kernel source exists
  late_window      the same step timed over iterations 81-100 of the workload's stated
                   100-iteration run (a network that has grown its edges), with the edge
                   counts at both ends of the window
  cpu_baseline     the CPU oracle timed on this host's cores on the first iterations of the
                   same workload (its find-winners loop on 16 threads); beside it
                   ``single_core``: the oracle per phase on one pinned core

--sweep prints one JSON line per (collision rule, m) for the sweep workload (100,000 units
on the noisy torus, m in {1, 64, 1,024, 16,384, 65,536}, 10 warm-up + 50 timed
iterations): throughput, conflict rate and, for the winner lock, the birthday estimate of
the conflict rate that the implicit lock on the winner implies for uniformly hit winners.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import shutil
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "signal-unit distance evals/s and signals/s at 1 GPU; % fp32 VALU peak"
FP32_PEAK_TFLOPS = 157.3     # 256 CUs x 2.4 GHz x 256 fp32 flop/clk; also the fp32 MFMA peak
F16_PEAK_TFLOPS = 2500.0     # dense binary16 matrix-core peak
EXECUTED_FLOPS_PER_PAIR = 32  # one 32x32x16 product (32768 flops) per 1,024 pairs
FLOPS_PER_EVAL = 8           # 3 sub + 3 mul + 2 add of one squared distance
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "find_winners_genus3_200k_traffic.json")
SCAN_KERNEL = "fh_scan"
SMALL_SCAN_KERNEL = "sm_scan"      # batches of at most SMALL_M signals take the small-batch scan
SMALL_M = 256
VALU_PLAIN_PEAK_TFLOPS = 39.32     # 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (no FMA, no packing)
SCAN_SOURCES = [os.path.join(ROOT, "paper_1503_08294_amd", "csrc", f)
                for f in ("find_f16.hip", "gsn_internal.h")]


def scan_source_hash() -> str:
    h = hashlib.sha256()
    for path in SCAN_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(launch_evals: int):
    """Per-launch HBM bytes of the scan kernel from the committed counter summary, or None
    if there is none or it was taken on another version of the kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        t = json.load(f)
    if t.get("source_sha256_16") != scan_source_hash() or t.get("launch_evals") != launch_evals:
        return None
    return t.get("bytes_per_launch")


def host_info() -> dict:
    """CPU model and core counts of this host (the oracle's timing context)."""
    model = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            if line.lower().startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count()
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "usable_cpus": usable}


def oracle_threads() -> int:
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count() or 1
    return max(1, min(16, usable))


def oracle_phases_child(args):
    """Child-process mode (no GPU, no torch): the oracle on ONE core, pinned, timed per
    phase over the first iterations of a workload, for each m in args.phase_m; prints one
    JSON object."""
    import numpy as np
    import oracle
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream
    wl = WORKLOADS[args.workload]
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    out = {"cpu": sorted(os.sched_getaffinity(0)), "threads": 1, "runs": []}
    for m in [int(v) for v in args.phase_m.split(",")]:
        cap = wl.capacity(m)
        p = oracle.Params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha, wl.err_beta,
                          cap["n_max"], cap["e_max"], m, lock_mode=args.phase_lock)
        o = oracle.Oracle(p, units, threads=1)
        stream = SignalStream(cloud, wl.signal_seed)
        t = {"find": 0.0, "resolve": 0.0, "adapt": 0.0, "edges": 0.0, "grow": 0.0}
        done = 0
        while done < args.phase_iters:
            sig = stream.next(m)
            t0 = time.perf_counter()
            w, sc, d1, _ = o.find_winners(sig)
            t1 = time.perf_counter()
            acc = o.resolve_conflicts(w, sc, d1)
            t2 = time.perf_counter()
            o.adapt(sig, w, sc, d1, acc)
            t3 = time.perf_counter()
            o.update_edges(w, sc, acc)
            t4 = time.perf_counter()
            if wl.grow:
                o.grow(done + 1, wl.insert_every)
            t5 = time.perf_counter()
            t["find"] += t1 - t0
            t["resolve"] += t2 - t1
            t["adapt"] += t3 - t2
            t["edges"] += t4 - t3
            t["grow"] += t5 - t4
            done += 1
            if sum(t.values()) > args.phase_budget:
                break
        total = sum(t.values())
        n = units.shape[1]
        out["runs"].append({"m": m, "iterations": done,
                            "phase_ms": {k: 1e3 * v / done for k, v in t.items()},
                            "fw_evals_per_s": m * n * done / t["find"],
                            "signals_per_s": m * done / total,
                            "evals_per_s": m * n * done / total})
    print(json.dumps(out), flush=True)


def single_core_oracle(workload: str, ms, iters: int, budget_s: float, lock_mode: int = 0):
    """Runs oracle_phases_child in a child process pinned to one core with taskset.  Call
    it before this process touches the GPU."""
    try:
        cpus = sorted(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        cpus = [0]
    cpu = cpus[-1]
    cmd = [sys.executable, os.path.abspath(__file__), "--oracle-phases",
           "--workload", workload, "--phase-m", ",".join(str(v) for v in ms),
           "--phase-iters", str(iters), "--phase-budget", str(budget_s),
           "--phase-lock", str(lock_mode)]
    if shutil.which("taskset"):
        cmd = ["taskset", "-c", str(cpu)] + cmd
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run(cmd, capture_output=True, text=True, env=env,
                       timeout=300 + 3 * budget_s * len(ms))
    if r.returncode != 0:
        print(r.stderr[-2000:], file=sys.stderr, flush=True)
        return {"error": f"oracle child exited with {r.returncode}"}
    res = json.loads(r.stdout.strip().splitlines()[-1])
    res["pinned_with"] = "taskset -c %d" % cpu if cmd[0] == "taskset" else "sched_setaffinity"
    return res


def cpu_baseline(wl, units, cloud, budget_s: float, lock_mode: int = 0, key_mode: int = 0,
                 m: int | None = None, max_iters: int = 200):
    """The oracle on the same initial units and the same seeded signal batches as the GPU
    run, whole iterations until about budget_s seconds have passed (at most 200)."""
    import oracle
    from paper_1503_08294_amd.clouds import SignalStream
    m = m or wl.m
    threads = oracle_threads()
    cap = wl.capacity(m)
    p = oracle.Params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha, wl.err_beta,
                      cap["n_max"], cap["e_max"], m, lock_mode=lock_mode,
                      key_mode=key_mode)
    o = oracle.Oracle(p, units, threads=threads)
    stream = SignalStream(cloud, wl.signal_seed)
    dt = 0.0
    done = 0
    accepted = 0
    while done < max_iters and (done == 0 or dt < budget_s):
        sig = stream.next(m)
        t0 = time.perf_counter()
        acc = o.iterate(sig)[4]
        if wl.grow:
            o.grow(done + 1, wl.insert_every)
        dt += time.perf_counter() - t0
        accepted += int(acc.sum())
        done += 1
    evals = m * units.shape[1] * done
    return {"value": evals / dt, "unit": "evals/s", "cores": threads, "kind": "oracle",
            "signals_per_s": m * done / dt, "accepted_per_s": accepted / dt,
            "sample": f"first {done} whole iterations of {wl.name} (N={units.shape[1]}, "
                      f"m={m}), oracle find-winners loop on {threads} threads, the rest "
                      "of the iteration sequential",
            "seconds": dt}


# The growing-network run: genus-3 cloud (4,000,000 points), two initial cloud points,
# m = smallest power of two above N capped at 8192, one GNG insertion every 100 signals,
# stop when a window of 65,536 signals has a mean squared winner distance below 1.5e-5.
SCHEDULE = dict(m_cap=8192, insert_every=100, qe_window=65536, max_signals=40_000_000,
                qe_threshold=1.5e-5, seed=3)
SCHEDULE_N_MAX = 200_000
SCHEDULE_CPU_SIGNALS = 2_000_000


def run_schedule_bench(args):
    import numpy as np
    import torch

    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, initial_units

    wl = WORKLOADS["genus3_200k"]
    print(f"[bench] generating the genus-3 cloud ({wl.n_points} points)", file=sys.stderr,
          flush=True)
    cloud = wl.make_cloud()
    units = initial_units(cloud, 2, wl.unit_seed)
    soa = np.ascontiguousarray(cloud.T)
    torch.cuda.set_device(0)
    dev_cloud = torch.from_numpy(soa).cuda()
    lock_mode = {"set": gsn.GSN_LOCK_SET, "winner": gsn.GSN_LOCK_WINNER,
                 "greedy": gsn.GSN_LOCK_SET_GREEDY}[args.lock]
    key_mode = gsn.GSN_KEY_INDEX if args.key == "index" else gsn.GSN_KEY_DIST_INDEX
    n_max = SCHEDULE_N_MAX
    params = gsn.make_params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha, wl.err_beta,
                             n_max, 4 * n_max + 16, SCHEDULE["m_cap"], lock_mode, key_mode)

    def one_run(max_signals):
        net = gsn.Network(params, torch.from_numpy(units).cuda())
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r = net.run_schedule(dev_cloud, gsn.make_schedule(**dict(SCHEDULE,
                                                                 max_signals=max_signals)))
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        if net.check() != 0:
            raise SystemExit(f"device status {net.check()} after the run")
        net.close()
        return r, el

    print("[bench] warmup run (first 1M signals)", file=sys.stderr, flush=True)
    one_run(1_000_000)
    print("[bench] timed run", file=sys.stderr, flush=True)
    r, el = one_run(SCHEDULE["max_signals"])
    out = {
        "metric": "growing-network run to the quantization-error threshold: signals/s",
        "value": r["signals"] / el,
        "unit": "signals/s",
        "n_gpus": 1,
        "steps": r["iterations"],
        "warmup": 1,
        "ms_per_step": 1e3 * el / r["iterations"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE,
        "data": "synthetic",
        "config": {"workload": "genus3_schedule", "cloud_points": wl.n_points,
                   "initial_units": 2, "n_max": n_max, **SCHEDULE,
                   "collision": {"lock": args.lock, "key": args.key},
                   "screen": SCREEN + " above 256 signals per iteration; binary32 direct "
                             "form at and below",
                   "parallelism": "single"},
        "seconds": el,
        "result": r,
        "accepted_per_s": r["accepted"] / el,
        "cpu_baseline": None,
    }
    if args.cpu_budget > 0:
        import oracle
        print(f"[bench] cpu baseline (first {SCHEDULE_CPU_SIGNALS} signals)", file=sys.stderr,
              flush=True)
        threads = oracle_threads()
        o = oracle.Oracle(oracle.Params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha,
                                        wl.err_beta, n_max, 4 * n_max + 16,
                                        SCHEDULE["m_cap"], lock_mode=lock_mode,
                                        key_mode=key_mode), units, threads=threads)
        t0 = time.perf_counter()
        ro = o.run_schedule(soa, oracle.Schedule(**dict(SCHEDULE,
                                                        max_signals=SCHEDULE_CPU_SIGNALS)))
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": ro["signals"] / dt, "unit": "signals/s",
                               "cores": threads, "kind": "oracle",
                               "sample": f"the first {ro['signals']} signals of the same run "
                                         f"(N 2 -> {ro['n_units']}), oracle find-winners on "
                                         f"{threads} threads", "seconds": dt}
        r1, el1 = one_run(SCHEDULE_CPU_SIGNALS)
        out["gpu_same_sample"] = {"signals_per_s": r1["signals"] / el1, "seconds": el1,
                                  "n_units": r1["n_units"]}
    print(json.dumps(out), flush=True)


def copy_calibration(nbytes: int, reps: int):
    """A plain device copy of known size, for scaling FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "reps": reps}), flush=True)



SCREEN = "f16-split MFMA screen, exact f32 direct-form recheck"
DTYPE = "f16-split MFMA screen + f32 recheck"
LATE_WINDOW = (81, 100)      # iterations timed on the grown network (stated run: 100)


def lock_modes(gsn, args):
    lock_mode = {"set": gsn.GSN_LOCK_SET, "winner": gsn.GSN_LOCK_WINNER,
                 "greedy": gsn.GSN_LOCK_SET_GREEDY}[args.lock]
    key_mode = gsn.GSN_KEY_INDEX if args.key == "index" else gsn.GSN_KEY_DIST_INDEX
    return lock_mode, key_mode


def tune(gsn, net, args):
    """Launch-configuration knobs from the command line (results never depend on them)."""
    if args.variant:
        net.tune(gsn.GSN_TUNE_VARIANT, args.variant)
    if args.split:
        net.tune(gsn.GSN_TUNE_SPLIT, args.split)
    if args.grab:
        net.tune(gsn.GSN_TUNE_GRAB, args.grab)
    if args.rebucket:
        net.tune(gsn.GSN_TUNE_REBUCKET, args.rebucket)


SCAN_TIMER_EVERY = 4   # inside the timed steps the scan carries an event pair every 4th step


def time_loop(torch, gsn, units, params, args, warm_batches, batches):
    """The same iterations through gsn_iterate_loop on a second network from the same start:
    the warm-up batches one gsn_iterate call each, a snapshot (gsn_export) imported back at
    once (so that both loop calls below start from the host state an import leaves), one
    loop call over ``batches`` (it records the loop's HIP graph and runs it: timed as the
    first call), the snapshot imported again, and the same loop call again: a replay of the
    recorded graph over the same iterations from the same state (the loop's rate; its end
    state must equal the first call's bit for bit).  No event timers (they do not record
    inside a loop)."""
    import numpy as np
    count, _, m = batches.shape
    net = gsn.Network(params, torch.from_numpy(units).cuda())
    tune(gsn, net, args)
    for sig in warm_batches:
        net.iterate(torch.from_numpy(np.ascontiguousarray(sig)).cuda())
    snap = net.export()
    net.import_state(snap["xyz"], snap["err"], snap["edges"])
    buf = torch.from_numpy(np.ascontiguousarray(batches)).cuda()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    net.iterate_loop(buf)
    torch.cuda.synchronize()
    first_s = time.perf_counter() - t0
    end1 = net.export()
    records = net.stat(gsn.GSN_STAT_LOOP_RECORDS)
    net.import_state(snap["xyz"], snap["err"], snap["edges"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    net.iterate_loop(buf)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    if net.check() != 0:
        raise SystemExit(f"device status {net.check()} after the loop")
    end2 = net.export()
    same = all(torch.equal(end1[k], end2[k]) for k in ("xyz", "err", "edges"))
    w = len(warm_batches)
    rec = {"iterations": [w + 1, w + count],
           "first_call_ms_per_step": 1e3 * first_s / count,
           "replayed": net.stat(gsn.GSN_STAT_LOOP_RECORDS) == records,
           "replay_equals_first_call": same,
           "ms_per_step": 1e3 * el / count, "evals_per_s": m * units.shape[1] * count / el,
           "signals_per_s": m * count / el, "edges_at_start": int(snap["edges"].shape[1]),
           "edges_at_end": int(end2["edges"].shape[1])}
    del net, buf
    return rec


def timed_steps(torch, gsn, net, step, first, count, scan_only=True):
    """Runs steps first .. first+count-1 between two synchronizations.  With scan_only the
    scan's HIP event pair is the only timer inside the window, recorded on every
    SCAN_TIMER_EVERY-th step (each pair of markers idles the stream a few microseconds), else
    every phase timer records on every step.  Returns the elapsed seconds, {timer: (mean ms
    per launch, launches)}, and the resolved and accepted signal counts."""
    for w in range(gsn.GSN_T_COUNT):
        gsn.gsn_timing_read(net.h, w)
    gsn.gsn_timing_select(net.h, (1 << gsn.GSN_T_FIND_SCAN) if scan_only
                          else (1 << gsn.GSN_T_COUNT) - 1)
    torch.cuda.synchronize()
    net.stat(gsn.GSN_STAT_CLEAR)
    every = SCAN_TIMER_EVERY if scan_only else 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(first, first + count):
        if every > 1:
            gsn.gsn_timing_enable(net.h, (t - first) % every == 0)
        else:
            gsn.gsn_timing_enable(net.h, True)
        step(t)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gsn.gsn_timing_enable(net.h, False)
    timers = {}
    for w in range(gsn.GSN_T_COUNT):
        ms, launches = gsn.gsn_timing_read(net.h, w)
        timers[w] = (ms / max(launches, 1), launches)
    resolved = net.stat(gsn.GSN_STAT_RESOLVED)
    accepted = net.stat(gsn.GSN_STAT_ACCEPTED)
    if net.check() != 0:
        raise SystemExit(f"device status {net.check()} after steps {first}..{first + count}")
    return elapsed, timers, resolved, accepted


def scan_roofline(m, n, scan_ms, launches, traffic):
    scan_s = max(scan_ms, 1e-9) * 1e-3
    achieved = FLOPS_PER_EVAL * m * n / scan_s / 1e12
    if m <= SMALL_M:
        # the small-batch scan: direct-form distances on the vector unit, one binary32
        # operation per lane and cycle (no fused multiply-add in the definition)
        return {"bound": "alu", "kernel": SMALL_SCAN_KERNEL, "dtype": "f32",
                "achieved": achieved, "peak": VALU_PLAIN_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / VALU_PLAIN_PEAK_TFLOPS, "traffic": None,
                "flops_per_launch": FLOPS_PER_EVAL * m * n, "avg_launch_ms": scan_ms,
                "launches_timed": launches,
                "peak_derivation": "256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz, one plain binary32 "
                                   "operation per lane per cycle"}
    return {"bound": "mfma", "kernel": SCAN_KERNEL, "dtype": "f16",
            "achieved": achieved, "peak": F16_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / F16_PEAK_TFLOPS, "traffic": traffic,
            "flops_per_launch": FLOPS_PER_EVAL * m * n,
            "avg_launch_ms": scan_ms, "launches_timed": launches,
            "executed_mfma_tflops": EXECUTED_FLOPS_PER_PAIR * m * n / scan_s / 1e12,
            "executed_mfma_frac": EXECUTED_FLOPS_PER_PAIR * m * n / scan_s / 1e12
                                  / F16_PEAK_TFLOPS,
            "algorithmic_rate_vs_fp32_peak": achieved / FP32_PEAK_TFLOPS}


def birthday_conflict_rate(n: int, m: int) -> float:
    """Expected discarded fraction when m signals hit N equally likely winners and one
    survives per winner: 1 - (N/m)(1 - (1 - 1/N)^m) ~ 1 - (N/m)(1 - e^(-m/N))."""
    return 1.0 - (n / m) * (1.0 - math.exp(m * math.log1p(-1.0 / n)))


def run_sweep(args):
    """The sweep workload: for each collision rule and each m, a fresh network of 100,000
    units, 10 warm-up and 50 timed iterations; one JSON line per record."""
    import numpy as np

    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream

    wl = WORKLOADS["torus_sweep"]
    ms = [int(v) for v in args.sweep_m.split(",")] if args.sweep_m else list(wl.sweep_m)
    locks = args.sweep_locks.split(",")
    single = None
    if args.cpu_budget > 0:
        # before this process touches the GPU: a pinned child process, one core
        print("[bench] single-core oracle per phase (pinned)", file=sys.stderr, flush=True)
        single = single_core_oracle(wl.name, ms, 5, min(args.cpu_budget, 6.0))

    import torch

    from paper_1503_08294_amd import gsn

    print(f"[bench] generating {wl.name}: {wl.n_points} cloud points, N={wl.n_units}",
          file=sys.stderr, flush=True)
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    n = units.shape[1]
    torch.cuda.set_device(0)
    host = host_info()
    warm, steps = 10, 50
    for lock in locks:
        args.lock = lock
        lock_mode, key_mode = lock_modes(gsn, args)
        for m in ms:
            print(f"[bench] sweep lock={lock} m={m}", file=sys.stderr, flush=True)
            stream = SignalStream(cloud, wl.signal_seed)
            dev_sig = torch.from_numpy(np.stack([stream.next(m)
                                                 for _ in range(warm + steps)])).cuda()
            cap = wl.capacity(m)
            params = gsn.make_params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha,
                                     wl.err_beta, cap["n_max"], cap["e_max"], m, lock_mode,
                                     key_mode)
            net = gsn.Network(params, torch.from_numpy(units).cuda())
            tune(gsn, net, args)
            prep = net.prepare_iterate([dev_sig[t] for t in range(warm + steps)])

            def step(t):
                prep(t)

            for t in range(warm):
                step(t)
            el, timers, resolved, accepted = timed_steps(torch, gsn, net, step, warm, steps)
            scan_ms, launches = timers[gsn.GSN_T_FIND_SCAN]
            loop_rec = None
            if not args.no_loop:
                batches = dev_sig.cpu().numpy()
                loop_rec = time_loop(torch, gsn, units, params, args, batches[:warm],
                                     batches[warm:warm + steps])
            rec = {
                "metric": "sweep: signals/s and conflict rate vs m at 1 GPU",
                "value": m * steps / el, "unit": "signals/s", "n_gpus": 1,
                "steps": steps, "warmup": warm, "ms_per_step": 1e3 * el / steps,
                "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
                "dtype": DTYPE, "data": "synthetic",
                "config": {"workload": wl.name, "n_units": n, "m_signals": m,
                           "cloud_points": wl.n_points, "cloud": "noisy torus",
                           "collision": {"lock": lock, "key": args.key},
                           "screen": SCREEN, "parallelism": "single"},
                "evals_per_s": m * n * steps / el,
                "accepted_per_s": accepted / el,
                "conflict_rate": 1.0 - accepted / max(resolved, 1),
                "roofline": scan_roofline(m, n, scan_ms, launches, None),
                "state_after": dict(zip(("units", "edges"), net.sizes())),
                "loop": loop_rec,
            }
            if lock_mode == gsn.GSN_LOCK_WINNER:
                rec["birthday_conflict_rate"] = birthday_conflict_rate(n, m)
                updates = net.stat(gsn.GSN_STAT_UPDATES)
                rec["update_rounds"] = ({"mean": net.stat(gsn.GSN_STAT_ROUNDS) / updates,
                                         "max": net.stat(gsn.GSN_STAT_ROUNDS_MAX)}
                                        if updates else None)
            if args.cpu_budget > 0:
                rec["cpu_baseline"] = cpu_baseline(wl, units, cloud, min(args.cpu_budget, 3.0),
                                                   lock_mode, key_mode, m=m, max_iters=60)
                rec["cpu_baseline"]["host"] = host
                if single and lock == "set":
                    rec["cpu_baseline"]["single_core"] = dict(
                        next((r for r in single.get("runs", []) if r["m"] == m), {}),
                        pinned_with=single.get("pinned_with"))
            net.close()
            del net, dev_sig, prep
            print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="genus3_200k")
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="seconds of CPU oracle work for the cpu_baseline leg (0 = skip)")
    ap.add_argument("--copy-calibration", type=int, default=0,
                    help="only run a plain device copy of this many bytes")
    ap.add_argument("--lock", choices=("set", "winner", "greedy"), default="set",
                    help="collision rule: lock set {b, s} + N(b) with one parallel update, "
                         "the winner alone with the survivors applied in key order, or the "
                         "lock sets taken greedily in key order")
    ap.add_argument("--key", choices=("dist", "index"), default="dist",
                    help="survivor priority: (winner distance, index) or the index alone")
    ap.add_argument("--grid-cell", type=float, default=0.0,
                    help="find winners with the paper's hash index (cubes of this side over "
                         "the cloud's box) instead of the exhaustive search; 0 = exhaustive")
    ap.add_argument("--grid-exact", action="store_true",
                    help="with --grid-cell: certify the index's result per signal and use the "
                         "exhaustive search where it cannot be certified (exact results)")
    ap.add_argument("--schedule", action="store_true",
                    help="instead of fixed-size steps, time one growing-network run "
                         "(gsn_run_schedule) from two units to the quantization-error "
                         "threshold on the genus-3 cloud")
    ap.add_argument("--sweep", action="store_true",
                    help="the sweep workload: one JSON line per collision rule and m")
    ap.add_argument("--sweep-m", default="", help="with --sweep: comma-separated m values")
    ap.add_argument("--sweep-locks", default="set,winner",
                    help="with --sweep: comma-separated collision rules")
    ap.add_argument("--variant", type=int, default=0,
                    help="find-winners kernel variant (GSN_TUNE_VARIANT; 0 = automatic)")
    ap.add_argument("--split", type=int, default=0,
                    help="unit chunks / partial rows of the scan (GSN_TUNE_SPLIT; 0 = automatic)")
    ap.add_argument("--grab", type=int, default=0,
                    help="batches per grab of the dynamic scan (GSN_TUNE_GRAB; 0 = default)")
    ap.add_argument("--rebucket", type=int, default=0,
                    help="find calls between rebuilds of the unit order (GSN_TUNE_REBUCKET)")
    ap.add_argument("--no-loop", action="store_true",
                    help="skip the record of the same iterations run through gsn_iterate_loop")
    ap.add_argument("--no-late-window", action="store_true",
                    help="skip the record of iterations 81-100")
    ap.add_argument("--oracle-iters", type=int, default=3,
                    help="iterations of the single-core oracle timing (bounded by its budget)")
    ap.add_argument("--oracle-budget", type=float, default=0.0,
                    help="seconds of single-core oracle work (0 = min(cpu-budget, 8))")
    # child-process mode of the single-core oracle timing (no GPU)
    ap.add_argument("--oracle-phases", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--phase-m", default="", help=argparse.SUPPRESS)
    ap.add_argument("--phase-iters", type=int, default=2, help=argparse.SUPPRESS)
    ap.add_argument("--phase-budget", type=float, default=10.0, help=argparse.SUPPRESS)
    ap.add_argument("--phase-lock", type=int, default=0, help=argparse.SUPPRESS)
    args = ap.parse_args()

    if args.oracle_phases:
        oracle_phases_child(args)
        return

    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(the path shards by signals across GPUs by design, but only one GPU is used "
              "here)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration, 5)
        return

    if args.schedule:
        run_schedule_bench(args)
        return

    if args.sweep:
        run_sweep(args)
        return

    import numpy as np

    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream

    wl = WORKLOADS[args.workload]
    single = None
    if args.cpu_budget > 0:
        # before this process touches the GPU: a pinned child process, one core
        print("[bench] single-core oracle per phase (pinned)", file=sys.stderr, flush=True)
        single = single_core_oracle(wl.name, [wl.m], args.oracle_iters,
                                    args.oracle_budget or min(args.cpu_budget, 8.0))

    import torch

    from paper_1503_08294_amd import gsn

    print(f"[bench] generating {wl.name}: {wl.n_points} cloud points, N={wl.n_units}, "
          f"m={wl.m}", file=sys.stderr, flush=True)
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    stream = SignalStream(cloud, wl.signal_seed)
    n, m = units.shape[1], wl.m
    # the timed steps, a few more with every phase timer on, one for the conflict rate at
    # their end, then (untimed) up to the late window of the stated run
    phase_steps = min(args.steps, 20)
    t_phase = args.warmup + args.steps
    t_last = t_phase + phase_steps
    late = None if args.no_late_window or args.grid_cell > 0 or wl.grow else LATE_WINDOW
    total = t_last + 1
    if late and total < late[0] - 1:
        total = late[1]
    else:
        late = None          # the timed steps already reach past the window's start
    host_sig = np.stack([stream.next(m) for _ in range(total)])      # (T, 3, m)

    torch.cuda.set_device(0)
    dev_sig = torch.from_numpy(host_sig).cuda()
    cap = wl.capacity()
    lock_mode, key_mode = lock_modes(gsn, args)
    params = gsn.make_params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha, wl.err_beta,
                             cap["n_max"], cap["e_max"], cap["m_max"], lock_mode, key_mode)
    net = gsn.Network(params, torch.from_numpy(units).cuda())
    tune(gsn, net, args)
    grid = grid_ws = None
    if args.grid_cell > 0:
        lo = cloud.min(axis=0) - np.float32(1e-3)
        hi = cloud.max(axis=0) + np.float32(1e-3)
        dims = [int(np.ceil((hi[a] - lo[a]) / args.grid_cell)) for a in range(3)]
        grid = gsn.make_grid([float(v) for v in lo], args.grid_cell, dims,
                             exact=args.grid_exact)
        grid_ws = net.grid_workspace(grid)

    # the timed loop makes one ctypes call per step: arguments marshalled beforehand
    prep = net.prepare_iterate([dev_sig[t] for t in range(total)]) if grid is None else None

    def step(t):
        if grid is None:
            prep(t)
        else:
            net.find_winners_grid(dev_sig[t], grid, grid_ws)
            net.update(dev_sig[t])
        if wl.grow:
            net.grow(t + 1, wl.insert_every)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    edges_before = net.sizes()[1]

    # inside the timed steps only the scan kernel carries an event pair (its average launch
    # duration is the roofline's denominator); each further event pair costs the stream a
    # few microseconds, so the per-phase times come from the steps after them
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    elapsed, timers, resolved, accepted_timed = timed_steps(torch, gsn, net, step,
                                                            args.warmup, args.steps)
    scan_ms, scan_launches = timers[gsn.GSN_T_FIND_SCAN]
    updates = net.stat(gsn.GSN_STAT_UPDATES)
    rounds = ({"mean": net.stat(gsn.GSN_STAT_ROUNDS) / updates,
               "max": net.stat(gsn.GSN_STAT_ROUNDS_MAX)} if updates else None)
    edges_after = net.sizes()[1]

    print(f"[bench] phase timers over {phase_steps} more steps", file=sys.stderr, flush=True)
    _, ptimers, _, _ = timed_steps(torch, gsn, net, step, t_phase, phase_steps,
                                   scan_only=False)
    phase = {}
    for name, w in (("find_scan", gsn.GSN_T_FIND_SCAN), ("find", gsn.GSN_T_FIND),
                    ("resolve", gsn.GSN_T_RESOLVE), ("adapt", gsn.GSN_T_ADAPT),
                    ("edges", gsn.GSN_T_EDGES), ("update_fused", gsn.GSN_T_UPDATE)):
        phase[name] = ptimers[w][0] if ptimers[w][1] else 0.0

    # one more untimed iteration to report the conflict rate at this state
    index_stats = None
    if grid is not None:
        # the index against the exhaustive search on this state and batch
        gw, gs_, gd1, _ = [t.clone() for t in net.find_winners_grid(dev_sig[t_last], grid,
                                                                    grid_ws)]
        ew, es, ed1, _ = net.find_winners(dev_sig[t_last])
        index_stats = {"cell": args.grid_cell, "dims": list(grid.dims),
                       "winner_differs": float((gw != ew).float().mean().item()),
                       "second_differs": float((gs_ != es).float().mean().item()),
                       "d1_excess_mean": float((gd1 - ed1).double().mean().item()),
                       "exhaustive_find_ms_same_state": None}
        gsn.gsn_timing_select(net.h, (1 << gsn.GSN_T_COUNT) - 1)
        gsn.gsn_timing_enable(net.h, True)
        for _ in range(10):
            net.find_winners(dev_sig[t_last])
        torch.cuda.synchronize()
        gsn.gsn_timing_enable(net.h, False)
        ms_ex, cnt_ex = gsn.gsn_timing_read(net.h, gsn.GSN_T_FIND)
        gsn.gsn_timing_read(net.h, gsn.GSN_T_FIND_SCAN)
        index_stats["exhaustive_find_ms_same_state"] = ms_ex / max(cnt_ex, 1)
        net.resolve_conflicts(m)
        net.adapt(dev_sig[t_last])
        net.update_edges(m)
        acc = net.buf.accepted[:m]
    else:
        acc = net.iterate(dev_sig[t_last])[4]
    conflict_at_end = 1.0 - float(acc.sum().item()) / m
    n_units, n_edges = net.sizes()

    late_rec = None
    if late:
        # continue the stated run (untimed) to the window, then time it
        for t in range(t_last + 1, late[0] - 1):
            step(t)
        torch.cuda.synchronize()
        e0 = net.sizes()[1]
        count = late[1] - late[0] + 1
        print(f"[bench] late window: iterations {late[0]}-{late[1]}", file=sys.stderr,
              flush=True)
        el, lt, res_l, acc_l = timed_steps(torch, gsn, net, step, late[0] - 1, count)
        late_rec = {"iterations": list(late), "ms_per_step": 1e3 * el / count,
                    "evals_per_s": m * n * count / el, "signals_per_s": m * count / el,
                    "accepted_per_s": acc_l / el,
                    "conflict_rate": 1.0 - acc_l / max(res_l, 1),
                    "scan_avg_launch_ms": lt[gsn.GSN_T_FIND_SCAN][0],
                    "edges_at_start": e0, "edges_at_end": net.sizes()[1]}

    loop_rec = None
    if grid is None and not wl.grow and not args.no_loop:
        count = min(args.steps, gsn.GSN_MAX_LOOP)
        loop_rec = time_loop(torch, gsn, units, params, args, host_sig[:args.warmup],
                             host_sig[args.warmup:args.warmup + count])

    ms_per_step = 1e3 * elapsed / args.steps
    traffic = load_traffic(m * n)
    out = {
        "metric": METRIC,
        "value": m * n * args.steps / elapsed,
        "unit": "evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE,
        "data": "synthetic",
        "config": {"workload": wl.name, "n_units": n, "m_signals": m,
                   "cloud_points": wl.n_points, "cloud": "genus-3 tube surface",
                   "iteration": "find+resolve+adapt+update_edges", "parallelism": "single",
                   "find": ("exhaustive" if grid is None else
                            f"hash index, cubes of side {args.grid_cell}" +
                            (", certified exact" if args.grid_exact else "")),
                   "screen": SCREEN if grid is None else None,
                   "timed_iterations": [args.warmup + 1, args.warmup + args.steps],
                   "collision": {"lock": args.lock, "key": args.key}},
        "signals_per_s": m * args.steps / elapsed,
        "accepted_per_s": accepted_timed / elapsed,
        "accepted_fraction": accepted_timed / max(resolved, 1),
        "conflict_rate": 1.0 - accepted_timed / max(resolved, 1),
        "conflict_rate_at_end": conflict_at_end,
        "edges_timed": [edges_before, edges_after],
        "fw_evals_per_s": m * n / (phase["find"] * 1e-3),
        "fw_algorithmic_rate_vs_fp32_peak": FLOPS_PER_EVAL * m * n / (phase["find"] * 1e-3)
                                            / 1e12 / FP32_PEAK_TFLOPS,
        "phase_ms": phase,
        "phase_steps": phase_steps,
        "state_after": {"units": n_units, "edges": n_edges},
        "late_window": late_rec,
        "loop": loop_rec,
        "update_rounds": rounds,
        "index": index_stats,
        "roofline": scan_roofline(m, n, scan_ms, scan_launches, traffic),
        "cpu_baseline": None,
    }
    if grid is not None:
        out["roofline"] = None   # the scan kernel does not run; see "index"
    if args.cpu_budget > 0:
        print(f"[bench] cpu baseline (~{args.cpu_budget:.0f} s)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, units, cloud, args.cpu_budget, lock_mode,
                                           key_mode)
        out["cpu_baseline"]["host"] = host_info()
        if single is not None:
            run = next((r for r in single.get("runs", []) if r["m"] == m), {})
            out["cpu_baseline"]["single_core"] = dict(run, pinned_with=single.get("pinned_with"),
                                                      kind="oracle", threads=1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
