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
  cpu_baseline     the CPU oracle timed on this host's cores on the first iterations of the
                   same workload
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
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


def cpu_baseline(wl, units, cloud, budget_s: float, lock_mode: int = 0, key_mode: int = 0):
    """The oracle on the same initial units and the same seeded signal batches as the GPU
    run, whole iterations until about budget_s seconds have passed (at most 200)."""
    import oracle
    from paper_1503_08294_amd.clouds import SignalStream
    threads = max(1, min(16, os.cpu_count() or 1))
    cap = wl.capacity()
    p = oracle.Params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha, wl.err_beta,
                      cap["n_max"], cap["e_max"], cap["m_max"], lock_mode=lock_mode,
                      key_mode=key_mode)
    o = oracle.Oracle(p, units, threads=threads)
    stream = SignalStream(cloud, wl.signal_seed)
    batches = [stream.next(wl.m) for _ in range(3)]
    dt = 0.0
    done = 0
    while done < 200 and dt < budget_s:
        sig = batches[done] if done < len(batches) else stream.next(wl.m)
        t0 = time.perf_counter()
        o.iterate(sig)
        if wl.grow:
            o.grow(done + 1, wl.insert_every)
        dt += time.perf_counter() - t0
        done += 1
    evals = wl.m * units.shape[1] * done
    return {"value": evals / dt, "unit": "evals/s", "cores": threads, "kind": "oracle",
            "signals_per_s": wl.m * done / dt,
            "sample": f"first {done} whole iterations of {wl.name} (N={units.shape[1]}, "
                      f"m={wl.m}), oracle find-winners on {threads} threads",
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
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "genus3_schedule", "cloud_points": wl.n_points,
                   "initial_units": 2, "n_max": n_max, **SCHEDULE,
                   "collision": {"lock": args.lock, "key": args.key},
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
        threads = max(1, min(16, os.cpu_count() or 1))
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
    args = ap.parse_args()

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

    import numpy as np
    import torch

    from paper_1503_08294_amd import gsn
    from paper_1503_08294_amd.clouds import WORKLOADS, SignalStream

    wl = WORKLOADS[args.workload]
    print(f"[bench] generating {wl.name}: {wl.n_points} cloud points, N={wl.n_units}, "
          f"m={wl.m}", file=sys.stderr, flush=True)
    cloud = wl.make_cloud()
    units = wl.make_units(cloud)
    stream = SignalStream(cloud, wl.signal_seed)
    # the timed steps, then a few more with every phase timer on, then one for the
    # conflict rate
    phase_steps = min(args.steps, 20)
    total = args.warmup + args.steps + phase_steps + 1
    host_sig = np.stack([stream.next(wl.m) for _ in range(total)])      # (T, 3, m)
    n, m = units.shape[1], wl.m

    torch.cuda.set_device(0)
    dev_sig = torch.from_numpy(host_sig).cuda()
    cap = wl.capacity()
    lock_mode = {"set": gsn.GSN_LOCK_SET, "winner": gsn.GSN_LOCK_WINNER,
                 "greedy": gsn.GSN_LOCK_SET_GREEDY}[args.lock]
    key_mode = gsn.GSN_KEY_INDEX if args.key == "index" else gsn.GSN_KEY_DIST_INDEX
    params = gsn.make_params(wl.eps_b, wl.eps_n, wl.max_age, wl.err_alpha, wl.err_beta,
                             cap["n_max"], cap["e_max"], cap["m_max"], lock_mode, key_mode)
    net = gsn.Network(params, torch.from_numpy(units).cuda())
    grid = grid_ws = None
    if args.grid_cell > 0:
        lo = cloud.min(axis=0) - np.float32(1e-3)
        hi = cloud.max(axis=0) + np.float32(1e-3)
        dims = [int(np.ceil((hi[a] - lo[a]) / args.grid_cell)) for a in range(3)]
        grid = gsn.make_grid([float(v) for v in lo], args.grid_cell, dims,
                             exact=args.grid_exact)
        grid_ws = net.grid_workspace(grid)

    def step(t):
        if grid is None:
            net.iterate(dev_sig[t])
        else:
            net.find_winners_grid(dev_sig[t], grid, grid_ws)
            net.resolve_conflicts(m)
            net.adapt(dev_sig[t])
            net.update_edges(m)
        if wl.grow:
            net.grow(t + 1, wl.insert_every)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    for w in range(gsn.GSN_T_COUNT):
        gsn.gsn_timing_read(net.h, w)
    # inside the timed steps only the scan kernel carries an event pair (its average launch
    # duration is the roofline's denominator); each further event pair costs the stream a
    # few microseconds, so the per-phase times come from the steps after them
    gsn.gsn_timing_select(net.h, 1 << gsn.GSN_T_FIND_SCAN)
    gsn.gsn_timing_enable(net.h, True)

    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    net.stat(gsn.GSN_STAT_CLEAR)
    t0 = time.perf_counter()
    for t in range(args.warmup, args.warmup + args.steps):
        step(t)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gsn.gsn_timing_enable(net.h, False)
    scan_ms_sum, scan_launches = gsn.gsn_timing_read(net.h, gsn.GSN_T_FIND_SCAN)
    scan_ms = scan_ms_sum / max(scan_launches, 1)
    resolved = net.stat(gsn.GSN_STAT_RESOLVED)
    accepted_timed = net.stat(gsn.GSN_STAT_ACCEPTED)
    updates = net.stat(gsn.GSN_STAT_UPDATES)
    rounds = ({"mean": net.stat(gsn.GSN_STAT_ROUNDS) / updates,
               "max": net.stat(gsn.GSN_STAT_ROUNDS_MAX)} if updates else None)
    if net.check() != 0:
        raise SystemExit(f"device status {net.check()} after the timed steps")

    print(f"[bench] phase timers over {phase_steps} more steps", file=sys.stderr, flush=True)
    gsn.gsn_timing_select(net.h, (1 << gsn.GSN_T_COUNT) - 1)
    gsn.gsn_timing_enable(net.h, True)
    t_phase = args.warmup + args.steps
    for t in range(t_phase, t_phase + phase_steps):
        step(t)
    torch.cuda.synchronize()
    gsn.gsn_timing_enable(net.h, False)
    phase = {}
    for name, w in (("find_scan", gsn.GSN_T_FIND_SCAN), ("find", gsn.GSN_T_FIND),
                    ("resolve", gsn.GSN_T_RESOLVE), ("adapt", gsn.GSN_T_ADAPT),
                    ("edges", gsn.GSN_T_EDGES), ("update_fused", gsn.GSN_T_UPDATE)):
        ms, cnt = gsn.gsn_timing_read(net.h, w)
        phase[name] = ms / max(cnt, 1)
    if net.check() != 0:
        raise SystemExit(f"device status {net.check()} after the phase steps")

    # one more untimed iteration to report the conflict rate at this state
    t_last = t_phase + phase_steps
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
    conflict_rate = 1.0 - float(acc.sum().item()) / m
    n_units, n_edges = net.sizes()

    ms_per_step = 1e3 * elapsed / args.steps
    scan_s = max(scan_ms, 1e-9) * 1e-3
    achieved = FLOPS_PER_EVAL * m * n / scan_s / 1e12
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
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "n_units": n, "m_signals": m,
                   "cloud_points": wl.n_points, "cloud": "genus-3 tube surface",
                   "iteration": "find+resolve+adapt+update_edges", "parallelism": "single",
                   "find": ("exhaustive" if grid is None else
                            f"hash index, cubes of side {args.grid_cell}" +
                            (", certified exact" if args.grid_exact else "")),
                   "collision": {"lock": args.lock, "key": args.key}},
        "signals_per_s": m * args.steps / elapsed,
        "accepted_per_s": accepted_timed / elapsed,
        "accepted_fraction": accepted_timed / max(resolved, 1),
        "fw_evals_per_s": m * n / (phase["find"] * 1e-3),
        "fw_frac_fp32_peak": FLOPS_PER_EVAL * m * n / (phase["find"] * 1e-3) / 1e12
                             / FP32_PEAK_TFLOPS,
        "phase_ms": phase,
        "phase_steps": phase_steps,
        "conflict_rate": conflict_rate,
        "state_after": {"units": n_units, "edges": n_edges},
        "update_rounds": rounds,
        "index": index_stats,
        "roofline": {"bound": "mfma", "kernel": SCAN_KERNEL, "dtype": "f16",
                     "achieved": achieved, "peak": F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / F16_PEAK_TFLOPS, "traffic": traffic,
                     "flops_per_launch": FLOPS_PER_EVAL * m * n,
                     "avg_launch_ms": scan_ms,
                     "launches_timed": scan_launches,
                     "executed_mfma_tflops": EXECUTED_FLOPS_PER_PAIR * m * n / scan_s / 1e12,
                     "executed_mfma_frac": EXECUTED_FLOPS_PER_PAIR * m * n / scan_s / 1e12
                                           / F16_PEAK_TFLOPS,
                     "achieved_vs_fp32_peak": achieved / FP32_PEAK_TFLOPS},
        "cpu_baseline": None,
    }
    if grid is not None:
        out["roofline"] = None   # the scan kernel does not run; see "index"
    if args.cpu_budget > 0:
        print(f"[bench] cpu baseline (~{args.cpu_budget:.0f} s)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, units, cloud, args.cpu_budget, lock_mode,
                                           key_mode)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
