"""Benchmark of the C3 hot path on one MI355X.

One step = c3_check: signature, exact vote on the signatures and
localization over R replica copies resident in HBM, in one call (the line
also reports the same outputs from the three separate calls c3_signature +
c3_consensus + c3_localize).  Default workload: R = 8
replicas of 1,073,807,360 bf16 parameters in layer-shaped tensors (16 layers
of a 2048/8192 transformer), chunk 1 MiB, with seeded faults on one replica.

Prints ONE JSON line on stdout (progress goes to stderr):
  value      replica GB/s fingerprinted + localized (R * S bytes / step time)
  roofline   the streaming signature kernel against MI355X HBM peak, timed
             with HIP events the library records around that kernel, and
             the read probe of the same access pattern as "achievable"
  parity     the oracle's records, votes and lists of the CPU sample
             against the GPU's
  cpu_baseline  the CPU oracle (single thread) on a bounded sample

Flags: --gpus N (only 1: the path runs on one GPU), --steps K, --warmup W
(default: untimed steps until at least 0.25 s and 10 steps have run, which
takes the GPU past the clock and power transient of its first launches;
the JSON reports the count), 
--config 1..7 (5: timing consensus of 32,768 ranks; 6: optimizer-boundary
check on 8 replicas of a 134M-parameter AdamW state; 7: out-of-band hang
localization, CPU only), --no-cpu-baseline,
--copy-calibration (adds a 1 GiB device copy used to scale rocprofv3
FETCH_SIZE / WRITE_SIZE counters).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "replica GB/s fingerprinted+localized; % of MI355X HBM peak"
# sources that define the streaming signature kernel: counter-based traffic
# figures are reported only while these are unchanged
SIG_SOURCES = ["paper_2608_11034_amd/csrc/c3_signature.hip", "paper_2608_11034_amd/csrc/c3_device.h",
               "paper_2608_11034_amd/csrc/c3_sigplan.h"]
# the same for the single-pass timing kernel
TIMING_SOURCES = ["paper_2608_11034_amd/csrc/c3_timing.hip", "paper_2608_11034_amd/csrc/c3_vote_row.h",
                  "paper_2608_11034_amd/csrc/c3_device.h"]


def traffic_file(workload: str, kernel: str = "signature_kernel") -> str:
    return os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(sources=SIG_SOURCES) -> str:
    h = hashlib.sha256()
    for p in sources:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, kernel: str = "signature_kernel", sources=SIG_SOURCES):
    """HBM bytes per launch from committed counter runs, if the kernel is unchanged."""
    try:
        with open(traffic_file(workload, kernel)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_hash") != kernel_source_hash(sources):
        return None
    return t.get("hbm_bytes_per_launch")


def copy_calibration(torch, dev):
    """Three 1 GiB device-to-device copies, whose counter readings scale
    FETCH_SIZE and WRITE_SIZE to bytes in a counter run."""
    log("[bench] copy calibration: 1 GiB device copy x3")
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()


def host_cpu():
    """Host CPU model (the kernel's model string, and lscpu's when it says
    more), the CPU family/model/stepping numbers, and the cores this process
    may run on."""
    import subprocess
    info = {}
    try:
        for ln in open("/proc/cpuinfo"):
            k, _, v = ln.partition(":")
            k = k.strip()
            if k in ("model name", "cpu family", "model", "stepping") and k not in info:
                info[k] = v.strip()
            if not ln.strip() and info:
                break
    except OSError:
        pass
    model = info.get("model name", "unknown")
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in out.splitlines():
            if ln.startswith("Model name:"):
                lm = ln.split(":", 1)[1].strip()
                if len(lm) > len(model):
                    model = lm
    except (OSError, subprocess.SubprocessError):
        pass
    return {"model": model, "family_model_stepping": [info.get("cpu family"), info.get("model"),
                                                      info.get("stepping")],
            "cores_available": len(os.sched_getaffinity(0))}


def records_match(g, ref):
    """GPU records [R, C] against the oracle's: bit-exact signature, counts,
    ids and absmax; fp64 sums within |d| <= max(1e-6 |ref|, 1e-12
    sqrt(n_finite sumsq)), sums of squares within 1e-6 relative.  Returns
    the number of records that differ."""
    import numpy as np
    exact = ((g["sig"] == ref["sig"]) & (g["n_elems"] == ref["n_elems"]) &
             (g["nan_count"] == ref["nan"]) & (g["inf_count"] == ref["inf"]) &
             (g["tensor"] == ref["tensor"]) & (g["chunk_in_tensor"] == ref["chunk"]) &
             (g["absmax"] == ref["absmax"]))
    n_fin = ref["n_elems"].astype(np.float64) - ref["nan"] - ref["inf"]
    floor = 1e-12 * np.sqrt(np.maximum(n_fin, 0) * np.maximum(ref["sumsq"], 0))
    s_ok = np.abs(g["sum"] - ref["sum"]) <= np.maximum(1e-6 * np.abs(ref["sum"]), floor)
    q_ok = np.abs(g["sumsq"] - ref["sumsq"]) <= 1e-6 * np.abs(ref["sumsq"])
    return int((~(exact & s_ok & q_ok)).sum())


def cpu_baseline(w, budget_s: float, gpu=None):
    """Oracle over the first chunks of every replica: bounded sample, one
    thread pinned to one host core.  With `gpu` (records [R, C] and the
    per-chunk status, bitmap and majority of the timed steps, as numpy), the
    oracle's records, votes and lists of the sample are compared with the
    GPU's for the same chunks."""
    import numpy as np
    import oracle
    import workloads

    # sample: whole leading tensors of each replica, up to ~budget_s of oracle work
    per_byte_s = 1.0 / 0.9e9          # oracle bf16 speed on one host core, rough
    target = int(budget_s / per_byte_s / w.R)
    metas, nbytes = [], 0
    for d, shape in w.metas:
        nb = int(np.prod(shape)) * workloads.ELEM_SIZE[d]
        if metas and nbytes + nb > target:
            break
        metas.append((d, shape))
        nbytes += nb
    T = len(metas)
    t0 = time.perf_counter()
    reps = [[workloads.host_bytes(w.replicas[r][t]) for t in range(T)] for r in range(w.R)]
    d2h = time.perf_counter() - t0
    affinity = os.sched_getaffinity(0)
    core = min(affinity)
    os.sched_setaffinity(0, {core})
    try:
        t0 = time.perf_counter()
        rec = oracle.signature(reps, metas, w.chunk_bytes)
        st, bm, mj = oracle.vote_exact(rec["sig"])
        loc = oracle.localize(st, bm, mj, w.R)
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, affinity)
    sample_bytes = nbytes * w.R
    Cs = rec["sig"].shape[1]
    out = {"value": sample_bytes / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
           "sample": f"first {T} tensors of all {w.R} replicas ({sample_bytes} bytes, "
                     f"{Cs} chunks), signature+vote+localize, {dt:.1f} s on host core {core}",
           "seconds": dt, "d2h_seconds": round(d2h, 3),
           "d2h_GBps": round(sample_bytes / d2h / 1e9, 2) if d2h > 0 else None,
           "host": host_cpu()}
    if gpu is not None:
        bad = records_match(gpu["records"][:, :Cs], rec)
        votes_ok = (np.array_equal(gpu["status"][:Cs], st) and
                    np.array_equal(gpu["bitmap"][:Cs], bm) and np.array_equal(gpu["maj"][:Cs], mj))
        o = gpu["outliers"]
        sel = o["chunk"] < Cs
        lists_ok = (o["chunk"][sel].tolist() == loc["unit"].tolist() and
                    o["replica"][sel].tolist() == loc["replica"].tolist() and
                    o["majority_replica"][sel].tolist() == loc["majority"].tolist())
        out["parity"] = {"ok": bad == 0 and votes_ok and lists_ok,
                         "records_compared": int(w.R * Cs), "records_differing": bad,
                         "chunks_compared": int(Cs), "votes_equal": bool(votes_ok),
                         "outlier_list_equal": bool(lists_ok)}
    return out


def timing_cpu_baseline(w, gpu):
    """The oracle's timing consensus (exact vote on the fingerprints,
    statistical vote on the step times, window confirmation) over the whole
    workload, one thread pinned to one host core; its per-unit results and
    verdicts are compared with the GPU's (`gpu`: numpy copies of the last
    call's outputs)."""
    import numpy as np
    import oracle

    T, G, R = w.T, w.G, w.R
    t0 = time.perf_counter()
    fp = w.fingerprints.cpu().numpy().reshape(T * G, R).view(np.uint64)
    tau = w.times.cpu().numpy().reshape(T * G, R)
    d2h = time.perf_counter() - t0
    affinity = os.sched_getaffinity(0)
    core = min(affinity)
    os.sched_setaffinity(0, {core})
    try:
        t0 = time.perf_counter()
        ost, obm, omj = oracle.vote_exact(fp, replica_axis=1)
        sst, sbm, smj = oracle.vote_statistical(tau, oracle.KAPPA_DEFAULT, replica_axis=1)
        ref = oracle.confirm(obm.reshape(T, G), sbm.reshape(T, G), R, 16)
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, affinity)
    nbytes = fp.nbytes + tau.nbytes
    units_ok = (np.array_equal(gpu["fp"][0], ost) and np.array_equal(gpu["fp"][1], obm) and
                np.array_equal(gpu["fp"][2], omj) and np.array_equal(gpu["t"][0], sst) and
                np.array_equal(gpu["t"][1], sbm) and np.array_equal(gpu["t"][2], smj))
    v = gpu["verdicts"]
    fields = (("flags", "flags"), ("first_divergent_iter", "first_div"),
              ("divergent_count", "div_count"), ("slow_count", "slow_count"),
              ("max_window_slow", "max_window"), ("first_straggler_window", "first_window"))
    bad = 0
    for k, rk in fields:
        bad = max(bad, int((np.asarray(v[k]) != np.asarray(ref[rk])).sum()))
    return {"value": nbytes / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"the whole workload: {R * G} ranks x {T} iterations ({nbytes} bytes of "
                      f"records), exact vote, statistical vote and window confirmation, "
                      f"{dt:.1f} s on host core {core}",
            "seconds": dt, "d2h_seconds": round(d2h, 3), "host": host_cpu(),
            "parity": {"ok": units_ok and bad == 0, "units_compared": int(T * G),
                       "per_unit_results_equal": bool(units_ok),
                       "ranks_compared": int(R * G), "verdict_fields_differing": bad}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5, 6, 7, 8])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--grid", type=int, default=0)
    ap.add_argument("--tile", type=int, default=0)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this hot path runs on one GPU (R replicas resident in one GPU's HBM); "
              "--gpus N > 1 is not supported", file=sys.stderr)
        sys.exit(2)

    if args.config == 7:
        return bench_hang(args)

    import torch
    import workloads
    from paper_2608_11034_amd import c3

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.config == 5:
        return bench_timing(args, torch, workloads, c3, dev)
    if args.config == 6:
        return bench_optimizer(args, torch, workloads, c3, dev)
    if args.config == 8:
        return bench_wide(args, torch, workloads, c3, dev)
    log(f"[bench] generating config {args.config}")
    w = workloads.make(args.config, device=dev, scale="full")
    torch.cuda.synchronize()
    total = w.total_bytes
    plan = c3.SignaturePlan(w.replicas, w.chunk_bytes, args.tile)
    C = plan.C
    outs = plan.new_check_outputs()
    rec, status, bitmap, maj, outl, und, cnt = outs
    cws = torch.empty(plan.check_workspace_size(), dtype=torch.uint8, device=dev)
    ws = plan.new_workspace()
    lws = torch.empty(c3.localize_workspace_size(C), dtype=torch.uint8, device=dev)

    def step(staged=False):
        # c3_check: signature, exact vote and localization in one call
        plan.run_check(outs, cws, grid_blocks=args.grid, plan_staged=staged)

    def step_three_calls(staged=False):
        # the same outputs from c3_signature + c3_consensus + c3_localize
        plan.run(rec, ws, grid_blocks=args.grid, plan_staged=staged)
        c3.consensus(rec, c3.EXACT, out=(status, bitmap, maj))
        c3.localize(status, bitmap, maj, rec, out=(outl, und, cnt), workspace=lws)

    def timed(staged, fn=step):
        """Mean ms per step over K back-to-back steps between one pair of
        events, and the wall time."""
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record()
        for _ in range(args.steps):
            fn(staged)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps, time.perf_counter() - t0

    def per_step(fn=step):
        """Median and minimum ms of single steps: K more steps with an event
        between consecutive ones.  Each event record idles the GPU a few
        microseconds, so these include one event; the mean above has none."""
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        torch.cuda.synchronize()
        evs[0].record()
        for i in range(args.steps):
            fn(False)
            evs[i + 1].record()
        torch.cuda.synchronize()
        per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
        return per[len(per) // 2], per[0]

    args.warmup = warm_up(torch, step, args.warmup)
    log(f"[bench] warmup {args.warmup} steps")
    counts = cnt.cpu().tolist()
    log(f"[bench] outliers={counts[0]} undecided={counts[1]} attributed_chunks={counts[2]}")

    log(f"[bench] timing {args.steps} steps")
    ms_per_step, wall = timed(staged=False)
    step_med, step_min = per_step()
    ms_back_to_back = ms_per_step
    cold = total < COLD_BELOW_BYTES
    if cold:
        # a working set the caches could hold: each step from HBM, timed alone
        ms_per_step, step_med, step_min = cold_calls(torch, lambda: step(False), args.steps, dev)
    value = total / (ms_per_step * 1e-3) / 1e9
    # the same steps when the plan staged by the previous call is reused
    ms_staged, _ = timed(staged=True)
    # the three separate calls, for comparison (same outputs)
    for _ in range(5):
        step_three_calls()
    ms_three, _ = timed(staged=False, fn=step_three_calls)
    med_three, _ = per_step(fn=step_three_calls)
    step()                       # leave c3_check's outputs for the parity check

    # dominant kernel: the streaming signature kernel, events recorded by the
    # library on the launch stream immediately around it
    log("[bench] timing the signature kernel alone")
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in evs:                       # materialize the HIP events
        a.record()
        b.record()
    torch.cuda.synchronize()
    # untimed steps enqueued just before the timed ones, so that the GPU is
    # not idle (and its clock not ramping) when the first timed one starts
    for _ in range(5):
        step(False)
    for a, b in evs:
        plan.run_check(outs, cws, ev_begin=a, ev_end=b, grid_blocks=args.grid)
    torch.cuda.synchronize()
    k_all = sorted(a.elapsed_time(b) for a, b in evs)
    k_ms = sum(k_all) / len(k_all)
    k_med, k_min = k_all[len(k_all) // 2], k_all[0]
    achieved = total / (k_ms * 1e-3) / 1e9

    # the read ceiling of the same access pattern: the library's read probe
    # (256 KiB tiles, 16 loads in flight per lane, nothing computed) over a
    # buffer of the same size, capped at 32 GiB, timed the same way
    log("[bench] timing the read probe")
    probe_bytes = min(total, 32 << 30) // 1024 * 1024
    probe_buf = torch.empty(probe_bytes, dtype=torch.uint8, device=dev)
    probe_cs = torch.empty(-(-probe_bytes // (256 << 10)), dtype=torch.int64, device=dev)
    for _ in range(3):
        c3.read_probe(probe_buf, 0, checksum=probe_cs)
    pevs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(args.steps)]
    for a, b in pevs:
        a.record()
        b.record()
    torch.cuda.synchronize()
    for _ in range(3):
        c3.read_probe(probe_buf, 0, checksum=probe_cs)
    for a, b in pevs:
        c3.read_probe(probe_buf, 0, checksum=probe_cs, ev_begin=a, ev_end=b)
    torch.cuda.synchronize()
    p_all = sorted(a.elapsed_time(b) for a, b in pevs)
    p_ms = sum(p_all) / len(p_all)
    achievable = probe_bytes / (p_ms * 1e-3) / 1e9
    del probe_buf, probe_cs

    if args.copy_calibration:
        copy_calibration(torch, dev)

    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline on a bounded sample")
        # the timed steps' own outputs (every step rewrites the same buffers)
        import numpy as np
        gpu = {"records": c3.records_numpy(rec), "status": status.cpu().numpy(),
               "bitmap": bitmap.cpu().numpy().view(np.uint64), "maj": maj.cpu().numpy(),
               "outliers": c3.outliers_numpy(outl, cnt)}
        cpu = cpu_baseline(w, args.cpu_budget, gpu)
        log(f"[bench] oracle {cpu['value']:.3f} GB/s over {cpu['seconds']:.1f} s; "
            f"parity {cpu['parity']}")
        cpu.pop("seconds")
        parity = cpu.pop("parity")

    traffic = measured_traffic(w.name)
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_median": round(step_med, 4),
        "ms_per_step_min": round(step_min, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64+f64",
        "data": "synthetic",
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "parity": parity,
        "config": {"workload": w.name, "R": w.R, "tensors_per_replica": len(w.metas),
                   "bytes_per_replica": w.bytes_per_replica, "replica_bytes_total": total,
                   "chunk_bytes": w.chunk_bytes, "chunks": C,
                   "input_dtype": "f32" if args.config in (1, 4) else "bf16",
                   "outliers": counts[0], "undecided": counts[1]},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "kernel": "signature_kernel",
                     "kernel_ms": round(k_ms, 4), "kernel_ms_median": round(k_med, 4),
                     "kernel_ms_min": round(k_min, 4), "algorithmic_bytes_per_launch": total,
                     "achievable": {"GBps": round(achievable, 2), "kernel": "read_probe_kernel",
                                    "bytes_per_launch": probe_bytes, "ms": round(p_ms, 4),
                                    "ms_median": round(p_all[len(p_all) // 2], 4),
                                    "ms_min": round(p_all[0], 4),
                                    "frac_of_peak": round(achievable / HBM_PEAK_GBS, 4)},
                     "frac_of_achievable": round(achieved / achievable, 4)},
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
        "timing": ("per call after a 1 GiB cache-evicting read" if cold
                   else "back-to-back calls between one pair of events"),
        "ms_per_step_back_to_back": round(ms_back_to_back, 4),
        "ms_per_step_plan_reused": round(ms_staged, 4),
        "value_plan_reused": round(total / (ms_staged * 1e-3) / 1e9, 2),
        "step": "c3_check (signature + exact vote + localize in one call)",
        "ms_per_step_three_calls": round(ms_three, 4),
        "ms_per_step_three_calls_median": round(med_three, 4),
        "value_three_calls": round(total / (ms_three * 1e-3) / 1e9, 2),
    }
    print(json.dumps(out), flush=True)


# Working sets below this size are timed call by call with the caches
# evicted first: reading 1 GiB before each call clears the 256 MB MALL and
# the L2s, so the call reads its inputs from HBM.  The eviction is a plain
# (cache-allocating) read, a torch reduction, rather than a write, so that
# no dirty lines are left for the timed call to write back.
COLD_BELOW_BYTES = 1 << 30
_scratch = {}


def cold_calls(torch, fn, steps, dev):
    """Per-call ms of `steps` calls, each after reading a 1 GiB buffer (not
    timed) and between its own pair of events: (mean, median, min)."""
    if dev not in _scratch:
        _scratch[dev] = torch.full((1 << 28,), 7, dtype=torch.int32, device=dev)
    junk = _scratch[dev]
    ts = []
    for i in range(steps):
        junk.sum()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b))
    ts.sort()
    return sum(ts) / len(ts), ts[len(ts) // 2], ts[0]


def warm_up(torch, step, warmup, min_s=0.25, min_steps=10):
    """Runs `warmup` untimed steps, or with None steps until min_s seconds and
    min_steps steps have passed; returns the count."""
    if warmup is not None:
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        return warmup
    n, t0 = 0, time.perf_counter()
    while n < min_steps or time.perf_counter() - t0 < min_s:
        step()
        torch.cuda.synchronize()
        n += 1
    return n


def _kernel_ms(torch, fn, reps):
    """Mean duration of a call that enqueues one kernel, by events around it."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    torch.cuda.synchronize()
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in evs) / reps


def bench_timing(args, torch, workloads, c3, dev):
    """Progress/timing consensus: exact vote on fingerprints, statistical vote
    on step times and temporal confirmation (c3_timing_consensus, one kernel
    on this shape), one step per pass over all records; per-unit results are
    written."""
    log("[bench] generating config 5")
    w = workloads.make(5, device=dev, scale="full")
    T, G, R = w.T, w.G, w.R
    U = T * G
    total = w.total_bytes
    fp_out = (torch.empty(U, dtype=torch.uint8, device=dev), torch.empty(U, dtype=torch.int64, device=dev),
              torch.empty(U, dtype=torch.int32, device=dev))
    t_out = (torch.empty(U, dtype=torch.uint8, device=dev), torch.empty(U, dtype=torch.int64, device=dev),
             torch.empty(U, dtype=torch.int32, device=dev))
    ver = torch.empty((R * G, 24), dtype=torch.uint8, device=dev)
    ws = torch.empty(c3.timing_consensus_workspace_size(R, G, T, 16), dtype=torch.uint8, device=dev)

    def step():
        c3.timing_consensus(w.fingerprints, w.times, window=16, out=(ver, fp_out, t_out),
                            workspace=ws)

    def step_verdicts_only():
        c3.timing_consensus(w.fingerprints, w.times, window=16, out=(ver, None, None),
                            workspace=ws)

    args.warmup = warm_up(torch, step, args.warmup)
    v = c3.verdicts_numpy(ver)
    strag = int(((v["flags"] & c3.RANK_STRAGGLER) != 0).sum())
    proto = int(((v["flags"] & c3.RANK_PROTOCOL) != 0).sum())
    log(f"[bench] stragglers={strag} protocol_outliers={proto}")

    def timed(fn):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    t0 = time.perf_counter()
    ms_b2b = timed(step)
    ms_verdicts_b2b = timed(step_verdicts_only)
    # the 403 MB of records are 1.6 times the 256 MB MALL: each call is timed
    # alone after a 1 GiB read that evicts the caches (back-to-back calls
    # keep part of the records and results cached)
    ms, ms_med, ms_min = cold_calls(torch, step, args.steps, dev)
    wall = time.perf_counter() - t0
    ms_verdicts, ms_verdicts_med, _ = cold_calls(torch, step_verdicts_only, args.steps, dev)
    # the three separate calls, for comparison
    sep_f = (torch.empty_like(fp_out[0]), torch.empty_like(fp_out[1]), torch.empty_like(fp_out[2]))
    sep_t = (torch.empty_like(t_out[0]), torch.empty_like(t_out[1]), torch.empty_like(t_out[2]))
    cws = torch.empty(max(c3.confirm_workspace_size(R, G, T), 256), dtype=torch.uint8, device=dev)

    def separate():
        c3.consensus(w.fingerprints, c3.EXACT, out=sep_f)
        c3.consensus(w.times, c3.STATISTICAL, out=sep_t)
        c3.confirm(sep_f[1].view(T, G), sep_t[1].view(T, G), R, 16, out=ver, workspace=cws)
    ms_sep_b2b = timed(separate)
    ms_sep, _, _ = cold_calls(torch, separate, args.steps, dev)
    if args.copy_calibration:
        copy_calibration(torch, dev)
    cpu = parity = None
    if not args.no_cpu_baseline:
        import numpy as np
        log("[bench] CPU oracle baseline over the whole workload")
        step()
        torch.cuda.synchronize()
        gpu = {"fp": (fp_out[0].cpu().numpy(), fp_out[1].cpu().numpy().view(np.uint64),
                      fp_out[2].cpu().numpy()),
               "t": (t_out[0].cpu().numpy(), t_out[1].cpu().numpy().view(np.uint64),
                     t_out[2].cpu().numpy()),
               "verdicts": c3.verdicts_numpy(ver)}
        cpu = timing_cpu_baseline(w, gpu)
        log(f"[bench] oracle {cpu['value']:.3f} GB/s over {cpu['seconds']:.1f} s; "
            f"parity {cpu['parity']}")
        parity = cpu.pop("parity")
    # the single pass reads the records once and writes the per-unit results
    # (status 1 + bitmap 8 + majority 4 bytes per unit and kind) and the
    # verdicts; the outlier masks stay in LDS
    pass_bytes = U * R * (8 + 4) + 2 * U * 13 + R * G * 24
    # without per-unit results: the records and the verdicts
    vo_bytes = U * R * (8 + 4) + R * G * 24
    out = {
        "metric": "timing+fingerprint records GB/s voted+confirmed",
        "value": round(total / (ms * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_step_median": round(ms_med, 4),
        "ms_per_step_min": round(ms_min, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64+f64",
        "data": "synthetic",
        "timing": "per call after a 1 GiB cache-evicting read",
        "config": {"workload": w.name, "ranks": R * G, "group": R, "iterations": T,
                   "record_bytes_total": total, "stragglers_found": strag,
                   "protocol_outliers_found": proto},
        "roofline": {"bound": "hbm", "achieved": round(pass_bytes / (ms * 1e-3) / 1e9, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(pass_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(w.name, "timing_pass_kernel", TIMING_SOURCES),
                     "kernel": "timing_pass_kernel (per-unit results)",
                     "kernel_ms": round(ms, 4), "algorithmic_bytes_per_launch": pass_bytes},
        "ms_per_step_back_to_back": round(ms_b2b, 4),
        "ms_per_step_verdicts_only": round(ms_verdicts, 4),
        "ms_per_step_verdicts_only_median": round(ms_verdicts_med, 4),
        "ms_per_step_verdicts_only_back_to_back": round(ms_verdicts_b2b, 4),
        "roofline_verdicts_only": {"bound": "hbm", "achieved": round(vo_bytes / (ms_verdicts * 1e-3) / 1e9, 2),
                                   "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                   "frac": round(vo_bytes / (ms_verdicts * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                   "kernel": "timing_pass_kernel", "algorithmic_bytes_per_launch": vo_bytes},
        "ms_per_step_separate_calls": round(ms_sep, 4),
        "ms_per_step_separate_calls_back_to_back": round(ms_sep_b2b, 4),
        "cpu_baseline": cpu,
        "parity": parity,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(out), flush=True)


def bench_wide(args, torch, workloads, c3, dev):
    """Votes over wide peer groups (gathered tables of 33 to 256 peers): per
    group size R, c3_consensus on 262,144 units, STATISTICAL on fp32 and fp64
    step times and EXACT on 64-bit fingerprints; mean ms per call between
    HIP events over `steps` calls.  Unless --no-cpu-baseline, the oracle
    votes the first `S` units of every table, one thread pinned to one host
    core, and its status, bitmap words and majority index are compared with
    the GPU's."""
    import numpy as np
    U = 1 << 18
    S = 1 << 14
    rows = []
    oracle_s = {}
    parity = {"ok": True, "units_compared_per_table": S, "tables": 0, "tables_differing": []}
    for R in (17, 33, 64, 65, 128, 129, 192, 256):
        tau32, fp = workloads.wide_votes(R, U, device=dev)
        tau64 = tau32.double()
        line = {"R": R}
        for name, ev, mode in (("stat_f32", tau32, c3.STATISTICAL), ("stat_f64", tau64, c3.STATISTICAL),
                               ("exact_u64", fp, c3.EXACT)):
            out = c3.consensus(ev, mode)
            warm_up(torch, lambda: c3.consensus(ev, mode, out=out), args.warmup or 5)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(args.steps):
                c3.consensus(ev, mode, out=out)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            line[name + "_ms"] = round(ms, 4)
            line[name + "_GBps"] = round(ev.numel() * ev.element_size() / (ms * 1e-3) / 1e9, 1)
            if name == "stat_f32":
                st = out[0].cpu()
                line["attributed_units"] = int((st == c3.ATTRIBUTED).sum())
            if not args.no_cpu_baseline:
                oracle_s[(R, name)] = wide_oracle_sample(ev, mode, out, R, S, c3, np, parity, name)
        rows.append(line)
        log(f"[bench] wide R={R}: {line}")
        del tau32, tau64, fp
    out = {"metric": "wide-group consensus ms per 262,144 units", "value": rows[-1]["stat_f32_ms"],
           "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup or 5,
           "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f32/f64/u64",
           "data": "synthetic",
           "config": {"workload": "wide_groups_units262144", "units": U, "layout": "unit-major [U][R]"},
           "per_R": rows, "cpu_baseline": None, "parity": None}
    if oracle_s:
        # the oracle at the headline's shape (R = 256, fp32 times), scaled from
        # its S-unit sample to the 262,144 units the value is quoted on
        t = oracle_s[(256, "stat_f32")]
        out["cpu_baseline"] = {
            "value": round(t * (U / S) * 1e3, 1), "unit": "ms", "cores": 1, "kind": "oracle",
            "sample": f"the first {S} of {U} units of every table, each table voted once; "
                      f"the value scales R = 256 fp32 ({t:.2f} s) to {U} units; "
                      f"{sum(oracle_s.values()):.1f} s in all",
            "per_table_seconds": {f"R{r}_{k}": round(v, 4) for (r, k), v in oracle_s.items()},
            "host": host_cpu()}
        out["parity"] = parity
    print(json.dumps(out), flush=True)


def wide_oracle_sample(ev, mode, out, R, S, c3, np, parity, name):
    """Oracle vote over the first S units of one wide table on one pinned
    host core; records in `parity` whether the GPU's outputs agree.  Returns
    the oracle's seconds."""
    import oracle

    host = ev[:S].cpu().numpy()
    if host.dtype == np.int64:
        host = host.view(np.uint64)
    affinity = os.sched_getaffinity(0)
    os.sched_setaffinity(0, {min(affinity)})
    try:
        t0 = time.perf_counter()
        if mode == c3.EXACT:
            ost, obm, omj = oracle.vote_exact(host, replica_axis=1)
        else:
            ost, obm, omj = oracle.vote_statistical(host, oracle.KAPPA_DEFAULT, replica_axis=1)
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, affinity)
    words = c3.bitmap_words(R)
    g_bm = out[1].cpu().numpy().view(np.uint64).reshape(-1, words)[:S]
    same = (np.array_equal(out[0][:S].cpu().numpy(), ost) and
            np.array_equal(g_bm, obm.reshape(S, words)) and
            np.array_equal(out[2][:S].cpu().numpy(), omj))
    parity["tables"] += 1
    if not same:
        parity["ok"] = False
        parity["tables_differing"].append(f"R{R}_{name}")
    return dt


def bench_optimizer(args, torch, workloads, c3, dev):
    """Optimizer-boundary check: one step = one scheduled check on the next
    rotating 64K-element slice (AdamW replay on R replicas, signatures of the
    4 input and 3 output slices per replica, exact vote, localize)."""
    log("[bench] generating config 6")
    w = workloads.make(6, device=dev, scale="full")
    torch.cuda.synchronize()
    chk = c3.OptimizerBoundaryCheck(*w.state, slice_elems=w.slice_elems, tile_bytes=args.tile)
    tile = chk.st.tile_bytes or 65536
    hp = c3.adamw_hparams(w.hparams["lr"], w.hparams["betas"], w.hparams["eps"],
                          w.hparams["weight_decay"], w.hparams["step"])
    n_slices = -(-w.numel // w.slice_elems)
    k0 = w.fault_slices[0]
    found = {}
    for k in sorted(set(w.fault_slices)):
        res = chk.run(k, hp)
        torch.cuda.synchronize()
        o = c3.outliers_numpy(res[4], res[6])
        found[k] = sorted({(chk.UNITS[int(u)], int(r)) for u, r in zip(o["chunk"], o["replica"])})
    log(f"[bench] outliers at the faulted slices: {found}")
    wk = [0]

    def warm_step():
        chk.run(k0 + wk[0], hp)
        wk[0] += 1
    args.warmup = warm_up(torch, warm_step, args.warmup)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    for i in range(args.steps):
        chk.run(k0 + i, hp)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    n = w.slice_elems
    R = w.R
    # Per-kernel durations in the check's launch configuration (slice k0, row
    # stride S, the same signature tile).  These kernels last microseconds:
    # a per-launch event pair would add several microseconds of its own, and
    # the host needs about as long to enqueue one call as the GPU to run it.
    # So a 4 GiB device copy is queued first, a run of back-to-back launches
    # is enqueued behind it between one pair of HIP events on the launch
    # stream, and the interval is divided by the run's length.
    head_src = torch.empty(1 << 32, dtype=torch.uint8, device=dev)
    head_dst = torch.empty_like(head_src)
    batch = 64

    def batch_ms(fn):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        fn(0, None, None)
        torch.cuda.synchronize()
        head_dst.copy_(head_src)
        a.record()
        for i in range(batch):
            fn(i, a if i == 0 else None, b if i == batch - 1 else None)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / batch

    k_adamw = batch_ms(lambda i, x, y: c3.adamw_slice(*w.state, k0 * n, n, hp, out=chk.updated,
                                                       out_stride=n, _tables=chk.tables))
    views = [[x[r][k0 * n:(k0 + 1) * n] for x in w.state] + [chk.updated[r, j] for j in range(3)]
             for r in range(R)]
    plan = c3.SignaturePlan(views, n * 4, tile)
    rec = plan.new_records()
    sws = plan.new_workspace()
    plan.run(rec, sws)
    # the staged plan is reused (no fetch kernel); the library records the
    # first event right before the first signature kernel, and the last one
    # is recorded again after the loop, behind the last partial combine
    k_sig = batch_ms(lambda i, a, b: plan.run(rec, sws, plan_staged=True, ev_begin=a, ev_end=b))
    del head_src, head_dst
    adamw_bytes = R * n * 28                 # read p, g, m, v; write p', m', v'
    sig_bytes = R * 7 * n * 4                # the seven signed slices per replica
    kern = {"adamw_slice_vec4_kernel": (k_adamw, adamw_bytes),
            "signature_kernel+finalize_kernel": (k_sig, sig_bytes)}
    dom = max(kern, key=lambda k: kern[k][0])
    d_ms, d_bytes = kern[dom]
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline on a bounded sample of checks")
        from oracle import adamw as oadamw
        n_host = 8
        host = [[t[(k0 % n_slices) * n:(k0 % n_slices + n_host) * n].cpu().numpy() for t in x]
                for x in w.state]
        t1 = time.perf_counter()
        done = 0
        while done < 1 or time.perf_counter() - t1 < args.cpu_budget:
            oadamw.boundary_check(host, done % n_host, w.hparams, n)
            done += 1
        dt = time.perf_counter() - t1
        cpu = {"value": round(done / dt, 3), "unit": "checks/s", "cores": 1, "kind": "oracle",
               "sample": f"{done} checks over {n_host} resident 64K-element slices of all {R} "
                         f"replicas (AdamW replay, 56 slice signatures, vote, localize), {dt:.1f} s",
               "host": host_cpu()}
    res = {
        "metric": "optimizer-boundary checks/s (64K-element AdamW slice, 8 replicas)",
        "value": round(1e3 / ms, 1),
        "unit": "checks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+u64",
        "data": "synthetic",
        "config": {"workload": w.name, "R": R, "params_per_replica": w.numel,
                   "slice_elems": n, "slices": n_slices, "tile_bytes": tile,
                   "outliers_at_fault_slices": {str(k): v for k, v in found.items()}},
        "roofline": {"bound": "hbm", "achieved": round(d_bytes / (d_ms * 1e-3) / 1e9, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(d_bytes / (d_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None, "kernel": dom, "kernel_ms": round(d_ms, 4),
                     "algorithmic_bytes_per_launch": d_bytes},
        "kernels": {k: {"ms": round(v[0], 4), "algorithmic_bytes": v[1],
                        "GBps": round(v[1] / (v[0] * 1e-3) / 1e9, 1)} for k, v in kern.items()},
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(res), flush=True)


def bench_hang(args):
    """Out-of-band hang localization on the host CPU: the native cost of the
    progress path, and the time from a frozen rank to every observer's
    verdict in a 4-rank Gloo drill (one step per drill)."""
    import statistics
    import subprocess

    from paper_2608_11034_amd import build as pbuild
    from paper_2608_11034_amd import oob_drill
    log("[bench] native progress path")
    native = json.loads(subprocess.run([pbuild.OOB_BENCH, "2000000"], check=True,
                                       capture_output=True, text=True, timeout=300).stdout)
    native.pop("sink", None)
    silence = 0.5
    runs = max(1, min(args.steps, 5))
    lat, classes = [], []
    for i in range(runs):
        log(f"[bench] freeze drill {i + 1}/{runs}")
        res = oob_drill.run_drill("freeze", world=4, at_step=5, silence_s=silence)
        lat += list(res["latency_s"].values())
        classes += [(v or {}).get("class") for v in res["verdicts"].values()]
    over = [t - silence for t in lat]
    out = {
        "metric": "hang localization latency beyond the silence threshold (frozen rank -> verdict)",
        "value": round(statistics.median(over), 4) if over else None,
        "unit": "s",
        "n_gpus": 0,
        "steps": runs,
        "warmup": 0,
        "ms_per_step": None,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": "gloo_drill_4ranks_freeze", "ranks": 4, "silence_threshold_s": silence,
                   "poll_s": 0.005, "verdicts": classes},
        "latency_s": {"min": round(min(lat), 4), "median": round(statistics.median(lat), 4),
                      "max": round(max(lat), 4)} if lat else None,
        "native": native,
        "roofline": None,
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
