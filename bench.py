"""Benchmark of the batched serving simulator on one MI355X.

Workload: the heavy-trace configuration -- 64 models with power-law (0.9)
rates summing to 1000 req/s, Gamma CV 4, one hour (about 3.6 M requests),
8192 candidate placements of 16 groups x (S=4, k=2), SLO scale 5, per-request
outputs kept for 16 of the placements.  One step = one batched call that
simulates every placement over the whole trace (dispatch, stage recurrence,
admission, counting, digests, per-request outputs); inputs are resident in HBM
before the timed region.

Prints ONE JSON line: events/s (request x placement pairs per second), the
roofline of the simulator kernel, and the CPU oracle's rate on a bounded
sample of the same workload (single thread).

Also reported, as "sweep": the SLO-curve sweep workload -- one fixed
placement (the 32-model / 64-device greedy search's best, 64 single-device
groups) over a 16 x 16 x 16 grid of rate scale, CV and SLO scale, every grid
point with its own 10-minute trace (4096 segments, about 4.4e8 requests) --
timed the same way, with its HBM roofline (each segment is read once).

The oracle's rate is taken on one pinned core (median of 3 runs over a
sample of jobs), and every job of the heavy trace and of the sweep is then
recomputed by the oracle on the host's cores and compared ("parity_full").
As "small_configs": the 4-model tiny case and one 512-job greedy step, timed
and compared with the oracle on every job.

And, as "search": wall time and simulated events of two placement searches
(reduced and full Alg. 2) on the 32-model / 64-device workload and of the
fast heuristic on its 10 uniform partitions beside the greedy's results; as
"batching": the dynamic-batching simulator on the batching experiment's shape
for maximum batch sizes 1-8; as "peaks_measured": the fp64 vector and
device-memory read ceilings measured on this machine, beside the published
figures the roofline objects use.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--cpu-sample J] [--no-cpu] [--no-parity-full]
                    [--no-small] [--no-sweep] [--no-search] [--no-batching] [--no-peaks]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "simulated request×placement events/sec on 1 GPU; % of HBM/VALU roofline"
# fp64 vector lane-operations per second on MI355X: 256 CUs x 4 SIMDs x 16
# fp64 lanes x 2.4 GHz = 3.93e13 (the 78.6 TFLOP/s figure counts an FMA as 2;
# the simulator issues no FMA, only max / add / compare / multiply).
PEAK_FP64_OPS = 256 * 4 * 16 * 2.4e9
HBM_PEAK = 8.0e12

# HBM traffic of one launch of the simulator kernels: rocprofv3 --pmc
# FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by what the same
# counter reads for a plain 1 GiB device copy.  The figures belong to the
# kernel sources (and compile flags) whose SHA-256 is recorded here; once those
# change, traffic is reported as null until it is measured again.
KERNEL_SOURCES = ["paper_2302_11665_amd/csrc/sim_api.hip", "paper_2302_11665_amd/csrc/sim_kernel.hpp",
                  "paper_2302_11665_amd/csrc/sim_launch.hip", "paper_2302_11665_amd/csrc/sim_launch.hpp",
                  "paper_2302_11665_amd/csrc/sim_shared.hpp", "paper_2302_11665_amd/csrc/sim_spec.hip"]
MEASURED_TRAFFIC = {
    "sources_sha256": "684637c3137697b219070a57f8d6c86345014f155cb72e55f014cddc6114a889",
    # one step of the heavy-trace workload runs the segment-speculative
    # pipeline (configuration check, pass 0, reconciliation rounds, output
    # rows, digest): its counters summed over the step's dispatches
    "kernel": "spec_pass0<4, 32, true, 64, true> + spec_round_fast<16, 4> + spec_rows<4, 32, true, 64> "
              "(row pieces and the final step) + spec_cfg_check (+ the variants that return at once)",
    "fetch_kib": 2218171.63, "write_kib": 5990707.06,
    "fetch_scale": 1048576.0 / 524301.90, "write_scale": 1048576.0 / 1048576.0,
}
MEASURED_TRAFFIC_SWEEP = {
    "sources_sha256": "684637c3137697b219070a57f8d6c86345014f155cb72e55f014cddc6114a889",
    "kernel": "seg_kernel<1>",
    "fetch_kib": 2595524.38, "write_kib": 14218.69,
    "fetch_scale": 1048576.0 / 524301.90, "write_scale": 1048576.0 / 1048576.0,
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def host_threads():
    """Oracle worker threads: the CPUs this process may run on, at most 16 (a
    one-GPU share of the host)."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def host_cpu_info():
    """CPU model, clocks and counts of the host the oracle runs on."""
    model = mhz = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                k, _, v = line.partition(":")
                k = k.strip()
                if k == "model name" and model is None:
                    model = v.strip()
                elif k == "cpu MHz" and mhz is None:
                    mhz = float(v)
    except (OSError, ValueError):
        pass
    max_mhz = None
    try:
        with open("/sys/devices/system/cpu/cpu0/cpufreq/cpuinfo_max_freq") as f:
            max_mhz = int(f.read().strip()) / 1000.0
    except (OSError, ValueError):
        pass
    return {"cpu_model": model, "cpu_mhz": mhz, "cpu_max_mhz": max_mhz, "nproc": os.cpu_count(),
            "affinity_cpus": len(os.sched_getaffinity(0))}


def oracle_cpu_baseline(lib, N, jobs, one_job, runs=3):
    """The oracle as it stands, single-threaded and pinned to one core: the
    same jobs `runs` times, the median run's events/s."""
    cpus = sorted(os.sched_getaffinity(0))
    core = cpus[0]
    os.sched_setaffinity(0, {core})
    times = []
    try:
        for r in range(runs):
            t0 = time.perf_counter()
            for j in jobs:
                one_job(j)
            times.append(time.perf_counter() - t0)
            log(f"cpu oracle run {r + 1}/{runs}: {len(jobs)} jobs in {times[-1]:.2f}s")
    finally:
        os.sched_setaffinity(0, set(cpus))
    med = sorted(times)[len(times) // 2]
    return {"value": round(len(jobs) * N / med, 1), "unit": "events/s", "cores": 1, "kind": "oracle",
            "pinned_core": core, "runs_s": [round(x, 3) for x in times], "statistic": f"median of {runs} runs",
            **host_cpu_info()}


def oracle_parity_full(jobs, one_job, check, label):
    """Every job recomputed by the oracle on host_threads() threads (the
    oracle's C calls release the GIL) and compared by check(j, result), which
    returns the number of mismatching fields."""
    from concurrent.futures import ThreadPoolExecutor
    nthreads = host_threads()
    jobs = list(jobs)
    mism, bad = 0, []
    t0 = time.perf_counter()
    with ThreadPoolExecutor(nthreads) as ex:
        for q, (j, r) in enumerate(zip(jobs, ex.map(one_job, jobs))):
            k = check(j, r)
            if k:
                mism += k
                if len(bad) < 8:
                    bad.append(int(j))
            if (q + 1) % 1024 == 0 or q + 1 == len(jobs):
                log(f"{label} full parity: {q + 1}/{len(jobs)} jobs, {mism} mismatches, "
                    f"{time.perf_counter() - t0:.1f}s")
    return {"jobs": len(jobs), "mismatches": mism, "first_bad_jobs": bad, "cores": nthreads,
            "wall_s": round(time.perf_counter() - t0, 2), "kind": "oracle, every job"}


def algorithmic_ops(pb):
    """fp64 operations the definition needs per launch: per request of a hosted
    model, (H - 1) dispatch compares over its H hosting groups, S max + S add in
    the stage chain, one add for the deadline and one compare; plus one
    multiply per (job, model) for the SLO.  Placements here give every group
    the same configuration."""
    import numpy as np
    M = pb.d_single.shape[0]
    counts = np.bincount(pb.model, minlength=M).astype(np.float64)
    S = int(pb.cfg_stages[pb.group_cfg[0, 0]])
    hosts = np.zeros(pb.host_mask.shape, dtype=np.float64)
    hm = pb.host_mask
    for g in range(64):
        hosts += ((hm >> np.uint64(g)) & np.uint64(1)).astype(np.float64)
    per = np.where(hosts > 0, hosts - 1 + 2 * S + 2, 0.0)  # [P, M]
    ops_per_scale = float((per * counts[None, :]).sum()) + pb.group_cfg.shape[0] * M
    return ops_per_scale * pb.slo_scale.shape[0]


def sources_sha256():
    """SHA-256 over the kernel sources and the HIP compile flags."""
    import hashlib
    from paper_2302_11665_amd import build
    h = hashlib.sha256()
    for f in sorted(KERNEL_SOURCES):
        h.update(os.path.basename(f).encode())
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    h.update(" ".join(build.HIP_FLAGS).encode())
    return h.hexdigest()


def measured_traffic(m, default_workload):
    if not default_workload or m["sources_sha256"] is None or sources_sha256() != m["sources_sha256"]:
        return None
    return round((m["fetch_kib"] * m["fetch_scale"] + m["write_kib"] * m["write_scale"]) * 1024.0)


def algorithmic_bytes(pb):
    """Bytes the definition moves per launch: the trace read once (time f64 +
    model i32), the placement tables, the per-job outputs (served i64, attain
    f64, digest 2 x u64) and the per-request outputs of the selected jobs."""
    N, J = len(pb.t), pb.n_jobs
    return (12 * N + pb.group_cfg.nbytes + pb.host_mask.nbytes + pb.stage_lat.nbytes
            + J * (8 + 8 + 16) + 8 * N * len(pb.finish_jobs))


def sweep_placement():
    """The best placement of the 32-model / 64-device greedy search, stored
    with the search's result (inputs only: group configurations and hosting
    masks)."""
    import numpy as np
    with open(os.path.join(ROOT, "tests", "golden", "c3_greedy_oracle.json")) as f:
        fx = json.load(f)
    return (np.array(fx["best_group_cfg"], np.int32),
            np.array([int(x) for x in fx["best_host_mask"]], np.uint64))


def sweep_algorithmic_bytes(sp, n_finish_rows, stride):
    """Every segment read once (12 B per request), offsets and job records,
    per-job outputs and the per-request outputs of the selected jobs."""
    return (12 * len(sp.t) + sp.seg_offsets.nbytes + 16 * len(sp.job_segment)
            + 32 * len(sp.job_segment) + 8 * n_finish_rows * stride)


def bench_sweep(args, np, torch, api, problems):
    t0 = time.time()
    gcfg, hm = sweep_placement()
    sp = problems.c5_sweep(gcfg, hm)
    gen_s = time.time() - t0
    events = sp.events
    log(f"sweep: {len(sp.job_segment)} jobs, {events:.3e} events; built in {gen_s:.2f}s")
    t0 = time.time()
    ds = api.upload_sweep(sp)
    torch.cuda.synchronize()
    up_s = time.time() - t0
    for _ in range(args.warmup):
        api.run_sweep(ds)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev[0].record(stream)
    for k in range(args.steps):
        api.run_sweep(ds)
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps)]
    ms = float(np.mean(per))
    log(f"sweep: {ms:.3f} ms/step (min {min(per):.3f}, max {max(per):.3f})")
    nbytes = sweep_algorithmic_bytes(sp, len(ds.finish_jobs), ds.finish_stride)
    gbs = nbytes / (ms / 1000.0) / 1e9
    res = api.sweep_results(ds)
    del ds
    torch.cuda.empty_cache()
    parity = None
    if not args.no_cpu:
        import oracle
        lib = oracle.lib()
        lens = np.diff(sp.seg_offsets)
        fset = set(int(x) for x in sp.finish_jobs)

        def one(j):
            s = int(sp.job_segment[j])
            a, b = int(sp.seg_offsets[s]), int(sp.seg_offsets[s + 1])
            return lib.simulate_job(sp.t[a:b], sp.model[a:b], sp.d_single, sp.cfg_stages, sp.stage_lat,
                                    sp.group_cfg[sp.job_placement[j]], sp.host_mask[sp.job_placement[j]],
                                    sp.job_scale[j], want_finish=j in fset)

        def check(j, r):
            s, dg, fin = r
            n = int(lens[sp.job_segment[j]])
            bad = int(int(res["served"][j]) != s) + int(tuple(int(x) for x in res["digest"][j]) != dg)
            bad += int(res["attain"][j] != (s / n if n else 0.0))
            if fin is not None:
                bad += int(res["finish"][j][:n].tobytes() != fin.tobytes())
            return bad

        parity = oracle_parity_full(range(len(sp.job_segment)), one, check, "sweep")
        parity["finish_rows"] = len(fset)
    return {"workload": "SLO-curve sweep: 32 models, 64 single-device groups (greedy best), 16x16x16 grid of "
                        "rate scale x CV x SLO scale, own 600 s trace per point",
            "jobs": int(len(sp.job_segment)), "requests": int(len(sp.t)), "events": int(events),
            "ms_per_step": round(ms, 3), "value": round(events / (ms / 1000.0), 1), "unit": "events/s",
            "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                         "frac": round(gbs * 1e9 / HBM_PEAK, 5), "traffic": measured_traffic(MEASURED_TRAFFIC_SWEEP, True),
                         "algorithmic_bytes": int(nbytes)},
            "served_total": int(res["served"].sum()), "parity_full": parity,
            "trace_gen_s": round(gen_s, 3), "upload_s": round(up_s, 3)}


def bench_small(args, np, torch, api, problems):
    """The two small configurations: the 4-model tiny case (all 273 maps of 4
    models onto the partitions of 4 devices, Poisson 5 req/s per model, 60 s,
    SLO scale 5) and one greedy step of the 16-model case (64 single-replica
    candidates x 8 SLO scales, Gamma 4 req/s per model CV 3, 10 minutes).
    Each call timed with HIP events (mean of 20 after 3 warm-ups); every job
    compared with the oracle; the oracle's single-core rate over all jobs."""
    out = {}
    lib = None
    if not args.no_cpu:
        import oracle
        lib = oracle.lib()
    for name, pb in (("tiny_273_jobs", problems.c1_tiny()), ("greedy_step_512_jobs", problems.c2_greedy_step())):
        N, J, K = len(pb.t), pb.n_jobs, len(pb.slo_scale)
        dp = api.upload(pb, finish=False)
        for _ in range(3):
            api.run(dp)
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(21)]
        ev[0].record(stream)
        for k in range(20):
            api.run(dp)
            ev[k + 1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.mean([ev[k].elapsed_time(ev[k + 1]) for k in range(20)]))
        res = api.results(dp)
        rec = {"requests": N, "jobs": J, "events": N * J, "ms_per_call": round(ms, 4),
               "value": round(N * J / (ms / 1000.0), 1), "unit": "events/s"}
        if lib is not None:
            def one(j, pb=pb, K=K):
                p, k = divmod(int(j), K)
                return lib.simulate_job(pb.t, pb.model, pb.d_single, pb.cfg_stages, pb.stage_lat, pb.group_cfg[p],
                                        pb.host_mask[p], pb.slo_scale[k])

            def check(j, r, res=res, N=N):
                s, dg, _ = r
                return (int(int(res["served"][j]) != s) + int(tuple(int(x) for x in res["digest"][j]) != dg)
                        + int(res["attain"][j] != (s / N if N else 0.0)))

            rec["parity_full"] = oracle_parity_full(range(J), one, check, name)
            cb = oracle_cpu_baseline(lib, N, list(range(J)), one)
            rec["cpu_oracle_events_per_s"] = cb["value"]
            rec["speedup_vs_cpu_oracle"] = round(rec["value"] / cb["value"], 1)
        log(f"{name}: {ms:.3f} ms/call, {rec['value']:.3e} events/s")
        out[name] = rec
        del dp
    return out


def bench_search(args, np, torch, sim, problems):
    """Placement searches on the 32-model / 64-device workload (Gamma 4 req/s
    per model, CV 2, 20 minutes, SLO scale 5): the reduced Alg. 2 (Alg. 1 with
    beam 1 on each of the 10 uniform partitions), whose oracle run is stored
    with its wall time, and the full Alg. 2 with up to 3 model buckets."""
    with open(os.path.join(ROOT, "tests", "golden", "c3_greedy_oracle.json")) as f:
        fx = json.load(f)
    gp = problems.c3_greedy()
    N = len(gp.t)
    d = sim.to_device
    t, m, ds, L = d(gp.t), d(gp.model), d(gp.d_single), d(gp.stage_lat)
    cd = (gp.cfg_stages * gp.cfg_k).astype(np.int32)
    out = {"workload": "32 models (d ~ U[0.05,0.8] s, w ~ U[1,13] GB), 64 x 32 GB devices, Gamma 4 req/s/model "
                       "CV 2, 1200 s, SLO scale 5; configurations (S,k) with S*k in {1,2,4,8}",
           "requests": N}
    runs = [("alg2_reduced", dict(max_buckets=1, bucket_threshold=10.0, balance_ratio=float("inf"),
                                  device_unit=64, beam=1)),
            ("alg2_full", dict(max_buckets=3, bucket_threshold=0.4, balance_ratio=2.0, device_unit=16, beam=1))]
    for name, kw in runs:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r = sim.as_placement_search(t, m, ds, gp.cfg_stages, L, gp.weight_mib, cd, 64, kw["device_unit"],
                                    gp.meta["device_mem_mib"], kw["bucket_threshold"], kw["balance_ratio"],
                                    kw["max_buckets"], kw["beam"], gp.slo_scale)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ev = r["jobs_simulated"] * N
        opts = {k: ("inf" if isinstance(v, float) and v == float("inf") else v) for k, v in kw.items()}
        res = {"options": opts, "wall_s": round(wall, 3), "launches": r["launches"], "jobs": r["jobs_simulated"],
               "events": ev, "events_per_s": round(ev / wall, 1), "served": r["served"],
               "problems": r["n_problems"], "kept_splits": r["n_kept_splits"],
               "buckets": [{"models": b["models"], "devices": b["devices"], "cfg": b["cfg"], "served": b["served"]}
                           for b in r["buckets"]]}
        if name == "alg2_reduced":
            res["oracle_served"] = fx["best_served"]
            res["oracle_wall_s"] = round(fx["seconds"], 1)
            res["oracle_note"] = "the same search on the CPU oracle, 8 threads (stored with its result)"
            res["parity"] = r["served"] == fx["best_served"]
        log(f"search {name}: {wall:.2f}s, {r['launches']} launches, {r['jobs_simulated']} jobs, served {r['served']}")
        out[name] = res
    # the fast heuristic of Sec. 4.2 on the 10 uniform partitions (the reduced
    # Alg. 2 with the heuristic in place of Alg. 1: the partitions advance in
    # lockstep, one launch per step), next to Alg. 1 with beam 1 on the same
    # partitions; per partition, the heuristic's result is the oracle's
    # (computed on host threads), the greedy's the stored oracle result that
    # the native search reproduces step for step
    kw = dict(max_buckets=1, bucket_threshold=10.0, balance_ratio=float("inf"), device_unit=64, beam=0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r = sim.as_placement_search(t, m, ds, gp.cfg_stages, L, gp.weight_mib, cd, 64, kw["device_unit"],
                                gp.meta["device_mem_mib"], kw["bucket_threshold"], kw["balance_ratio"],
                                kw["max_buckets"], kw["beam"], gp.slo_scale)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gs = [p["best_served"] for p in fx["partitions"]]
    fh = {"wall_s": round(wall, 3), "launches": r["launches"], "jobs": r["jobs_simulated"],
          "events": r["jobs_simulated"] * N, "served": r["served"], "greedy_served": fx["best_served"],
          "ratio": round(r["served"] / fx["best_served"], 5) if fx["best_served"] else None,
          "greedy_served_by_partition": gs,
          "note": "Sec. 4.2 expects the heuristic's attainment at >= 98% of the greedy search's"}
    if not args.no_cpu:
        import oracle
        from concurrent.futures import ThreadPoolExecutor
        from oracle import greedy as og
        lib = oracle.lib()

        def one(part):
            t1 = time.perf_counter()
            b = og.fast_selection(lib, gp.t, gp.model, gp.d_single, gp.weight_mib, gp.cfg_stages, gp.stage_lat,
                                  part["group_cfg"], part["group_mem_mib"], gp.slo_scale)["best_served"]
            return b, time.perf_counter() - t1

        nthr = min(host_threads(), len(gp.partitions))
        t1 = time.perf_counter()
        with ThreadPoolExecutor(nthr) as ex:
            got = list(ex.map(one, gp.partitions))
        fs = [b for b, _ in got]
        # the oracle's C simulation releases the GIL: the partitions' times add
        # up to what one thread would take
        fh["oracle_wall_s"] = round(time.perf_counter() - t1, 3)
        fh["oracle_threads"] = nthr
        fh["oracle_one_thread_s"] = round(sum(x for _, x in got), 3)
        fh["oracle_heuristic_served_by_partition"] = fs
        fh["ratio_by_partition"] = [round(a / b, 5) if b else None for a, b in zip(fs, gs)]
        fh["parity"] = max(fs) == r["served"]
    log(f"search fast heuristic: {wall:.2f}s, {r['launches']} launches, served {r['served']} "
        f"vs greedy {fx['best_served']}")
    out["fast_heuristic"] = fh
    return out


def bench_batching(args, np, torch, sim, problems):
    """The dynamic-batching simulator (Sec. 6.5) on the batching experiment's
    shape: 32 models of 151 ms, Gamma 4 req/s per model CV 4 for 10 minutes,
    256 placements on 16 groups of 4 devices (S=4) x 8 SLO scales, for maximum
    batch sizes 1, 2, 4 and 8 at latency slope 1; each call timed with HIP
    events, plus the oracle's rate on a sample of jobs with sampled parity."""
    import oracle
    pb = problems.batching()
    N, J = len(pb.t), pb.n_jobs
    d = sim.to_device
    t, m, ds, L, gc, hm, sc = (d(pb.t), d(pb.model), d(pb.d_single), d(pb.stage_lat), d(pb.group_cfg),
                               d(pb.host_mask), d(pb.slo_scale))
    served = torch.empty(J, dtype=torch.int64, device="cuda")
    digest = torch.empty((J, 2), dtype=torch.int64, device="cuda")
    K = len(pb.slo_scale)
    out = {"workload": "batching experiment shape: 32 models x 151 ms, Gamma 4 req/s/model CV 4, 600 s; "
                       "256 placements of 16 groups (S=4) x 8 SLO scales 1..20; latency slope 1",
           "requests": N, "jobs": J, "events_per_call": N * J, "by_max_batch": {}}
    lib = oracle.lib() if not args.no_cpu else None
    sample = list(range(0, J, max(1, J // 8)))[:8]
    for B in (1, 2, 4, 8):
        call = lambda: sim.as_simulate_batched(t, m, ds, pb.cfg_stages, L, gc, hm, sc, B, 1.0, served, digest,
                                               queue_cap=128)
        try:
            call()
        except sim.SimError as e:
            out["by_max_batch"][str(B)] = {"error": str(e)}
            log(f"batching B={B}: {e}")
            continue
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        for k in range(3):
            call()
            ev[k + 1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.mean([ev[k].elapsed_time(ev[k + 1]) for k in range(3)]))
        s_np, dg = served.cpu().numpy(), sim.u64(digest)
        res = {"ms_per_call": round(ms, 3), "events_per_s": round(N * J / (ms / 1000.0), 1),
               "attainment_mean": round(float(s_np.sum()) / (N * J), 5)}
        if lib is not None:
            t0 = time.perf_counter()
            mism = 0
            for j in sample:
                p, k = divmod(j, K)
                so, dgo, _, _ = lib.simulate_job_batched(pb.t, pb.model, pb.d_single, pb.cfg_stages, pb.stage_lat,
                                                         pb.group_cfg[p], pb.host_mask[p], pb.slo_scale[k], B, 1.0)
                mism += int(so != int(s_np[j]) or dgo != tuple(int(x) for x in dg[j]))
            cpu_s = time.perf_counter() - t0
            res["cpu_oracle_events_per_s"] = round(len(sample) * N / cpu_s, 1)
            res["parity_sampled"] = {"jobs": len(sample), "mismatches": mism}
        log(f"batching B={B}: {ms:.2f} ms/call, mean attainment {res['attainment_mean']}")
        out["by_max_batch"][str(B)] = res
    return out


def measure_peaks(torch):
    """The two ceilings measured on this machine with the probe library: fp64
    vector lane-operations per second (v_max_f64 / v_add_f64 chains, the
    simulator's kind of work) and device-memory read bytes per second over an
    8 GiB buffer.  Quoted beside the published figures the roofline uses."""
    import ctypes
    from paper_2302_11665_amd import build as b
    if not os.path.exists(b.PROBE_LIB):
        raise RuntimeError(f"{b.PROBE_LIB} is not built; run __graft_entry__.build()")
    torch.cuda.synchronize()
    L = ctypes.CDLL(b.PROBE_LIB)
    L.as_probe_valu_f64.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    L.as_probe_hbm_read.argtypes = [ctypes.c_size_t, ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    ops, bps = ctypes.c_double(0.0), ctypes.c_double(0.0)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    if L.as_probe_valu_f64(cus * 8, 200000, 3, ctypes.byref(ops)) != 0:
        raise RuntimeError("fp64 VALU probe failed")
    if L.as_probe_hbm_read(8 << 30, 5, ctypes.byref(bps)) != 0:
        raise RuntimeError("device-memory read probe failed")
    return {"fp64_lane_ops_per_s": float(f"{ops.value:.4e}"),
            "fp64_frac_of_published": round(ops.value / PEAK_FP64_OPS, 4),
            "hbm_read_bytes_per_s": float(f"{bps.value:.4e}"),
            "hbm_frac_of_published": round(bps.value / HBM_PEAK, 4),
            "note": "probes: 8 independent v_max_f64+v_add_f64 chains per lane, "
                    f"{cus * 8} blocks of 256 threads; 16-byte grid-stride reads of 8 GiB; best of the timed runs"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--placements", type=int, default=8192)
    ap.add_argument("--duration", type=float, default=3600.0)
    ap.add_argument("--cpu-sample", type=int, default=64,
                    help="jobs timed on the CPU oracle (single core, median of 3 runs)")
    ap.add_argument("--no-cpu", action="store_true", help="no oracle work at all (baseline and parity)")
    ap.add_argument("--no-parity-full", action="store_true",
                    help="skip the every-job oracle comparison of the heavy-trace step")
    ap.add_argument("--no-small", action="store_true", help="skip the two small configurations")
    ap.add_argument("--no-sweep", action="store_true", help="skip the SLO-curve sweep workload")
    ap.add_argument("--no-search", action="store_true", help="skip the placement-search timings")
    ap.add_argument("--no-batching", action="store_true", help="skip the dynamic-batching timings")
    ap.add_argument("--no-peaks", action="store_true", help="skip the fp64 VALU and memory-read peak probes")
    ap.add_argument("--sweep-only", action="store_true",
                    help="time only the SLO-curve sweep (prints its object alone)")
    ap.add_argument("--calibrate-copy", type=float, default=0.0,
                    help="instead of the benchmark, run a plain device copy of this many GiB "
                         "(HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import numpy as np
    import torch

    if args.calibrate_copy > 0:
        n = int(args.calibrate_copy * (1 << 30)) // 8
        x = torch.empty(n, dtype=torch.float64, device="cuda")
        y = torch.empty_like(x)
        x.fill_(1.0)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_read": n * 8, "bytes_written": n * 8}))
        return

    from paper_2302_11665_amd import api, sim
    from paper_2302_11665_amd.workload import problems

    if args.sweep_only:
        print(json.dumps({"sweep": bench_sweep(args, np, torch, api, problems)}), flush=True)
        return

    t0 = time.time()
    pb = problems.c4_heavy(duration=args.duration, n_placements=args.placements)
    gen_s = time.time() - t0
    N, J = len(pb.t), pb.n_jobs
    events = N * J
    log(f"workload: {J} jobs x {N} requests = {events:.3e} events; trace+placements built in {gen_s:.2f}s")
    t0 = time.time()
    dp = api.upload(pb)
    torch.cuda.synchronize()
    up_s = time.time() - t0
    log(f"uploaded in {up_s:.2f}s; library {sim.as_version()}")

    for w in range(args.warmup):
        api.run(dp)
        torch.cuda.synchronize()
        log(f"warmup {w + 1}/{args.warmup} done")
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev[0].record(stream)
    for k in range(args.steps):
        api.run(dp)
        ev[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    per = [ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps)]
    ms = float(np.mean(per))
    log(f"timed {args.steps} steps: {ms:.2f} ms/step (min {min(per):.2f}, max {max(per):.2f}); wall {wall:.2f}s")
    value = events / (ms / 1000.0)
    res = api.results(dp)

    ops = algorithmic_ops(pb)
    achieved = ops / (ms / 1000.0) / 1e12
    peak = PEAK_FP64_OPS / 1e12
    roof = {"bound": "alu", "achieved": round(achieved, 4), "peak": round(peak, 2), "unit": "TFLOP/s",
            "frac": round(achieved / peak, 5),
            "traffic": measured_traffic(MEASURED_TRAFFIC, args.placements == 8192 and args.duration == 3600.0),
            "algorithmic_bytes": int(algorithmic_bytes(pb)),
            "ops_per_event": round(ops / events, 3),
            "note": "fp64 lane-ops (max/add/cmp/mul, no FMA) of the definition per step / mean step time; "
                    "the step is the speculative pipeline (pass 0, reconciliation rounds, digest); "
                    "traffic includes its workspace (accept bitmap, checkpoints)"}

    out = {"metric": METRIC, "value": round(value, 1), "unit": "events/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
           "data": "synthetic",
           "config": {"workload": "heavy trace: 64 models power-law(0.9) 1000 req/s Gamma CV4 1h; "
                                  "8192 placements of 16 groups (S=4,k=2); SLO scale 5",
                      "requests": N, "placements": pb.group_cfg.shape[0], "jobs": J,
                      "finish_jobs": int(len(pb.finish_jobs))},
           "roofline": roof, "trace_gen_s": round(gen_s, 3), "upload_s": round(up_s, 3)}

    if not args.no_cpu:
        import oracle
        if not os.path.exists(oracle.LIB_PATH):
            oracle.build()
        lib = oracle.lib()
        fset = set(int(x) for x in pb.finish_jobs)

        def one(j, finish=True):
            return lib.simulate_job(pb.t, pb.model, pb.d_single, pb.cfg_stages, pb.stage_lat, pb.group_cfg[j],
                                    pb.host_mask[j], pb.slo_scale[0], want_finish=finish and j in fset)

        def check(j, r):
            s, dg, fin = r
            bad = int(int(res["served"][j]) != s) + int(tuple(int(x) for x in res["digest"][j]) != dg)
            bad += int(res["attain"][j] != s / N)
            if fin is not None:
                bad += int(res["finish"][j].tobytes() != fin.tobytes())
            return bad

        if args.cpu_sample > 0:
            step = max(1, J // args.cpu_sample)
            sample = list(range(0, J, step))[: args.cpu_sample]
            cb = oracle_cpu_baseline(lib, N, sample, lambda j: one(j, False))
            cb["sample"] = (f"{len(sample)} of {J} jobs (every {step}th) x the full trace = {len(sample) * N:.3e} "
                            f"events per run, one thread pinned to one core")
            out["cpu_baseline"] = cb
            out["speedup_vs_cpu_oracle"] = round(value / cb["value"], 1)
        if not args.no_parity_full:
            pf = oracle_parity_full(range(J), one, check, "heavy trace")
            pf["finish_rows"] = len(fset)
            out["parity_full"] = pf
    if not args.no_small:
        out["small_configs"] = bench_small(args, np, torch, api, problems)
    if not args.no_sweep:
        del dp
        torch.cuda.empty_cache()
        out["sweep"] = bench_sweep(args, np, torch, api, problems)
    if not args.no_search:
        out["search"] = bench_search(args, np, torch, sim, problems)
    if not args.no_batching:
        out["batching"] = bench_batching(args, np, torch, sim, problems)
    if not args.no_peaks:
        out["peaks_measured"] = measure_peaks(torch)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
