"""Throughput of the batched frequency-controller hot path on one MI355X.

One step = projection (+ feature-row expansion), tree-ensemble prediction on
every (scenario, frequency, iteration) row, and frequency selection, for one
batch of synthetic scenarios already resident in HBM.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config c3] [--no-cpu-baseline]
                    [--cpu-procs C]

Prints one JSON line: whole-step throughput, per-stage HIP-event times (mean,
median, min over the K timed steps), the forest kernel's roofline record, the
oracle's CPU baseline (one thread, and C single-threaded processes), the
paper's binary-search controller on the same projection, the model compiled
to its input lattice (a separate mode with a one-time build), and the
admission-control what-ifs (one new query per scenario) on the same workload.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# 256 CUs x 4 SIMDs x 16 lanes per clock x 2.4 GHz: one non-packed VALU lane
# operation (an fp32 compare or add) per lane per clock
VALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
FOREST_KERNEL = "forest_grid_lds_kernel"
METRIC = "feature rows predicted/sec + scenarios/sec end-to-end; % of HBM peak"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(inp, F, rows, sel=None):
    """Bytes each stage must move at least (inputs read once, outputs written
    once) for one step of the fused pipeline (rows are never materialized).
    Selection stops at the first round of four frequencies with a feasible
    one, so with the step's results `sel` = (freq_idx, status, n_iters) its
    bytes are the IPS of the frequencies up to that round (all of them when
    none is feasible, none for lost / invalid scenarios) over the projected
    iterations, plus the deadline map."""
    S, H = inp["n_scenarios"], inp["horizon"]
    R = int(inp["req_offset"][-1])
    f = inp["forest"]
    n_leaf = 1 << f["depth"]
    forest_bytes = f["n_trees"] * n_leaf * (16 + 4 + 16)   # device nodes, leaves, boxes
    k1 = R * 25 + S * 8 + S * 8 + S * H * 16 + S * 8        # requests; offsets, caps; curves; scalars
    k2 = S * H * 8 + F * 4 + S * 4 + forest_bytes + rows * 4
    k3 = rows * 4 + S * H * 8 + S * 28
    if sel is not None:
        idx, st, n = (np.asarray(a, np.int64) for a in sel)
        evaluated = np.where(st == 0, np.minimum(F, 4 * (idx // 4 + 1)), np.where(st == 1, F, 0))
        k3 = int((evaluated * n).sum()) * 4 + int(n.sum()) * 8 + S * 28
    return dict(project=k1, predict=k2, select=k3)


def traffic_record(path):
    """HBM bytes per launch from a committed rocprofv3 traffic record, if it
    was taken on the current sources of its kernel."""
    if not os.path.exists(path):
        return None
    from paper_2408_05235_amd import prof_summary
    rec = json.load(open(path))
    names = rec.get("sources")
    if not names or rec.get("sources_sha256") != prof_summary.sources_sha256(names):
        return None
    return rec.get("bytes_per_launch")


def _host_info():
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return dict(cpu_model=model, nproc=os.cpu_count(), affinity=len(os.sched_getaffinity(0)))


def _oracle_scenarios(sub_inputs, budget_s, keep=False):
    """Run the oracle on whole scenarios, one after another, until the budget
    is spent; returns (scenarios done, rows done, seconds, results) where
    results (with `keep`) holds each scenario's IPS, index and status."""
    import oracle
    done, rows, t_used, kept = 0, 0, 0.0, []
    for sub in sub_inputs:
        t0 = time.perf_counter()
        r = oracle.end_to_end(sub)
        t_used += time.perf_counter() - t0
        done += 1
        rows += sub["n_freqs"] * sub["horizon"]
        if keep:
            kept.append(dict(ips=r["ips"][0], freq_idx=int(r["freq_idx"][0]), status=int(r["status"][0])))
        if t_used >= budget_s:
            break
    return done, rows, t_used, kept


def cpu_baseline(inp, budget_s=12.0, max_scen=64, procs=0):
    """The oracle timed on whole scenarios of the workload (s = 0, s = S-1,
    then a seeded random order) for about `budget_s` seconds on one thread;
    with `procs` > 1 also as that many single-threaded processes, each on its
    own scenarios, for the same budget (rows of all processes / longest one)."""
    from paper_2408_05235_amd import synth
    S = inp["n_scenarios"]
    order = list(dict.fromkeys([0, S - 1] + list(np.random.default_rng(0).permutation(S))))
    done, rows, t_used = 0, 0, 0.0
    results = {}
    for s in order[:max_scen]:
        d, r, t, kept = _oracle_scenarios([synth.subset(inp, [s])], budget_s, keep=True)
        done, rows, t_used = done + d, rows + r, t_used + t
        results[int(s)] = kept[0]
        if t_used >= budget_s:
            break
    out = dict(value=rows / t_used, unit="rows/s", cores=1, kind="oracle",
               sample=f"{done} of {S} scenarios (all stages, single thread), {t_used:.1f} s",
               scenarios_per_s=done / t_used, **_host_info())
    out["_results"] = results
    if procs > 1 and S >= 2 * procs:
        import multiprocessing as mp
        per = max(2, (max_scen * 2) // procs)
        jobs = [[synth.subset(inp, [s]) for s in order[w::procs][:per]] for w in range(procs)]
        t0 = time.perf_counter()
        with mp.get_context("spawn").Pool(procs) as pool:
            res = pool.starmap(_oracle_scenarios, [(j, budget_s, False) for j in jobs])
        wall = time.perf_counter() - t0
        n = sum(r[0] for r in res)
        tot_rows = sum(r[1] for r in res)
        t_max = max(r[2] for r in res)
        out["sharded"] = dict(value=tot_rows / t_max, unit="rows/s", cores=procs, kind="oracle",
                              sample=f"{n} of {S} scenarios in {procs} single-threaded processes, "
                                     f"longest {t_max:.1f} s of oracle time ({wall:.1f} s wall with start-up)")
    return out


def oracle_parity(ctl, results):
    """The last timed step's IPS, frequency index and status against the
    oracle's on the scenarios the CPU baseline ran (bit for bit)."""
    idx = ctl.sel["freq_idx"].cpu().numpy()
    st = ctl.sel["status"].cpu().numpy().view(np.uint32)
    bad = []
    for s, r in results.items():
        ips = ctl.ips[s].cpu().numpy()
        if not (np.array_equal(ips.view(np.uint32), r["ips"].view(np.uint32))
                and int(idx[s]) == r["freq_idx"] and int(st[s]) == r["status"]):
            bad.append(s)
    return {"scenarios": len(results), "mismatched": bad[:16], "ok": not bad,
            "compared": "IPS of every (frequency, iteration) row, frequency index, status"}


def copy_bandwidth_gbs(mib=2048, reps=5):
    """Device-to-device copy bandwidth measured on this GPU (read + write
    bytes per second of a plain torch copy), the practical HBM ceiling."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    del src, dst
    return 2 * n * 4 / (best / 1e3) / 1e9


def d2h_results_ms(ctl, reps=5):
    """Copy of the per-scenario results (frequency index and status, S int32
    each) to pinned host memory, reported apart from the step."""
    import torch
    S = ctl.d["n_scenarios"]
    host = torch.empty((2, S), dtype=torch.int32, pin_memory=True)
    ts = []
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        host[0].copy_(ctl.sel["freq_idx"], non_blocking=True)
        host[1].copy_(ctl.sel["status"], non_blocking=True)
        torch.cuda.synchronize()
        ts.append((time.perf_counter() - t0) * 1e3)
    return float(np.median(ts))


def adjust_lengths_bench(inp, dev_in, steps, copy_gbs):
    """The scoreboard stage of Sec. 4.6 (predicted lengths inflated by 11/10,
    limited to 4096 tokens) over every request of the workload; HBM-bound:
    8 bytes read and 4 written per request, 16 read per scenario."""
    import torch

    from paper_2408_05235_amd import api
    S, R = inp["n_scenarios"], int(inp["req_offset"][-1])
    d = dev_in
    pred = (d["generated"].to(torch.int64) + d["remaining"]).to(torch.int32)
    num = torch.full((S,), 11, dtype=torch.int32, device="cuda:0")
    den = torch.full((S,), 10, dtype=torch.int32, device="cuda:0")
    mt = torch.full((S,), 4096, dtype=torch.int32, device="cuda:0")
    out = torch.empty(R, dtype=torch.int32, device="cuda:0")
    api.tl_adjust_lengths(d["req_offset"], d["generated"], pred, num, den, mt, out)
    torch.cuda.synchronize()
    ev = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        api.tl_adjust_lengths(d["req_offset"], d["generated"], pred, num, den, mt, out)
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    byt = 12 * R + 16 * S
    return {"requests": R, "ms_median": ms, "gbs": byt / (ms / 1e3) / 1e9,
            "frac_of_copy": byt / (ms / 1e3) / 1e9 / copy_gbs, "frac_of_hbm_peak": byt / (ms / 1e3) / 1e9 / HBM_PEAK_GBS}


def materialized_rows_bench(inp, dev_in, forest, ctl, steps, copy_gbs, sample_rows=1 << 20):
    """The path that writes the feature rows out (a separate mode, not the
    headline): tl_project with rows, HBM-write-bound at 4·n_features bytes
    per (s, f, j) row on top of its curve bytes, against the HBM peak and the
    measured copy; then the generic row kernel (tl_forest_predict, every tree
    walked from the root for every row) on the first `sample_rows` rows,
    checked against the grid path's IPS of the same rows."""
    import torch

    from paper_2408_05235_amd import api
    S, H, F, nf = inp["n_scenarios"], inp["horizon"], inp["n_freqs"], inp["n_features"]
    rows = S * F * H
    mctl = api.Controller(dev_in, forest, materialize_rows=True)
    mctl.project()
    torch.cuda.synchronize()
    ev = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        mctl.project()
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    byt = algorithmic_bytes(inp, F, rows)["project"] + rows * nf * 4
    n = min(sample_rows, rows)
    x = mctl.buf["rows"].view(-1, nf)[:n]
    out = torch.empty(n, dtype=torch.float32, device="cuda:0")
    forest.tl_forest_predict(x, out)
    torch.cuda.synchronize()
    same = bool(torch.equal(out, ctl.ips.view(-1)[:n]))
    ev = []
    for _ in range(max(1, steps // 2)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        forest.tl_forest_predict(x, out)
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    pms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del mctl, x, out
    torch.cuda.empty_cache()
    gbs = byt / (ms / 1e3) / 1e9
    return {"rows_bytes": rows * nf * 4, "project_ms": ms, "project_gbs": gbs, "frac_of_hbm_peak": gbs / HBM_PEAK_GBS,
            "frac_of_copy": gbs / copy_gbs,
            "row_kernel": {"rows": n, "ms": pms, "rows_per_s": n / (pms / 1e3), "same_ips_as_grid": same}}


LATTICE_FILE = os.path.join(ROOT, "profiles", "lattice_{}_traffic.json")


def lattice_bench(inp, cfg, ctl, steps, warmup, admission=None, max_gib=24):
    """The model compiled to its input lattice (a separate mode, not the
    headline): one-time build over (engine sizes x batch 0..max x the F
    frequencies x KV 0..capacity), then the step's prediction as a table
    lookup with identical values.  Reports the build time, the lookup's
    HIP-event time, the step with it (project + lookup + select), and the
    lookup kernel's HBM roofline (algorithmic bytes: 4 written + 4 read per
    row, 8 per (scenario, iteration)).  The binary search and, when
    `admission` is given (a function of the lattice), admission control are
    timed again with M read from the table.  Batch bound: the step's largest
    batch plus one, the batch a what-if query can add."""
    import torch

    from paper_2408_05235_amd import api
    S, H, F = inp["n_scenarios"], inp["horizon"], inp["n_freqs"]
    kv_max = int(cfg["kv_capacity"])
    b_max = int(ctl.buf["batch"].max().item()) + 1
    engines = [1.0, 2.0, 4.0, 8.0] if inp["n_features"] == 4 else None
    n_e = len(engines) if engines else 1
    gib = n_e * (b_max + 1) * F * 4096 * (kv_max // 4096 + 1) * 4 / 2 ** 30
    if gib > max_gib:
        return {"skipped": f"table would take {gib:.1f} GiB (bench limit {max_gib})"}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    lat = api.Lattice(ctl.forest, ctl.d["freqs_mhz"], kv_max, b_max, engines)
    torch.cuda.synchronize()
    build_s = time.perf_counter() - t0
    out = torch.empty_like(ctl.ips)
    call = lambda: lat.tl_lattice_predict_grid(ctl.buf["kv"], ctl.buf["batch"], ctl.d["engine_size"], out)
    for _ in range(max(1, warmup)):
        call()
    torch.cuda.synchronize()
    same = bool(torch.equal(out, ctl.ips))
    ev = []
    for _ in range(steps):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record()
        ctl.project()
        e[1].record()
        call()
        e[2].record()
        tl_sel = api.tl_select_freq(out, ctl.buf["deadline_at"], ctl.buf["n_iters"], ctl.d["tbt_slo_ns"],
                                    ctl.buf["flags"], ctl.sel)
        e[3].record()
        ev.append(e)
    torch.cuda.synchronize()
    st = np.array([[x[i].elapsed_time(x[i + 1]) for i in range(3)] for x in ev])
    step_ms = float(np.median(st.sum(axis=1)))
    look_ms = float(np.median(st[:, 1]))
    rows = S * F * H
    byt = 8 * rows + 8 * S * H
    achieved = byt / (look_ms / 1e3) / 1e9
    traffic = traffic_record(LATTICE_FILE.format(cfg["name"].split("_")[0]))
    # the binary search with M read from the table
    for _ in range(max(1, warmup)):
        ctl.select_binary(lat)
    torch.cuda.synchronize()
    ev_b = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ctl.select_binary(lat)
        e1.record()
        ev_b.append((e0, e1))
    torch.cuda.synchronize()
    bin_ms = float(np.median([a.elapsed_time(b) for a, b in ev_b]))
    res = {"table_gib": lat.nbytes / 2 ** 30, "build_s": build_s, "bounds": {"kv_max": kv_max, "batch_max": b_max},
           "binary_search_ms": bin_ms,
           "admission": admission(lat) if admission else None,
           "lookup_ms": look_ms, "step_ms": step_ms, "rows_per_s": rows / (step_ms / 1e3),
           "same_ips_as_direct": same,
           "roofline": {"kernel": "lattice_gather_kernel", "bound": "hbm", "achieved": achieved,
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic}}
    lat.close()
    return res


def search_evaluations(freq_idx, status, F):
    """Model evaluations per scenario of one binary search (Sec. 4.5) as the
    library runs it, from its results: a searched scenario ends with lo ==
    hi == its index, which fixes every probe's outcome (feasible iff the index
    is at most the probe), hence the number of probes, plus the check of lo
    when hi stayed at F-1; scenarios settled by their flags (lost, invalid)
    evaluate nothing."""
    out = np.zeros(len(freq_idx), np.int64)
    for k, (v, st) in enumerate(zip(np.asarray(freq_idx).tolist(), np.asarray(status).tolist())):
        if st >= 2:
            continue
        lo, hi, n = 0, F - 1, 0
        while lo < hi:
            mid = lo + (hi - lo) // 2
            n += 1
            if v <= mid:
                hi = mid
            else:
                lo = mid + 1
        out[k] = n + (hi == F - 1)
    return out


def binary_search_bench(ctl, steps, warmup):
    """The controller as the paper states it (Sec. 4.5): binary search over the
    frequencies, the model evaluated only at probed frequencies, on the
    projection of the last timed step; timed with HIP events, and compared
    with the exhaustive selection of that step (the two agree wherever
    feasibility is monotone in the frequency)."""
    import torch
    for _ in range(max(1, warmup)):
        ctl.select_binary()
    torch.cuda.synchronize()
    ev = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        idx, st = ctl.select_binary()
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    bi, ei = idx.cpu().numpy(), ctl.sel["freq_idx"].cpu().numpy()
    S, H = ctl.d["n_scenarios"], ctl.d["horizon"]
    F = ctl.d["freqs_mhz"].numel()
    probes = int(np.ceil(np.log2(F))) + 1 if F > 1 else 1
    evals = int(search_evaluations(bi, st.cpu().numpy(), F).sum())
    return {"ms_mean": float(ms.mean()), "ms_median": float(np.median(ms)), "ms_min": float(ms.min()),
            "rows_evaluated_per_call": H * evals, "rows_evaluated_bound": S * H * probes,
            "scenarios_per_s": S / (ms.mean() / 1e3), "same_index_as_exhaustive": float((bi == ei).mean())}


def admission_bench(inp, cfg, dev_in, forest, steps, warmup, lattice=None):
    """Admission control (Sec. 4.3.2) of one new query per scenario of the same
    workload: projection with the query, the model at the maximum frequency on
    every projected iteration, checks 1-3 (one tl_admit call), timed like the
    step with HIP events on the launch stream."""
    import torch

    from paper_2408_05235_amd import api, synth
    cand = synth.make_candidates(cfg, inp)
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dt).view(np.int64 if dt == np.uint64 else dt)).cuda()
    cp, cl, cd = t(cand["cand_prompt"], np.int32), t(cand["cand_len"], np.int32), t(cand["cand_deadline_ns"], np.uint64)
    d = dev_in
    fmax = float(inp["freqs_mhz"][-1])
    res = None

    def call():
        nonlocal res
        res = api.tl_admit(forest, fmax, d["tbt_slo_ns"], cp, cl, d["req_offset"], d["prompt"], d["generated"],
                           d["remaining"], d["arrival"], d["kv_capacity"], d["horizon"], d["block_tokens"],
                           d["deadline_ns"], d["lost"], d["batch_cap"], d["engine_size"], cd, res, lattice=lattice)

    for _ in range(max(1, warmup)):
        call()
    torch.cuda.synchronize()
    ms = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        call()
        e1.record()
        ms.append((e0, e1))
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in ms])
    S, H = inp["n_scenarios"], inp["horizon"]
    dec = np.bincount(res["decision"].cpu().numpy(), minlength=6)
    return {"what_ifs": S, "ms_mean": float(ms.mean()), "ms_median": float(np.median(ms)), "ms_min": float(ms.min()),
            "what_ifs_per_s": S / (ms.mean() / 1e3), "rows_per_s": S * H / (ms.mean() / 1e3),
            "decisions": dict(zip(("admit", "admit_lost", "queue_capacity", "queue_tbt", "queue_e2e", "invalid"),
                                  dec.tolist()))}


def _clock_record():
    """Clock state of the first AMD GPU as the driver reports it in sysfs
    (clocks are left at their defaults): performance level and the current
    shader / memory clock levels.  Read from files; no other program runs."""
    import glob
    out = {}
    for dev in sorted(glob.glob("/sys/class/drm/card*/device")):
        try:
            if open(os.path.join(dev, "vendor")).read().strip() != "0x1002":
                continue
        except OSError:
            continue
        for name in ("power_dpm_force_performance_level", "pp_dpm_sclk", "pp_dpm_mclk"):
            try:
                lines = open(os.path.join(dev, name)).read().split("\n")
            except OSError as e:
                out[name] = f"unreadable: {e.strerror}"
                continue
            cur = [ln.strip() for ln in lines if ln.strip().endswith("*")]
            out[name] = (cur[0] if cur else " ".join(ln.strip() for ln in lines if ln.strip()))[:120]
        break
    return out or {"error": "no AMD GPU in /sys/class/drm"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="c3")
    ap.add_argument("--lattice-max-gib", type=float, default=24,
                    help="largest model table the lattice mode builds (larger ones are reported as skipped)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-procs", type=int, default=min(16, len(os.sched_getaffinity(0))),
                    help="processes for the sharded oracle run (0 or 1: single thread only)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy a buffer of this size once (a known-size "
                         "kernel for scaling hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(scenarios are independent: shard them across GPUs, one process each)", file=sys.stderr)
        sys.exit(2)

    from paper_2408_05235_amd import configs, synth

    cfg = configs.get_config(args.config)
    t0 = time.perf_counter()
    inp = synth.make_inputs(cfg)
    log(f"inputs {cfg['name']}: {time.perf_counter() - t0:.1f}s, {int(inp['req_offset'][-1])} requests")
    # host-side work that starts other processes runs before the GPU is touched
    cpu_base = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        cpu_base = cpu_baseline(inp, procs=args.cpu_procs)
    clocks = _clock_record()

    import torch

    from paper_2408_05235_amd import api

    torch.cuda.set_device(0)
    dev_in = api.upload(inp, "cuda:0")
    forest = api.Forest.from_dict(inp["forest"])
    ctl = api.Controller(dev_in, forest)
    S, H, F = inp["n_scenarios"], inp["horizon"], inp["n_freqs"]
    rows = S * F * H
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        ctl.step()
    torch.cuda.synchronize()
    log("warmup done")

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        e = ev[k]
        e[0].record()
        ctl.project()
        e[1].record()
        ctl.predict()
        e[2].record()
        ctl.select()
        e[3].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    log(f"timed {args.steps} steps in {wall:.2f}s")
    copy_gbs = copy_bandwidth_gbs()

    st = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(3)] for e in ev])  # ms
    step_ev = np.array([e[0].elapsed_time(e[3]) for e in ev])
    stage_ms = st.mean(axis=0)
    step_ms = wall * 1e3 / args.steps
    byt = algorithmic_bytes(inp, F, rows, (ctl.sel["freq_idx"].cpu().numpy(), ctl.sel["status"].cpu().numpy(),
                                           np.clip(ctl.buf["n_iters"].cpu().numpy(), 0, H)))
    tot_bytes = sum(byt.values())

    f = inp["forest"]
    # algorithmic work of the forest stage: every (row, tree) pair needs at
    # least its leaf accumulated (one fp32 add); walks that leaf reuse avoids
    # are not counted, so this is the floor any implementation must execute
    ops_per_row = f["n_trees"]
    forest_s = stage_ms[1] / 1e3
    achieved = ops_per_row * rows / forest_s / 1e12
    traffic = traffic_record(os.path.join(ROOT, "profiles", f"forest_{cfg['name'].split('_')[0]}_traffic.json"))

    out = {
        "metric": METRIC,
        "value": rows / (step_ms / 1e3),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg["name"], "scenarios": S, "horizon": H, "freqs": F,
                   "rows_per_step": rows, "trees": f["n_trees"], "depth": f["depth"],
                   "features": inp["n_features"], "requests": int(inp["req_offset"][-1])},
        "scenarios_per_s": S / (step_ms / 1e3),
        "hbm_frac_end_to_end": tot_bytes / (step_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
        "hbm_copy_gbs_measured": copy_gbs,
        "stages_ms": {"project": stage_ms[0], "predict": stage_ms[1], "select": stage_ms[2]},
        "stages_ms_median": dict(zip(("project", "predict", "select"), np.median(st, axis=0).tolist())),
        "stages_ms_min": dict(zip(("project", "predict", "select"), st.min(axis=0).tolist())),
        "step_ms_events": {"median": float(np.median(step_ev)), "min": float(step_ev.min())},
        "gpu": {"name": torch.cuda.get_device_properties(0).name,
                "compute_units": torch.cuda.get_device_properties(0).multi_processor_count,
                "clocks": clocks},
        "stage_hbm_gbs": {k: byt[k] / (v / 1e3) / 1e9 for k, v in
                          zip(("project", "predict", "select"), stage_ms)},
        "forest_rows_per_s": rows / forest_s,
        "forest_node_visits_per_s_equiv": rows * f["n_trees"] * f["depth"] / forest_s,
        "roofline": {"kernel": FOREST_KERNEL, "bound": "alu", "achieved": achieved,
                     "peak": VALU_PEAK_TOPS, "unit": "Tops/s", "frac": achieved / VALU_PEAK_TOPS,
                     "traffic": traffic, "ops_per_row": ops_per_row,
                     "ops_note": "one fp32 leaf add per (row, tree); peak = non-packed VALU lane ops"},
    }
    out["results_d2h_ms"] = d2h_results_ms(ctl)
    out["adjust_lengths"] = adjust_lengths_bench(inp, dev_in, args.steps, copy_gbs)
    log("length stage done")
    out["materialized_rows"] = materialized_rows_bench(inp, dev_in, forest, ctl, args.steps, copy_gbs)
    log("materialized rows done")
    out["lattice"] = lattice_bench(inp, cfg, ctl, args.steps, args.warmup,
                                   lambda lat: admission_bench(inp, cfg, dev_in, forest, args.steps, args.warmup, lat),
                                   max_gib=args.lattice_max_gib)
    log("lattice mode done")
    out["binary_search"] = binary_search_bench(ctl, args.steps, args.warmup)
    log("binary search done")
    out["admission"] = admission_bench(inp, cfg, dev_in, forest, args.steps, args.warmup)
    log("admission done")
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = n * 4
        del src, dst
    parity_ok = True
    if cpu_base is not None:
        out["cpu_baseline"] = cpu_base
        out["cpu_baseline"]["parity"] = oracle_parity(ctl, cpu_base.pop("_results"))
        parity_ok = out["cpu_baseline"]["parity"]["ok"]
    forest.close()
    print(json.dumps(out), flush=True)
    if not parity_ok:
        log("the timed step's results differ from the oracle's on the baseline scenarios")
        sys.exit(1)


if __name__ == "__main__":
    main()
