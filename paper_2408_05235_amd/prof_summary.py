"""Summarize rocprofv3 CSV output into the short text files kept in profiles/.

    python -m paper_2408_05235_amd.prof_summary stats  <kernel_stats.csv> <out.md> <command>
    python -m paper_2408_05235_amd.prof_summary trace  <kernel_trace.csv> <out.md> <command>
    python -m paper_2408_05235_amd.prof_summary traffic <fetch_counter_collection.csv> \
        <write_counter_collection.csv> <kernel substring> <copy bytes> <out.json> <command>

    python -m paper_2408_05235_amd.prof_summary counters <out.md> <kernel substring> <command> \
        <counter_collection.csv> [<counter_collection.csv> ...]

`traffic` turns FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the first
dispatch of one kernel into bytes per launch, each scaled by what the same counter reads for the last
copy dispatch of the run, a copy of known size (the counters' byte formulas
need not match the request sizes a kernel uses).

`counters` takes every counter of the given runs at the first dispatch of one
kernel (the timed step's) and derives the rates kept beside the kernel statistics: LDS bank
conflict cycles per cycle of indexed LDS activity, and per LDS instruction.
L2 hit rate from TCC_HIT and TCC_MISS (rocprofv3 has no L2CacheHit for gfx950).
Derived counters that rocprofv3 computes itself (VALUBusy, VALUUtilization,
both percentages) are reported as it gives them.
"""
from __future__ import annotations

import csv
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))


def _short(name):
    if "rocprim" in name:
        # library sort kernels: keep the stage name of the config
        import re
        m = re.search(r"wrapped_([a-z_]+?)_config", name)
        return "rocprim " + (m.group(1) if m else "kernel") + " (radix sort of the work order)"
    return name.replace("tl::(anonymous namespace)::", "").replace("void ", "").split("(")[0]


def kernel_stats(csv_path, out_md, command, title=""):
    rows = list(csv.DictReader(open(csv_path)))
    lines = [f"# {title or 'rocprofv3 kernel statistics'}", "", "Command:", "", "```", command, "```", "",
             "| kernel | calls | average ms | min ms | max ms | share |", "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {_short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e6:.3f} | "
                     f"{float(r['MinNs']) / 1e6:.3f} | {float(r['MaxNs']) / 1e6:.3f} | "
                     f"{float(r['Percentage']):.2f}% |")
    open(out_md, "w").write("\n".join(lines) + "\n")
    return rows


def trace_stats(trace_csv, out_md, command, title=""):
    """Kernel statistics from a kernel trace, one line per (kernel, launch
    grid): launches of one kernel at different sizes (the controller step and
    a lattice build, say) are kept apart."""
    groups = {}
    for r in csv.DictReader(open(trace_csv)):
        grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
        wg = int(r["Workgroup_Size_X"]) * int(r["Workgroup_Size_Y"]) * int(r["Workgroup_Size_Z"])
        ns = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        groups.setdefault((r["Kernel_Name"], grid // max(wg, 1), wg), []).append(ns)
    total = sum(sum(v) for v in groups.values())
    rows = sorted(groups.items(), key=lambda kv: -sum(kv[1]))
    lines = [f"# {title or 'rocprofv3 kernel statistics'}", "", "Command:", "", "```", command, "```", "",
             "| kernel | workgroups x threads | calls | average ms | min ms | max ms | share |",
             "|---|---|---|---|---|---|---|"]
    for (name, n_wg, wg), v in rows:
        lines.append(f"| {_short(name)} | {n_wg} x {wg} | {len(v)} | {sum(v) / len(v) / 1e6:.3f} | "
                     f"{min(v) / 1e6:.3f} | {max(v) / 1e6:.3f} | {100.0 * sum(v) / total:.2f}% |")
    open(out_md, "w").write("\n".join(lines) + "\n")
    return rows


def _per_dispatch(csv_path, counter):
    out = []
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] == counter:
            out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    agg = {}
    for d, k, v in out:
        agg.setdefault(d, [k, 0.0])[1] += v
    return [(d, k, v) for d, (k, v) in sorted(agg.items())]


# the sources each profiled kernel is built from: a traffic record is used
# only while all of them still hash the same
KERNEL_SOURCES = {
    "forest_grid_lds": ["forest.hip", "forest_walk.h", "tl_internal.h", "record_format.h", "device_util.h",
                        "host_forest.cpp", "api.cpp"],
    "lattice_gather": ["lattice.hip", "tl_internal.h", "record_format.h", "device_util.h", "api.cpp"],
}


def sources_sha256(names):
    h = hashlib.sha256()
    for n in names:
        h.update(n.encode())
        h.update(open(os.path.join(PKG, "csrc", n), "rb").read())
    return h.hexdigest()


def traffic(fetch_csv, write_csv, kernel, copy_bytes, out_json, command):
    res = {}
    for name, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        disp = _per_dispatch(path, counter)
        copies = [v for d, k, v in disp if "copyBuffer" in k]
        if not copies:
            raise SystemExit(f"no copy dispatch in {path}")
        scale = copy_bytes / (copies[-1] * 1024.0)
        vals = [v for d, k, v in disp if kernel in k]
        if not vals:
            raise SystemExit(f"no dispatch of {kernel} in {path}")
        # the first dispatch: the timed step's (later ones may be other uses
        # of the same kernel, such as building a lattice table)
        res[name] = dict(kib_per_launch=vals[0], copy_kib=copies[-1], scale=scale,
                         bytes_per_launch=vals[0] * 1024.0 * scale)
    names = KERNEL_SOURCES[kernel]
    rec = dict(kernel=kernel, command=command, copy_bytes=copy_bytes,
               fetch=res["fetch"], write=res["write"],
               bytes_per_launch=res["fetch"]["bytes_per_launch"] + res["write"]["bytes_per_launch"],
               sources=names, sources_sha256=sources_sha256(names))
    json.dump(rec, open(out_json, "w"), indent=1)
    return rec


def counters(out_md, kernel, command, csv_paths):
    vals = {}
    names = set()
    for path in csv_paths:
        for r in csv.DictReader(open(path)):
            if kernel not in r["Kernel_Name"]:
                continue
            names.add(r["Kernel_Name"])
            key = (r["Counter_Name"], path, int(r["Dispatch_Id"]))
            vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
    if not vals:
        raise SystemExit(f"no dispatch of {kernel} in {csv_paths}")
    # the first dispatch of each run: the timed step's (later ones may be
    # other uses of the kernel, such as building a lattice table)
    first = {}
    for (c, path, d) in sorted(vals):
        first.setdefault((c, path), d)
    vals = {k: v for k, v in vals.items() if first[(k[0], k[1])] == k[2]}
    per = {}
    for (c, _, _), v in vals.items():
        per.setdefault(c, []).append(v)
    avg = {c: sum(v) / len(v) for c, v in per.items()}
    n_disp = {c: len(v) for c, v in per.items()}
    lines = [f"# rocprofv3 counters of {_short(sorted(names)[0])}", "", "Command:", "", "```", command, "```", "",
             "| counter | dispatches | average per dispatch |", "|---|---|---|"]
    for c in sorted(avg):
        lines.append(f"| {c} | {n_disp[c]} | {avg[c]:.6g} |")
    derived = []
    if "SQ_LDS_BANK_CONFLICT" in avg and avg.get("SQ_LDS_IDX_ACTIVE"):
        derived.append(("LDS bank-conflict cycles / indexed-LDS-active cycles",
                        avg["SQ_LDS_BANK_CONFLICT"] / avg["SQ_LDS_IDX_ACTIVE"]))
    if "SQ_LDS_BANK_CONFLICT" in avg and avg.get("SQ_INSTS_LDS"):
        derived.append(("LDS bank-conflict cycles per LDS instruction",
                        avg["SQ_LDS_BANK_CONFLICT"] / avg["SQ_INSTS_LDS"]))
    if avg.get("TCC_HIT_sum", 0) + avg.get("TCC_MISS_sum", 0) > 0:
        derived.append(("L2 hit rate, % (TCC_HIT / (TCC_HIT + TCC_MISS))",
                        100.0 * avg["TCC_HIT_sum"] / (avg["TCC_HIT_sum"] + avg["TCC_MISS_sum"])))
    if derived:
        lines += ["", "| derived | value |", "|---|---|"]
        lines += [f"| {k} | {v:.4g} |" for k, v in derived]
    open(out_md, "w").write("\n".join(lines) + "\n")
    return avg, derived


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        trace_stats(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5] if len(sys.argv) > 5 else "")
    elif sys.argv[1] == "stats":
        kernel_stats(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5] if len(sys.argv) > 5 else "")
    elif sys.argv[1] == "traffic":
        print(json.dumps(traffic(sys.argv[2], sys.argv[3], sys.argv[4], int(sys.argv[5]), sys.argv[6],
                                 sys.argv[7]), indent=1))
    elif sys.argv[1] == "counters":
        print(counters(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5:]))
    else:
        raise SystemExit(__doc__)
