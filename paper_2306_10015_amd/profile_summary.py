"""Summarise rocprofv3 CSV output of one kernel into the short text files kept
under profiles/ (measurement tooling; not used by the engine).

    python -m paper_2306_10015_amd.profile_summary --name engine_kernel_opt6.7b \\
        --unit engine_dense.hip --kernel engine_kernel \\
        --trace out/trace --fetch out/fetch --write out/write \\
        --copy-fetch out/copy_fetch --copy-write out/copy_write --valu out/valu \\
        --elements 6648897536 --elem-bytes 2 --records 1,1,1,64,256 --commands cmds.txt

(each directory being the -d output of one rocprofv3 run: see the commands
listed at the top of every summary).

FETCH_SIZE and WRITE_SIZE are scaled by what the same counters read for a
plain device copy of known size (--copy-*), per dispatch. VALU busy follows
rocprofv3's derived metric, 100 * SQ_ACTIVE_INST_VALU / CUs / GRBM_GUI_ACTIVE
cycles, with GRBM_GUI_ACTIVE summed over the 8 XCDs in the CSV; it counts a
cycle in which a second VALU instruction issued beside the first (a
transcendental on its own unit) twice, so it exceeds 100 where instructions
co-issue: the main pipe's busy share is that figure times (1 - the
SQ_ACTIVE_INST_VALU2 share). GRBM_GUI_ACTIVE per XCD over the dispatch's
duration is the clock it ran at (exact for long dispatches; the counted run's
durations of short ones include collection overhead). Instruction
counts are per lane: SQ_INSTS_VALU counts wave instructions, times 64 lanes,
over the elements (x records for the engine) of the dispatch; transcendental
ones (SQ_INSTS_VALU_TRANS_F32) are given apart, since they issue on a unit of
their own.

The summary is stamped with a hash of the kernel's translation unit and every
header it includes (directly or not): a later change to any of those files
makes the figures stale, and bench.py then stops quoting them.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2306_10015_amd", "csrc")
CUS, XCDS = 256, 8
_INCLUDE = re.compile(r'^\s*#\s*include\s+"([^"]+)"', re.M)


def unit_sources(unit: str) -> list[str]:
    """The translation unit csrc/<unit> and every header of this repository it
    includes, directly or through other headers (repository-relative paths,
    sorted)."""
    seen: set[str] = set()
    todo = [os.path.normpath(os.path.join(CSRC, unit))]
    while todo:
        path = todo.pop()
        if path in seen:
            continue
        seen.add(path)
        with open(path) as f:
            text = f.read()
        for inc in _INCLUDE.findall(text):
            cand = os.path.normpath(os.path.join(os.path.dirname(path), inc))
            if os.path.exists(cand):
                todo.append(cand)
    return sorted(os.path.relpath(p, ROOT) for p in seen)


def source_hash(unit: str) -> str:
    """sha256 over the unit's sources (unit_sources order: path, then bytes)."""
    h = hashlib.sha256()
    for rel in unit_sources(unit):
        h.update(rel.encode() + b"\0")
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def one(d: str, suffix: str) -> str:
    hits = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
    if not hits:
        raise FileNotFoundError(f"no *{suffix} under {d}")
    return hits[0]


def dispatches(d: str, name_filter: str | None = None):
    out = collections.OrderedDict()
    for r in csv.DictReader(open(one(d, "counter_collection.csv"))):
        if name_filter and not re.search(name_filter, r["Kernel_Name"]):
            continue
        k = int(r["Dispatch_Id"])
        e = out.setdefault(k, {"name": r["Kernel_Name"], "grid": int(r["Grid_Size"]),
                               "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
        e[r["Counter_Name"]] = float(r["Counter_Value"])
    return out


def biggest(dis: dict, counter: str) -> float:
    return max(e[counter] for e in dis.values())


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--name", required=True)
    ap.add_argument("--unit", required=True, help="translation unit under csrc/ the kernel is compiled from")
    ap.add_argument("--kernel", required=True, help="regular expression selecting the kernel's dispatches")
    ap.add_argument("--trace")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--valu")
    ap.add_argument("--elements", type=int, required=True, help="elements one dispatch processes")
    ap.add_argument("--elem-bytes", type=float, required=True,
                    help="storage bytes per element (NF4: 0.5625 = half a code byte + 4/64 of an absmax)")
    ap.add_argument("--alg-bytes", type=float,
                    help="algorithmic bytes per dispatch (default: elements x elem-bytes read and written)")
    ap.add_argument("--copy-bytes", type=float,
                    help="bytes each way of the copy probe's dispatch (default: half the algorithmic bytes)")
    ap.add_argument("--records", default="", help="records per dispatch, cycling (e.g. 1,1,1,64,256); "
                                                  "empty for kernels without records (per element)")
    ap.add_argument("--timed", default="",
                    help="A:B — the kernel's dispatches A .. B-1 of the traced run (in launch order) are the "
                         "bench's timed region: their average duration is reported apart")
    ap.add_argument("--bench-json", help="the JSON line bench.py printed in the traced run")
    ap.add_argument("--commands", help="text file with the commands that made the inputs")
    ap.add_argument("--outdir", default=os.path.join(ROOT, "profiles"))
    a = ap.parse_args()
    alg = round(a.alg_bytes if a.alg_bytes else 2 * a.elements * a.elem_bytes)
    lines = [f"# {a.name}", ""]
    summary = {"kernel": a.kernel, "kernel_unit": a.unit, "kernel_sources": unit_sources(a.unit),
               "kernel_source_sha256": source_hash(a.unit), "alg_bytes_per_dispatch": alg,
               "elements_per_dispatch": a.elements}
    if a.commands:
        lines += ["Commands (run from the repository root on an MI355X machine):", "", "```"]
        lines += [l.rstrip() for l in open(a.commands) if l.strip()]
        lines += ["```", ""]
    if a.trace:
        lines += ["## Kernel trace (rocprofv3 --kernel-trace --stats)", "",
                  "| kernel | calls | average ns | min ns | max ns | % time |", "|---|---|---|---|---|---|"]
        for r in csv.DictReader(open(one(a.trace, "kernel_stats.csv"))):
            name = r["Name"] if len(r["Name"]) <= 100 else r["Name"][:80] + " ..."
            lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']):.0f} | "
                         f"{r['MinNs']} | {r['MaxNs']} | {float(r['Percentage']):.2f} |")
            if re.search(a.kernel, r["Name"]):
                summary.setdefault("trace_average_ns", {})[r["Name"]] = float(r["AverageNs"])
        lines.append("")
        if a.timed:
            lo, hi = (int(x) for x in a.timed.split(":"))
            rows = [r for r in csv.DictReader(open(one(a.trace, "kernel_trace.csv")))
                    if re.search(a.kernel, r["Kernel_Name"])]
            rows.sort(key=lambda r: int(r["Start_Timestamp"]))
            sel = rows[lo:hi]
            ns = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in sel]
            avg = sum(ns) / len(ns)
            summary["timed_region"] = {"dispatches": f"{lo}:{hi}", "average_ns": avg}
            lines += [f"Timed region of the traced bench run: the kernel's dispatches {lo}..{hi - 1} in launch "
                      f"order ({len(ns)} dispatches) average **{avg:.0f} ns** "
                      f"(min {min(ns)}, max {max(ns)})."]
            if a.bench_json:
                bj = json.loads(open(a.bench_json).read().strip().splitlines()[-1])
                rl = bj["roofline"]
                lines += [f"The same run's bench line: avg_launch_ms {rl['avg_launch_ms']:.4f} "
                          f"(HIP events over the timed region / launches), "
                          f"ms_per_step {bj['ms_per_step']:.3f}, value {bj['value']:.4g} {bj['unit']}; "
                          f"trace / events = {avg / 1e6 / rl['avg_launch_ms']:.4f}."]
                summary["timed_region"]["bench_avg_launch_ms"] = rl["avg_launch_ms"]
            lines.append("")
    if a.fetch and a.write and a.copy_fetch and a.copy_write:
        f = dispatches(a.fetch, a.kernel)
        w = dispatches(a.write, a.kernel)
        cf = dispatches(a.copy_fetch)
        cw = dispatches(a.copy_write)
        # the copy probe moves a buffer of known size: the largest dispatch is it
        cf_kib = biggest(cf, "FETCH_SIZE")
        cw_kib = biggest(cw, "WRITE_SIZE")
        copy_bytes_each = a.copy_bytes or alg / 2  # read this many, write this many
        fscale = copy_bytes_each / (cf_kib * 1024)
        wscale = copy_bytes_each / (cw_kib * 1024)
        fk = [e["FETCH_SIZE"] for e in f.values()]
        wk = [e["WRITE_SIZE"] for e in w.values()]
        fb = sum(fk) / len(fk) * 1024 * fscale
        wb = sum(wk) / len(wk) * 1024 * wscale
        summary.update({"fetch_kib_raw": sum(fk) / len(fk), "write_kib_raw": sum(wk) / len(wk),
                        "fetch_scale": fscale, "write_scale": wscale,
                        "hbm_bytes_per_dispatch": fb + wb, "traffic_over_alg": (fb + wb) / alg})
        lines += ["## HBM traffic per dispatch (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE)", "",
                  f"- plain copy of a buffer ({copy_bytes_each / 1e6:.2f} MB each way): "
                  f"FETCH_SIZE {cf_kib:.0f} KiB, WRITE_SIZE {cw_kib:.0f} KiB -> scale factors "
                  f"fetch x{fscale:.3f}, write x{wscale:.3f}",
                  f"- kernel dispatches: {len(fk)}; FETCH_SIZE {min(fk):.0f}..{max(fk):.0f} KiB raw, "
                  f"WRITE_SIZE {min(wk):.0f}..{max(wk):.0f} KiB raw",
                  f"- scaled: read {fb / 1e6:.2f} MB + write {wb / 1e6:.2f} MB = {(fb + wb) / 1e6:.2f} MB "
                  f"per dispatch; algorithmic {alg / 1e6:.2f} MB (ratio {(fb + wb) / alg:.4f})", ""]
    if a.valu:
        v = dispatches(a.valu, a.kernel)
        recs = [int(x) for x in a.records.split(",")] if a.records else []
        per = "param-seed" if recs else "element"
        lines += ["## VALU (rocprofv3 --pmc SQ_ACTIVE_INST_VALU SQ_INSTS_VALU SQ_ACTIVE_INST_VALU2 "
                  "SQ_INSTS_VALU_TRANS_F32 ... GRBM_GUI_ACTIVE)", "",
                  f"| dispatch | records | ns | GHz | VALU busy % | dual-issue share % | main pipe busy % | "
                  f"VALU instr per {per} | of them transcendental | non-transcendental |",
                  "|---|---|---|---|---|---|---|---|---|---|"]
        rows = []
        for i, (k, e) in enumerate(v.items()):
            cyc = e["GRBM_GUI_ACTIVE"] / XCDS
            busy = 100 * e["SQ_ACTIVE_INST_VALU"] / CUS / cyc
            dual = 100 * e.get("SQ_ACTIVE_INST_VALU2", 0) / max(e["SQ_ACTIVE_INST_VALU"], 1)
            r = recs[i % len(recs)] if recs else 0
            units = a.elements * (r if recs else 1)
            ips = e["SQ_INSTS_VALU"] * 64 / units
            tps = e.get("SQ_INSTS_VALU_TRANS_F32", 0.0) * 64 / units
            ghz = cyc / e["ns"]
            rows.append((r, busy, dual, ips, tps, ghz))
            lines.append(f"| {k} | {r if recs else '-'} | {e['ns']} | {ghz:.2f} | {busy:.1f} | {dual:.1f} | "
                         f"{busy * (1 - dual / 100):.1f} | {ips:.3f} | {tps:.3f} | {ips - tps:.3f} |")
        lines.append("")
        by = collections.defaultdict(list)
        for r, busy, dual, ips, tps, ghz in rows:
            by[r].append((busy, dual, ips, tps, ghz))
        summary["valu_by_records"] = {
            str(r): {"busy_pct": sum(x[0] for x in vals) / len(vals),
                     "dual_issue_pct": sum(x[1] for x in vals) / len(vals),
                     "main_pipe_busy_pct": sum(x[0] * (1 - x[1] / 100) for x in vals) / len(vals),
                     "clock_ghz": sum(x[4] for x in vals) / len(vals),
                     f"instr_per_{per.replace('-', '_')}": sum(x[2] for x in vals) / len(vals),
                     f"trans_per_{per.replace('-', '_')}": sum(x[3] for x in vals) / len(vals)}
            for r, vals in by.items()}
    lines += [f"Kernel `{a.kernel}` compiled from `{a.unit}`; sources "
              + ", ".join(f"`{s}`" for s in summary["kernel_sources"]) + ".", "",
              f"Kernel sources sha256: `{summary['kernel_source_sha256']}`", ""]
    os.makedirs(a.outdir, exist_ok=True)
    with open(os.path.join(a.outdir, a.name + ".md"), "w") as fh:
        fh.write("\n".join(lines))
    with open(os.path.join(a.outdir, a.name + ".json"), "w") as fh:
        json.dump(summary, fh, indent=1)
    print("\n".join(lines))


if __name__ == "__main__":
    main()
