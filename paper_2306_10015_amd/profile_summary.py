"""Summarise rocprofv3 CSV output of the engine into the short text files kept
under profiles/ (measurement tooling; not used by the engine).

    python -m paper_2306_10015_amd.profile_summary --name engine_kernel_opt125m \\
        --trace out/prof_trace --fetch out/prof_fetch \\
        --write out/prof_write --copy-fetch out/prof_copy_fetch \\
        --copy-write out/prof_copy_write --valu out/prof_valu \\
        --elements 123581952 --elem-bytes 4 --records 1,1,1,8,32 --commands cmds.txt

(each directory being the -d output of one rocprofv3 run: see the commands
listed at the top of every summary).

FETCH_SIZE and WRITE_SIZE are scaled by what the same counters read for a
plain device copy of known size (--copy-*), per dispatch. VALU busy follows
rocprofv3's derived metric, 100 * SQ_ACTIVE_INST_VALU / CUs / GRBM_GUI_ACTIVE
cycles, with GRBM_GUI_ACTIVE summed over the 8 XCDs in the CSV.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL_SOURCES = ["paper_2306_10015_amd/csrc/kernels.hip", "paper_2306_10015_amd/csrc/engine.hpp",
                  "paper_2306_10015_amd/csrc/records.hpp", "paper_2306_10015_amd/csrc/nf4.hpp",
                  "paper_2306_10015_amd/csrc/launch.hpp"]
CUS, XCDS = 256, 8


def source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
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
        if name_filter and name_filter not in r["Kernel_Name"]:
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
    ap.add_argument("--kernel", default="engine_kernel")
    ap.add_argument("--trace")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--valu")
    ap.add_argument("--elements", type=int, required=True)
    ap.add_argument("--elem-bytes", type=float, required=True,
                    help="storage bytes per element (NF4: 0.5625 = half a code byte + 4/64 of an absmax)")
    ap.add_argument("--copy-bytes", type=float,
                    help="bytes each way of the copy probe's dispatch (default: the engine's algorithmic read)")
    ap.add_argument("--records", default="", help="records per dispatch, cycling (e.g. 1,1,1,8,32)")
    ap.add_argument("--instr-per-param-seed", type=float, default=15.5)
    ap.add_argument("--commands", help="text file with the commands that made the inputs")
    ap.add_argument("--outdir", default=os.path.join(ROOT, "profiles"))
    a = ap.parse_args()
    alg = round(2 * a.elements * a.elem_bytes)
    lines = [f"# {a.name}", ""]
    summary = {"kernel_source_sha256": source_hash(), "alg_bytes_per_dispatch": alg}
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
        lines.append("")
    if a.fetch and a.write and a.copy_fetch and a.copy_write:
        f = dispatches(a.fetch, a.kernel)
        w = dispatches(a.write, a.kernel)
        cf = dispatches(a.copy_fetch)
        cw = dispatches(a.copy_write)
        copy_bytes_each = None
        # the copy probe moves the parameter buffer: the largest dispatch is it
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
                        "hbm_bytes_per_dispatch": fb + wb})
        lines += ["## HBM traffic per dispatch (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE)", "",
                  f"- plain copy of the same buffer ({copy_bytes_each / 1e6:.2f} MB each way): "
                  f"FETCH_SIZE {cf_kib:.0f} KiB, WRITE_SIZE {cw_kib:.0f} KiB -> scale factors "
                  f"fetch x{fscale:.3f}, write x{wscale:.3f}",
                  f"- engine dispatches: {len(fk)}; FETCH_SIZE {min(fk):.0f}..{max(fk):.0f} KiB raw, "
                  f"WRITE_SIZE {min(wk):.0f}..{max(wk):.0f} KiB raw",
                  f"- scaled: read {fb / 1e6:.2f} MB + write {wb / 1e6:.2f} MB = {(fb + wb) / 1e6:.2f} MB "
                  f"per dispatch; algorithmic {alg / 1e6:.2f} MB (ratio {(fb + wb) / alg:.4f})", ""]
    if a.valu:
        v = dispatches(a.valu, a.kernel)
        recs = [int(x) for x in a.records.split(",")] if a.records else []
        lines += ["## VALU (rocprofv3 --pmc SQ_ACTIVE_INST_VALU SQ_INSTS_VALU SQ_ACTIVE_INST_VALU2 "
                  "SQ_INSTS_VALU_TRANS_F32 ... GRBM_GUI_ACTIVE)", "",
                  "| dispatch | records | ns | VALU busy % | dual-issue share % | VALU instr per param-seed |",
                  "|---|---|---|---|---|---|"]
        rows = []
        for i, (k, e) in enumerate(v.items()):
            cyc = e["GRBM_GUI_ACTIVE"] / XCDS
            busy = 100 * e["SQ_ACTIVE_INST_VALU"] / CUS / cyc
            dual = 100 * e.get("SQ_ACTIVE_INST_VALU2", 0) / max(e["SQ_ACTIVE_INST_VALU"], 1)
            r = recs[i % len(recs)] if recs else 0
            ips = e["SQ_INSTS_VALU"] * 64 / (a.elements * r) if r else float("nan")
            rows.append((r, busy, dual, ips))
            lines.append(f"| {k} | {r} | {e['ns']} | {busy:.1f} | {dual:.1f} | {ips:.2f} |")
        lines.append("")
        by = collections.defaultdict(list)
        for r, busy, dual, ips in rows:
            by[r].append((busy, dual, ips))
        summary["valu_by_records"] = {str(r): {"busy_pct": sum(x[0] for x in vals) / len(vals),
                                               "dual_issue_pct": sum(x[1] for x in vals) / len(vals),
                                               "instr_per_param_seed": sum(x[2] for x in vals) / len(vals)}
                                      for r, vals in by.items()}
        lines += [f"Minimal VALU instructions per param-seed of the method on gfx950: "
                  f"{a.instr_per_param_seed}.", ""]
    lines += [f"Kernel sources sha256: `{summary['kernel_source_sha256']}`", ""]
    os.makedirs(a.outdir, exist_ok=True)
    with open(os.path.join(a.outdir, a.name + ".md"), "w") as fh:
        fh.write("\n".join(lines))
    if "hbm_bytes_per_dispatch" in summary:
        with open(os.path.join(a.outdir, a.name + "_traffic.json"), "w") as fh:
            json.dump(summary, fh, indent=1)
    print("\n".join(lines))


if __name__ == "__main__":
    main()
