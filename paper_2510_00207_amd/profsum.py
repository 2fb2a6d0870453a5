"""Summaries of rocprofv3 output for the measurements kept under profiles/.

    python -m paper_2510_00207_amd.profsum trace DIR --out FILE.md --command "..."
        kernel-trace statistics (run_kernel_stats.csv) as a markdown table

    python -m paper_2510_00207_amd.profsum traffic FETCH_DIR WRITE_DIR --probe-mib N
            --out FILE.json --md FILE.md --command "..."
        HBM bytes per dispatch from two PMC passes (FETCH_SIZE, then WRITE_SIZE,
        KiB per dispatch), each scaled by what the same counter reads for the
        plain copy of N MiB that bench.py --copy-probe N runs last; the grouped
        GEMM's average over its launches is stored with a hash of the kernel
        source, so a later kernel change is detected and the figure dropped.

    python -m paper_2510_00207_amd.profsum mfma DIR --out FILE.md --command "..."
        MFMA busy share of the expert GEMMs (or of the kernels whose names
        match --match) from one PMC pass with
        SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE: GRBM_GUI_ACTIVE is summed
        over the 8 XCDs, so a dispatch's cycles are GRBM_GUI_ACTIVE / 8 and its
        MFMA busy share is SQ_VALU_MFMA_BUSY_CYCLES / (cycles * 1024 SIMDs);
        the clock is cycles / duration.

Reads CSV files only; runs nothing on the GPU.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
GEMM_SOURCES = ("csrc/gemm.hip", "csrc/common.hpp")
GEMM_KERNEL = "gemm_dma_kernel"
GATE_GEMM = ", 6, "  # epilogue 6: the gate backward's dW_g partials, not an expert GEMM


def expert_gemm(name: str) -> bool:
    return name.startswith(GEMM_KERNEL) and GATE_GEMM not in name


def gemm_source_hash() -> str:
    h = hashlib.sha256()
    for rel in GEMM_SOURCES:
        with open(os.path.join(PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def short_name(name: str) -> str:
    name = re.sub(r"^void ", "", name).replace("flowmoe::(anonymous namespace)::", "")
    return re.sub(r"\((flowmoe|GemmParams|unsigned|int const|float const|HIP_vector).*$", "", name)


def cmd_trace(a) -> None:
    rows = list(csv.DictReader(open(os.path.join(a.dir, "run_kernel_stats.csv"))))
    lines = [f"# {a.title}", "", "Command (run from the repository root on one MI355X):", "",
             f"    {a.command}", "",
             "| kernel | calls | avg us | min us | max us | total ms |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        nm = short_name(r["Name"])
        if nm.startswith("at::") or "rocclr" in nm:
            continue
        lines.append(f"| `{nm}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.3f} |")
    if a.note:
        lines += ["", a.note]
    open(a.out, "w").write("\n".join(lines) + "\n")


def _pmc(dirname: str, counter: str):
    """dispatch id -> (short kernel name, counter value in bytes)"""
    out = {}
    for r in csv.DictReader(open(os.path.join(dirname, "run_counter_collection.csv"))):
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        nm, v = short_name(r["Kernel_Name"]), float(r["Counter_Value"]) * 1024.0
        out[d] = (nm, out.get(d, (nm, 0.0))[1] + v)
    return out


def cmd_traffic(a) -> None:
    fetch, write = _pmc(a.fetch_dir, "FETCH_SIZE"), _pmc(a.write_dir, "WRITE_SIZE")
    probe = float(a.probe_mib) * 2**20

    def probe_value(tab):  # the copy probe is the last copy kernel of the run
        copies = [d for d, (nm, _) in tab.items() if "copyBuffer" in nm or "copy" in nm.lower()]
        return tab[max(copies)][1]

    f_scale, w_scale = probe / probe_value(fetch), probe / probe_value(write)
    per = collections.defaultdict(lambda: [[], []])
    for d, (nm, v) in fetch.items():
        per[nm][0].append(v * f_scale)
    for d, (nm, v) in write.items():
        per[nm][1].append(v * w_scale)
    kernels = {}
    for nm, (fv, wv) in sorted(per.items()):
        if nm.startswith("at::") or "rocclr" in nm:
            continue
        kernels[nm] = {"dispatches": len(fv), "fetch_bytes": sum(fv) / max(1, len(fv)),
                       "write_bytes": sum(wv) / max(1, len(wv))}
    gemm = [(sum(per[nm][0]) + sum(per[nm][1]), len(per[nm][0])) for nm in per if expert_gemm(nm)]
    tot, n = sum(g[0] for g in gemm), sum(g[1] for g in gemm)
    res = {"gemm_source_sha256": gemm_source_hash(), "command": a.command,
           "probe_mib": a.probe_mib, "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "gemm_bytes_per_launch": tot / max(1, n), "gemm_launches": n, "kernels": kernels}
    json.dump(res, open(a.out, "w"), indent=1)
    if a.md:
        lines = [f"# {a.title}", "", "Commands (run from the repository root on one MI355X), one pass per counter:", "",
                 f"    {a.command}", "",
                 f"Calibration: the {a.probe_mib} MiB copy probe read FETCH_SIZE x{f_scale:.3f} and "
                 f"WRITE_SIZE x{w_scale:.3f} of its true bytes; the figures below are scaled by those "
                 "factors (MiB per dispatch).", "",
                 "| kernel | dispatches | fetch MiB | write MiB |", "|---|---|---|---|"]
        for nm, k in kernels.items():
            lines.append(f"| `{nm}` | {k['dispatches']} | {k['fetch_bytes'] / 2**20:.1f} | "
                         f"{k['write_bytes'] / 2**20:.1f} |")
        lines += ["", f"Expert GEMMs ({GEMM_KERNEL}), average over their {n} launches: "
                      f"{res['gemm_bytes_per_launch'] / 2**20:.1f} MiB of HBM traffic per launch."]
        open(a.md, "w").write("\n".join(lines) + "\n")


def cmd_mfma(a) -> None:
    per = collections.defaultdict(dict)
    for r in csv.DictReader(open(os.path.join(a.dir, "run_counter_collection.csv"))):
        d = int(r["Dispatch_Id"])
        c = per[d]
        c["name"] = short_name(r["Kernel_Name"])
        c["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        c[r["Counter_Name"]] = c.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    agg = collections.defaultdict(lambda: [0, 0.0, 0.0, 0.0])  # launches, busy, cycles, ns
    pick = (lambda nm: re.search(a.match, nm)) if a.match else expert_gemm
    for c in per.values():
        if not pick(c["name"]) or "SQ_VALU_MFMA_BUSY_CYCLES" not in c:
            continue
        g = agg[c["name"]]
        g[0] += 1
        g[1] += c["SQ_VALU_MFMA_BUSY_CYCLES"]
        g[2] += c["GRBM_GUI_ACTIVE"] / 8.0
        g[3] += c["ns"]
    lines = [f"# {a.title}", "", "Command (run from the repository root on one MI355X):", "",
             f"    {a.command}", "",
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (cycles x 1024 SIMDs), cycles = "
             "GRBM_GUI_ACTIVE / 8 (the counter is summed over the 8 XCDs); clock = cycles / "
             "duration.", "",
             "| kernel | launches | avg us | clock GHz | MFMA busy |", "|---|---|---|---|---|"]
    tb = tc = 0.0
    for nm, (n, busy, cyc, ns) in sorted(agg.items()):
        tb += busy
        tc += cyc
        lines.append(f"| `{nm}` | {n} | {ns / n / 1e3:.1f} | {cyc / ns:.2f} | "
                     f"{busy / (cyc * 1024):.3f} |")
    if tc > 0:
        what = "matching" if a.match else "expert GEMM"
        lines += ["", f"All {what} launches together: MFMA busy {tb / (tc * 1024):.3f}."]
    if a.note:
        lines += ["", a.note]
    open(a.out, "w").write("\n".join(lines) + "\n")


def main() -> None:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("dir")
    t.add_argument("--out", required=True)
    t.add_argument("--title", default="Kernel trace")
    t.add_argument("--command", required=True)
    t.add_argument("--note", default="")
    p = sub.add_parser("traffic")
    p.add_argument("fetch_dir")
    p.add_argument("write_dir")
    p.add_argument("--probe-mib", type=int, required=True)
    p.add_argument("--out", required=True)
    p.add_argument("--md", default="")
    p.add_argument("--title", default="HBM traffic per dispatch")
    p.add_argument("--command", required=True)
    m = sub.add_parser("mfma")
    m.add_argument("dir")
    m.add_argument("--out", required=True)
    m.add_argument("--title", default="MFMA busy share of the expert GEMMs")
    m.add_argument("--command", required=True)
    m.add_argument("--note", default="")
    m.add_argument("--match", default="",
                   help="regex over kernel names (default: the expert GEMMs)")
    a = ap.parse_args()
    {"trace": cmd_trace, "traffic": cmd_traffic, "mfma": cmd_mfma}[a.cmd](a)


if __name__ == "__main__":
    main()
