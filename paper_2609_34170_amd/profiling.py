"""Summaries of rocprofv3 output for profiles/.

    python -m paper_2609_34170_amd.profiling stats <kernel_stats.csv> <out.md> --title T --command C [--bench-line F]
    python -m paper_2609_34170_amd.profiling traffic <fetch_dir> <write_dir> --kernel K --workload W
                                                     --regex R --algorithmic-bytes B --command-fetch C1 --command-write C2
    python -m paper_2609_34170_amd.profiling counters <pmc_dir> <out.md> --title T --command C

``stats`` turns a ``--kernel-trace --stats`` kernel table into a markdown table.
``counters`` summarises a ``--pmc`` pass of SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE,
SQ_LDS_IDX_ACTIVE, SQ_LDS_BANK_CONFLICT, SQ_INSTS_VALU and SQ_INSTS_VALU_MFMA_MOPS_BF16
per kernel: MFMA busy = busy cycles summed over SIMDs / (GUI-active cycles x SIMDs),
the GUI-active cycles of a dispatch being the largest over the XCDs.
``traffic`` reads two ``--pmc`` runs (FETCH_SIZE, then WRITE_SIZE, in KiB per
dispatch) of a program that also ran plain device copies of 512 MiB
(``bench.py --copy-calibration 512``): each counter is scaled by the bytes a
copy moves over what the counter reads for it, and the kernel's bytes per
launch are recorded in profiles/traffic.json with the sha256 of the kernel's
source files (bench.py reports the figure only while they match).
"""

from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_34170_amd", "csrc")
COPY_KERNEL = "copyBuffer"
COPY_BYTES = 512 << 20

# source files of each kernel class (the traffic record's hash)
KERNEL_SOURCES = {
    "persistent_layers": ["persistent.hip", "persistent.h", "common.h", "kernels.h"],
    "gemm": ["gemm.hip", "common.h", "kernels.h"],
    "attn": ["attention.hip", "common.h", "kernels.h"],
}


def sources_sha256(kernel: str):
    key = "persistent_layers" if kernel.startswith("persistent") else kernel.split("<")[0].rstrip("0123456789x")
    key = "gemm" if key.startswith("gemm") else key
    files = KERNEL_SOURCES.get(key)
    if not files:
        return None
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _rows(path):
    with open(path, newline="") as fh:
        return list(csv.DictReader(fh))


def _col(row, *names):
    for n in names:
        if n in row:
            return row[n]
    raise KeyError(f"none of {names} in {list(row)}")


def stats_markdown(csv_path, title, command, bench_line=None, top=14):
    rows = _rows(csv_path)
    out = [f"# {title}", "", "Command (from the repository root, on one MI355X):", "", "    " + command, ""]
    if bench_line:
        out += [f"Whole run (create + warmup + timed + latency + eager profile steps). bench line of this run: {bench_line}.",
                ""]
    out += ["Durations in microseconds.", "", "| kernel | calls | total ms | avg us | min us | max us | % |",
            "|---|---:|---:|---:|---:|---:|---:|"]
    rows.sort(key=lambda r: -float(_col(r, "TotalDurationNs")))
    for r in rows[:top]:
        name = _col(r, "Name", "KernelName", "Kernel_Name")
        name = name if len(name) <= 80 else name[:78] + ".."
        out.append("| `{}` | {} | {:.2f} | {:.2f} | {:.2f} | {:.2f} | {:.2f} |".format(
            name, _col(r, "Calls"), float(_col(r, "TotalDurationNs")) / 1e6, float(_col(r, "AverageNs")) / 1e3,
            float(_col(r, "MinNs")) / 1e3, float(_col(r, "MaxNs")) / 1e3, float(_col(r, "Percentage"))))
    return "\n".join(out) + "\n"


def _counter_means(pmc_dir, counter, regex):
    """Mean counter value (KiB per dispatch) of the kernels matching regex, and of the copy kernel."""
    files = glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {pmc_dir}")
    pat = re.compile(regex)
    per = {}
    for f in files:
        for r in _rows(f):
            if _col(r, "Counter_Name") != counter:
                continue
            name = _col(r, "Kernel_Name")
            key = "copy" if COPY_KERNEL in name else ("kernel" if pat.search(name) else None)
            if key is None:
                continue
            disp = _col(r, "Dispatch_Id")
            per.setdefault(key, {}).setdefault(disp, 0.0)
            per[key][disp] += float(_col(r, "Counter_Value"))
    if "copy" not in per or "kernel" not in per:
        raise RuntimeError(f"{counter}: missing copy or kernel dispatches in {pmc_dir}")
    # the calibration copies are the largest copy dispatches (the program's own
    # small copies -- uploads, context publications -- are left out)
    big = max(per["copy"].values())
    cal = [v for v in per["copy"].values() if v >= 0.5 * big]
    mean = lambda d: sum(d.values()) / len(d)
    return mean(per["kernel"]), len(per["kernel"]), sum(cal) / len(cal)


def traffic(fetch_dir, write_dir, kernel, workload, regex, algo_bytes, cmd_fetch, cmd_write, avg_us=None):
    fk, fn, fc = _counter_means(fetch_dir, "FETCH_SIZE", regex)
    wk, wn, wc = _counter_means(write_dir, "WRITE_SIZE", regex)
    fscale = COPY_BYTES / 1024.0 / fc  # a copy reads COPY_BYTES
    wscale = COPY_BYTES / 1024.0 / wc  # and writes COPY_BYTES
    fb = fk * 1024.0 * fscale
    wb = wk * 1024.0 * wscale
    entry = {"kernel": kernel, "workload": workload, "sources_sha256": sources_sha256(kernel),
             "fetch_kib_raw": round(fk, 1), "write_kib_raw": round(wk, 1), "fetch_scale": round(fscale, 4),
             "write_scale": round(wscale, 4), "fetch_bytes": int(fb), "write_bytes": int(wb),
             "bytes_per_launch": int(fb + wb)}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    rec = {"note": "HBM-side bytes per launch from rocprofv3 FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each "
                   "scaled by the same counter on a 512 MiB device copy; valid while the kernel sources hash to "
                   "sources_sha256", "entries": []}
    if os.path.exists(path):
        with open(path) as fh:
            rec = json.load(fh)
    rec["entries"] = [e for e in rec["entries"] if not (e["kernel"] == kernel and e["workload"] == workload)]
    rec["entries"].append(entry)
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    md = [f"# HBM traffic of `{kernel}` -- workload {workload}", "",
          "Two rocprofv3 counter passes over the same program (one counter per pass), each also running five plain",
          "512 MiB device copies (`bench.py --copy-calibration 512`, `__amd_rocclr_copyBuffer`) as the calibration",
          "of known size.  From the repository root, on one MI355X:", "", "    " + cmd_fetch, "    " + cmd_write, "",
          "| counter | 512 MiB copy (KiB/dispatch) | scale to bytes moved | kernel (KiB/dispatch, mean) | dispatches | bytes per launch |",
          "|---|---:|---:|---:|---:|---:|",
          f"| FETCH_SIZE | {fc:,.0f} | {fscale:.3f} | {fk:,.0f} | {fn} | {fb / 1e9:.3f} GB |",
          f"| WRITE_SIZE | {wc:,.0f} | {wscale:.3f} | {wk:,.0f} | {wn} | {wb / 1e9:.3f} GB |", "",
          f"Traffic per launch {(fb + wb) / 1e9:.3f} GB against {algo_bytes / 1e9:.3f} GB of algorithmic bytes "
          f"({(fb + wb) / algo_bytes:.2f}x)."]
    if avg_us:
        md.append(f"Average kernel duration in the same build: {avg_us:.1f} us.")
    md.append("The record in `traffic.json` carries the sha256 of the kernel's sources; bench.py reports the figure "
              "only while they match.")
    return entry, "\n".join(md) + "\n"


# MI355X: 256 compute units of 4 SIMDs in 8 XCDs
CUS, SIMDS, XCDS = 256, 1024, 8


def counters_markdown(pmc_dir, title, command):
    """Per kernel: dispatches, MFMA busy, LDS active, LDS bank conflicts per LDS-active cycle,
    VALU instructions per bf16 MFMA op (the counters are summed over the XCDs' instances;
    GRBM_GUI_ACTIVE, the same on every XCD, is divided by their count)."""
    files = glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {pmc_dir}")
    agg, disp = {}, {}
    for f in files:
        for r in _rows(f):
            name = _col(r, "Kernel_Name")
            name = name if len(name) <= 70 else name[:68] + ".."
            c = _col(r, "Counter_Name")
            agg.setdefault(name, {}).setdefault(c, 0.0)
            agg[name][c] += float(_col(r, "Counter_Value"))
            disp.setdefault(name, set()).add(_col(r, "Dispatch_Id"))
    out = [f"# {title}", "", "Command (from the repository root, on one MI355X):", "", "    " + command, "",
           "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE per XCD x 1024 SIMDs); LDS active =",
           "SQ_LDS_IDX_ACTIVE / (GRBM_GUI_ACTIVE per XCD x 256 CUs); conflicts = SQ_LDS_BANK_CONFLICT /",
           "SQ_LDS_IDX_ACTIVE; GRBM_GUI_ACTIVE is reported summed over the 8 XCDs.", "",
           "| kernel | dispatches | GPU-active us / dispatch | MFMA busy | LDS active | LDS bank conflicts | VALU instr / bf16 MFMA op |",
           "|---|---:|---:|---:|---:|---:|---:|"]
    for name, d in sorted(agg.items(), key=lambda kv: -kv[1].get("GRBM_GUI_ACTIVE", 0.0)):
        n = len(disp[name])
        gui = d.get("GRBM_GUI_ACTIVE", 0.0) / XCDS  # cycles, summed over dispatches
        if gui <= 0:
            continue
        mfma = d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (gui * SIMDS)
        lds = d.get("SQ_LDS_IDX_ACTIVE", 0.0) / (gui * CUS)
        conf = d.get("SQ_LDS_BANK_CONFLICT", 0.0) / max(d.get("SQ_LDS_IDX_ACTIVE", 0.0), 1.0)
        ops = d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
        valu = d.get("SQ_INSTS_VALU", 0.0) / ops if ops > 0 else float("nan")
        out.append(f"| `{name}` | {n} | {gui / n / 2400.0:.1f} | {mfma * 100:.1f}% | {lds * 100:.1f}% | "
                   f"{conf * 100:.1f}% | {valu:.3f} |")
    out.append("")
    out.append("GPU-active microseconds assume the 2.4 GHz clock.")
    return "\n".join(out) + "\n"


def main(argv=None):
    p = argparse.ArgumentParser()
    sub = p.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("out")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--bench-line")
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("out")
    t.add_argument("--kernel", required=True)
    t.add_argument("--workload", required=True)
    t.add_argument("--regex", required=True)
    t.add_argument("--algorithmic-bytes", type=float, required=True)
    t.add_argument("--command-fetch", required=True)
    t.add_argument("--command-write", required=True)
    t.add_argument("--avg-us", type=float)
    c = sub.add_parser("counters")
    c.add_argument("pmc_dir")
    c.add_argument("out")
    c.add_argument("--title", required=True)
    c.add_argument("--command", required=True)
    a = p.parse_args(argv)
    if a.cmd == "counters":
        with open(a.out, "w") as fh:
            fh.write(counters_markdown(a.pmc_dir, a.title, a.command))
    elif a.cmd == "stats":
        with open(a.out, "w") as fh:
            fh.write(stats_markdown(a.csv, a.title, a.command, a.bench_line))
    else:
        entry, md = traffic(a.fetch_dir, a.write_dir, a.kernel, a.workload, a.regex, a.algorithmic_bytes,
                            a.command_fetch, a.command_write, a.avg_us)
        with open(a.out, "w") as fh:
            fh.write(md)
        print(json.dumps(entry))
    return 0


if __name__ == "__main__":
    sys.exit(main())
