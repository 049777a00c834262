"""Summaries of rocprofv3 CSV output for the committed profile notes.

Three sub-commands, each reading the CSV files rocprofv3 writes with
``--output-format csv`` under a run's output directory:

``stats DIR --title T --command C``
    Markdown table of the ``*_kernel_stats.csv`` of a ``--kernel-trace --stats``
    run (calls, total, average, share per kernel).

``traffic --fetch DIR1 --write DIR2 --kernel K --copy-kernel C --copy-bytes N``
    JSON summary of HBM traffic per dispatch of the kernel whose name contains
    K, from a ``--pmc FETCH_SIZE`` run (DIR1) and a ``--pmc WRITE_SIZE`` run
    (DIR2) of the same program.  Both counters are in KiB per dispatch; each is
    scaled by (N bytes / what the same counter reads for the copy kernel C,
    which reads N bytes and writes N bytes), so the figures are in bytes of the
    copy's own accounting.  The summary records a hash of the sources listed
    with ``--source`` so that a reader can tell when the kernel has changed
    since the counters were taken.

``mfma DIR --kernels K1,K2,... --workload W``
    JSON summary of the matrix-core utilisation of the kernels whose names
    contain one of K1, K2, ... (the CNN stage), from a ``--pmc
    SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_MFMA SQ_INSTS_VALU GRBM_GUI_ACTIVE`` run:
    per kernel the busy fraction SQ_VALU_MFMA_BUSY_CYCLES / (cycles x SIMDs),
    cycles being GRBM_GUI_ACTIVE / XCDs, and over the stage the same with
    busy and cycles summed over its dispatches.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys


def _rows(directory: str, suffix: str):
    files = sorted(glob.glob(os.path.join(directory, "**", "*" + suffix), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {directory}")
    for f in files:
        with open(f, newline="") as fh:
            yield from csv.DictReader(fh)


def short_name(name: str) -> str:
    """Kernel name without namespaces, return type and parameter list."""
    s = name.replace("nsc::(anonymous namespace)::", "").replace("(anonymous namespace)::", "")
    if s.startswith("void "):
        s = s[5:]
    depth = 0
    for i, ch in enumerate(s):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return s[:i]
    return s


def sources_hash(paths) -> str:
    h = hashlib.sha256()
    for p in sorted(paths):
        with open(p, "rb") as fh:
            h.update(os.path.basename(p).encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def cmd_stats(a) -> None:
    rows = list(_rows(a.dir, "kernel_stats.csv"))
    out = [f"# {a.title}", "", "Command (from the repository root, on one MI355X):", "", "```",
           a.command, "```", "",
           "rocprofv3 kernel statistics (durations in microseconds):", "",
           "| kernel | calls | total us | average us | min us | max us | % |",
           "|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append("| `{}` | {} | {:.1f} | {:.3f} | {:.3f} | {:.3f} | {:.2f} |".format(
            short_name(r["Name"]), r["Calls"], float(r["TotalDurationNs"]) / 1e3,
            float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
            float(r["Percentage"])))
    text = "\n".join(out) + "\n"
    if a.out:
        with open(a.out, "w") as fh:
            fh.write(text)
    sys.stdout.write(text)


def _per_dispatch(directory: str, counter: str):
    """{kernel name: [value per dispatch]} for one counter (values summed over
    the rows a dispatch has)."""
    acc = {}
    for r in _rows(directory, "counter_collection.csv"):
        if r.get("Counter_Name") != counter:
            continue
        key = (r["Kernel_Name"], r.get("Dispatch_Id") or r.get("Correlation_Id"))
        acc[key] = acc.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for (name, _), v in sorted(acc.items(), key=lambda kv: int(kv[0][1] or 0)):
        out.setdefault(name, []).append(v)
    return out


def _pick(table, pattern: str, what: str, skip: int = 0):
    """The one kernel matching pattern: its mean per dispatch, in dispatch
    order after the first `skip` dispatches."""
    names = [n for n in table if pattern in n]
    if len(names) != 1:
        raise SystemExit(f"{what}: {len(names)} kernels match {pattern!r}: {names[:5]}")
    vals = table[names[0]][skip:]
    return names[0], sum(vals) / len(vals), len(vals)


def cmd_traffic(a) -> None:
    fetch = _per_dispatch(a.fetch, "FETCH_SIZE")
    write = _per_dispatch(a.write, "WRITE_SIZE")
    kname, f_kib, nf = _pick(fetch, a.kernel, "FETCH_SIZE kernel", a.skip_first)
    _, w_kib, nw = _pick(write, a.kernel, "WRITE_SIZE kernel", a.skip_first)
    cname, cf_kib, _ = _pick(fetch, a.copy_kernel, "FETCH_SIZE copy")
    _, cw_kib, _ = _pick(write, a.copy_kernel, "WRITE_SIZE copy")
    sf = a.copy_bytes / (cf_kib * 1024.0)
    sw = a.copy_bytes / (cw_kib * 1024.0)
    fetch_b = f_kib * 1024.0 * sf
    write_b = w_kib * 1024.0 * sw
    res = {
        "kernel": short_name(kname),
        "workload": a.workload,
        "dispatches": {"fetch_run": nf, "write_run": nw},
        "fetch_kib_per_dispatch": f_kib,
        "write_kib_per_dispatch": w_kib,
        "copy_kernel": short_name(cname),
        "copy_bytes": a.copy_bytes,
        "copy_fetch_kib": cf_kib,
        "copy_write_kib": cw_kib,
        "scale_fetch": sf,
        "scale_write": sw,
        "fetch_bytes": fetch_b,
        "write_bytes": write_b,
        "traffic_bytes": fetch_b + write_b,
        "algorithmic_bytes": a.algorithmic_bytes,
        "traffic_over_algorithmic": (fetch_b + write_b) / a.algorithmic_bytes
        if a.algorithmic_bytes else None,
        "sources": sorted(os.path.relpath(p) for p in a.source),
        "sources_sha256_16": sources_hash(a.source) if a.source else None,
        "commands": a.command,
    }
    text = json.dumps(res, indent=1) + "\n"
    if a.out:
        with open(a.out, "w") as fh:
            fh.write(text)
    sys.stdout.write(text)


SIMDS = 1024  # MI355X: 256 compute units x 4 SIMDs
XCDS = 8      # GRBM_GUI_ACTIVE counts once per XCD
CLOCK_HZ = 2.4e9


def cmd_mfma(a) -> None:
    busy = _per_dispatch(a.dir, "SQ_VALU_MFMA_BUSY_CYCLES")
    gui = _per_dispatch(a.dir, "GRBM_GUI_ACTIVE")
    mfma = _per_dispatch(a.dir, "SQ_INSTS_MFMA")
    valu = _per_dispatch(a.dir, "SQ_INSTS_VALU")
    pats = [k for k in a.kernels.split(",") if k]
    kernels, tot_busy, tot_cyc = {}, 0.0, 0.0
    for name in sorted(busy):
        if not any(p in name for p in pats):
            continue
        cyc = [g / XCDS for g in gui[name]]
        b, c = sum(busy[name]), sum(cyc)
        n_m, n_v = sum(mfma.get(name, [0.0])), sum(valu.get(name, [0.0]))
        kernels[short_name(name)] = {
            "dispatches": len(cyc),
            "avg_ms": c / len(cyc) / CLOCK_HZ * 1e3,
            "mfma_busy": b / (c * SIMDS) if c else None,
            "mfma_insts_per_dispatch": n_m / len(cyc),
            "valu_insts_per_mfma": n_v / n_m if n_m else None,
        }
        tot_busy += b
        tot_cyc += c
    res = {
        "workload": a.workload,
        "kernels": kernels,
        "stage_mfma_busy": tot_busy / (tot_cyc * SIMDS) if tot_cyc else None,
        "note": "busy = SQ_VALU_MFMA_BUSY_CYCLES / ((GRBM_GUI_ACTIVE / 8) x 1024 SIMDs): the "
                "issued matrix-core work, hi / lo passes and K padding included",
        "sources": sorted(os.path.relpath(p) for p in a.source),
        "sources_sha256_16": sources_hash(a.source) if a.source else None,
        "commands": a.command,
    }
    text = json.dumps(res, indent=1) + "\n"
    if a.out:
        with open(a.out, "w") as fh:
            fh.write(text)
    sys.stdout.write(text)


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--out")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--copy-kernel", required=True)
    t.add_argument("--copy-bytes", type=float, required=True)
    t.add_argument("--algorithmic-bytes", type=float, default=0.0)
    t.add_argument("--skip-first", type=int, default=0,
                   help="leave out the kernel's first dispatches (set-up work of the run)")
    t.add_argument("--workload", default="")
    t.add_argument("--source", action="append", default=[])
    t.add_argument("--command", action="append", default=[])
    t.add_argument("--out")
    m = sub.add_parser("mfma")
    m.add_argument("dir")
    m.add_argument("--kernels", required=True)
    m.add_argument("--workload", default="")
    m.add_argument("--source", action="append", default=[])
    m.add_argument("--command", action="append", default=[])
    m.add_argument("--out")
    a = ap.parse_args(argv)
    {"stats": cmd_stats, "traffic": cmd_traffic, "mfma": cmd_mfma}[a.cmd](a)


if __name__ == "__main__":
    main()
