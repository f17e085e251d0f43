"""HBM traffic per kernel launch from rocprofv3 counter runs, and kernel-time
summaries from rocprofv3 kernel-trace statistics.

Reads the counter-collection CSVs of two `rocprofv3 --pmc FETCH_SIZE` and
`rocprofv3 --pmc WRITE_SIZE` runs of `bench.py --copy-calibration`, scales
each kernel's mean counter (KiB per dispatch) by what the same counter reads
for the plain copy of a known size in the same run, and writes the result
(with the hash of the kernel sources it was taken on) for bench.py:

    python -m paper_2606_14782_amd.counters --fetch DIR --write DIR \
        --out profiles/traffic.json --md profiles/traffic_<workload>.md

With --trace DIR it instead summarises the *kernel_stats.csv of a
`rocprofv3 --kernel-trace --stats` run into a markdown table (--md).
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
COPY_BYTES = 1 << 30

# demangled kernel name -> name used by the library's own timing
_NAMES = [
    (r"bacon::k_pass<0,", "window_lse"),
    (r"bacon::k_pass<1,", "window_score"),
    (r"bacon::k_pass<2,", "window_score_calib"),
    (r"bacon::k_lse_merge\b", "lse_merge"),
    (r"bacon::k_krpass<0,", "window_lse_kr"),
    (r"bacon::k_krpass<2,", "window_score_calib_kr"),
    (r"bacon::k_krdual<", "window_score_calib_lse_kr"),
    (r"bacon::k_pass_dual<", "window_score_calib_lse"),
    (r"bacon::k_single<", "window_score_single"),
    (r"bacon::k_sel_a\b", "segment_calib_cand"),
    (r"bacon::k_sel_b\b", "segment_score_final"),
    (r"bacon::k_segcal\b", "segment_calib"),
    (r"bacon::k_segscore\b", "segment_score"),
    (r"bacon::k_segcand\b", "segment_cand"),
    (r"bacon::k_segfinal\b", "final_topk"),
    (r"bacon::k_compact\b", "compact"),
    (r"bacon::k_select<1>", "select_calib"),
    (r"bacon::k_select<2>", "select_topk"),
    (r"bacon::k_elem\b", "calib_elem"),
    (r"bacon::k_alloc\b", "head_alloc"),
]


def _code_only(text: str) -> str:
    """The source with comments and blank lines removed (no string literal in
    the kernel sources holds a comment marker)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = (re.sub(r"//.*", "", ln).rstrip() for ln in text.splitlines())
    return "\n".join(ln for ln in lines if ln)


def source_sha() -> str:
    """Hash of the kernel sources' code (comments aside); counters taken on
    other code are stale."""
    h = hashlib.sha256()
    for f in ("kernels.hip", "internal.h"):
        with open(os.path.join(HERE, "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def library_name(kernel: str) -> str | None:
    for pat, name in _NAMES:
        if re.search(pat, kernel):
            return name
    return None


def _rows(d: str):
    files = sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True))
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    for f in files:
        with open(f, newline="") as fh:
            yield from csv.DictReader(fh)


def per_kernel(d: str, counter: str):
    """Mean counter value per dispatch (KiB) for each kernel name."""
    acc = defaultdict(list)
    for r in _rows(d):
        if r.get("Counter_Name") != counter:
            continue
        acc[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return {k: (sum(v) / len(v), len(v)) for k, v in acc.items()}


def copy_kib(stats) -> float:
    """Counter of the calibration copy: torch's elementwise multiply by 1."""
    cands = [(v, k) for k, (v, n) in stats.items() if "Mul" in k and library_name(k) is None]
    if not cands:
        raise SystemExit("calibration copy kernel not found (run bench.py --copy-calibration)")
    return max(cands)[0]


def trace_summary(d: str, md: str, command: str, title: str) -> None:
    """Markdown table of the per-kernel statistics of a kernel-trace run."""
    files = sorted(glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True))
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {d}")
    rows = []
    for f in files:
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                calls = int(float(r.get("Calls", 0)))
                tot = float(r.get("TotalDurationNs", 0.0))
                avg = float(r.get("AverageNs", tot / max(calls, 1)))
                rows.append((tot, r.get("Name", "?"), calls, avg, float(r.get("MinNs", 0.0)),
                             float(r.get("MaxNs", 0.0))))
    total = sum(x[0] for x in rows) or 1.0
    lines = [f"# {title}", "", f"command (from /tmp with TMPDIR=/tmp): `{command}`", "",
             f"kernel sources: {source_sha()}", "",
             "| kernel | library name | calls | avg us | min us | max us | share |",
             "|---|---|---|---|---|---|---|"]
    for tot, name, calls, avg, mn, mx in sorted(rows, reverse=True):
        short = name if len(name) <= 60 else name[:57] + "..."
        lib = library_name(name) or "(torch / runtime)"
        lines.append(f"| `{short}` | {lib} | {calls} | {avg / 1e3:.2f} | {mn / 1e3:.2f} | "
                     f"{mx / 1e3:.2f} | {100 * tot / total:.1f}% |")
    with open(md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def sq_summary(dirs, md: str, command: str, title: str) -> None:
    """Markdown table of the mean per-dispatch value of every counter of one
    or more --pmc runs (e.g. SQ_ counters), per library kernel."""
    agg = {}
    for d in dirs:
        for r in _rows(d):
            name = library_name(r["Kernel_Name"])
            if name is not None:
                agg.setdefault(name, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    counters = sorted({c for cs in agg.values() for c in cs})
    lines = [f"# {title}", "", f"commands (from /tmp with TMPDIR=/tmp): `{command}`", "",
             f"kernel sources: {source_sha()}", "",
             "Mean value per dispatch, summed over the device (cycle counters in the units "
             "rocprofv3 reports).", "",
             "| kernel | " + " | ".join(counters) + " |",
             "|---|" + "---|" * len(counters)]
    for name in sorted(agg):
        cs = agg[name]
        cells = [f"{sum(cs[c]) / len(cs[c]):.0f}" if c in cs else "" for c in counters]
        lines.append(f"| {name} | " + " | ".join(cells) + " |")
    with open(md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--sq", nargs="*")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--out")
    ap.add_argument("--trace")
    ap.add_argument("--title", default="Kernel durations")
    ap.add_argument("--md", required=True)
    ap.add_argument("--command", default="")
    args = ap.parse_args()
    if args.sq:
        sq_summary(args.sq, args.md, args.command, args.title)
        return
    if args.trace:
        trace_summary(args.trace, args.md, args.command, args.title)
        return
    if not (args.fetch and args.write and args.out):
        raise SystemExit("--fetch, --write and --out are required without --trace")
    fs, ws = per_kernel(args.fetch, "FETCH_SIZE"), per_kernel(args.write, "WRITE_SIZE")
    ffac = COPY_BYTES / (copy_kib(fs) * 1024.0)
    wfac = COPY_BYTES / (copy_kib(ws) * 1024.0)
    kernels = {}
    for k in sorted(set(fs) | set(ws)):
        name = library_name(k)
        if name is None:
            continue
        fb = fs.get(k, (0.0, 0))[0] * 1024.0 * ffac
        wb = ws.get(k, (0.0, 0))[0] * 1024.0 * wfac
        e = kernels.setdefault(name, {"fetch_bytes": 0.0, "write_bytes": 0.0, "dispatches": 0,
                                      "variants": []})
        n = fs.get(k, (0, 0))[1]
        # several template instances of one library name: dispatch-weighted mean
        tot = e["dispatches"] + n
        if tot:
            e["fetch_bytes"] = (e["fetch_bytes"] * e["dispatches"] + fb * n) / tot
            e["write_bytes"] = (e["write_bytes"] * e["dispatches"] + wb * n) / tot
        e["dispatches"] = tot
        e["variants"].append(k)
    for e in kernels.values():
        e["bytes_per_launch"] = e["fetch_bytes"] + e["write_bytes"]
    rec = {"source_sha": source_sha(), "copy_bytes": COPY_BYTES,
           "copy_factor": {"fetch": ffac, "write": wfac}, "command": args.command,
           "kernels": kernels}
    with open(args.out, "w") as fh:
        json.dump(rec, fh, indent=1)
    lines = [f"# HBM traffic per launch (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
             f"kernel sources: {rec['source_sha']}", "",
             f"command: `{args.command}`", "",
             f"copy calibration: {COPY_BYTES} B read + written; counter scale factors "
             f"fetch {ffac:.4f}, write {wfac:.4f}", "",
             "| kernel | dispatches | fetch MB | write MB | total MB |", "|---|---|---|---|---|"]
    for name, e in sorted(kernels.items()):
        lines.append(f"| {name} | {e['dispatches']} | {e['fetch_bytes'] / 1e6:.2f} | "
                     f"{e['write_bytes'] / 1e6:.2f} | {e['bytes_per_launch'] / 1e6:.2f} |")
    with open(args.md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
