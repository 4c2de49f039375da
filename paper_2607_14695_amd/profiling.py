"""Reduce rocprofv3 output for the denoise kernels to short text summaries.

Two inputs are used:

* the kernel-trace statistics CSV (``--kernel-trace --stats``), which gives
  calls and average duration per kernel;
* two counter-collection CSVs, one from a ``--pmc FETCH_SIZE`` run and one from
  a ``--pmc WRITE_SIZE`` run of the same command. Each gives KiB per dispatch.

The counters are calibrated against a plain elementwise copy of known size,
launched in the same process before the workload (``bench.py
--calibrate-copy``: 256 MiB read and 256 MiB written per launch). Each
counter's factor is the copy's true bytes divided by what the counter reported
for the copy. The factor then scales the same counter for the kernel of
interest.

The traffic record written here carries a digest of the kernel's source files.
``bench.py`` reports the measured traffic only while that digest still matches
the sources, so a stale figure is never attached to a changed kernel.

Usage::

    python -m paper_2607_14695_amd.profiling --stats KT_kernel_stats.csv \\
        --fetch FETCH_counter_collection.csv --write WRITE_counter_collection.csv \\
        --kernel "attn_pair_kernel<256>" --kernel-class attention --workload pi0_chunk_bf16 \\
        --command-kt "..." --command-fetch "..." --command-write "..." \\
        --out-md profiles/attention_pi0_chunk_bf16.md \\
        --out-json profiles/traffic_pi0_chunk_bf16.json

The JSON file holds one record per kernel class of the workload.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
from typing import Dict, List, Optional, Tuple

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")

# source files that determine each kernel class's machine code
KERNEL_SOURCES: Dict[str, Tuple[str, ...]] = {
    "attention": ("attention.hip", "common.h", "kernels.h"),
    "attn_merge": ("attention.hip", "common.h", "kernels.h"),
    "gemm_qkv": ("gemm.hip", "common.h", "kernels.h"),
    "gemm_o": ("gemm.hip", "common.h", "kernels.h"),
    "gemm_gate_up": ("gemm.hip", "common.h", "kernels.h"),
    "gemm_down": ("gemm.hip", "common.h", "kernels.h"),
    "resid_norm": ("norm_ring.hip", "common.h", "kernels.h"),
    "embed_norm": ("norm_ring.hip", "common.h", "kernels.h"),
    "final_euler": ("norm_ring.hip", "common.h", "kernels.h"),
    "frame_proj": ("gemm.hip", "common.h", "kernels.h"),
    "ring_write": ("norm_ring.hip", "common.h", "kernels.h"),
    "modulation": ("gemm.hip", "norm_ring.hip", "common.h", "kernels.h"),
    "all": ("attention.hip", "gemm.hip", "norm_ring.hip", "reflex_api.hip", "common.h", "kernels.h"),
}

COPY_BYTES = 256 << 20  # bytes read, and bytes written, by one calibration copy
# The copy is torch.mul over 64 Mi fp32 elements; torch's vectorized
# elementwise kernel runs one thread per 4 elements.  Other multiplies in the
# same run (weight initialisation) share the kernel name, so a dispatch is
# the copy only when its grid matches as well.
COPY_PATTERN = re.compile(r"MulFunctor")
COPY_GRID = (COPY_BYTES // 4) // 4


def source_digest(kernel_class: str) -> str:
    """sha256 over the source files of a kernel class (names and contents)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel_class]:
        h.update(name.encode())
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _rows(path: str) -> List[dict]:
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def counter_per_dispatch(path: str, counter: str, kernel_pattern: str) -> Tuple[float, int, float]:
    """(average value per matching dispatch, matching dispatches, copy value).

    A dispatch can be listed once per counter instance; values of one
    dispatch are summed first."""
    per_dispatch: Dict[Tuple[str, str], float] = {}
    names: Dict[Tuple[str, str], str] = {}
    grids: Dict[Tuple[str, str], int] = {}
    for r in _rows(path):
        if r["Counter_Name"] != counter:
            continue
        key = (r["Dispatch_Id"], r.get("Agent_Id", ""))
        per_dispatch[key] = per_dispatch.get(key, 0.0) + float(r["Counter_Value"])
        names[key] = r["Kernel_Name"]
        grids[key] = int(r["Grid_Size"])
    pat = re.compile(kernel_pattern)
    vals = [v for k, v in per_dispatch.items() if pat.search(names[k])]
    copies = [v for k, v in per_dispatch.items() if COPY_PATTERN.search(names[k]) and grids[k] == COPY_GRID]
    if not vals:
        raise ValueError(f"no dispatch of {kernel_pattern!r} with counter {counter} in {path}")
    if not copies:
        raise ValueError(f"no calibration copy dispatch in {path}")
    return sum(vals) / len(vals), len(vals), sorted(copies)[len(copies) // 2]


def kernel_stats(path: str) -> List[dict]:
    out = []
    for r in _rows(path):
        out.append({"name": r["Name"], "calls": int(r["Calls"]), "total_ns": float(r["TotalDurationNs"]),
                    "avg_ns": float(r["AverageNs"]), "min_ns": float(r["MinNs"]), "max_ns": float(r["MaxNs"]),
                    "pct": float(r["Percentage"])})
    out.sort(key=lambda d: -d["total_ns"])
    return out


def _short(name: str) -> str:
    name = re.sub(r"^void ", "", name)
    depth, cut = 0, len(name)
    for i in range(len(name) - 1, -1, -1):  # strip the outermost trailing "( ... )"
        if name[i] == ")":
            depth += 1
        elif name[i] == "(":
            depth -= 1
            if depth == 0:
                cut = i
                break
    name = name[:cut] if name.endswith(")") else name
    return name if len(name) <= 90 else name[:87] + "..."


def dispatch_groups(trace_csv: str) -> List[dict]:
    """Kernel-trace dispatches grouped by (kernel, grid size): the same kernel
    launched for different workloads (batch sizes) keeps separate rows."""
    groups: Dict[Tuple[str, str], List[float]] = {}
    for r in _rows(trace_csv):
        if r.get("Kind", "KERNEL_DISPATCH") != "KERNEL_DISPATCH":
            continue
        key = (r["Kernel_Name"], r["Grid_Size_X"])
        groups.setdefault(key, []).append(float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
    out = []
    for (name, grid), d in groups.items():
        out.append({"name": name, "grid": int(grid), "calls": len(d), "avg_ns": sum(d) / len(d),
                    "min_ns": min(d), "max_ns": max(d), "total_ns": sum(d)})
    out.sort(key=lambda x: -x["total_ns"])
    return out


def groups_markdown(groups: List[dict], command: str, limit: int = 24) -> str:
    lines = ["| kernel | grid (threads) | calls | avg us | min us | max us |", "|---|---|---|---|---|---|"]
    for d in groups[:limit]:
        lines.append(f"| `{_short(d['name'])}` | {d['grid']} | {d['calls']} | {d['avg_ns'] / 1e3:.2f} | "
                     f"{d['min_ns'] / 1e3:.2f} | {d['max_ns'] / 1e3:.2f} |")
    return f"Command:\n\n```\n{command}\n```\n\n" + "\n".join(lines) + "\n"


def stats_markdown(stats: List[dict], command: str, limit: int = 20) -> str:
    lines = ["| kernel | calls | avg us | min us | max us | % of GPU time |", "|---|---|---|---|---|---|"]
    for d in stats[:limit]:
        lines.append(f"| `{_short(d['name'])}` | {d['calls']} | {d['avg_ns'] / 1e3:.2f} | {d['min_ns'] / 1e3:.2f} | "
                     f"{d['max_ns'] / 1e3:.2f} | {d['pct']:.2f} |")
    return f"Command:\n\n```\n{command}\n```\n\n" + "\n".join(lines) + "\n"


def main(argv: Optional[List[str]] = None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--stats", required=True)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--kernel", required=True, help="regex selecting the kernel's dispatches")
    ap.add_argument("--kernel-class", required=True, choices=sorted(KERNEL_SOURCES))
    ap.add_argument("--workload", required=True)
    ap.add_argument("--command-kt", required=True)
    ap.add_argument("--command-fetch", default="")
    ap.add_argument("--command-write", default="")
    ap.add_argument("--out-md", required=True)
    ap.add_argument("--out-json")
    ap.add_argument("--trace", help="kernel-trace CSV: add a table grouped by (kernel, grid size)")
    args = ap.parse_args(argv)

    stats = kernel_stats(args.stats)
    pat = re.compile(args.kernel)
    mine = [d for d in stats if pat.search(d["name"])]
    md = [f"# rocprofv3 summary: {args.kernel_class} on {args.workload}\n",
          "## Kernel trace statistics\n", stats_markdown(stats, args.command_kt)]
    if args.trace:
        md += ["## Dispatches grouped by kernel and grid size\n", groups_markdown(dispatch_groups(args.trace), args.command_kt)]
    rec = None
    if args.fetch and args.write:
        f_avg, f_n, f_copy = counter_per_dispatch(args.fetch, "FETCH_SIZE", args.kernel)
        w_avg, w_n, w_copy = counter_per_dispatch(args.write, "WRITE_SIZE", args.kernel)
        f_fac = COPY_BYTES / (f_copy * 1024.0)
        w_fac = COPY_BYTES / (w_copy * 1024.0)
        total = f_avg * 1024.0 * f_fac + w_avg * 1024.0 * w_fac
        rec = {
            "workload": args.workload, "kernel_class": args.kernel_class, "kernel_regex": args.kernel,
            "digest": source_digest(args.kernel_class),
            "fetch_kib_per_dispatch": round(f_avg, 3), "write_kib_per_dispatch": round(w_avg, 3),
            "dispatches": [f_n, w_n],
            "copy_fetch_kib": f_copy, "copy_write_kib": w_copy,
            "fetch_factor": round(f_fac, 4), "write_factor": round(w_fac, 4),
            "hbm_bytes_per_launch": round(total),
            "avg_duration_us": round(mine[0]["avg_ns"] / 1e3, 3) if mine else None,
            "commands": {"kernel_trace": args.command_kt, "fetch": args.command_fetch, "write": args.command_write},
        }
        md += ["## HBM traffic from counters\n",
               f"Commands:\n\n```\n{args.command_fetch}\n{args.command_write}\n```\n",
               "| quantity | value |", "|---|---|",
               f"| calibration copy FETCH_SIZE (KiB, 256 MiB read) | {f_copy:.1f} |",
               f"| calibration copy WRITE_SIZE (KiB, 256 MiB written) | {w_copy:.1f} |",
               f"| fetch factor | {f_fac:.4f} |", f"| write factor | {w_fac:.4f} |",
               f"| {args.kernel_class} FETCH_SIZE per dispatch (KiB, raw) | {f_avg:.1f} ({f_n} dispatches) |",
               f"| {args.kernel_class} WRITE_SIZE per dispatch (KiB, raw) | {w_avg:.1f} ({w_n} dispatches) |",
               f"| {args.kernel_class} calibrated HBM bytes per launch | {total / 1e6:.3f} MB |", ""]
    with open(args.out_md, "w") as f:
        f.write("\n".join(md))
    if rec is not None and args.out_json:
        # one file per workload, one record per kernel class (a rerun for a
        # class replaces that class's record only)
        try:
            with open(args.out_json) as f:
                doc = json.load(f)
        except (OSError, ValueError):
            doc = {}
        records = doc.get("records", {})
        records[args.kernel_class] = rec
        with open(args.out_json, "w") as f:
            json.dump({"workload": args.workload, "records": records}, f, indent=1)
            f.write("\n")


def load_traffic(path: str, kernel_class: str) -> Optional[int]:
    """HBM bytes per launch of one kernel class from a workload's traffic
    file, or None when there is no record for the class or the class's
    sources changed since the counters were taken."""
    try:
        with open(path) as f:
            doc = json.load(f)
    except (OSError, ValueError):
        return None
    rec = doc.get("records", {}).get(kernel_class)
    if rec is None:
        return None
    cls = rec.get("digest_class", kernel_class)
    if cls not in KERNEL_SOURCES or rec.get("digest") != source_digest(cls):
        return None
    return int(rec["hbm_bytes_per_launch"])





# ---------------------------------------------------------------------------
# per-workload summary: every kernel of one workload's run, by class
# ---------------------------------------------------------------------------
SIMDS = 1024          # 256 CUs x 4 SIMDs
CLOCK_GHZ = 2.4       # MI355X peak engine clock
MFMA_PEAK_TFLOPS = 2500.0

_EPI_CLASS = {"4": "gemm_qkv", "2": "gemm_gate_up", "5": "frame_proj", "1": "modulation", "3": "modulation"}


def _epi(name: str) -> Optional[str]:
    """Epilogue template argument of a GEMM kernel name (its first argument,
    or the third for the skinny kernels)."""
    m = re.search(r"gemm_(\w+)<([^>]*)>", name)
    if not m:
        return None
    args = [a.strip() for a in m.group(2).split(",")]
    if m.group(1) in ("skinny_lds",):
        return args[2] if len(args) > 2 else None
    if m.group(1) in ("skinny", "tiled"):
        return args[3] if m.group(1) == "skinny" and len(args) > 3 else (args[1] if len(args) > 1 else None)
    return args[0]


def classify(names: List[str]) -> List[str]:
    """Kernel class of each dispatch of one run, in dispatch order.  The fp32
    GEMM after the attention (or its merge) is the output projection, the one
    after the gate|up GEMM the down projection."""
    out, prev = [], ""
    for n in names:
        if "reflex::" not in n:
            c = "other"
        elif re.search(r"attn(16p|16|_pair)?_kernel", n):
            c = "attention"
        elif "attn_merge" in n:
            c = "attn_merge"
        elif "resid_norm" in n:
            c = "resid_norm"
        elif "final_euler" in n:
            c = "final_euler"
        elif "embed_norm" in n:
            c = "embed_norm"
        elif "ring_write" in n:
            c = "ring_write"
        elif "cond_kernel" in n:
            c = "modulation"
        elif "gemm_" in n:
            e = _epi(n)
            if e == "0":
                c = "gemm_o" if prev in ("attention", "attn_merge") else ("gemm_down" if prev == "gemm_gate_up"
                                                                          else "gemm_f32")
            else:
                c = _EPI_CLASS.get(e, "gemm")
        else:
            c = re.sub(r".*reflex::(\w+).*", r"\1", n)
        out.append(c)
        if c != "other":
            prev = c
    return out


def _dispatches(path: str) -> List[dict]:
    """Counter CSV -> one record per dispatch: name, grid, duration, counters."""
    recs: Dict[str, dict] = {}
    order: List[str] = []
    for r in _rows(path):
        k = r["Dispatch_Id"]
        if k not in recs:
            recs[k] = {"name": r["Kernel_Name"], "grid": int(r["Grid_Size"]),
                       "dur_ns": float(r["End_Timestamp"]) - float(r["Start_Timestamp"]), "c": {}}
            order.append(k)
        c = recs[k]["c"]
        c[r["Counter_Name"]] = c.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [recs[k] for k in sorted(order, key=lambda x: int(x))]


def _trace_dispatches(path: str) -> List[dict]:
    out = []
    for r in _rows(path):
        if r.get("Kind", "KERNEL_DISPATCH") != "KERNEL_DISPATCH":
            continue
        out.append({"name": r["Kernel_Name"], "grid": int(r["Grid_Size_X"]) * int(r.get("Grid_Size_Y", 1) or 1)
                    * int(r.get("Grid_Size_Z", 1) or 1),
                    "dur_ns": float(r["End_Timestamp"]) - float(r["Start_Timestamp"]),
                    "start": float(r["Start_Timestamp"])})
    out.sort(key=lambda d: d["start"])
    return out


def _copy_value(disp: List[dict], counter: str) -> float:
    vals = [d["c"][counter] for d in disp if COPY_PATTERN.search(d["name"]) and d["grid"] == COPY_GRID
            and counter in d["c"]]
    if not vals:
        raise ValueError(f"no calibration copy dispatch with {counter}")
    return sorted(vals)[len(vals) // 2]


STAMP_PATTERN = re.compile(r"stamp_kernel")


def stamp_validation(trace: str, stamp_us: Dict[str, float]) -> List[dict]:
    """Per kernel class: the kernel-trace durations of the dispatches that the
    in-graph class timing stamped (a library dispatch right after two stamp
    kernels) against the stamp figure the same run reported."""
    tr = _trace_dispatches(trace)
    tcls = classify([d["name"] for d in tr])
    acc: Dict[str, List[float]] = {}
    for i in range(2, len(tr)):
        if tcls[i] != "other" and STAMP_PATTERN.search(tr[i - 1]["name"]) and \
                STAMP_PATTERN.search(tr[i - 2]["name"]):
            acc.setdefault(tcls[i], []).append(tr[i]["dur_ns"] / 1e3)
    rows = []
    for c, durs in acc.items():
        if c in stamp_us:
            t = sum(durs) / len(durs)
            rows.append({"class": c, "stamped": len(durs), "trace_us": t, "stamp_us": stamp_us[c],
                         "ratio": stamp_us[c] / t})
    rows.sort(key=lambda r: r["class"])
    return rows


def summarize(workload: str, trace: str, fetch: str, write: str, mfma: str, commands: Dict[str, str],
              out_md: str, out_json: Optional[str], stamp_trace: Optional[str] = None,
              stamp_us: Optional[Dict[str, float]] = None) -> dict:
    """Per (class, kernel, grid): dispatches, average duration (kernel trace),
    calibrated HBM bytes per dispatch (FETCH_SIZE and WRITE_SIZE runs), MFMA
    busy fraction (SQ_VALU_MFMA_BUSY_CYCLES over duration x clock x SIMDs) and
    MFMA TFLOP/s (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 flops)."""
    tr = _trace_dispatches(trace)
    tcls = classify([d["name"] for d in tr])
    groups: Dict[Tuple[str, str, int], dict] = {}

    def grp(c, d):
        key = (c, _short(d["name"]), d["grid"])
        return groups.setdefault(key, {"n": 0, "dur": 0.0, "fetch": [], "write": [], "busy": [], "mops": [],
                                       "cdur": []})

    for c, d in zip(tcls, tr):
        if c == "other":
            continue
        g = grp(c, d)
        g["n"] += 1
        g["dur"] += d["dur_ns"]
    fd, wd, md = _dispatches(fetch), _dispatches(write), _dispatches(mfma)
    f_fac = COPY_BYTES / (_copy_value(fd, "FETCH_SIZE") * 1024.0)
    w_fac = COPY_BYTES / (_copy_value(wd, "WRITE_SIZE") * 1024.0)
    for disp, field in ((fd, "fetch"), (wd, "write"), (md, "mfma")):
        for c, d in zip(classify([x["name"] for x in disp]), disp):
            if c == "other":
                continue
            g = grp(c, d)
            if field == "fetch":
                g["fetch"].append(d["c"]["FETCH_SIZE"] * 1024.0 * f_fac)
            elif field == "write":
                g["write"].append(d["c"]["WRITE_SIZE"] * 1024.0 * w_fac)
            else:
                g["busy"].append(d["c"].get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0))
                g["mops"].append(d["c"].get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0))
                g["cdur"].append(d["dur_ns"])
    avg = lambda xs: sum(xs) / len(xs) if xs else None  # noqa: E731
    rows = []
    for (c, name, grid), g in groups.items():
        if g["n"] == 0:
            continue
        dur = g["dur"] / g["n"]
        hbm = (avg(g["fetch"]) or 0.0) + (avg(g["write"]) or 0.0) if g["fetch"] and g["write"] else None
        busy = avg(g["busy"])
        cdur = avg(g["cdur"])
        rows.append({"class": c, "kernel": name, "grid": grid, "dispatches": g["n"], "avg_us": dur / 1e3,
                     "total_us": g["dur"] / 1e3, "hbm_bytes": hbm,
                     "hbm_gbs": hbm / dur if hbm is not None else None,
                     "mfma_busy": busy / (cdur * CLOCK_GHZ * SIMDS) if busy is not None and cdur else None,
                     "mfma_tflops": (avg(g["mops"]) * 512) / (cdur * 1e3) if g["mops"] and cdur else None})
    rows.sort(key=lambda r: -r["total_us"])
    lines = [f"# rocprofv3 summary: {workload}\n",
             "Every kernel of a profiled run of the workload (ring filled, then ticks of frame write + chunk "
             "through the captured graphs), grouped by kernel class, kernel and grid.  Durations from the "
             "kernel trace.  HBM bytes per dispatch: FETCH_SIZE and WRITE_SIZE (KiB) of their own runs, each "
             f"scaled by what it reads for a plain 256 MiB copy in the same process (factors {f_fac:.4f} and "
             f"{w_fac:.4f}).  MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES / (duration x {CLOCK_GHZ} GHz x {SIMDS} "
             "SIMDs), from the counter run's own durations; MFMA TFLOP/s: SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 "
             "flops / duration.\n",
             "Commands:\n", "```"] + [f"{k}: {v}" for k, v in commands.items()] + ["```\n",
             "| class | kernel | grid (threads) | dispatches | avg us | total us | HBM MB / dispatch | HBM GB/s | "
             "MFMA busy | MFMA TFLOP/s |", "|---|---|---|---|---|---|---|---|---|---|"]
    fmt = lambda v, f: (f % v) if v is not None else "-"  # noqa: E731
    for r in rows:
        lines.append(f"| {r['class']} | `{r['kernel']}` | {r['grid']} | {r['dispatches']} | {r['avg_us']:.2f} | "
                     f"{r['total_us']:.1f} | {fmt(r['hbm_bytes'] and r['hbm_bytes'] / 1e6, '%.3f')} | "
                     f"{fmt(r['hbm_gbs'], '%.1f')} | {fmt(r['mfma_busy'] and 100 * r['mfma_busy'], '%.1f %%')} | "
                     f"{fmt(r['mfma_tflops'], '%.1f')} |")
    if stamp_trace and stamp_us:
        lines += ["", "In-graph class timing against the trace of the same dispatches: the benchmark's per-class "
                  "durations come from wall-clock stamp kernels around each launch inside the chunk's graph "
                  "(reflex_profile_graph).  The stamp run (command `stamps`) makes that measurement under the "
                  "kernel tracer; per class, the stamp figure it reported against the traced durations of the "
                  "stamped dispatches themselves.", "",
                  "| class | stamped dispatches | trace avg us | stamp avg us | stamp / trace |",
                  "|---|---|---|---|---|"]
        for r in stamp_validation(stamp_trace, stamp_us):
            lines.append(f"| {r['class']} | {r['stamped']} | {r['trace_us']:.2f} | {r['stamp_us']:.2f} | "
                         f"{r['ratio']:.3f} |")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    if out_json:
        # one traffic record per class: its most time-consuming kernel; the
        # attention record covers the kernel and its split merge (one unit per layer)
        best: Dict[str, dict] = {}
        for r in rows:
            if r["class"] not in best and r["hbm_bytes"] is not None:
                best[r["class"]] = r
        records = {}
        for c, r in best.items():
            cls = c if c in KERNEL_SOURCES else "all"
            hbm = r["hbm_bytes"]
            dur = r["avg_us"]
            if c == "attention" and "attn_merge" in best:
                hbm += best["attn_merge"]["hbm_bytes"]
                dur += best["attn_merge"]["avg_us"]
            records[c] = {"workload": workload, "kernel_class": c, "kernel": r["kernel"], "grid": r["grid"],
                          "digest": source_digest(cls), "digest_class": cls,
                          "hbm_bytes_per_launch": round(hbm), "avg_duration_us": round(dur, 3),
                          "mfma_busy": r["mfma_busy"] and round(r["mfma_busy"], 4)}
        with open(out_json, "w") as f:
            json.dump({"workload": workload, "fetch_factor": round(f_fac, 4), "write_factor": round(w_fac, 4),
                       "commands": commands, "records": records}, f, indent=1)
            f.write("\n")
    return {"rows": rows}


def main_summarize(argv: Optional[List[str]] = None) -> None:
    ap = argparse.ArgumentParser(description="per-workload kernel summary from a kernel trace and counter runs")
    ap.add_argument("--workload", required=True)
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--mfma", required=True)
    ap.add_argument("--command", action="append", default=[], help="NAME=COMMAND, repeated")
    ap.add_argument("--out-md", required=True)
    ap.add_argument("--out-json")
    ap.add_argument("--stamp-trace", help="kernel trace of a `bench.py --profile-workload W --stamps` run")
    ap.add_argument("--stamp-log", help="that run's output: its JSON line holds stamp_us")
    a = ap.parse_args(argv)
    cmds = dict(c.split("=", 1) for c in a.command)
    stamp_us = None
    if a.stamp_log:
        with open(a.stamp_log) as f:
            for line in f:
                if line.startswith("{") and "stamp_us" in line:
                    stamp_us = json.loads(line)["stamp_us"]
    summarize(a.workload, a.trace, a.fetch, a.write, a.mfma, cmds, a.out_md, a.out_json, a.stamp_trace, stamp_us)


if __name__ == "__main__":
    import sys

    if len(sys.argv) > 1 and sys.argv[1] == "summarize":
        main_summarize(sys.argv[2:])
    else:
        main()
