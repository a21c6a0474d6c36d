"""Summarise rocprofv3 output of a benchmark run into a short text record.

    python -m paper_2609_07816_amd.rocprof_summary --name NAME --unit-kernels K1,K2,.. \\
        --first-kernel K1 --trace DIR --fetch DIR --write DIR --copy-fetch DIR \\
        --copy-write DIR --copy-bytes N --algorithmic-bytes N --commands FILE [--sq DIR ...]

A unit (one forward call, one decode step, one gain scan) is a group of consecutive dispatches
of the kernels named in --unit-kernels; the kernel trace is cut into units at every dispatch of
--first-kernel. A unit's span runs from its first dispatch's start to its last dispatch's end;
the per-kernel duration statistics come from the same trace.

The per-dispatch FETCH_SIZE and WRITE_SIZE counters (KiB) of every kernel of a unit are summed
per unit, and the same two counters of a plain device copy of N bytes give each counter's scale
on this device (bytes moved / counter bytes); a unit's HBM traffic is its counters times those
scales; each kernel's counted bytes over its average duration give its achieved bandwidth
(FETCH_SIZE counts what leaves the L2 for the memory fabric, last-level cache hits included, so
this bounds the HBM rate from above). Optional --sq directories hold further counter runs (SQ_* and the like), reported per
kernel as averages per dispatch. Writes profiles/NAME.md (with the commands that produced the
data) and profiles/NAME.json (read by bench.py, together with the hash of the kernel sources it
describes).
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
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
CSRC = os.path.join(ROOT, "paper_2609_07816_amd", "csrc")


def source_hash(names=None) -> str:
    """Hash of the library's HIP sources and headers that define and launch the kernels a
    summary measured (`names`, file names under csrc/; default: all of them). A summary is stale
    once any of those files has changed."""
    if names is None:
        names = [n for n in os.listdir(CSRC) if n.endswith((".hip", ".h"))]
    h = hashlib.sha256()
    for name in sorted(names):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def _all(dirname: str, pattern: str):
    hits = sorted(glob.glob(os.path.join(dirname, "**", pattern), recursive=True))
    if not hits:
        raise FileNotFoundError(f"{pattern} under {dirname}")
    return hits


class Units:
    def __init__(self, kernels, first, window=None):
        self.kernels = kernels
        self.first = first
        self.window = window  # (a, b): keep units a..b-1 only

    def short(self, name: str):
        for key in self.kernels:
            if key in name:
                return key
        return None

    def group(self, rows, key_start):
        """Rows (dicts) in dispatch order, grouped into units."""
        groups = []
        for r in rows:
            k = self.short(r["Kernel_Name"])
            if k is None:
                continue
            if k == self.first or not groups:
                groups.append([])
            groups[-1].append((k, r))
        if self.window:
            groups = groups[self.window[0]:self.window[1]]
        return groups


def trace_units(dirname, units):
    rows = []
    for f in _all(dirname, "*kernel_trace.csv"):
        rows += list(csv.DictReader(open(f)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    return units.group(rows, "Start_Timestamp")


def counter_rows(dirname):
    rows = []
    for f in _all(dirname, "*counter_collection.csv"):
        rows += list(csv.DictReader(open(f)))
    rows.sort(key=lambda r: int(r.get("Dispatch_Id", 0)))
    return rows


def counter_per_unit(dirname, units, counter):
    """Average over units of the per-unit sum of one counter, and its per-kernel averages."""
    rows = [r for r in counter_rows(dirname) if r["Counter_Name"].startswith(counter)]
    per_disp = collections.OrderedDict()
    for r in rows:  # one value per (dispatch, counter); sum dimension instances if repeated
        key = (int(r.get("Dispatch_Id", 0)), r["Kernel_Name"])
        per_disp[key] = per_disp.get(key, 0.0) + float(r["Counter_Value"])
    disp_rows = [{"Kernel_Name": k[1], "v": v} for k, v in per_disp.items()]
    groups = units.group(disp_rows, None)
    steady = groups[1:] if len(groups) > 1 else groups
    sums = [sum(r["v"] for _, r in g) for g in steady]
    perk = collections.defaultdict(list)
    for g in steady:
        for k, r in g:
            perk[k].append(r["v"])
    if not sums:
        raise ValueError(f"no unit kernels in {dirname}")
    return sum(sums) / len(sums), {k: sum(v) / len(v) for k, v in perk.items()}, len(steady)


def copy_kib(dirname: str, kernel: str):
    rows = counter_rows(dirname)
    vals = [float(r["Counter_Value"]) for r in rows if kernel in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"no dispatch of {kernel} in {dirname}")
    return sum(vals) / len(vals)


def sq_counters(dirs, units):
    """Per-kernel averages per dispatch of every counter in the given runs."""
    out = collections.defaultdict(dict)
    for d in dirs:
        rows = counter_rows(d)
        acc = collections.defaultdict(lambda: collections.defaultdict(float))
        for r in rows:
            k = units.short(r["Kernel_Name"])
            if k is None:
                continue
            acc[(k, r["Counter_Name"])][int(r.get("Dispatch_Id", 0))] += float(r["Counter_Value"])
        for (k, c), per in acc.items():
            vals = list(per.values())
            out[k][c] = sum(vals) / len(vals)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--name", required=True)
    ap.add_argument("--title", default="")
    ap.add_argument("--unit-kernels", required=True, help="comma-separated kernel names")
    ap.add_argument("--first-kernel", required=True)
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--copy-fetch", required=True)
    ap.add_argument("--copy-write", required=True)
    ap.add_argument("--copy-kernel", default="copyBuffer")
    ap.add_argument("--copy-bytes", type=int, required=True)
    ap.add_argument("--algorithmic-bytes", type=int, required=True)
    ap.add_argument("--sq", nargs="*", default=[])
    ap.add_argument("--window", default="", help="a:b as a python slice of the run's units "
                    "(negative counts from the end; the first kept unit is still dropped as a "
                    "warm-up)")
    ap.add_argument("--notes", default="", help="text file appended to the summary")
    ap.add_argument("--commands", required=True, help="text file with the commands that ran")
    ap.add_argument("--sources", default="", help="comma-separated csrc/ files that define and "
                    "launch the measured kernels (default: all of csrc/)")
    args = ap.parse_args()

    window = None
    if args.window:  # python slice bounds: "a:b", "-n:" (the last n units), "-n:-1"
        a, b = args.window.split(":")
        window = (int(a) if a else None, int(b) if b else None)
    units = Units(args.unit_kernels.split(","), args.first_kernel, window)
    groups = trace_units(args.trace, units)
    steady = groups[1:] if len(groups) > 1 else groups  # the first unit pays first-use costs
    spans = [max(int(r["End_Timestamp"]) for _, r in g) -
             min(int(r["Start_Timestamp"]) for _, r in g) for g in steady]
    span_ns = sum(spans) / len(spans)
    per = collections.defaultdict(list)
    for g in steady:
        for k, r in g:
            per[k].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    stats = {k: dict(calls=len(v), avg_ns=sum(v) / len(v), min_ns=min(v), max_ns=max(v))
             for k, v in per.items()}
    fk, fkk, nf = counter_per_unit(args.fetch, units, "FETCH_SIZE")
    wk, wkk, nw = counter_per_unit(args.write, units, "WRITE_SIZE")
    cfk = copy_kib(args.copy_fetch, args.copy_kernel)
    cwk = copy_kib(args.copy_write, args.copy_kernel)
    f_scale = args.copy_bytes / (cfk * 1024.0)
    w_scale = args.copy_bytes / (cwk * 1024.0)
    read_b = fk * 1024.0 * f_scale
    write_b = wk * 1024.0 * w_scale
    sq = sq_counters(args.sq, units) if args.sq else {}
    sources = sorted(args.sources.split(",")) if args.sources else None
    rec = dict(unit=args.title or args.name, kernel_source_sha256=source_hash(sources),
               kernel_sources=sources,
               units=len(steady), span_ns=span_ns, kernels=stats,
               fetch_kib_per_unit=fk, write_kib_per_unit=wk, counter_units=[nf, nw],
               fetch_kib_per_kernel=fkk, write_kib_per_kernel=wkk,
               copy_bytes=args.copy_bytes, copy_fetch_kib=cfk, copy_write_kib=cwk,
               fetch_scale=f_scale, write_scale=w_scale, hbm_read_bytes=read_b,
               hbm_write_bytes=write_b, traffic_bytes=read_b + write_b,
               algorithmic_bytes=args.algorithmic_bytes, counters_per_kernel=sq)
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", args.name + ".json"), "w") as f:
        json.dump(rec, f, indent=1)
    cmds = open(args.commands).read().strip()
    gb = 1e9
    order = sorted(stats.items(), key=lambda kv: -kv[1]["avg_ns"] * kv[1]["calls"])
    def moved(k, v):  # the kernel's counted bytes over its average duration, and of 8 TB/s
        gbs = (fkk.get(k, 0) * f_scale + wkk.get(k, 0) * w_scale) * 1024 / v["avg_ns"]
        return f"{gbs:.0f} GB/s ({gbs / HBM_PEAK_GBS:.2f})"

    krows = "\n".join(
        f"| {k} | {v['calls']} | {v['avg_ns'] / 1e3:.1f} us | {v['min_ns'] / 1e3:.1f} us | "
        f"{v['max_ns'] / 1e3:.1f} us | {fkk.get(k, 0) * f_scale * 1024 / gb:.4f} GB | "
        f"{wkk.get(k, 0) * w_scale * 1024 / gb:.4f} GB | {moved(k, v)} |" for k, v in order)
    sq_md = ""
    if sq:
        names = sorted({c for d in sq.values() for c in d})
        sq_md = "\n## Counters per dispatch (rocprofv3 --pmc)\n\n| counter | " + \
            " | ".join(k for k, _ in order) + " |\n|---|" + "---|" * len(order) + "\n"
        for c in names:
            sq_md += f"| {c} | " + " | ".join(
                f"{sq.get(k, {}).get(c, float('nan')):.4g}" for k, _ in order) + " |\n"
    notes = open(args.notes).read().strip() + "\n" if args.notes else ""
    md = f"""# {args.name}

Unit: {args.title or args.name}.
Kernel source sha256 ({', '.join(sources) if sources else 'all of csrc/'}):
`{rec['kernel_source_sha256']}`

## Span and kernels (rocprofv3 --kernel-trace --stats)

Average span of {len(steady)} units (first dispatch start to last dispatch end, the first unit of
the run excluded): **{span_ns / 1e3:.1f} us**.

| kernel | dispatches | average | min | max | HBM read / dispatch | HBM write / dispatch | read + write / average (of 8 TB/s) |
|---|---|---|---|---|---|---|---|
{krows}

## HBM bytes per unit (rocprofv3 --pmc, one counter per run)

| counter | unit (KiB) | plain copy of {args.copy_bytes / 2**30:.2f} GiB (KiB) | scale (bytes moved / counter bytes) | unit bytes |
|---|---|---|---|---|
| FETCH_SIZE | {fk:.0f} | {cfk:.0f} | {f_scale:.4f} | {read_b / gb:.4f} GB |
| WRITE_SIZE | {wk:.0f} | {cwk:.0f} | {w_scale:.4f} | {write_b / gb:.4f} GB |

Traffic per unit: {(read_b + write_b) / gb:.4f} GB; algorithmic bytes per unit:
{args.algorithmic_bytes / gb:.4f} GB (ratio {(read_b + write_b) / args.algorithmic_bytes:.3f}).
Achieved on algorithmic bytes at the traced span: {args.algorithmic_bytes / (span_ns * 1e-9) / gb:.1f} GB/s.
{sq_md}
{notes}
## Commands (run from the repository root on the GPU host, TMPDIR=/tmp)

```
{cmds}
```
"""
    with open(os.path.join(ROOT, "profiles", args.name + ".md"), "w") as f:
        f.write(md)
    print(json.dumps({k: v for k, v in rec.items() if k not in ("kernels", "counters_per_kernel")}))


if __name__ == "__main__":
    main()
