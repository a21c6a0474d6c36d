"""Summarise rocprofv3 CSV output of the forward benchmark into a short text record.

    python -m paper_2609_07816_amd.rocprof_summary --name NAME --kernel SUBSTR \\
        --trace DIR --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR \\
        --copy-bytes N --commands FILE

Reads the kernel-trace statistics (average duration of the kernel whose name contains SUBSTR),
the per-dispatch FETCH_SIZE and WRITE_SIZE counters (KiB) of that kernel, and the same two
counters for a plain device copy of N bytes. The copy gives the scale of each counter on this
device (bytes moved / counter bytes); the kernel's HBM traffic per launch is its counters times
those scales. Writes profiles/NAME.md (with the commands that produced the data) and
profiles/NAME.json (read by bench.py, together with the hash of the kernel source it describes).
"""

from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_07816_amd", "csrc")


def source_hash() -> str:
    """Hash of every HIP source and header of the library (a summary is stale once any of the
    kernels it measured has changed)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def _one(dirname: str, pattern: str) -> str:
    hits = glob.glob(os.path.join(dirname, "**", pattern), recursive=True)
    if not hits:
        raise FileNotFoundError(f"{pattern} under {dirname}")
    return sorted(hits)[0]


def counter_kib(dirname: str, kernel: str):
    rows = list(csv.DictReader(open(_one(dirname, "*counter_collection.csv"))))
    vals = [float(r["Counter_Value"]) for r in rows if kernel in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"no dispatch of {kernel} in {dirname}")
    return sum(vals) / len(vals), len(vals)


def trace_stats(dirname: str, kernel: str):
    for r in csv.DictReader(open(_one(dirname, "*kernel_stats.csv"))):
        if kernel in r["Name"]:
            return dict(name=r["Name"], calls=int(r["Calls"]),
                        avg_ns=float(r["AverageNs"]), min_ns=float(r["MinNs"]),
                        max_ns=float(r["MaxNs"]))
    raise ValueError(f"{kernel} not in the kernel statistics of {dirname}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--name", required=True)
    ap.add_argument("--kernel", required=True)
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--copy-fetch", required=True)
    ap.add_argument("--copy-write", required=True)
    ap.add_argument("--copy-kernel", default="copyBuffer")
    ap.add_argument("--copy-bytes", type=int, required=True)
    ap.add_argument("--algorithmic-bytes", type=int, required=True)
    ap.add_argument("--commands", required=True, help="text file with the commands that ran")
    args = ap.parse_args()

    tr = trace_stats(args.trace, args.kernel)
    fk, nf = counter_kib(args.fetch, args.kernel)
    wk, nw = counter_kib(args.write, args.kernel)
    cfk, _ = counter_kib(args.copy_fetch, args.copy_kernel)
    cwk, _ = counter_kib(args.copy_write, args.copy_kernel)
    f_scale = args.copy_bytes / (cfk * 1024.0)
    w_scale = args.copy_bytes / (cwk * 1024.0)
    read_b = fk * 1024.0 * f_scale
    write_b = wk * 1024.0 * w_scale
    rec = dict(kernel=tr["name"], kernel_source_sha256=source_hash(), trace=tr,
               fetch_kib_per_dispatch=fk, write_kib_per_dispatch=wk, dispatches=[nf, nw],
               copy_bytes=args.copy_bytes, copy_fetch_kib=cfk, copy_write_kib=cwk,
               fetch_scale=f_scale, write_scale=w_scale, hbm_read_bytes=read_b,
               hbm_write_bytes=write_b, traffic_bytes=read_b + write_b,
               algorithmic_bytes=args.algorithmic_bytes)
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", args.name + ".json"), "w") as f:
        json.dump(rec, f, indent=1)
    cmds = open(args.commands).read().strip()
    gb = 1e9
    md = f"""# {args.name}

Kernel: `{tr['name']}`
Kernel source sha256: `{rec['kernel_source_sha256']}`

## Duration (rocprofv3 --kernel-trace --stats)

| calls | average | min | max |
|---|---|---|---|
| {tr['calls']} | {tr['avg_ns'] / 1e3:.1f} us | {tr['min_ns'] / 1e3:.1f} us | {tr['max_ns'] / 1e3:.1f} us |

## HBM bytes per dispatch (rocprofv3 --pmc, one counter per run)

| counter | kernel (KiB/dispatch) | plain copy of {args.copy_bytes / 2**30:.2f} GiB (KiB) | scale (bytes moved / counter bytes) | kernel bytes |
|---|---|---|---|---|
| FETCH_SIZE | {fk:.0f} | {cfk:.0f} | {f_scale:.4f} | {read_b / gb:.4f} GB |
| WRITE_SIZE | {wk:.0f} | {cwk:.0f} | {w_scale:.4f} | {write_b / gb:.4f} GB |

Traffic per launch: {(read_b + write_b) / gb:.4f} GB; algorithmic bytes per launch:
{args.algorithmic_bytes / gb:.4f} GB (ratio {(read_b + write_b) / args.algorithmic_bytes:.3f}).
Achieved on algorithmic bytes at the traced average: {args.algorithmic_bytes / (tr['avg_ns'] * 1e-9) / gb:.1f} GB/s.

## Commands (run from the repository root on the GPU host, TMPDIR=/tmp)

```
{cmds}
python -m paper_2609_07816_amd.rocprof_summary --name {args.name} --kernel {args.kernel} \\
    --trace {args.trace} --fetch {args.fetch} --write {args.write} \\
    --copy-fetch {args.copy_fetch} --copy-write {args.copy_write} \\
    --copy-bytes {args.copy_bytes} --algorithmic-bytes {args.algorithmic_bytes} \\
    --commands <file with the commands above>
```
"""
    with open(os.path.join(ROOT, "profiles", args.name + ".md"), "w") as f:
        f.write(md)
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
