"""Summarise rocprofv3 output of the forward benchmark into a short text record.

    python -m paper_2609_07816_amd.rocprof_summary --name NAME --first-kernel SUBSTR \\
        --trace DIR --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR \\
        --copy-bytes N --algorithmic-bytes N --commands FILE

One forward is the walk kernel, preceded for a packed batch by the kernel that orders its
sequences and, for an in-place variance update, by a copy of the initial variances. The kernel
trace is cut into forwards at every dispatch whose name contains SUBSTR (the forward's first
kernel); a forward's span runs from its first dispatch's start to the last end before the next
forward. The per-kernel duration statistics come from the same trace.

The per-dispatch FETCH_SIZE and WRITE_SIZE counters (KiB) of every kernel of the forward are
summed per forward, and the same two counters of a plain device copy of N bytes give each
counter's scale on this device (bytes moved / counter bytes); the forward's HBM traffic is its
counters times those scales. Writes profiles/NAME.md (with the commands that produced the data)
and profiles/NAME.json (read by bench.py, together with the hash of the kernel sources it
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
CSRC = os.path.join(ROOT, "paper_2609_07816_amd", "csrc")
FORWARD_KERNELS = ("walk_kernel", "order_kernel", "copy_floats_kernel")


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


def short(name: str) -> str:
    for key in FORWARD_KERNELS:
        if key in name:
            return key.rstrip("_")
    return name[:40]


def is_forward(name: str) -> bool:
    return any(key in name for key in FORWARD_KERNELS)


def forwards(dirname: str, first: str):
    """Dispatches of the kernel trace grouped into forwards (lists of (name, start, end))."""
    rows = list(csv.DictReader(open(_one(dirname, "*kernel_trace.csv"))))
    ev = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"])
                for r in rows if is_forward(r["Kernel_Name"]))
    groups = []
    for s, e, n in ev:
        if first in n or not groups:
            groups.append([])
        groups[-1].append((n, s, e))
    return groups


def kernel_stats(groups):
    per = collections.defaultdict(list)
    for g in groups:
        for n, s, e in g:
            per[short(n)].append(e - s)
    return {k: dict(calls=len(v), avg_ns=sum(v) / len(v), min_ns=min(v), max_ns=max(v))
            for k, v in per.items()}


def counter_per_forward(dirname: str, first: str):
    """Sum over one forward of a counter's per-dispatch values (KiB), averaged over forwards."""
    rows = list(csv.DictReader(open(_one(dirname, "*counter_collection.csv"))))
    rows = [r for r in rows if is_forward(r["Kernel_Name"])]
    rows.sort(key=lambda r: int(r.get("Dispatch_Id", 0)))
    sums = []
    for r in rows:
        if first in r["Kernel_Name"] or not sums:
            sums.append(0.0)
        sums[-1] += float(r["Counter_Value"])
    if not sums:
        raise ValueError(f"no forward kernels in {dirname}")
    return sum(sums) / len(sums), len(sums)


def copy_kib(dirname: str, kernel: str):
    rows = list(csv.DictReader(open(_one(dirname, "*counter_collection.csv"))))
    vals = [float(r["Counter_Value"]) for r in rows if kernel in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"no dispatch of {kernel} in {dirname}")
    return sum(vals) / len(vals)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--name", required=True)
    ap.add_argument("--first-kernel", default="walk_kernel")
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

    groups = forwards(args.trace, args.first_kernel)
    steady = groups[1:] if len(groups) > 1 else groups  # the first forward pays first-use costs
    spans = [max(e for _, _, e in g) - min(s for _, s, _ in g) for g in steady]
    span_ns = sum(spans) / len(spans)
    stats = kernel_stats(steady)
    fk, nf = counter_per_forward(args.fetch, args.first_kernel)
    wk, nw = counter_per_forward(args.write, args.first_kernel)
    cfk = copy_kib(args.copy_fetch, args.copy_kernel)
    cwk = copy_kib(args.copy_write, args.copy_kernel)
    f_scale = args.copy_bytes / (cfk * 1024.0)
    w_scale = args.copy_bytes / (cwk * 1024.0)
    read_b = fk * 1024.0 * f_scale
    write_b = wk * 1024.0 * w_scale
    rec = dict(unit="one forward call (every kernel of the call)",
               kernel_source_sha256=source_hash(), forwards=len(steady),
               forward_span_ns=span_ns, kernels=stats,
               fetch_kib_per_forward=fk, write_kib_per_forward=wk, counter_forwards=[nf, nw],
               copy_bytes=args.copy_bytes, copy_fetch_kib=cfk, copy_write_kib=cwk,
               fetch_scale=f_scale, write_scale=w_scale, hbm_read_bytes=read_b,
               hbm_write_bytes=write_b, traffic_bytes=read_b + write_b,
               algorithmic_bytes=args.algorithmic_bytes)
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", args.name + ".json"), "w") as f:
        json.dump(rec, f, indent=1)
    cmds = open(args.commands).read().strip()
    gb = 1e9
    order = sorted(stats.items(), key=lambda kv: -kv[1]["avg_ns"] * kv[1]["calls"])
    krows = "\n".join(
        f"| {k} | {v['calls']} | {v['avg_ns'] / 1e3:.1f} us | {v['min_ns'] / 1e3:.1f} us | "
        f"{v['max_ns'] / 1e3:.1f} us |" for k, v in order)
    md = f"""# {args.name}

Unit: one forward call (every kernel of the call; here the walk kernel alone).
Kernel source sha256 (all of csrc/): `{rec['kernel_source_sha256']}`

## Forward span (rocprofv3 --kernel-trace --stats)

Average span of {len(steady)} forwards (first dispatch start to last dispatch end, the first
forward of the run excluded): **{span_ns / 1e3:.1f} us**.

| kernel | dispatches | average | min | max |
|---|---|---|---|---|
{krows}

## HBM bytes per forward (rocprofv3 --pmc, one counter per run)

| counter | forward (KiB) | plain copy of {args.copy_bytes / 2**30:.2f} GiB (KiB) | scale (bytes moved / counter bytes) | forward bytes |
|---|---|---|---|---|
| FETCH_SIZE | {fk:.0f} | {cfk:.0f} | {f_scale:.4f} | {read_b / gb:.4f} GB |
| WRITE_SIZE | {wk:.0f} | {cwk:.0f} | {w_scale:.4f} | {write_b / gb:.4f} GB |

Traffic per forward: {(read_b + write_b) / gb:.4f} GB; algorithmic bytes per forward:
{args.algorithmic_bytes / gb:.4f} GB (ratio {(read_b + write_b) / args.algorithmic_bytes:.3f}). Every
workgroup of a head (one per block of value columns) reads the head's q, k, alpha and omega;
the blocks of one head run on one XCD, so all but the first read should hit its L2, and
traffic above the algorithmic bytes counts the reads that did not.
Achieved on algorithmic bytes at the traced span: {args.algorithmic_bytes / (span_ns * 1e-9) / gb:.1f} GB/s.

## Commands (run from the repository root on the GPU host, TMPDIR=/tmp)

```
{cmds}
python -m paper_2609_07816_amd.rocprof_summary --name {args.name} \\
    --first-kernel {args.first_kernel} --trace {args.trace} --fetch {args.fetch} \\
    --write {args.write} --copy-fetch {args.copy_fetch} --copy-write {args.copy_write} \\
    --copy-bytes {args.copy_bytes} --algorithmic-bytes {args.algorithmic_bytes} \\
    --commands <file with the commands above>
```
"""
    with open(os.path.join(ROOT, "profiles", args.name + ".md"), "w") as f:
        f.write(md)
    print(json.dumps({k: v for k, v in rec.items() if k != "kernels"}))


if __name__ == "__main__":
    main()
