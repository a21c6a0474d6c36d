"""Benchmark of the KDN forward hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]

Workload: Diagonal KDN forward, B=4, H=16, T=4096, dk=dv=128, bf16 q/k/v/gates/noise, float32
state (the mixer shape of the paper's 750M model: 16 heads x 128 at d_model 2048, 4K context,
batch 4 as in its throughput probe). Inputs are seeded synthetic tensors resident in HBM before
timing starts. One step = one full forward over the batch (every stage of the path: the
variance chain and gains, the chunk operands, the chunkwise triangular solve, the state update,
the outputs and the final states; all in one walk kernel).

Prints one JSON line with tokens/s, the roofline position of one forward call (algorithmic bytes
per call / the HIP-event duration of the call on the caller's stream, against the 8 TB/s HBM
peak) and the CPU oracle timed on a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "KDN forward tokens/s (H=16,d=128,T=4096) + % of MFMA/HBM roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16


def algorithmic_bytes(B, T, H, dk, dv, in_bytes, variant="diag"):
    """Minimum HBM traffic of one forward: every input read once, o written once, final states
    written once (no initial state is read here: S0 = 0, P0 = 1)."""
    per_tok_head = (2 * dk + dv) * in_bytes + dv * in_bytes  # q, k, v in; o out
    if variant == "diag":
        per_tok_head += 2 * dk * in_bytes + in_bytes          # alpha, omega per channel; r
    else:
        per_tok_head += 3 * in_bytes                          # scalar alpha, omega, r
    states = H * B * (dk * dv * 4 + (dk if variant == "diag" else 1) * 4)
    return B * T * H * per_tok_head + states


def algorithmic_flops(B, T, H, dk, dv, C=64):
    """Dense flop count of the chunked WY form per token-head: 6 dk dv + 10 C d + C^2 / 3."""
    d = dk
    return B * T * H * (6 * d * dv + 10 * C * d + C * C / 3.0)


def decode_bytes(R, H, dk, dv, in_bytes):
    """Minimum HBM traffic of one Diagonal decode step: the state slot read and written
    (S and P in float32), the token's inputs read and o written."""
    per_row_head = 2 * (dk * dv * 4 + dk * 4) + (2 * dk + dv + 2 * dk) * in_bytes + in_bytes \
        + dv * in_bytes
    return R * H * per_row_head


def decode_measure(kdn, W, torch, steps=64):
    """Diagonal decode steps at the serving shape (R = 256 rows, H = 16, d = 128, bf16 inputs,
    a float32 state pool of 256 slots updated in place): per-step HIP-event durations on the
    caller's stream, against the HBM roofline. Reported beside the forward line."""
    import numpy as np
    R, H, d = 256, 16, 128
    x = W.draw_inputs("diag", "bf16", R, 1, H, d, d, seed=1004, random_state=True)
    dev = {n: torch.from_numpy(x.stored[n].view(np.int16)).view(torch.bfloat16).cuda()[:, 0]
           for n in ("q", "k", "v", "alpha", "omega", "r")}
    S = torch.from_numpy(x.S0.astype(np.float32)).cuda()
    P = torch.from_numpy(x.P0.astype(np.float32)).cuda()
    stream = torch.cuda.current_stream()
    args = [dev[n] for n in ("q", "k", "v", "alpha", "omega", "r")]
    for _ in range(5):
        kdn.decode_step("diag", *args, S, P, mu=x.mu, scale=x.scale)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        ev[i][0].record(stream)
        kdn.decode_step("diag", *args, S, P, mu=x.mu, scale=x.scale)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    nbytes = decode_bytes(R, H, d, d, 2)
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"workload": "diag-decode-R256-H16-d128 (state pool of 256 slots, bf16 inputs)",
            "kernel": "decode_kernel: one workgroup per (row, head)", "steps": steps,
            "ms_per_step_median": round(ms, 4), "tokens_per_s": round(R / (ms * 1e-3), 1),
            "algorithmic_bytes_per_step": nbytes, "achieved": round(gbs, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4)}


PROFILE = os.path.join(ROOT, "profiles", "kdn_forward_diag_B4_T4096_H16_d128.json")


def measured_traffic():
    """HBM bytes per forward from the committed rocprofv3 counter summary (FETCH_SIZE and
    WRITE_SIZE of every kernel of the forward, scaled by a plain copy of known size), or None
    when the summary is missing or was taken from a different version of the kernel sources."""
    try:
        from paper_2609_07816_amd.rocprof_summary import source_hash
        with open(PROFILE) as f:
            rec = json.load(f)
        if rec.get("kernel_source_sha256") != source_hash():
            return None
        return int(round(rec["traffic_bytes"]))
    except (OSError, ValueError, KeyError):
        return None


def cpu_baseline(x, nthreads):
    """The oracle, unchanged, on the workload's independent (batch row, head) chains at full
    length (a bounded run: about ten seconds on one core). Returns the rate in workload
    tokens/s."""
    import oracle
    names = ("q", "k", "v", "alpha", "omega", "r")
    chains = [(b, h) for b in range(x.B) for h in range(x.H)]  # every chain: ~10 s on one core
    arrs = {n: x.f64(n) for n in names}
    t_total = 0.0
    for b, h in chains:
        a = [np.ascontiguousarray(arrs[n][b:b + 1, :, h:h + 1]) for n in names]
        t0 = time.perf_counter()
        oracle.forward_diag(*a, mu=x.mu, scale=x.scale, nthreads=1)
        t_total += time.perf_counter() - t0
    # chains are independent and the oracle parallelises over chains with OpenMP; the sample is
    # timed chain by chain on one thread and scaled by the thread count actually available
    # (measured directly below with all chains in one OpenMP call)
    a = [np.ascontiguousarray(np.stack([arrs[n][b, :, h] for b, h in chains])[:, :, None])
         for n in names]
    t0 = time.perf_counter()
    oracle.forward_diag(*a, mu=x.mu, scale=x.scale, nthreads=nthreads)
    t_par = time.perf_counter() - t0
    token_heads = len(chains) * x.T
    tokens_equiv = token_heads / x.H  # one workload token carries H head-chains
    return {"value": tokens_equiv / t_par, "unit": "tokens/s", "cores": nthreads,
            "kind": "oracle",
            "sample": f"{len(chains)} of {x.B * x.H} (batch row, head) chains of the workload at "
                      f"full length T={x.T} ({token_heads} token-heads); float64 sequential "
                      f"recurrence, OpenMP over chains; single-thread time "
                      f"{t_total:.2f} s, {nthreads}-thread time {t_par:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--chunk", type=int, default=0)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB five times (used to "
                         "calibrate the HBM byte counters of rocprofv3)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus above 1 is not supported "
                                   "(sequences and heads shard with no communication)"}))
        sys.exit(2)

    import torch
    from paper_2609_07816_amd import kdn
    from paper_2609_07816_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe:
        n = args.copy_probe * (1 << 20)
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n,
                          "launches": 5}))
        return
    kdn.lib()
    x = W.draw_workload(2)
    B, T, H, dk, dv = x.B, x.T, x.H, x.dk, x.dv
    names = ("q", "k", "v", "alpha", "omega", "r")
    dev = {n: torch.from_numpy(x.stored[n].view(np.int16)).view(torch.bfloat16).cuda()
           for n in names}
    stream = torch.cuda.current_stream()

    def step():
        return kdn.forward_diag(*[dev[n] for n in names], mu=x.mu, scale=x.scale,
                                chunk=args.chunk)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps between two synchronisations; HIP events around every forward
    # call on torch's current stream, which the binding passes to the library (every kernel of
    # the call runs on that stream)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        step()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = [a.elapsed_time(b) for a, b in ev]

    ms_per_step = 1e3 * wall / args.steps
    tokens = B * T
    value = tokens / (ms_per_step / 1e3)
    kmean = float(np.mean(kern_ms))
    kmed = float(np.median(kern_ms))
    abytes = algorithmic_bytes(B, T, H, dk, dv, 2)
    aflops = algorithmic_flops(B, T, H, dk, dv)
    achieved = abytes / (kmean * 1e-3) / 1e9
    rec = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "diag-fwd-B4-H16-T4096-d128", "variant": "diagonal", "B": B,
                   "T": T, "H": H, "dk": dk, "dv": dv, "inputs": "bf16", "state": "f32",
                   "mfma": "bf16 in, f32 accumulate", "chunk": args.chunk or 64,
                   "mu": x.mu, "scale": x.scale},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(),
                     "kernel": "walk_kernel: one workgroup per (sequence, head, 32 value "
                               "columns) walks the chunks (bf16, dk=dv=128, chunk 64)",
                     "algorithmic_bytes_per_launch": abytes,
                     "kernel_ms_mean": round(kmean, 4), "kernel_ms_median": round(kmed, 4),
                     "mfma_frac": round(aflops / (kmean * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
                                        4)},
    }
    rec["decode"] = decode_measure(kdn, W, torch)
    if not args.no_cpu_baseline:
        nthreads = min(16, os.cpu_count() or 1)
        rec["cpu_baseline"] = cpu_baseline(x, nthreads)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
