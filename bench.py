"""Benchmark of the KDN forward hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--only WHAT]

Headline workload: Diagonal KDN forward, B=4, H=16, T=4096, dk=dv=128, bf16 q/k/v/gates/noise,
float32 state (the mixer shape of the paper's 750M model: 16 heads x 128 at d_model 2048, 4K
context, batch 4 as in its throughput probe). Inputs are seeded synthetic tensors resident in HBM
before timing starts. One step = one full forward over the batch: every stage of the path (the
chunk summaries of the variance chain, the log-depth carry scan, the per-chunk prep of the gains
and the chunk operands, and the walk that carries the memory through the chunks).

Prints one JSON line: tokens/s of the headline forward, the roofline position of one forward call
(algorithmic bytes per call / the GPU time per call, from HIP events on the caller's stream around
the K back-to-back calls of the timed region, against the 8 TB/s HBM peak), the CPU oracle timed
on a bounded sample of the same workload, and one object per other workload of the path (the
isotropic forward, the packed variable-length batch, the decode workload's prefill and decode
steps, the gain scan alone, the backward, the layer forward with its maps fused), timed the same
way (decode: events around every call, whose host side would otherwise set the pace).
The larger workloads draw their inputs on the GPU with the same laws (timing only; their parity
is checked by the tests on host-drawn inputs).

The default warmup is 200 untimed forward calls (about 60 ms): the GPU raises its clocks only
after some tens of milliseconds of load, and five warmup calls leave the timed steps about 9%
slower than the same calls at steady clocks.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "KDN forward tokens/s (H=16,d=128,T=4096) + % of MFMA/HBM roofline"
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense float32 (the backward's products)
FORWARD_KERNELS = "forward call: 4 kernels (chunk summaries, log-depth carry scan, per-chunk " \
                  "prep, walk over the chunks)"


# ---------------------------------------------------------------------------------------------
# algorithmic work
# ---------------------------------------------------------------------------------------------

def forward_bytes(tokens, N, H, dk, dv, es, variant, apc=True, with_init=False):
    """Minimum HBM traffic of one forward: every input read once, o written once, the final
    states written once (and the initial states read once when given)."""
    if variant == "diag":
        per = (2 * dk + dv) * es + 2 * dk * es + es            # q, k, v; alpha, omega; r
    else:
        per = (2 * dk + dv) * es + (dk if apc else 1) * es + 2 * es  # q, k, v; alpha; omega, r
    per += dv * es                                              # o
    nst = dk if variant == "diag" else 1
    states = N * H * (dk * dv * 4 + nst * 4)
    return tokens * H * per + states * (2 if with_init else 1)


def forward_flops(tokens, H, dk, dv, C=64):
    """Dense flop count of the chunked WY form per token-head: 6 dk dv + 10 C d + C^2 / 3."""
    return tokens * H * (6 * dk * dv + 10 * C * dk + C * C / 3.0)


def decode_bytes(R, H, dk, dv, es, variant):
    """Minimum HBM traffic of one decode step: the state slot read and written (S and P in
    float32), the token's inputs read and o written."""
    nst = dk if variant == "diag" else 1
    per = 2 * (dk * dv * 4 + nst * 4) + (2 * dk + dv) * es + dk * es \
        + (dk if variant == "diag" else 1) * es + es + dv * es
    return R * H * per


def gain_bytes(tokens, H, dk, es):
    """Minimum traffic of the gain scan alone (diagonal): k, alpha, omega and r read once, the
    gains written once in float32."""
    return tokens * H * (3 * dk * es + es + 4 * dk)


def gain_iso_bytes(tokens, H, dk, es, apc):
    """Minimum traffic of the isotropic gain scan alone: k (and alpha per channel) read once,
    the per-head alpha, omega and r read once, beta written once in float32."""
    return tokens * H * (dk * es * (2 if apc else 1) + (2 if apc else 3) * es + 4)


# ---------------------------------------------------------------------------------------------
# inputs drawn on the GPU (same laws as paper_2609_07816_amd/workloads.py)
# ---------------------------------------------------------------------------------------------

def gpu_inputs(torch, variant, B, T, H, dk, dv, seed, apc=True, random_state=False, N=None):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    f32, bf = torch.float32, torch.bfloat16

    def normal(shape):
        return torch.randn(shape, generator=g, device="cuda", dtype=f32)

    def unit(x):
        return (x / x.norm(dim=-1, keepdim=True)).to(bf)

    sp = torch.nn.functional.softplus
    d = {"q": unit(normal((B, T, H, dk))), "k": unit(normal((B, T, H, dk))),
         "v": normal((B, T, H, dv)).to(bf)}
    ashape = (B, T, H, dk) if (variant == "diag" or apc) else (B, T, H)
    d["alpha"] = torch.sigmoid(normal(ashape) + 2.0).to(bf)
    oshape = (B, T, H, dk) if variant == "diag" else (B, T, H)
    d["omega"] = (sp(normal(oshape)) + 1e-3).to(bf)
    d["r"] = (sp(normal((B, T, H))) + 1e-3).to(bf)
    if random_state:
        n = B if N is None else N
        d["S0"] = 0.02 * normal((n, H, dk, dv))
        pshape = (n, H, dk) if variant == "diag" else (n, H)
        d["P0"] = torch.rand(pshape, generator=g, device="cuda") * 0.9 + 0.1
    return d


NAMES = ("q", "k", "v", "alpha", "omega", "r")


def time_calls(torch, fn, steps, warmup, per_call=False, reps=5, warm_s=0.1):
    """Milliseconds per call on torch's current stream (the stream the binding passes to the
    library; every kernel of a call runs on it).

    Untimed calls first: `warmup` of them, and more until `warm_s` seconds of GPU work have
    passed (the GPU's clocks rise only after some tens of milliseconds of load). Then by
    default `reps` regions of `steps` back-to-back calls, HIP events around each region; one
    value (region time / steps) per region. per_call=True: events around every call instead,
    one value per call (for calls short enough that the host, not the GPU, would set the pace
    of back-to-back calls; each pair of timing events adds a few microseconds of its own)."""
    stream = torch.cuda.current_stream()
    t0, n = time.perf_counter(), 0
    while n < warmup or time.perf_counter() - t0 < warm_s:
        fn()
        n += 1
        if n % 16 == 0:
            torch.cuda.synchronize()  # the host's clock follows the GPU's progress
    torch.cuda.synchronize()
    if per_call:
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        for a, b in ev:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in ev]
    out = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(steps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        out.append(a.elapsed_time(b) / steps)
    return out


def summary(ms, nbytes, tokens, extra=None):
    med, mean = float(np.median(ms)), float(np.mean(ms))
    gbs = nbytes / (mean * 1e-3) / 1e9
    rec = {"ms_median": round(med, 4), "ms_mean": round(mean, 4),
           "tokens_per_s": round(tokens / (med * 1e-3), 1), "algorithmic_bytes": int(nbytes),
           "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": round(gbs / HBM_PEAK_GBS, 4)}
    if extra:
        rec.update(extra)
    return rec


# ---------------------------------------------------------------------------------------------
# the other workloads of the path
# ---------------------------------------------------------------------------------------------

def bench_iso(torch, kdn, steps):
    """Workload 1: isotropic forward, B4 H16 T2048 d128, scalar gates, bf16."""
    B, T, H, d = 4, 2048, 16, 128
    x = gpu_inputs(torch, "iso", B, T, H, d, d, seed=1001, apc=False)
    ms = time_calls(torch, lambda: kdn.forward_iso(*[x[n] for n in NAMES], mu=float(d),
                                                   scale=d ** -0.5), steps, 3)
    return summary(ms, forward_bytes(B * T, B, H, d, d, 2, "iso", apc=False), B * T,
                   {"workload": "iso-fwd-B4-H16-T2048-d128 (scalar gates)",
                    "kernels": FORWARD_KERNELS})


def bench_gain_iso(torch, kdn, steps, copies=4):
    """The isotropic gain scan alone (kdn_gain_iso) at workload 1's shape (B4 H16 T2048 d128
    bf16), with scalar gates (workload 1's) and with gates per channel, on `copies` copies of the
    inputs taken in turn (as for the diagonal gain scan)."""
    B, T, H, d = 4, 2048, 16, 128
    out = {}
    for apc in (False, True):
        x = gpu_inputs(torch, "iso", B, T, H, d, d, seed=1001, apc=apc)
        names = ("k", "alpha", "omega", "r")
        sets = [x] + [{n: x[n].clone() for n in names} for _ in range(copies - 1)]
        turn = [0]

        def call():
            y = sets[turn[0] % copies]
            turn[0] += 1
            return kdn.gain_iso(y["k"], y["alpha"], y["omega"], y["r"], mu=float(d),
                                want_phat=False)

        ms = time_calls(torch, call, steps, 3)
        gates = "per channel" if apc else "scalar"
        out["gates_per_channel" if apc else "scalar_gates"] = summary(
            ms, gain_iso_bytes(B * T, H, d, 2, apc), B * T,
            {"workload": f"iso-gain-scan-B4-H16-T2048-d128 ({gates} gates, beta out, float32)",
             "inputs": f"{copies} copies taken in turn"})
    return out


def bench_varlen(torch, kdn, W, steps):
    """Workload 3: diagonal forward over 32 packed sequences of U[256, 8192] tokens, random
    initial states, bf16."""
    H, d = 16, 128
    lens = W.draw_lengths(32, 256, 8192, seed=1003)
    T = int(lens.sum())
    x = gpu_inputs(torch, "diag", 1, T, H, d, d, seed=1003, random_state=True, N=len(lens))
    cu = torch.zeros(len(lens) + 1, dtype=torch.int32, device="cuda")
    cu[1:] = torch.from_numpy(np.cumsum(lens).astype(np.int32)).cuda()
    ms = time_calls(torch, lambda: kdn.forward_diag(*[x[n] for n in NAMES], S0=x["S0"],
                                                    P0=x["P0"], cu_seqlens=cu, mu=float(d),
                                                    scale=d ** -0.5), steps, 3)
    return summary(ms, forward_bytes(T, len(lens), H, d, d, 2, "diag", with_init=True), T,
                   {"workload": f"diag-varlen-32seq-U256-8192-H16-d128 ({T} tokens)",
                    "kernels": FORWARD_KERNELS})


# decode steps before each decode variant's 64 timed steps: a fixed count (about 0.1 s of
# steps), so that the timed steps keep fixed positions in a profiler's trace
DECODE_WARMUP = 1200


def bench_decode_workload(torch, kdn, steps):
    """Workload 4: B256 T1024 prefill of every row (diagonal, bf16), then decode steps of both
    variants on 256 rows; also the diagonal step on a pool of 1024 slots (4x the state the
    Infinity Cache can hold), rows mapped to every fourth slot."""
    R, H, d, T = 256, 16, 128, 1024
    out = {}
    x = gpu_inputs(torch, "diag", R, T, H, d, d, seed=1004)
    ms = time_calls(torch, lambda: kdn.forward_diag(*[x[n] for n in NAMES], mu=float(d),
                                                    scale=d ** -0.5), max(3, steps // 4), 1)
    out["prefill"] = summary(ms, forward_bytes(R * T, R, H, d, d, 2, "diag"), R * T,
                             {"workload": "diag-fwd-B256-H16-T1024-d128 (the decode prefill)",
                              "kernels": FORWARD_KERNELS})
    del x
    torch.cuda.empty_cache()
    for variant in ("diag", "iso"):
        st = gpu_inputs(torch, variant, R, 1, H, d, d, seed=1104, apc=True, random_state=True)
        args = [st[n][:, 0].contiguous() for n in NAMES]
        S, P = st["S0"], st["P0"]
        ms = time_calls(torch, lambda: kdn.decode_step(variant, *args, S, P, mu=float(d),
                                                       scale=d ** -0.5), 64, DECODE_WARMUP,
                        per_call=True, warm_s=0.0)
        out[f"decode_{variant}"] = summary(
            ms, decode_bytes(R, H, d, d, 2, variant), R,
            {"workload": f"{variant}-decode-R256-H16-d128 (state pool of 256 slots, 256 MiB)",
             "kernel": "decode_kernel: one workgroup per (row, head)"})
    st = gpu_inputs(torch, "diag", R, 1, H, d, d, seed=1105, random_state=True, N=4 * R)
    args = [st[n][:, 0].contiguous() for n in NAMES]
    slots = torch.arange(0, 4 * R, 4, dtype=torch.int32, device="cuda")
    ms = time_calls(torch, lambda: kdn.decode_step("diag", *args, st["S0"], st["P0"],
                                                   slot_idx=slots, mu=float(d),
                                                   scale=d ** -0.5), 64, DECODE_WARMUP,
                    per_call=True, warm_s=0.0)
    out["decode_diag_pool1024"] = summary(
        ms, decode_bytes(R, H, d, d, 2, "diag"), R,
        {"workload": "diag-decode-R256-H16-d128, rows on every fourth slot of a 1024-slot pool "
                     "(1 GiB of state)", "kernel": "decode_kernel"})
    return out


def bench_gain(torch, kdn, x, steps, copies=4):
    """The gain scan alone (kdn_gain_diag) at the headline shape: chunk summaries, carry scan
    and emission of the float32 gains. The calls take `copies` copies of the inputs in turn
    (4 x 201 MB, more than the 256 MB last-level cache), so that every call reads its inputs
    from HBM, as the first call on fresh inputs does."""
    B, T, H, d = x["k"].shape
    names = ("k", "alpha", "omega", "r")
    sets = [x] + [{n: x[n].clone() for n in names} for _ in range(copies - 1)]
    turn = [0]

    def call():
        y = sets[turn[0] % copies]
        turn[0] += 1
        return kdn.gain_diag(y["k"], y["alpha"], y["omega"], y["r"], mu=float(d),
                             want_phat=False)

    ms = time_calls(torch, call, steps, 3)
    return summary(ms, gain_bytes(B * T, H, d, 2), B * T,
                   {"workload": "diag-gain-scan-B4-H16-T4096-d128 (kappa out, float32)",
                    "inputs": f"{copies} copies taken in turn",
                    "kernels": "gain scan: chunk summaries, carry scan, emission"})


def backward_bytes(tokens, H, dk, dv, es):
    """Minimum traffic of one diagonal backward: the forward's inputs and dO read once, the
    float32 gradients of q, k, v, alpha, omega and r written once."""
    return tokens * H * ((5 * dk + 2 * dv) * es + es + (4 * dk + dv + 1) * 4)


def backward_flops(tokens, H, dk, dv, C=64):
    """Dense flop count (a multiply-add is two) of the chunked backward per token-head, products
    with a triangular factor counted at half:
      replay: T and B (2 C dk), (I + T)^-1 (2 C^2 / 3);
      forward walk: X = V - Kbar S, S update (2 x 2 dk dv), Delta = A X (C dv);
      reverse walk: Ktail dS_out, dS_in's two products (3 x 2 dk dv), B^T dO and A^T dDelta
        (2 x C dv);
      gradients: Psi S_in^T, dO S_in^T, Delta dS_out^T (3 x 2 dk dv), dO Delta^T and
        Psi Delta^T (2 x C dv), the four T/B terms (4 C dk)."""
    return tokens * H * (16 * dk * dv + 5 * C * dv + 6 * C * dk + 2 * C * C / 3.0)


def bench_backward(torch, kdn, x, steps):
    """kdn_backward at the headline shape, with random incoming adjoints of o, S_T and P_T."""
    B, T, H, d = x["k"].shape
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    dO = torch.randn((B, T, H, d), generator=g, device="cuda").to(torch.bfloat16)
    dS = torch.randn((B, H, d, d), generator=g, device="cuda")
    dP = torch.randn((B, H, d), generator=g, device="cuda")
    ms = time_calls(torch, lambda: kdn.backward("diag", *[x[n] for n in NAMES], mu=float(d),
                                                dO=dO, dS_T=dS, dP_T=dP), steps, 3)
    flops = backward_flops(B * T, H, d, d)
    mean = float(np.mean(ms))
    return summary(ms, backward_bytes(B * T, H, d, d, 2), B * T,
                   {"workload": "diag-bwd-B4-H16-T4096-d128 (float32 gradients)",
                    "flops": flops, "mfma_peak_tflops": FP32_MFMA_PEAK_TFLOPS,
                    "mfma_frac": round(flops / (mean * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4),
                    "kernels": "backward: chunk summaries, carry scan, per-chunk replay, forward "
                               "walk, reverse walk, per-chunk gradients, variance-adjoint scan, "
                               "per-token gain gradients"})


def bench_layer(torch, kdn, steps):
    """The layer forward (kdn_forward_layer: gate pre-activations, q/k L2 norm, effective-write
    output) at the headline shape, and beside it the same layer done unfused: the maps as torch
    elementwise ops, then the plain forward."""
    B, T, H, d = 4, 4096, 16, 128
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    bf = torch.bfloat16

    def normal(shape, shift=0.0):
        return (torch.randn(shape, generator=g, device="cuda") + shift).to(bf)

    q, k, v = normal((B, T, H, d)), normal((B, T, H, d)), normal((B, T, H, d))
    a_pre, w_pre, r_pre = normal((B, T, H, d), 2.0), normal((B, T, H, d)), normal((B, T, H))
    sp = torch.nn.functional.softplus

    def fused():
        return kdn.forward_layer("diag", q, k, v, a_pre, w_pre, r_pre, mu=float(d),
                                 gates_preact=True, r_min=0.01, qk_l2norm=True,
                                 want_beta_eff=True)

    def unfused():
        qn = (q.float() / q.float().norm(dim=-1, keepdim=True)).to(bf)
        kn = (k.float() / k.float().norm(dim=-1, keepdim=True)).to(bf)
        a = torch.sigmoid(a_pre.float()).to(bf)
        w = sp(w_pre.float()).to(bf)
        r = (0.01 + sp(r_pre.float())).to(bf)
        return kdn.forward_diag(qn, kn, v, a, w, r, mu=float(d))

    ms = time_calls(torch, fused, steps, 3)
    ms_u = time_calls(torch, unfused, steps, 3)
    rec = summary(ms, forward_bytes(B * T, B, H, d, d, 2, "diag") + B * T * H * 4, B * T,
                  {"workload": "diag-layer-fwd-B4-H16-T4096-d128 (pre-activation gates, q/k "
                               "L2 norm, beta_eff out)",
                   "kernels": "layer forward: the forward's 4 kernels with the maps fused"})
    rec["unfused_ms_median"] = round(float(np.median(ms_u)), 4)
    rec["unfused"] = "torch sigmoid / softplus / L2 norm in float32, rounded to bf16, then the " \
                     "plain forward"
    return rec


# ---------------------------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of the headline workload
# ---------------------------------------------------------------------------------------------

def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(x, nthreads):
    """The oracle, unchanged, on the workload's independent (batch row, head) chains at full
    length: all 64 chains in one OpenMP call on nthreads threads, and one chain alone on one
    thread. Returns the rate in workload tokens/s."""
    import oracle
    arrs = {n: x.f64(n) for n in NAMES}
    chains = [(b, h) for b in range(x.B) for h in range(x.H)]
    a1 = [np.ascontiguousarray(arrs[n][0:1, :, 0:1]) for n in NAMES]
    t0 = time.perf_counter()
    oracle.forward_diag(*a1, mu=x.mu, scale=x.scale, nthreads=1)
    t_one = time.perf_counter() - t0
    a = [np.ascontiguousarray(np.stack([arrs[n][b, :, h] for b, h in chains])[:, :, None])
         for n in NAMES]
    t0 = time.perf_counter()
    oracle.forward_diag(*a, mu=x.mu, scale=x.scale, nthreads=nthreads)
    t_par = time.perf_counter() - t0
    token_heads = len(chains) * x.T
    return {"value": round(token_heads / x.H / t_par, 1), "unit": "tokens/s",
            "cores": nthreads, "kind": "oracle", "nproc": os.cpu_count(),
            "cpu_model": cpu_model(),
            "sample": f"all {len(chains)} (batch row, head) chains of the headline workload at "
                      f"full length T={x.T} ({token_heads} token-heads, one workload token = "
                      f"{x.H} token-heads); float64 sequential recurrence, OpenMP over chains on "
                      f"{nthreads} threads: {t_par:.2f} s; one chain on one thread: "
                      f"{t_one:.2f} s"}


PROFILE = os.path.join(ROOT, "profiles", "kdn_forward_diag_B4_T4096_H16_d128.json")


def measured_traffic():
    """HBM bytes per forward from the committed rocprofv3 counter summary (FETCH_SIZE and
    WRITE_SIZE of every kernel of the forward, scaled by a plain copy of known size), or None
    when the summary is missing or was taken from a different version of the kernel sources."""
    try:
        from paper_2609_07816_amd.rocprof_summary import source_hash
        with open(PROFILE) as f:
            rec = json.load(f)
        if rec.get("kernel_source_sha256") != source_hash(rec.get("kernel_sources")):
            return None
        return int(round(rec["traffic_bytes"]))
    except (OSError, ValueError, KeyError):
        return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--chunk", type=int, default=0)
    ap.add_argument("--only", default="all",
                    choices=["all", "headline", "iso", "varlen", "decode", "gain", "gain_iso",
                             "backward", "layer"],
                    help="run only the headline forward or one other workload (profiling runs)")
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
    if args.only in ("iso", "varlen", "decode", "layer", "gain_iso"):
        fn = {"iso": lambda: bench_iso(torch, kdn, args.steps),
              "gain_iso": lambda: bench_gain_iso(torch, kdn, args.steps),
              "varlen": lambda: bench_varlen(torch, kdn, W, args.steps),
              "decode": lambda: bench_decode_workload(torch, kdn, args.steps),
              "layer": lambda: bench_layer(torch, kdn, args.steps)}[args.only]
        print(json.dumps({args.only: fn()}), flush=True)
        return

    x = W.draw_workload(2)
    B, T, H, dk, dv = x.B, x.T, x.H, x.dk, x.dv
    dev = {n: torch.from_numpy(x.stored[n].view(np.int16)).view(torch.bfloat16).cuda()
           for n in NAMES}
    if args.only == "gain":
        print(json.dumps({"gain": bench_gain(torch, kdn, dev, args.steps)}), flush=True)
        return
    if args.only == "backward":
        print(json.dumps({"backward": bench_backward(torch, kdn, dev, args.steps)}), flush=True)
        return

    def step():
        return kdn.forward_diag(*[dev[n] for n in NAMES], mu=x.mu, scale=x.scale,
                                chunk=args.chunk)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps between two synchronisations, back to back on torch's current
    # stream, which the binding passes to the library (every kernel of the call runs on that
    # stream); HIP events around the region give the GPU's time per call
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kmean = ev0.elapsed_time(ev1) / args.steps

    ms_per_step = 1e3 * wall / args.steps
    tokens = B * T
    value = tokens / (ms_per_step / 1e3)
    abytes = forward_bytes(B * T, B, H, dk, dv, 2, "diag")
    aflops = forward_flops(B * T, H, dk, dv)
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
                   "mfma": "bf16 in, f32 accumulate", "chunk": 64,
                   "mu": x.mu, "scale": x.scale},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(),
                     "kernel": FORWARD_KERNELS + "; bf16, dk=dv=128, chunk 64",
                     "algorithmic_bytes_per_launch": abytes,
                     "kernel_ms_mean": round(kmean, 4),
                     "mfma_frac": round(aflops / (kmean * 1e-3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
                                        4)},
    }
    if args.only == "all":
        rec["workloads"] = {"iso_forward": bench_iso(torch, kdn, args.steps),
                            "varlen_forward": bench_varlen(torch, kdn, W, args.steps),
                            "gain_scan": bench_gain(torch, kdn, dev, args.steps),
                            "gain_scan_iso": bench_gain_iso(torch, kdn, args.steps),
                            "backward": bench_backward(torch, kdn, dev, args.steps),
                            "layer_forward": bench_layer(torch, kdn, args.steps)}
        rec["workloads"].update(bench_decode_workload(torch, kdn, args.steps))
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(x, min(16, os.cpu_count() or 1))
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
