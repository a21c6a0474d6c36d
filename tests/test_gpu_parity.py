"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle on identical seeded
inputs. Bounds: relative L2 error <= 1e-5 for float32 inputs and <= 2e-2 for bf16 inputs, over
o, S_T and P_T (gains: <= 1e-5, they are float32 arithmetic on identical inputs).
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import (NAMES, TOL, dev_tensor, host_f64, rel_l2, run_gpu_forward,
                      run_oracle_forward, run_oracle_packed_seq, to_device)
from paper_2609_07816_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_07816_amd import kdn
    kdn.lib()  # fail loudly when the library is missing


def check(name, got, ref, tol):
    err = rel_l2(got, ref)
    print(f"  {name}: rel-L2 {err:.3e} (bound {tol:g})", flush=True)
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert err <= tol, f"{name}: rel-L2 {err:.3e} > {tol:g}"


def compare_forward(x, chunk=0, tol=None):
    tol = TOL[x.dtype] if tol is None else tol
    o, S, P = run_gpu_forward(x, chunk)
    ref = run_oracle_forward(x)
    check("o", o, ref["o"], tol)
    check("S_T", S, ref["S_T"], tol)
    check("P_T", P, ref["P_T"], tol)


# ---------------------------------------------------------------------------------------------
# workload 0 and small multi-chunk cases
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
@pytest.mark.parametrize("chunk", [64, 0])
def test_forward_tiny_f32(variant, apc, chunk):
    compare_forward(W.draw_workload(0, variant, apc), chunk)


@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
@pytest.mark.parametrize("T", [150, 64, 17])
def test_forward_f32_multichunk_ragged(variant, apc, T):
    x = W.draw_inputs(variant, "f32", 2, T, 3, 32, 32, seed=41, alpha_per_channel=apc,
                      random_state=True)
    compare_forward(x)


@pytest.mark.parametrize("dk,dv", [(128, 128), (128, 64), (64, 128), (16, 128), (32, 16),
                                   (16, 16)])
def test_forward_f32_head_sizes(dk, dv):
    x = W.draw_inputs("diag", "f32", 1, 100, 2, dk, dv, seed=42, random_state=True)
    compare_forward(x)


@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
def test_forward_bf16_ragged(variant, apc):
    x = W.draw_inputs(variant, "bf16", 2, 200, 2, 128, 128, seed=43, alpha_per_channel=apc)
    compare_forward(x)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_forward_packed_ragged(variant, dtype):
    lens = [1, 63, 64, 0, 65, 130, 7]
    d = 32 if dtype == "f32" else 128
    x = W.draw_inputs(variant, dtype, 1, sum(lens), 2, d, d, seed=44, lengths=lens,
                      random_state=True)
    compare_forward(x)


@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
def test_forward_long_f32(variant, apc):
    # 71 chunks of 64 per sequence (the last one partial): the variance carry crosses a block of
    # 64 chunks of the log-depth scan, and the walk carries S through every chunk, from given
    # initial states
    x = W.draw_inputs(variant, "f32", 2, 4500, 2, 32, 32, seed=47, alpha_per_channel=apc,
                      random_state=True)
    compare_forward(x)


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_forward_long_packed_f32(variant):
    # packed sequences of 11, 1, 66, 0, 17 and 6 chunks (one empty, several with a partial last
    # chunk; one crosses a 64-chunk block of the carry scan), walked longest first
    lens = [700, 3, 4200, 0, 1040, 333]
    x = W.draw_inputs(variant, "f32", 1, sum(lens), 2, 32, 32, seed=48, lengths=lens,
                      random_state=True)
    compare_forward(x)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_forward_composition(variant, dtype):
    """Two chained calls carrying (S, P) equal one call over the whole sequence (composition,
    with the split inside a chunk)."""
    from paper_2609_07816_amd import kdn
    d = 64
    x = W.draw_inputs(variant, dtype, 2, 300, 2, d, d, seed=45, random_state=True)
    dd = to_device(x)
    f = kdn.forward_diag if variant == "diag" else kdn.forward_iso
    o, S, P = f(*[dd[n] for n in NAMES], S0=dd["S0"], P0=dd["P0"], mu=x.mu, scale=x.scale)
    cut = 157
    part = [dd[n][:, :cut].contiguous() for n in NAMES]
    rest = [dd[n][:, cut:].contiguous() for n in NAMES]
    o1, S1, P1 = f(*part, S0=dd["S0"], P0=dd["P0"], mu=x.mu, scale=x.scale)
    o2, S2, P2 = f(*rest, S0=S1, P0=P1, mu=x.mu, scale=x.scale)
    torch.cuda.synchronize()
    check("o (two calls vs one)", host_f64(torch.cat([o1, o2], dim=1)), host_f64(o), TOL[dtype])
    check("S_T (two calls vs one)", host_f64(S2), host_f64(S), TOL[dtype])
    check("P_T (two calls vs one)", host_f64(P2), host_f64(P), TOL[dtype])


@pytest.mark.parametrize("packed", [False, True])
def test_determinism_bitwise(packed):
    if packed:
        lens = [300, 0, 1000, 64, 5, 700]
        x = W.draw_inputs("diag", "bf16", 1, sum(lens), 2, 128, 128, seed=46, lengths=lens,
                          random_state=True)
    else:
        x = W.draw_inputs("diag", "bf16", 2, 300, 2, 128, 128, seed=46)
    a = run_gpu_forward(x)
    for _ in range(10):
        b = run_gpu_forward(x)
        for u, w in zip(a, b):
            assert np.array_equal(u, w)


# ---------------------------------------------------------------------------------------------
# gain scan alone
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
@pytest.mark.parametrize("packed", [False, True])
def test_gain_scan(variant, apc, dtype, packed):
    from paper_2609_07816_amd import kdn
    if packed:
        lens = [5, 64, 200, 0, 129]
        x = W.draw_inputs(variant, dtype, 1, sum(lens), 3, 64, 64, seed=47, lengths=lens,
                          alpha_per_channel=apc, random_state=True)
    else:
        x = W.draw_inputs(variant, dtype, 2, 300, 3, 64, 64, seed=47, alpha_per_channel=apc,
                          random_state=True)
    d = to_device(x)
    f = kdn.gain_diag if variant == "diag" else kdn.gain_iso
    g, ph, P = f(d["k"], d["alpha"], d["omega"], d["r"], P0=d["P0"], cu_seqlens=d["cu"],
                 mu=x.mu)
    torch.cuda.synchronize()
    ref = run_oracle_forward(x, traces=True)
    gname, pname = ("kappa", "phat") if variant == "diag" else ("beta", "bhat")
    check(gname, host_f64(g), ref[gname], 1e-5)
    check(pname, host_f64(ph), ref[pname], 1e-5)
    check("P_T", host_f64(P), ref["P_T"], 1e-5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 128])
@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_gain_scan_head_sizes(variant, d, dtype):
    """Head sizes 32 (half the lanes of the diagonal kernels idle) and 128 (two channels per
    lane) on a packed batch whose chunks end at every offset class: 1, 3, 64, 130, 191."""
    from paper_2609_07816_amd import kdn
    lens = [3, 64, 130, 1, 191]
    x = W.draw_inputs(variant, dtype, 1, sum(lens), 2, d, d, seed=65, lengths=lens,
                      random_state=True)
    dd = to_device(x)
    f = kdn.gain_diag if variant == "diag" else kdn.gain_iso
    g, ph, P = f(dd["k"], dd["alpha"], dd["omega"], dd["r"], P0=dd["P0"], cu_seqlens=dd["cu"],
                 mu=x.mu)
    torch.cuda.synchronize()
    ref = run_oracle_forward(x, traces=True)
    gname, pname = ("kappa", "phat") if variant == "diag" else ("beta", "bhat")
    check(gname, host_f64(g), ref[gname], 1e-5)
    check(pname, host_f64(ph), ref[pname], 1e-5)
    check("P_T", host_f64(P), ref["P_T"], 1e-5)


def test_gain_scan_full_workload_sampled():
    """The Diagonal gain scan at B4 T4096 H16 d128 bf16 (the gain bench's shape) in the launch
    configuration the bench times; three (row, head) chains against the oracle."""
    from paper_2609_07816_amd import kdn
    x = W.draw_workload(2)
    d = to_device(x)
    g0, _, _ = kdn.gain_diag(d["k"], d["alpha"], d["omega"], d["r"], P0=d["P0"], mu=x.mu,
                             want_phat=False)
    g, ph, P = kdn.gain_diag(d["k"], d["alpha"], d["omega"], d["r"], P0=d["P0"], mu=x.mu)
    torch.cuda.synchronize()
    assert torch.equal(g0, g), "kappa must not depend on whether p_hat is written"
    chains = [(0, 0), (x.B - 1, x.H - 1), (1, 7)]
    g, ph, P = host_f64(g), host_f64(ph), host_f64(P)
    for (b, h), ref in zip(chains, run_oracle_forward(x, chains=chains, traces=True)):
        print(f" chain (b={b}, h={h})", flush=True)
        check("kappa", g[b:b + 1, :, h:h + 1], ref["kappa"], 1e-5)
        check("phat", ph[b:b + 1, :, h:h + 1], ref["phat"], 1e-5)
        check("P_T", P[b:b + 1, h:h + 1], ref["P_T"], 1e-5)


def test_many_heads_gain_and_forward():
    """H = 66000 heads (more than a grid's y or z extent may hold), T = 3, d = 16: the gain
    scans and the forward index their workgroups over (chunk, head) in one grid dimension."""
    from paper_2609_07816_amd import kdn
    H = 66000
    for variant in ("diag", "iso"):
        x = W.draw_inputs(variant, "f32", 1, 3, H, 16, 16, seed=66, random_state=True)
        d = to_device(x)
        f = kdn.gain_diag if variant == "diag" else kdn.gain_iso
        g, ph, P = f(d["k"], d["alpha"], d["omega"], d["r"], P0=d["P0"], mu=x.mu)
        o, S, P2 = run_gpu_forward(x)
        torch.cuda.synchronize()
        ref = run_oracle_forward(x, traces=True)
        gname = "kappa" if variant == "diag" else "beta"
        check(f"{variant} {gname}", host_f64(g), ref[gname], 1e-5)
        check(f"{variant} P_T (gain)", host_f64(P), ref["P_T"], 1e-5)
        check(f"{variant} o", o, ref["o"], TOL["f32"])
        check(f"{variant} P_T (forward)", P2, ref["P_T"], TOL["f32"])


# ---------------------------------------------------------------------------------------------
# decode
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
@pytest.mark.parametrize("d", [16, 128])
def test_decode_steps(variant, apc, dtype, d):
    from paper_2609_07816_amd import kdn
    R, H, slots, steps = 5, 3, 7, 6
    g = np.random.default_rng([48, d])
    S = (0.1 * g.standard_normal((slots, H, d, d))).astype(np.float32)
    P = g.uniform(0.1, 1.0, (slots, H, d) if variant == "diag" else (slots, H)).astype(np.float32)
    slot_idx = np.array([6, 0, -1, 3, 2], dtype=np.int32)
    S_ref, P_ref = S.astype(np.float64), P.astype(np.float64)
    S_dev, P_dev = torch.from_numpy(S).cuda(), torch.from_numpy(P).cuda()
    si = torch.from_numpy(slot_idx).cuda()
    o_prev = None
    for step in range(steps):
        x = W.draw_inputs(variant, dtype, R, 1, H, d, d, seed=49, stream=100 + step,
                          alpha_per_channel=apc)
        dd = to_device(x)
        o_dev = torch.zeros((R, H, d), dtype=dd["k"].dtype, device="cuda")
        kdn.decode_step(variant, *[dd[n][:, 0].contiguous() for n in NAMES], S_dev, P_dev,
                        slot_idx=si, mu=x.mu, scale=x.scale, o=o_dev)
        o_ref = oracle.decode_step(variant, *[x.f64(n)[:, 0] for n in NAMES], S_ref, P_ref,
                                   slot_idx=slot_idx, mu=x.mu, scale=x.scale)
        torch.cuda.synchronize()
        o = host_f64(o_dev)
        check(f"o step {step}", o, o_ref, TOL[dtype])
        assert np.all(o[2] == 0.0), "skipped row must be left untouched"
    check("S", host_f64(S_dev), S_ref, TOL[dtype])
    check("P", host_f64(P_dev), P_ref, TOL[dtype])
    untouched = [1, 4, 5]
    assert np.array_equal(host_f64(S_dev)[untouched], S.astype(np.float64)[untouched])


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_decode_chain_equals_forward(variant):
    from paper_2609_07816_amd import kdn
    x = W.draw_inputs(variant, "f32", 3, 40, 2, 32, 32, seed=50)
    o_f, S_f, P_f = run_gpu_forward(x)
    d = to_device(x)
    S = torch.zeros((3, 2, 32, 32), device="cuda")
    P = torch.ones((3, 2, 32) if variant == "diag" else (3, 2), device="cuda")
    outs = []
    for t in range(40):
        o = kdn.decode_step(variant, *[d[n][:, t].contiguous() for n in NAMES], S, P,
                            mu=x.mu, scale=x.scale)
        outs.append(host_f64(o))
    torch.cuda.synchronize()
    check("o", np.stack(outs, axis=1), o_f, 1e-5)
    check("S", host_f64(S), S_f, 1e-5)
    check("P", host_f64(P), P_f, 1e-5)


# ---------------------------------------------------------------------------------------------
# full-size workloads, checked on sampled chains
# ---------------------------------------------------------------------------------------------

def _sample_chains(B, H, k=6, seed=0):
    g = np.random.default_rng(seed)
    picks = {(0, 0), (B - 1, H - 1)}
    while len(picks) < k:
        picks.add((int(g.integers(B)), int(g.integers(H))))
    return sorted(picks)


@pytest.mark.parametrize("wid", [1, 2])
def test_full_workload_sampled(wid):
    x = W.draw_workload(wid)
    o, S, P = run_gpu_forward(x)
    chains = _sample_chains(x.B, x.H, seed=wid)
    refs = run_oracle_forward(x, chains=chains)
    for (b, h), ref in zip(chains, refs):
        print(f" chain (b={b}, h={h})")
        check("o", o[b:b + 1, :, h:h + 1], ref["o"], TOL[x.dtype])
        check("S_T", S[b:b + 1, h:h + 1], ref["S_T"], TOL[x.dtype])
        check("P_T", P[b:b + 1, h:h + 1], ref["P_T"], TOL[x.dtype])


def test_full_workload_packed_sampled():
    x = W.draw_workload(3)
    o, S, P = run_gpu_forward(x)
    lens = np.diff(x.cu_seqlens)
    picks = [int(np.argmin(lens)), int(np.argmax(lens)), 7, 20]
    for n in picks:
        heads = [0, 5, 15]
        ref = run_oracle_packed_seq(x, n, heads)
        t0, t1 = int(x.cu_seqlens[n]), int(x.cu_seqlens[n + 1])
        print(f" sequence {n} (length {t1 - t0})")
        check("o", o[:, t0:t1][:, :, heads], ref["o"], TOL[x.dtype])
        check("S_T", S[n:n + 1][:, heads], ref["S_T"], TOL[x.dtype])
        check("P_T", P[n:n + 1][:, heads], ref["P_T"], TOL[x.dtype])
