"""GPU parity on the method's numeric edge cases and on paths the workloads do not reach:
small and unit gates, zero process noise, tiny observation noise, long sequences whose variance
carry crosses blocks of 64 chunks, the decode workload at its full size, and guard bands around
every output (nothing is written outside the caller's buffers, also for a cu_seqlens that
overshoots the batch). Bounds as in test_gpu_parity.py."""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import (NAMES, TOL, host_f64, rel_l2, run_gpu_forward, run_oracle_forward,
                      to_device)
from paper_2609_07816_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_07816_amd import kdn
    kdn.lib()


def check(name, got, ref, tol):
    err = rel_l2(got, ref)
    print(f"  {name}: rel-L2 {err:.3e} (bound {tol:g})", flush=True)
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert err <= tol, f"{name}: rel-L2 {err:.3e} > {tol:g}"


LAWS = {
    # per-channel gates uniform on [0.01, 0.3]: the decay over a 64-token chunk reaches 1e-128
    "small_gates": dict(alpha_law=("uniform", 0.01, 0.3)),
    "unit_gates": dict(alpha_law=("const", 1.0)),
    "zero_process_noise": dict(omega_law=("const", 0.0)),
    "tiny_r": dict(r_law=("const", 1e-3)),
}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
@pytest.mark.parametrize("law", list(LAWS))
def test_edge_laws(law, variant, apc, dtype):
    d = 32 if dtype == "f32" else 128
    x = W.draw_inputs(variant, dtype, 1, 8192, 2, d, d, seed=60, alpha_per_channel=apc,
                      random_state=True, **LAWS[law])
    o, S, P = run_gpu_forward(x)
    ref = run_oracle_forward(x)
    check("o", o, ref["o"], TOL[dtype])
    check("S_T", S, ref["S_T"], TOL[dtype])
    check("P_T", P, ref["P_T"], TOL[dtype])


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_gates_below_exactness_floor_stay_finite(variant):
    # a fifth of the gates at 1e-6: some decays over 8 tokens fall below 2^-126, where the
    # midpoint references saturate; every output must stay finite, and the state and variances
    # (which the saturated factors do not touch) must still match
    x = W.draw_inputs(variant, "f32", 1, 1000, 2, 32, 32, seed=61,
                      alpha_law=("spikes", 0.9, 1e-6, 0.2), random_state=True)
    o, S, P = run_gpu_forward(x)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S)) and np.all(np.isfinite(P))
    ref = run_oracle_forward(x)
    check("P_T", P, ref["P_T"], 1e-5)


# ---------------------------------------------------------------------------------------------
# gain scan across blocks of 64 chunks
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
@pytest.mark.parametrize("packed", [False, True])
def test_gain_scan_long(variant, apc, dtype, packed):
    from paper_2609_07816_amd import kdn
    if packed:
        lens = [int(v) for v in W.draw_lengths(6, 256, 8192, seed=62)] + [8300]
        x = W.draw_inputs(variant, dtype, 1, sum(lens), 2, 16, 16, seed=62, lengths=lens,
                          alpha_per_channel=apc, random_state=True)
    else:
        x = W.draw_inputs(variant, dtype, 2, 8300, 2, 16, 16, seed=62, alpha_per_channel=apc,
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


# ---------------------------------------------------------------------------------------------
# the decode workload at full size: prefill of every row, then 64 steps
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_decode_workload4_full(variant):
    """256 rows x H16 x d128: a T = 1024 bf16 prefill of all 256 rows through the forward, then
    64 decode steps over every row. 16 rows (the first, the last and 14 drawn ones) are checked
    against the oracle after the prefill, at every decode step, and at the end."""
    from paper_2609_07816_amd import kdn
    R, H, d, T, steps = 256, 16, 128, 1024, 64
    pre = W.draw_decode_prefill(variant, R=R, H=H, d=d, T=T)
    dpre = to_device(pre)
    f = kdn.forward_diag if variant == "diag" else kdn.forward_iso
    _, S_dev, P_dev = f(*[dpre[n] for n in NAMES], mu=pre.mu, scale=pre.scale)
    torch.cuda.synchronize()
    g = np.random.default_rng(64)
    rows = sorted({0, R - 1} | set(int(v) for v in g.choice(np.arange(1, R - 1), 14,
                                                            replace=False)))
    sub = [pre.f64(n)[rows] for n in NAMES]
    fo = oracle.forward_diag if variant == "diag" else oracle.forward_iso
    ref = fo(*sub, mu=pre.mu, scale=pre.scale)
    S_ref, P_ref = ref["S_T"].copy(), ref["P_T"].copy()
    check("prefill S_T (sampled rows)", host_f64(S_dev)[rows], S_ref, TOL["bf16"])
    check("prefill P_T (sampled rows)", host_f64(P_dev)[rows], P_ref, TOL["bf16"])
    for s in range(steps):
        x = W.draw_decode_step(variant, s)
        dd = to_device(x)
        o = kdn.decode_step(variant, *[dd[n][:, 0].contiguous() for n in NAMES], S_dev, P_dev,
                            mu=x.mu, scale=x.scale)
        o_ref = oracle.decode_step(variant, *[x.f64(n)[rows, 0] for n in NAMES], S_ref, P_ref,
                                   mu=x.mu, scale=x.scale)
        torch.cuda.synchronize()
        check(f"o step {s} (sampled rows)", host_f64(o)[rows], o_ref, TOL["bf16"])
    check("S after decode", host_f64(S_dev)[rows], S_ref, TOL["bf16"])
    check("P after decode", host_f64(P_dev)[rows], P_ref, TOL["bf16"])


# ---------------------------------------------------------------------------------------------
# guard bands
# ---------------------------------------------------------------------------------------------

GUARD = 4096  # bytes of canary on each side of every output


def _guarded(shape, dtype, dev="cuda"):
    """A tensor view with GUARD bytes of 0xA5 canary before and after it."""
    es = torch.tensor([], dtype=dtype).element_size()
    n = int(np.prod(shape))
    pad = GUARD // es
    buf = torch.empty(n + 2 * pad, dtype=dtype, device=dev)
    buf.view(torch.uint8).fill_(0xA5)
    return buf, buf[pad:pad + n].view(shape), pad


def _canary_ok(buf, pad):
    b = buf.view(torch.uint8)
    es = buf.element_size()
    head, tail = b[:pad * es], b[b.numel() - pad * es:]
    return bool(torch.all(head == 0xA5)) and bool(torch.all(tail == 0xA5))


@pytest.mark.parametrize("variant", ["diag", "iso"])
@pytest.mark.parametrize("overshoot", [False, True])
def test_guard_bands(variant, overshoot):
    from paper_2609_07816_amd import kdn
    lens = [100, 0, 300, 37]
    x = W.draw_inputs(variant, "bf16", 1, sum(lens), 2, 64, 64, seed=65, lengths=lens,
                      random_state=True)
    d = to_device(x)
    N, T, H, dk, dv = len(lens), sum(lens), 2, 64, 64
    cu = d["cu"].clone()
    if overshoot:
        # broken device contract: sequences overlap, one claims tokens past the batch, and
        # their chunks add up to more than the workspace was sized for; the kernels clamp every
        # span to the batch and cap the chunk count, so all writes stay inside the buffers
        cu = torch.tensor([0, T, 0, T + 500, 0], dtype=torch.int32, device="cuda")
    ob, o, po = _guarded((1, T, H, dv), torch.bfloat16)
    sb, S, ps = _guarded((N, H, dk, dv), torch.float32)
    pshape = (N, H, dk) if variant == "diag" else (N, H)
    pb, P, pp = _guarded(pshape, torch.float32)
    L = kdn.lib()
    ws_bytes = L.kdn_forward_workspace_bytes(0 if variant == "diag" else 1, N, 1, T, H, dk, dv,
                                             kdn.KDN_BF16, 1, 0)
    wb, ws, pw = _guarded((ws_bytes,), torch.uint8)
    import ctypes
    args = [kdn._ptr(d[n]) for n in NAMES] + [kdn._ptr(d["S0"]), kdn._ptr(d["P0"]),
                                              kdn._ptr(o), kdn._ptr(S), kdn._ptr(P),
                                              kdn._ptr(cu), N, 1, T, H, dk, dv, kdn.KDN_BF16]
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    tail = [ctypes.c_float(x.mu), ctypes.c_float(x.scale), 0, kdn._ptr(ws), ws_bytes, stream]
    if variant == "diag":
        st = L.kdn_forward_diag(*args, *tail)
    else:
        st = L.kdn_forward_iso(*args, 1, *tail)
    assert st == kdn.KDN_OK, L.kdn_last_error().decode()
    torch.cuda.synchronize()
    for name, b, pad in (("o", ob, po), ("S_T", sb, ps), ("P_T", pb, pp), ("workspace", wb, pw)):
        assert _canary_ok(b, pad), f"{name}: a write landed outside the buffer"
    if not overshoot:
        ref = run_oracle_forward(x)
        check("o", host_f64(o), ref["o"], TOL["bf16"])
        check("S_T", host_f64(S), ref["S_T"], TOL["bf16"])
