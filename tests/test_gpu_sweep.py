"""A seeded random sweep over the configuration space, every case through the C ABI against the
oracle on identical inputs: the forward (o, S_T, P_T), the gain scan alone (kappa/beta, p_hat/
b_hat, P_T), one decode step from the initial states (rows of empty sequences skipped through
the slot map) and, for every fourth case, the backward.

The axes: variant and gate mode, input dtype, head sizes d_k and d_v, batch or packed lengths
(empty, one-token and chunk-boundary sequences among them), initial states given or not, and mu
and scale at or away from their defaults. Bounds as in the other parity tests: rel-L2 1e-5 for
float32 inputs and 2e-2 for bf16 inputs on the forward and decode; 1e-5 for the float32 gain
scan and gradients from identical inputs.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import NAMES, TOL, dev_tensor, host_f64, rel_l2, run_oracle_forward, to_device
from paper_2609_07816_amd import workloads as W

pytestmark = pytest.mark.gpu

NCASES = 24
GRADS = ("dq", "dk", "dv", "dalpha", "domega", "dr", "dS0", "dP0")


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


def draw_case(i):
    g = np.random.default_rng([70, i])
    variant, apc = [("diag", True), ("iso", True), ("iso", False)][i % 3]
    dtype = ("f32", "bf16")[(i // 3) % 2]
    dk, dv = (int(v) for v in g.choice([16, 32, 64, 128], size=2))
    H = int(g.integers(1, 4))
    packed = bool(g.integers(0, 2))
    random_state = bool(g.integers(0, 2))
    mu = float(dk) if g.integers(0, 2) else float(g.uniform(0.5, 2.0) * dk)
    scale = float(dk ** -0.5) if g.integers(0, 2) else float(g.uniform(0.1, 1.0))
    common = dict(seed=700 + i, alpha_per_channel=apc, random_state=random_state, mu=mu,
                  scale=scale)
    if packed:
        lens = [int(v) for v in g.choice([0, 1, 17, 63, 64, 65, 150, 200],
                                         size=int(g.integers(1, 6)))]
        if sum(lens) == 0:
            lens[0] = 5
        return W.draw_inputs(variant, dtype, 1, sum(lens), H, dk, dv, lengths=lens, **common)
    B, T = int(g.integers(1, 4)), int(g.integers(1, 260))
    return W.draw_inputs(variant, dtype, B, T, H, dk, dv, **common)


def describe(x):
    shape = (f"packed {np.diff(x.cu_seqlens).tolist()}" if x.cu_seqlens is not None
             else f"B{x.B} T{x.T}")
    return (f"{x.variant}{'' if x.alpha_per_channel else ' scalar gates'} {x.dtype} {shape} "
            f"H{x.H} dk{x.dk} dv{x.dv} mu {x.mu:.3g} scale {x.scale:.3g} "
            f"{'random' if x.S0 is not None else 'default'} initial states")


def token_rows(x):
    """Token 0 of every sequence (rows of empty sequences: zeros, slot -1)."""
    if x.cu_seqlens is None:
        return {n: x.stored[n][:, 0] for n in NAMES}, np.arange(x.B, dtype=np.int32)
    cu = x.cu_seqlens
    rows = {}
    for n in NAMES:
        a = x.stored[n][0]
        rows[n] = np.stack([a[min(int(cu[s]), x.T - 1)] for s in range(len(cu) - 1)])
    slots = np.array([s if cu[s + 1] > cu[s] else -1 for s in range(len(cu) - 1)],
                     dtype=np.int32)
    return rows, slots


@pytest.mark.parametrize("i", range(NCASES))
def test_sweep(i):
    from paper_2609_07816_amd import kdn
    x = draw_case(i)
    print(f" case {i}: {describe(x)}", flush=True)
    tol = TOL[x.dtype]
    d = to_device(x)
    ntok = x.T if x.cu_seqlens is None else int(x.cu_seqlens[-1])

    # forward
    f = kdn.forward_diag if x.variant == "diag" else kdn.forward_iso
    o, S, P = f(*[d[n] for n in NAMES], S0=d["S0"], P0=d["P0"], cu_seqlens=d["cu"], mu=x.mu,
                scale=x.scale)
    torch.cuda.synchronize()
    ref = run_oracle_forward(x, traces=True)
    check("o", host_f64(o)[:, :ntok], ref["o"][:, :ntok], tol)
    check("S_T", host_f64(S), ref["S_T"], tol)
    check("P_T", host_f64(P), ref["P_T"], tol)

    # gain scan alone
    fg = kdn.gain_diag if x.variant == "diag" else kdn.gain_iso
    gn, ph, P2 = fg(d["k"], d["alpha"], d["omega"], d["r"], P0=d["P0"], cu_seqlens=d["cu"],
                    mu=x.mu)
    torch.cuda.synchronize()
    gname, pname = ("kappa", "phat") if x.variant == "diag" else ("beta", "bhat")
    check(gname, host_f64(gn)[:, :ntok], ref[gname][:, :ntok], 1e-5)
    check(pname, host_f64(ph)[:, :ntok], ref[pname][:, :ntok], 1e-5)
    check("P_T (gain scan)", host_f64(P2), ref["P_T"], 1e-5)

    # one decode step per sequence from the initial states
    rows, slots = token_rows(x)
    N = x.N
    pshape = (N, x.H, x.dk) if x.variant == "diag" else (N, x.H)
    S0 = x.S0 if x.S0 is not None else np.zeros((N, x.H, x.dk, x.dv), np.float32)
    P0 = x.P0 if x.P0 is not None else np.ones(pshape, np.float32)
    S_dev, P_dev = torch.from_numpy(S0.copy()).cuda(), torch.from_numpy(P0.copy()).cuda()
    od = kdn.decode_step(x.variant, *[dev_tensor(rows[n], x.dtype) for n in NAMES], S_dev, P_dev,
                         slot_idx=torch.from_numpy(slots).cuda(), mu=x.mu, scale=x.scale)
    torch.cuda.synchronize()
    S_ref, P_ref = S0.astype(np.float64), P0.astype(np.float64)
    o_ref = oracle.decode_step(x.variant, *[W.to_f64(rows[n], x.dtype) for n in NAMES], S_ref,
                               P_ref, slot_idx=slots, mu=x.mu, scale=x.scale)
    live = slots >= 0
    check("decode o", host_f64(od)[live], o_ref[live], tol)
    check("decode S", host_f64(S_dev), S_ref, tol)
    check("decode P", host_f64(P_dev), P_ref, tol)

    # backward
    if i % 4 == 0:
        g = np.random.default_rng([71, i])
        dO = W.round_to(g.standard_normal((x.B, x.T, x.H, x.dv)), x.dtype)
        dS = g.standard_normal((N, x.H, x.dk, x.dv)).astype(np.float32)
        dP = g.standard_normal(pshape).astype(np.float32)
        got = kdn.backward(x.variant, *[d[n] for n in NAMES], S0=d["S0"], P0=d["P0"],
                           cu_seqlens=d["cu"], mu=x.mu, scale=x.scale,
                           dO=dev_tensor(dO, x.dtype), dS_T=torch.from_numpy(dS).cuda(),
                           dP_T=torch.from_numpy(dP).cuda())
        torch.cuda.synchronize()
        bref = oracle.backward(x.variant, *[x.f64(n) for n in NAMES], S0=x.S0, P0=x.P0,
                               cu_seqlens=x.cu_seqlens, mu=x.mu, scale=x.scale,
                               dO=W.to_f64(dO, x.dtype), dS_T=dS, dP_T=dP)
        for name in GRADS:
            gv, rv = host_f64(got[name]), bref[name]
            if name not in ("dS0", "dP0"):
                gv, rv = gv[:, :ntok], rv[:, :ntok]
            check(name, gv, rv, 1e-5)
