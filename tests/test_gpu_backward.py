"""GPU parity of kdn_backward (through the C ABI) against the oracle's reverse-mode adjoint
(oracle.backward, itself pinned by finite differences) on identical seeded inputs and identical
incoming adjoints dO, dS_T, dP_T.

Bound: relative L2 error <= 1e-5 on every gradient, for float32 and bf16 inputs alike: the
backward computes in float32 whatever the input dtype (bf16 inputs are exact in float32), so its
error is float32 rounding accumulated over sums of at most a chunk's 64 tokens, dk or dv terms,
the same budget as the forward's float32 bound.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import NAMES, dev_tensor, host_f64, rel_l2, to_device
from paper_2609_07816_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 1e-5
GRADS = ("dq", "dk", "dv", "dalpha", "domega", "dr", "dS0", "dP0")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_07816_amd import kdn
    kdn.lib()  # fail loudly when the library is missing


def check(name, got, ref, tol=TOL):
    err = rel_l2(got, ref)
    print(f"  {name}: rel-L2 {err:.3e} (bound {tol:g})", flush=True)
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert err <= tol, f"{name}: rel-L2 {err:.3e} > {tol:g}"


def adjoints(x, seed, with_state=True):
    g = np.random.default_rng(seed)
    dO = W.round_to(g.standard_normal((x.B, x.T, x.H, x.dv)), x.dtype)
    pshape = (x.N, x.H, x.dk) if x.variant == "diag" else (x.N, x.H)
    dS = g.standard_normal((x.N, x.H, x.dk, x.dv)).astype(np.float32) if with_state else None
    dP = g.standard_normal(pshape).astype(np.float32) if with_state else None
    return dO, dS, dP


def compare_backward(x, seed=0, with_state=True, tol=TOL):
    from paper_2609_07816_amd import kdn
    dO, dS, dP = adjoints(x, seed, with_state)
    d = to_device(x)
    got = kdn.backward(x.variant, d["q"], d["k"], d["v"], d["alpha"], d["omega"], d["r"],
                       S0=d["S0"], P0=d["P0"], cu_seqlens=d["cu"], mu=x.mu, scale=x.scale,
                       dO=dev_tensor(dO, x.dtype),
                       dS_T=None if dS is None else torch.from_numpy(dS).cuda(),
                       dP_T=None if dP is None else torch.from_numpy(dP).cuda())
    torch.cuda.synchronize()
    ref = oracle.backward(x.variant, *[x.f64(n) for n in NAMES], S0=x.S0, P0=x.P0,
                          cu_seqlens=x.cu_seqlens, mu=x.mu, scale=x.scale,
                          dO=W.to_f64(dO, x.dtype), dS_T=dS, dP_T=dP)
    for name in GRADS:
        g = host_f64(got[name])
        r = ref[name]
        if x.cu_seqlens is not None and name not in ("dS0", "dP0"):
            n_tok = int(x.cu_seqlens[-1])
            g, r = g[:, :n_tok], r[:, :n_tok]
        check(name, g, r, tol)


@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
def test_backward_tiny_f32(variant, apc):
    compare_backward(W.draw_workload(0, variant, apc), seed=90)


@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
@pytest.mark.parametrize("T", [150, 64, 17])
def test_backward_f32_multichunk_ragged(variant, apc, T):
    x = W.draw_inputs(variant, "f32", 2, T, 3, 32, 32, seed=91, alpha_per_channel=apc,
                      random_state=True)
    compare_backward(x, seed=91)


def test_backward_output_adjoint_only():
    x = W.draw_inputs("diag", "f32", 2, 130, 2, 32, 32, seed=92)
    compare_backward(x, seed=92, with_state=False)


@pytest.mark.parametrize("dk,dv", [(128, 128), (64, 128), (128, 64), (16, 32), (32, 16)])
def test_backward_f32_head_sizes(dk, dv):
    x = W.draw_inputs("diag", "f32", 1, 100, 2, dk, dv, seed=93, random_state=True)
    compare_backward(x, seed=93)


@pytest.mark.parametrize("variant,apc", [("diag", True), ("iso", True), ("iso", False)])
def test_backward_bf16(variant, apc):
    x = W.draw_inputs(variant, "bf16", 2, 200, 2, 128, 128, seed=94, alpha_per_channel=apc,
                      random_state=True)
    compare_backward(x, seed=94)


@pytest.mark.parametrize("variant", ["diag", "iso"])
def test_backward_packed_ragged(variant):
    lens = [1, 63, 64, 0, 65, 130, 7]
    x = W.draw_inputs(variant, "f32", 1, sum(lens), 2, 32, 32, seed=95, lengths=lens,
                      random_state=True)
    compare_backward(x, seed=95)


def test_backward_small_gates_and_zero_noise():
    """Gates down to 0.01 (decays far below the float32 range over a chunk), omega = 0 and a
    tiny r: every decay ratio stays at most one."""
    x = W.draw_inputs("diag", "f32", 1, 200, 2, 32, 32, seed=96, random_state=True,
                      alpha_law=("uniform", 0.01, 0.3), omega_law=("const", 0.0),
                      r_law=("uniform", 1e-3, 2e-3))
    compare_backward(x, seed=96)


# ---------------------------------------------------------------------------------------------
# full-size workloads (the isotropic B4 T2048 and the diagonal B4 T4096 at H16 d128, bf16), the
# backward run once over the whole batch, checked on sampled (batch row, head) chains: each
# chain's gradients depend on that chain's inputs and adjoints only, so the oracle runs on the
# sampled slices alone
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("wid", [1, 2])
def test_backward_full_workload_sampled(wid):
    from paper_2609_07816_amd import kdn
    x = W.draw_workload(wid)
    dO, dS, dP = adjoints(x, seed=100 + wid)
    d = to_device(x)
    got = kdn.backward(x.variant, d["q"], d["k"], d["v"], d["alpha"], d["omega"], d["r"],
                       S0=d["S0"], P0=d["P0"], mu=x.mu, scale=x.scale,
                       dO=dev_tensor(dO, x.dtype), dS_T=torch.from_numpy(dS).cuda(),
                       dP_T=torch.from_numpy(dP).cuda())
    torch.cuda.synchronize()
    chains = [(0, 0), (x.B - 1, x.H - 1), (1, 7)]
    for b, h in chains:
        tok = (slice(b, b + 1), slice(None), slice(h, h + 1))
        st = (slice(b, b + 1), slice(h, h + 1))
        ins = [x.f64(n)[tok] for n in NAMES]
        ref = oracle.backward(x.variant, *ins, S0=None if x.S0 is None else x.S0[st],
                              P0=None if x.P0 is None else x.P0[st], mu=x.mu, scale=x.scale,
                              dO=W.to_f64(dO, x.dtype)[tok], dS_T=dS[st], dP_T=dP[st])
        print(f" chain (b={b}, h={h})", flush=True)
        for name in GRADS:
            sl = st if name in ("dS0", "dP0") else tok
            check(name, host_f64(got[name][sl]), ref[name])
