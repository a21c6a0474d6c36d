"""The C ABI on the host (no GPU): the library loads, exports every entry point declared in
include/kdn.h, and rejects bad arguments with the documented status before touching a device."""

import ctypes

import pytest

from paper_2609_07816_amd import kdn

F = ctypes.c_float


@pytest.fixture(scope="module")
def L():
    return kdn.lib()


def test_exports_every_declared_symbol(L):
    names = kdn.declared_symbols()
    assert len(names) >= 10
    for name in names:
        assert hasattr(L, name), f"{name} declared in include/kdn.h but not exported"


def test_status_strings(L):
    for code, name in enumerate(["KDN_OK", "KDN_ERR_INVALID_ARG", "KDN_ERR_UNSUPPORTED",
                                 "KDN_ERR_WORKSPACE", "KDN_ERR_HIP"]):
        assert L.kdn_status_string(code).decode() == name
    assert L.kdn_version().decode().startswith("kdn-mi355x")


# fake, never-dereferenced device addresses: argument checks run before any launch
def P(i):
    return ctypes.c_void_p(0x1000000 * (i + 1))


def fwd(L, variant=0, ptrs=None, N=1, B=1, T=8, H=2, dk=64, dv=64, dtype=1, mu=64.0,
        scale=0.125, chunk=0, cu=None, S0=None, S_T=None, P0=None, P_T=None):
    p = [P(i) for i in range(7)] if ptrs is None else ptrs
    args = p[:6] + [S0, P0, p[6], S_T, P_T, cu, N, B, T, H, dk, dv, dtype]
    if variant == 0:
        return L.kdn_forward_diag(*args, F(mu), F(scale), chunk, None, 0, None)
    return L.kdn_forward_iso(*args, 1, F(mu), F(scale), chunk, None, 0, None)


@pytest.mark.parametrize("variant", [0, 1])
def test_forward_argument_errors(L, variant):
    assert fwd(L, variant, ptrs=[None] + [P(i) for i in range(6)]) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, T=0) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, N=2, B=1) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, cu=P(20), N=2, B=2) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, mu=0.0) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, mu=-1.0) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, scale=0.0) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, dtype=7) == kdn.KDN_ERR_INVALID_ARG
    assert fwd(L, variant, dk=48) == kdn.KDN_ERR_UNSUPPORTED
    assert fwd(L, variant, dv=256) == kdn.KDN_ERR_UNSUPPORTED
    assert fwd(L, variant, chunk=24) == kdn.KDN_ERR_UNSUPPORTED
    assert fwd(L, variant, chunk=16) == kdn.KDN_ERR_UNSUPPORTED
    assert fwd(L, variant, chunk=32) == kdn.KDN_ERR_UNSUPPORTED
    # output aliasing an input
    p = [P(i) for i in range(7)]
    p[6] = p[2]
    assert fwd(L, variant, ptrs=p) == kdn.KDN_ERR_INVALID_ARG
    # partial overlap of the state output with the state input
    base = 0x7000000
    assert fwd(L, variant, S0=ctypes.c_void_p(base), S_T=ctypes.c_void_p(base + 64)) \
        == kdn.KDN_ERR_INVALID_ARG
    assert "S_T" in L.kdn_last_error().decode()


def test_decode_argument_errors(L):
    p = [P(i) for i in range(9)]

    def dec(variant=0, ptrs=p, slot=None, o=P(10), R=4, slots=4, H=2, dk=64, dv=64, dtype=1):
        return L.kdn_decode_step(variant, *ptrs[:6], ptrs[6], ptrs[7], slot, o, R, slots, H,
                                 dk, dv, dtype, 1, F(64.0), F(0.125), None)

    assert dec(variant=2) == kdn.KDN_ERR_INVALID_ARG
    assert dec(o=None) == kdn.KDN_ERR_INVALID_ARG
    assert dec(R=5, slots=4) == kdn.KDN_ERR_INVALID_ARG        # no slot map, too many rows
    assert dec(dk=8) == kdn.KDN_ERR_UNSUPPORTED
    assert dec(o=p[0]) == kdn.KDN_ERR_INVALID_ARG              # o aliases q


def test_gain_argument_errors(L):
    p = [P(i) for i in range(5)]
    st = L.kdn_gain_diag(*p[:4], None, p[4], None, None, None, 1, 1, 8, 2, 64, 1, F(64.0), None,
                         0, None)
    assert st == kdn.KDN_ERR_WORKSPACE
    need = L.kdn_gain_workspace_bytes(0, 1, 1, 8, 2, 64)
    assert need > 0
    st = L.kdn_gain_diag(*p[:4], None, p[4], None, None, None, 1, 1, 8, 2, 64, 1, F(-1.0),
                         P(30), need, None)
    assert st == kdn.KDN_ERR_INVALID_ARG
    # an input tensor of 2 GiB or more (T = 2^20, H = 16, d 128 bf16: 4 GiB) is refused before
    # the workspace is even looked at
    for f in (L.kdn_gain_diag, L.kdn_gain_iso):
        args = [*p[:4], None, p[4], None, None, None, 1, 1, 1 << 20, 16, 128, 1]
        if f is L.kdn_gain_iso:
            args.append(1)
        st = f(*args, F(64.0), None, 0, None)
        assert st == kdn.KDN_ERR_UNSUPPORTED


def test_forward_workspace(L):
    # the forward refuses a missing or short workspace before launching anything
    assert fwd(L, 0) == kdn.KDN_ERR_WORKSPACE
    need = L.kdn_forward_workspace_bytes(0, 1, 1, 8, 2, 64, 64, 1, 0, 0)
    assert need > 0
    p = [P(i) for i in range(7)]
    args = p[:6] + [None, None, p[6], None, None, None, 1, 1, 8, 2, 64, 64, 1]
    assert L.kdn_forward_diag(*args, F(64.0), F(0.125), 0, P(40), need - 1, None) \
        == kdn.KDN_ERR_WORKSPACE


def rec_bytes(dk, es):
    """Bytes of one (chunk, head) record of the prep: K_bar, Q_bar, P_tail^T (64 x dk each),
    L^-1 and A_qk (64 x 64 each) in the operand precision, and gamma_C (dk float32), rounded up
    to 256."""
    raw = 3 * 64 * dk * es + 2 * 64 * 64 * es + 4 * dk
    return (raw + 255) // 256 * 256


def al256(x):
    return (x + 255) // 256 * 256


def test_workspace_queries(L):
    # fixed length: maxch = N * ceil(T / 64) chunks; per chunk and head a float4 summary and a
    # float2 carry per variance channel, and one prep record
    N, T, H, dk = 4, 4096, 16, 128
    maxch = N * 64
    want = al256(maxch * H * dk * 16) + al256(maxch * H * dk * 8) + maxch * H * rec_bytes(dk, 2)
    assert L.kdn_forward_workspace_bytes(0, N, N, T, H, dk, 128, 1, 0, 0) == want
    assert L.kdn_forward_workspace_bytes(0, N, N, T, H, dk, 128, 1, 0, 64) == want
    want_iso = al256(maxch * H * 16) + al256(maxch * H * 8) + maxch * H * rec_bytes(dk, 2)
    assert L.kdn_forward_workspace_bytes(1, N, N, T, H, dk, 128, 1, 0, 0) == want_iso
    want_f32 = al256(maxch * H * dk * 16) + al256(maxch * H * dk * 8) + \
        maxch * H * rec_bytes(dk, 4)
    assert L.kdn_forward_workspace_bytes(0, N, N, T, H, dk, 128, 0, 0, 0) == want_f32
    # packed: maxch = T / 64 + N, plus the chunk-offset table and the walk order
    Np, Tp = 32, 135000
    maxp = Tp // 64 + Np
    want_p = al256((Np + 1) * 4) + al256(Np * 4) + al256(maxp * H * dk * 16) + \
        al256(maxp * H * dk * 8) + maxp * H * rec_bytes(dk, 2)
    assert L.kdn_forward_workspace_bytes(0, Np, 1, Tp, H, dk, 128, 1, 1, 0) == want_p
    # rejected arguments give 0
    assert L.kdn_forward_workspace_bytes(0, 4, 4, 4096, 16, 128, 128, 1, 0, 32) == 0
    assert L.kdn_forward_workspace_bytes(0, 4, 4, 4096, 16, 48, 128, 1, 0, 0) == 0
    assert L.kdn_forward_workspace_bytes(0, 0, 4, 4096, 16, 128, 128, 1, 0, 0) == 0
    assert L.kdn_forward_workspace_bytes(2, 4, 4, 4096, 16, 128, 128, 1, 0, 0) == 0
    small = L.kdn_gain_workspace_bytes(0, 1, 1, 64, 1, 128)
    big = L.kdn_gain_workspace_bytes(0, 4, 4, 4096, 16, 128)
    assert big > small > 0


def test_layer_argument_errors(L):
    p = [P(i) for i in range(7)]
    args = p[:6] + [None, None, p[6], None, None, None, 1, 1, 8, 2, 64, 64, 1, 1, F(64.0),
                    F(0.125)]
    need = L.kdn_forward_workspace_bytes(0, 1, 1, 8, 2, 64, 64, 1, 0, 0)
    ws = [P(40), need, None]
    opts = kdn.LayerOpts(1, 0.0, 0, None, None)          # gates_preact needs r_min > 0
    assert L.kdn_forward_layer(0, *args, ctypes.byref(opts), *ws) == kdn.KDN_ERR_INVALID_ARG
    assert "r_min" in L.kdn_last_error().decode()
    opts = kdn.LayerOpts(1, 0.01, 1, None, 0x1000000 * 3)  # beta_eff inside v
    assert L.kdn_forward_layer(0, *args, ctypes.byref(opts), *ws) == kdn.KDN_ERR_INVALID_ARG
    assert "beta_eff" in L.kdn_last_error().decode()
    opts = kdn.LayerOpts(0, 0.0, 0, 0x7000000, 0x7000000)  # beta_eff aliases mu_t
    assert L.kdn_forward_layer(0, *args, ctypes.byref(opts), *ws) == kdn.KDN_ERR_INVALID_ARG
    assert L.kdn_forward_layer(2, *args, None, *ws) == kdn.KDN_ERR_INVALID_ARG
    assert L.kdn_forward_layer(0, *args, None, P(40), need - 1, None) == kdn.KDN_ERR_WORKSPACE
    dec = [0] + [P(i) for i in range(8)] + [None, P(10), 4, 4, 2, 64, 64, 1, 1, F(64.0),
                                            F(0.125)]
    opts = kdn.LayerOpts(1, -1.0, 0, None, None)
    assert L.kdn_decode_step_layer(*dec, ctypes.byref(opts), None) == kdn.KDN_ERR_INVALID_ARG
    opts = kdn.LayerOpts(0, 0.0, 0, None, 0x1000000 * 11)  # beta_eff inside o
    assert L.kdn_decode_step_layer(*dec, ctypes.byref(opts), None) == kdn.KDN_ERR_INVALID_ARG


def test_misaligned_tensors_rejected(L):
    """Tensors of d_k or d_v columns are moved in 16-byte pieces: a pointer off a 16-byte
    boundary is refused before any launch (per-head scalars such as r have no such rule)."""
    off = ctypes.c_void_p(0x1000000 + 8)
    p = [P(i) for i in range(7)]
    assert fwd(L, ptrs=[off] + p[1:]) == kdn.KDN_ERR_INVALID_ARG
    assert "q must be 16-byte aligned" in L.kdn_last_error().decode()
    assert fwd(L, ptrs=p[:6] + [off]) == kdn.KDN_ERR_INVALID_ARG
    assert "o must be" in L.kdn_last_error().decode()
    # r (one value per token and head) may sit anywhere: the call reaches the workspace check
    assert fwd(L, ptrs=p[:5] + [ctypes.c_void_p(0x6000002)] + p[6:]) == kdn.KDN_ERR_WORKSPACE
    g = [P(i) for i in range(10, 18)]
    bwd = [0] + p[:6] + [None, None, None, 1, 1, 8, 2, 64, 64, 1, 1, F(64.0), F(0.125), None,
                         None, None]
    ws = [P(40), 1 << 40, None]
    g_bad = list(g)
    g_bad[2] = ctypes.c_void_p(0x1b000004)
    assert L.kdn_backward(*bwd, *g_bad, *ws) == kdn.KDN_ERR_INVALID_ARG
    assert "dv must be 16-byte aligned" in L.kdn_last_error().decode()
    dec = [0] + p[:6] + [ctypes.c_void_p(0x8000004), P(8), None, P(10), 4, 4, 2, 64, 64, 1, 1,
                         F(64.0), F(0.125), None]
    assert L.kdn_decode_step(*dec) == kdn.KDN_ERR_INVALID_ARG
    assert "S must be 16-byte aligned" in L.kdn_last_error().decode()
