"""Pins of the oracle's Kalman Associative Memory (oracle.forward_kam, the exact filter with a
dense covariance; Prop. "Kalman Associative Memory") against independent references (no GPU):
the information-form Gaussian conditioning of tests/bruteforce.py run over whole trajectories,
and the Diagonal KDN oracle in the case where the dense filter stays diagonal (one-hot keys,
diagonal initial covariance, information scale 1).
"""

import numpy as np
import pytest

import bruteforce as bf
import oracle

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def chain(x):
    x = np.asarray(x, dtype=np.float64)
    return x[None, :, None, ...]


@pytest.mark.parametrize("dk,dv,T,seed", [(5, 3, 9, 0), (4, 6, 12, 1), (7, 2, 5, 2)])
def test_kam_trajectory_equals_information_form_filter(dk, dv, T, seed):
    g = np.random.default_rng([50, seed])
    q, k = g.standard_normal((2, T, dk))
    v = g.standard_normal((T, dv))
    a = g.uniform(0.3, 1.0, (T, dk))
    w = g.uniform(0.01, 0.5, (T, dk))
    r = g.uniform(0.1, 2.0, T)
    S0 = g.standard_normal((dk, dv))
    X = g.standard_normal((dk, dk))
    P0 = X @ X.T / dk + 0.2 * np.eye(dk)
    out = oracle.forward_kam(chain(q), chain(k), chain(v), chain(a), chain(w), chain(r),
                             S0=S0[None, None], P0=P0[None, None], scale=0.6)
    S, P = S0.copy(), P0.copy()
    for t in range(T):
        S_hat, P_hat = bf.predict(S, P, np.diag(a[t]), np.diag(w[t]))
        S, P, _ = bf.condition(S_hat, P_hat, k[t], v[t], r[t])
        np.testing.assert_allclose(out["o"][0, t, 0], 0.6 * S.T @ q[t], rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(out["S_T"][0, 0], S, rtol=1e-9, atol=1e-11)
    np.testing.assert_allclose(out["P_T"][0, 0], P, rtol=1e-9, atol=1e-12)


def test_kam_stays_diagonal_on_one_hot_keys_and_equals_diagonal_kdn():
    """With one-hot keys, a diagonal initial covariance and diagonal D, Omega, the dense filter
    never leaves the diagonal family, so it is Diagonal KDN at information scale mu = 1."""
    g = np.random.default_rng(51)
    T, dk, dv = 30, 6, 4
    k = np.zeros((T, dk))
    k[np.arange(T), g.integers(0, dk, T)] = g.uniform(0.5, 2.0, T)
    q = g.standard_normal((T, dk))
    v = g.standard_normal((T, dv))
    a = g.uniform(0.5, 1.0, (T, dk))
    w = g.uniform(0.01, 0.3, (T, dk))
    r = g.uniform(0.1, 1.0, T)
    p0 = g.uniform(0.2, 1.5, dk)
    args = [chain(x) for x in (q, k, v, a, w, r)]
    kam = oracle.forward_kam(*args, P0=np.diag(p0)[None, None], scale=0.5)
    dia = oracle.forward_diag(*args, P0=p0[None, None], mu=1.0, scale=0.5)
    P = kam["P_T"][0, 0]
    np.testing.assert_array_equal(P - np.diag(np.diag(P)), 0.0)
    np.testing.assert_allclose(np.diag(P), dia["P_T"][0, 0], rtol=1e-12)
    np.testing.assert_allclose(kam["o"], dia["o"], rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(kam["S_T"], dia["S_T"], rtol=1e-11, atol=1e-13)


def test_kam_covariance_symmetric_positive_and_packed_batches_separate():
    g = np.random.default_rng(52)
    lens = [5, 0, 11]
    T, H, dk, dv = sum(lens), 2, 4, 3
    x = [g.standard_normal((1, T, H, dk)), g.standard_normal((1, T, H, dk)),
         g.standard_normal((1, T, H, dv)), g.uniform(0.4, 1.0, (1, T, H, dk)),
         g.uniform(0.01, 0.3, (1, T, H, dk)), g.uniform(0.2, 1.0, (1, T, H))]
    cu = np.array([0, 5, 5, 16], dtype=np.int32)
    out = oracle.forward_kam(*x, cu_seqlens=cu)
    for n in range(3):
        for h in range(H):
            P = out["P_T"][n, h]
            np.testing.assert_allclose(P, P.T, rtol=1e-12, atol=1e-14)
            assert np.all(np.linalg.eigvalsh(P) > 0)
        t0, t1 = cu[n], cu[n + 1]
        one = oracle.forward_kam(*[a[:, t0:t1] for a in x]) if t1 > t0 else None
        if one is not None:
            np.testing.assert_array_equal(out["o"][:, t0:t1], one["o"])
            np.testing.assert_array_equal(out["P_T"][n], one["P_T"][0])
    np.testing.assert_array_equal(out["P_T"][1], np.broadcast_to(np.eye(dk), (H, dk, dk)))


def test_kam_batch_rows_and_heads_are_independent_chains():
    """A fixed-length batch of two rows equals the two rows run alone (the row offset of every
    token); heads likewise."""
    g = np.random.default_rng(53)
    B, T, H, dk, dv = 2, 7, 2, 3, 2
    x = [g.standard_normal((B, T, H, dk)), g.standard_normal((B, T, H, dk)),
         g.standard_normal((B, T, H, dv)), g.uniform(0.4, 1.0, (B, T, H, dk)),
         g.uniform(0.01, 0.3, (B, T, H, dk)), g.uniform(0.2, 1.0, (B, T, H))]
    both = oracle.forward_kam(*x)
    for b in range(B):
        for h in range(H):
            one = oracle.forward_kam(*[a[b:b + 1, :, h:h + 1] for a in x])
            np.testing.assert_array_equal(both["o"][b:b + 1, :, h:h + 1], one["o"])
            np.testing.assert_array_equal(both["S_T"][b, h], one["S_T"][0, 0])
            np.testing.assert_array_equal(both["P_T"][b, h], one["P_T"][0, 0])
