"""Pins for the oracle's gradients (CPU only): torch autograd through fp64
masked attention (a library routine), central finite differences of the
fp64 forward, and closed forms of the softmax Jacobian."""
import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W


def _mask(rp, ci, N):
    m = np.zeros((N, N), dtype=bool)
    for i in range(N):
        m[i, ci[rp[i]:rp[i + 1]]] = True
    return m


@pytest.mark.parametrize("N,d,seed", [(9, 4, 0), (33, 16, 1), (64, 32, 2)])
def test_gradients_match_torch_autograd(oracle, N, d, seed):
    rng = np.random.default_rng(seed)
    rp, ci = W.random_csr(rng, N, max_deg=N, empty_frac=0.1, dup_frac=0.2)
    Q, K, V, G = (rng.standard_normal((N, d)) for _ in range(4))
    scale = 0.3
    dQ, dK, dV = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, scale)
    m = torch.from_numpy(_mask(rp, ci, N))
    t = [torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (Q, K, V)]
    S = scale * (t[0] @ t[1].T)
    S = S.masked_fill(~m, float("-inf"))
    rows = m.any(dim=1)
    P = torch.zeros_like(S)
    P[rows] = torch.softmax(S[rows], dim=1)
    O = P @ t[2]
    (O * torch.from_numpy(G)).sum().backward()
    for got, ref in zip((dQ, dK, dV), t):
        np.testing.assert_allclose(got, ref.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_gradients_match_finite_differences(oracle):
    rng = np.random.default_rng(3)
    N, d = 12, 3
    rp, ci = W.random_csr(rng, N, max_deg=6, empty_frac=0.1)
    Q, K, V, G = (rng.standard_normal((N, d)) for _ in range(4))
    scale = 0.7
    grads = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, scale)
    h = 1e-6
    for which in range(3):
        base = [Q, K, V]
        for idx in np.ndindex(N, d):
            plus = [x.copy() for x in base]
            minus = [x.copy() for x in base]
            plus[which][idx] += h
            minus[which][idx] -= h
            Lp = (oracle.attention_f64_exact(rp, ci, *plus, scale) * G).sum()
            Lm = (oracle.attention_f64_exact(rp, ci, *minus, scale) * G).sum()
            assert abs((Lp - Lm) / (2 * h) - grads[which][idx]) < 1e-7


def test_constant_keys_give_zero_query_gradient(oracle):
    """All K rows equal: every score of a row is the same, so the softmax
    Jacobian's rows sum to zero against a constant K: dQ = 0."""
    rng = np.random.default_rng(4)
    N, d = 40, 8
    rp, ci = W.random_csr(rng, N, max_deg=12)
    Q, V, G = (rng.standard_normal((N, d)) for _ in range(3))
    K = np.tile(rng.standard_normal(d), (N, 1))
    dQ, _, _ = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, 1.3)
    assert np.abs(dQ).max() < 1e-12


def test_single_neighbour_rows(oracle):
    """P = 1 on a single-neighbour row: no score gradient, dV_j = sum of G_i
    over the rows that point at j."""
    rng = np.random.default_rng(5)
    N, d = 30, 5
    j = rng.integers(0, N, size=N).astype(np.int32)
    rp = np.arange(N + 1, dtype=np.int32)
    Q, K, V, G = (rng.standard_normal((N, d)) for _ in range(4))
    dQ, dK, dV = oracle.attention_bwd_f64(rp, j, Q, K, V, G, 0.9)
    assert np.abs(dQ).max() < 1e-13 and np.abs(dK).max() < 1e-13
    ref = np.zeros((N, d))
    np.add.at(ref, j, G)
    np.testing.assert_allclose(dV, ref, rtol=0, atol=1e-13)


def test_binary16_entry_widens_exactly(oracle):
    rng = np.random.default_rng(6)
    N, d = 20, 8
    rp, ci = W.random_csr(rng, N, max_deg=7)
    X = [rng.standard_normal((N, d)).astype(np.float16) for _ in range(4)]
    a = oracle.attention_bwd_f64(rp, ci, *X, 0.5)
    b = oracle.attention_bwd_f64(rp, ci, *[x.astype(np.float64) for x in X], 0.5)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_constant_values_give_zero_score_gradients(oracle):
    """All V rows equal: O_i = V for every non-empty row whatever P is, so
    dP_ij = G_i . V is the same for all j of a row and equals delta_i: dS = 0,
    hence dQ = dK = 0, while dV still receives sum_i P_ij G_i."""
    rng = np.random.default_rng(7)
    N, d = 50, 6
    rp, ci = W.random_csr(rng, N, max_deg=10, empty_frac=0.1)
    Q, K, G = (rng.standard_normal((N, d)) for _ in range(3))
    V = np.tile(rng.standard_normal(d), (N, 1))
    dQ, dK, dV = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, 0.8)
    assert np.abs(dQ).max() < 1e-12 and np.abs(dK).max() < 1e-12
    # dV sums to the sum of G over non-empty rows (each P row sums to one)
    nonempty = np.diff(rp) > 0
    np.testing.assert_allclose(dV.sum(axis=0), G[nonempty].sum(axis=0), atol=1e-11)


def test_scale_derivative_identity(oracle):
    """The scores are scale * Q_i . K_j, so dL/dscale = sum dS_ij Q_i . K_j,
    which equals <dQ, Q> / scale and <dK, K> / scale; the derivative is
    checked against a central difference in the scale itself."""
    rng = np.random.default_rng(8)
    N, d = 25, 4
    rp, ci = W.random_csr(rng, N, max_deg=8, empty_frac=0.1)
    Q, K, V, G = (rng.standard_normal((N, d)) for _ in range(4))
    s = 0.6
    dQ, dK, _ = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, s)
    h = 1e-6
    fd = ((oracle.attention_f64_exact(rp, ci, Q, K, V, s + h) * G).sum()
          - (oracle.attention_f64_exact(rp, ci, Q, K, V, s - h) * G).sum()) / (2 * h)
    assert abs((dQ * Q).sum() / s - fd) < 1e-7
    assert abs((dK * K).sum() / s - fd) < 1e-7


def test_empty_rows_and_unreferenced_columns(oracle):
    """An empty row has O = 0 independent of its Q, so its dQ row is 0; a
    node no row points at contributes to no output, so its dK and dV rows
    are 0."""
    rng = np.random.default_rng(9)
    N, d = 40, 5
    rp, ci = W.random_csr(rng, N, max_deg=6, empty_frac=0.3)
    ci = np.where(ci < 3, ci + 3, ci).astype(np.int32)   # nodes 0, 1, 2 unreferenced
    Q, K, V, G = (rng.standard_normal((N, d)) for _ in range(4))
    dQ, dK, dV = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, 0.5)
    empty = np.diff(rp) == 0
    assert empty.any() and np.all(dQ[empty] == 0)
    unref = np.ones(N, dtype=bool)
    unref[ci] = False
    assert unref.any()
    assert np.all(dK[unref] == 0) and np.all(dV[unref] == 0)
