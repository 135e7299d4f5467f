"""The sampled-row method of the large GPU parity tests (tests/_subproblem):
on small random patterns the oracle's outputs and gradients on the
sub-problem equal, exactly, those of the whole problem on the sampled rows
and keys (CPU only)."""
import numpy as np
import pytest

from paper_2505_08098_amd import workloads as W
from _subproblem import rows_attending, rows_subproblem, sample_keys


@pytest.mark.parametrize("seed", range(3))
def test_subproblem_is_exact(oracle, seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(50, 400))
    rp, ci = W.random_csr(rng, N, max_deg=min(N, 40), empty_frac=0.1, dup_frac=0.2)
    Q, K, V, G = (rng.standard_normal((N, 32)).astype(np.float16) for _ in range(4))
    full = oracle.attention_bwd_f64(rp, ci, Q, K, V, G, 0.2)
    fo = oracle.attention_f64(rp, ci, Q, K, V, 0.2)
    S = sample_keys(rp, ci, 15, 3, rng)
    R = np.union1d(S, rows_attending(rp, ci, S))
    mrp, mci, U = rows_subproblem(rp, ci, R)
    assert oracle.check_csr(mrp, mci, U.size) == 0
    sub = oracle.attention_bwd_f64(mrp, mci, Q[U], K[U], V[U], G[U], 0.2)
    so = oracle.attention_f64(mrp, mci, Q[U], K[U], V[U], 0.2)
    iR, iS = np.searchsorted(U, R), np.searchsorted(U, S)
    assert np.array_equal(so[iR], fo[R])
    assert np.array_equal(sub[0][iR], full[0][R])
    assert np.array_equal(sub[1][iS], full[1][S])
    assert np.array_equal(sub[2][iS], full[2][S])


def test_sample_keys_holds_the_hubs():
    rng = np.random.default_rng(4)
    N = 1000
    rp, ci = W.random_csr(rng, N, max_deg=5)
    ci[::3] = 7       # node 7 is referenced by many rows
    S = sample_keys(rp, ci, 10, 1, rng)
    assert 7 in S and 0 in S and N - 1 in S
    assert set(rows_attending(rp, ci, [7]).tolist()) == set(
        np.repeat(np.arange(N), np.diff(rp))[ci == 7].tolist())
