"""Exact oracle checks on sampled rows of large patterns.

The oracle runs on a small problem cut out of the pattern: the sampled rows
keep their full neighbour lists, every node they reference is present (with
an empty list of its own), so the operator's output on a sampled row and its
gradient contributions are exactly those of the whole problem.
"""
import numpy as np


def _neighbours(rp, ci, rows):
    """Concatenated neighbour lists of `rows` (in the given order) and the
    list lengths."""
    rp = np.asarray(rp, dtype=np.int64)
    lens = rp[rows + 1] - rp[rows]
    starts = np.repeat(rp[rows], lens)
    offs = np.arange(int(lens.sum()), dtype=np.int64) - np.repeat(np.cumsum(lens) - lens, lens)
    return np.asarray(ci)[starts + offs], lens


def rows_subproblem(rp, ci, rows):
    """(mrp, mci, U): a CSR over the nodes U (sorted global ids) in which the
    sorted distinct `rows` keep their neighbour lists and every other node of
    U has none; local id of a global node x is searchsorted(U, x)."""
    rows = np.unique(np.asarray(rows, dtype=np.int64))
    nb, lens = _neighbours(rp, ci, rows)
    U = np.unique(np.concatenate([rows, nb.astype(np.int64)]))
    deg = np.zeros(U.size, dtype=np.int64)
    deg[np.searchsorted(U, rows)] = lens
    mrp = np.zeros(U.size + 1, dtype=np.int64)
    np.cumsum(deg, out=mrp[1:])
    mci = np.searchsorted(U, nb).astype(np.int32)
    return mrp.astype(np.int32), mci, U


def rows_attending(rp, ci, keys):
    """Rows whose neighbour list holds one of `keys` (the rows of A^T)."""
    hit = np.isin(np.asarray(ci), np.asarray(keys))
    owner = np.repeat(np.arange(len(rp) - 1, dtype=np.int64), np.diff(np.asarray(rp)))
    return np.unique(owner[hit])


def sample_keys(rp, ci, n_random, n_hubs, rng):
    """n_random uniformly drawn nodes plus the n_hubs nodes referenced by the
    most rows (the heaviest rows of A^T), sorted and distinct."""
    N = len(rp) - 1
    indeg = np.bincount(np.asarray(ci), minlength=N)
    hubs = np.argsort(indeg, kind="stable")[-n_hubs:]
    return np.unique(np.concatenate([rng.integers(0, N, size=n_random), hubs,
                                     [0, N - 1]]).astype(np.int64))
