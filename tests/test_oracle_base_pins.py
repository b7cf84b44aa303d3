"""Pins of the BASE-layer oracle (oracle/base.py): brute force over every
balanced assignment of tiny inputs, invariants of optimality, and special cases
with a known answer.  CPU only."""

import itertools

import numpy as np
import pytest

import oracle


def brute_force(L):
    N, E = L.shape
    c = N // E
    best = -np.inf
    for perm in itertools.permutations(range(N)):
        ids = np.array([perm[i] // c for i in range(N)])
        best = max(best, L[np.arange(N), ids].sum())
    return best


@pytest.mark.parametrize("N,E,seed", [(4, 2, 0), (6, 3, 1), (6, 2, 2), (8, 4, 3), (8, 2, 4), (6, 1, 5)])
def test_base_against_brute_force(N, E, seed):
    L = np.random.default_rng(seed).integers(-3, 4, (N, E)).astype(np.float64)
    ids, total = oracle.base_assign(L)
    assert np.bincount(ids, minlength=E).tolist() == [N // E] * E
    assert total == brute_force(L)
    assert total == L[np.arange(N), ids].sum()


def test_base_invariants():
    rng = np.random.default_rng(7)
    N, E = 96, 8
    L = rng.standard_normal((N, E))
    ids, total = oracle.base_assign(L)
    assert (np.bincount(ids, minlength=E) == N // E).all()
    # no exchange of two tokens between their experts improves the total
    own = L[np.arange(N), ids]
    swap = L[:, ids]                                         # swap[i, j] = L[i, ids[j]]
    assert (own[:, None] + own[None, :] >= swap + swap.T - 1e-12).all()
    # adding a constant to one expert's column changes nothing (every expert takes N / E)
    L2 = L.copy()
    L2[:, 3] += 5.0
    assert abs(oracle.base_assign(L2)[1] - (total + 5.0 * N / E)) < 1e-9
    # it is never worse than top-1 routing restricted to a balanced result
    assert total <= L.max(axis=1).sum() + 1e-12


def test_base_special_cases():
    # one expert: everything goes to it
    L = np.arange(6, dtype=np.float64).reshape(6, 1)
    assert oracle.base_assign(L)[0].tolist() == [0] * 6
    # scores already balanced by top-1: the top-1 routing is the answer
    L = np.array([[5.0, 0.0], [0.0, 5.0], [4.0, 1.0], [1.0, 4.0]])
    ids, total = oracle.base_assign(L)
    assert ids.tolist() == [0, 1, 0, 1] and total == 18.0
    # every token prefers expert 0: the two with the smallest loss for moving go to expert 1
    L = np.array([[9.0, 1.0], [9.0, 8.5], [9.0, 0.0], [9.0, 8.0]])
    ids, total = oracle.base_assign(L)
    assert ids.tolist() == [0, 1, 0, 1] and total == 9 + 8.5 + 9 + 8
    with pytest.raises(ValueError):
        oracle.base_assign(np.zeros((5, 2)))
    w = oracle.base_weights(np.array([[0.0, 2.0]]), [1])
    assert abs(w[0] - 1 / (1 + np.exp(-2.0))) < 1e-15
