"""Pins of the oracle's further gates (Sec. 3.1): hierarchical top-k (R19),
Dense-To-Sparse noisy tempered logits (R20) and the balanced hash table (R21),
against brute force, library routines, the Gumbel-max identity, hand-computed
cases and the list-scheduling bound.  CPU only."""

import itertools

import numpy as np
import pytest
import torch

import oracle


@pytest.mark.parametrize("E,groups,k", [(4, 2, 1), (6, 3, 2), (8, 2, 3), (12, 4, 3), (8, 8, 1), (12, 1, 4)])
def test_htopk_against_group_maxima_and_stable_sort(E, groups, k):
    rng = np.random.default_rng(E * 10 + groups + k)
    L = rng.integers(0, 3, (300, E)).astype(np.float64)  # dense ties
    ids = oracle.select(L, oracle.GATE_HTOPK, k, groups)
    Gs = E // groups
    gmax = L.reshape(300, groups, Gs).max(axis=2)
    for s in range(300):
        g = int(np.argmax(gmax[s]))  # first maximum: the lower group on ties
        part = L[s, g * Gs:(g + 1) * Gs]
        want = g * Gs + np.argsort(-part, kind="stable")[:k]
        assert ids[s].tolist() == want.tolist(), (s, L[s], ids[s])


def test_htopk_with_one_group_is_topk_and_contains_the_best():
    rng = np.random.default_rng(4)
    L = rng.standard_normal((200, 16))
    assert np.array_equal(oracle.select(L, oracle.GATE_HTOPK, 3, 1), oracle.select(L, oracle.GATE_TOPK, 3))
    ids = oracle.select(L, oracle.GATE_HTOPK, 2, 4)
    top1 = oracle.select(L, oracle.GATE_TOPK, 1)[:, 0]
    assert (ids[:, 0] == top1).all()
    assert (ids[:, 0] // 4 == ids[:, 1] // 4).all()
    w1 = oracle.gate_weights(L, ids, oracle.GATE_HTOPK, 1)
    np.testing.assert_allclose(w1.sum(axis=1), 1.0, rtol=1e-15)
    p = torch.softmax(torch.tensor(L), dim=1).numpy()
    np.testing.assert_allclose(oracle.gate_weights(L, ids, oracle.GATE_HTOPK, 0), p[np.arange(200)[:, None], ids],
                               rtol=1e-13)


def test_dense_to_sparse_gumbel_max_identity():
    # with tau = 1, the argmax of L + g (g standard Gumbel) is distributed as softmax(L)
    L = np.array([0.5, -1.0, 1.2, 0.0, 0.3], dtype=np.float32)
    n = 200000
    rng = np.random.default_rng(7)
    g = -np.log(-np.log(rng.random((n, L.size)))).astype(np.float32)
    noisy = oracle.noisy_logits_f32(np.broadcast_to(L, (n, L.size)), g, 1.0)
    winners = np.argmax(noisy, axis=1)
    freq = np.bincount(winners, minlength=L.size) / n
    p = np.exp(L.astype(np.float64) - L.max())
    p /= p.sum()
    assert (np.abs(freq - p) <= 4 * np.sqrt(p * (1 - p) / n)).all(), (freq, p)


def test_dense_to_sparse_temperature_and_rounding():
    L = np.array([[1.0, 3.0, -2.0, 0.5]], dtype=np.float32)
    # a power-of-two temperature scales exactly; order and gaps scale with it
    out = oracle.noisy_logits_f32(L, None, 0.25)
    assert np.array_equal(out, L * 4)
    # the sum is rounded to fp32 before the division: 1 + 2^-24 ties to 1, then / 3
    one = np.array([[1.0]], dtype=np.float32)
    tiny = np.array([[2.0 ** -24]], dtype=np.float32)
    assert oracle.noisy_logits_f32(one, tiny, 3.0)[0, 0] == np.float32(1.0) / np.float32(3.0)
    # a lower temperature sharpens the Switch weight of the best expert
    ids = oracle.select(L.astype(np.float64), oracle.GATE_TOPK, 1)
    w_hot = oracle.gate_weights(oracle.noisy_logits_f32(L, None, 1.0).astype(np.float64), ids, oracle.GATE_TOPK, 0)
    w_cold = oracle.gate_weights(oracle.noisy_logits_f32(L, None, 0.1).astype(np.float64), ids, oracle.GATE_TOPK, 0)
    assert w_cold[0, 0] > w_hot[0, 0] > 0.5


def test_balanced_table_hand_case():
    # loads: t0 (5) -> e0; t1 (4) -> e1; t2 (3) -> e1 [4 < 5]; t3 (3) -> e0 [5 < 7];
    # t4 (2) -> e1 [7 < 8]; t5 (1) -> e0 [8 < 9]: final loads 9 and 9
    assert oracle.balanced_hash_table([5, 4, 3, 3, 2, 1], 2).tolist() == [0, 1, 1, 0, 1, 0]
    # equal frequencies go in id order, equal loads to the lower expert
    assert oracle.balanced_hash_table([1, 1, 1, 1, 1], 3).tolist() == [0, 1, 2, 0, 1]
    assert oracle.table_hash_ids([4, 0, 2], np.array([0, 1, 1, 0, 1])).tolist() == [[1], [0], [1]]


def test_balanced_table_bounds_against_brute_force():
    rng = np.random.default_rng(9)
    for trial in range(60):
        vocab = int(rng.integers(1, 8))
        E = int(rng.integers(1, 4))
        freq = rng.integers(0, 20, vocab).astype(np.float64)
        table = oracle.balanced_hash_table(freq, E)
        load = np.bincount(table, weights=freq, minlength=E)
        assert load.sum() == freq.sum() and ((table >= 0) & (table < E)).all()
        # the last token placed went to the least loaded expert
        assert load.max() - load.min() <= freq.max() + 1e-12
        best = min(max(np.bincount(np.array(a), weights=freq, minlength=E)) for a in
                   itertools.product(range(E), repeat=vocab))
        assert load.max() <= (4.0 / 3.0 - 1.0 / (3.0 * E)) * best + 1e-9, (freq, E, load, best)


def test_balanced_table_zipf_balance():
    ranks = np.arange(1, 50258, dtype=np.float64)
    p = ranks ** -1.1
    p /= p.sum()
    table = oracle.balanced_hash_table(p, 128)
    load = np.bincount(table, weights=p, minlength=128)
    # the most frequent token alone holds 13.9 % of the mass, so no assignment
    # can have a smaller largest load; the greedy one reaches exactly that
    assert abs(load.max() - p.max()) < 1e-12
    assert (table == table[0]).sum() == 1 and abs(load.sum() - 1.0) < 1e-12


@pytest.mark.parametrize("kind,normalize,k,groups", [(oracle.GATE_HTOPK, 1, 2, 4), (oracle.GATE_HTOPK, 0, 3, 2)])
def test_htopk_and_temperature_gradient_central_differences(kind, normalize, k, groups):
    rng = np.random.default_rng(13)
    S, E, tau = 4, 8, 0.7
    Lraw = rng.standard_normal((S, E)) * 2
    g = rng.standard_normal((S, E))
    t = float(np.float32(tau))
    Lf = (Lraw + g) / t
    ids = oracle.select(Lf, kind, k, groups)
    dw = rng.standard_normal((S, k))
    dL, _ = oracle.gate_dlogits(Lf, ids, dw, kind, normalize, temperature=tau)
    h = 1e-6
    fd = np.zeros_like(Lraw)
    for s in range(S):
        for e in range(E):
            Lp, Lm = Lraw.copy(), Lraw.copy()
            Lp[s, e] += h
            Lm[s, e] -= h
            fp = (dw * oracle.gate_weights((Lp + g) / t, ids, kind, normalize)).sum()
            fm = (dw * oracle.gate_weights((Lm + g) / t, ids, kind, normalize)).sum()
            fd[s, e] = (fp - fm) / (2 * h)
    np.testing.assert_allclose(dL, fd, atol=1e-7)
