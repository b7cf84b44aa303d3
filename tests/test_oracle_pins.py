"""Pins for the CPU oracle: hand cases, brute force, closed forms, library
cross-checks and invariants.  None of these re-types the oracle's formulas; each
checks it against something the paper or the mathematics fixes."""

import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st
from hypothesis.extra import numpy as hnp

import oracle
from oracle import GATE_HASH, GATE_KTOP1, GATE_TOPK

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------- bf16

def test_bf16_hand_cases():
    for case in golden("bf16_rne.json")["cases"]:
        v = float.fromhex(case["value"])
        got = int(oracle.f64_to_bf16(np.array([v]))[0])
        assert got == int(case["bits"], 16), case
        # decoding the expected pattern gives a value within half a spacing
        back = float(oracle.bf16_to_f64(np.array([got], dtype=np.uint16))[0])
        assert math.copysign(1.0, back) == math.copysign(1.0, v)


def test_bf16_matches_torch_from_f32():
    rng = np.random.default_rng(11)
    v = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-38).astype(np.float32),
        (rng.standard_normal(2000) * 1e30).astype(np.float32),
        # exact ties: low 16 bits 0x8000 on odd and even upper halves
        (np.arange(0x3F800000, 0x3F800000 + 64 * 0x10000, 0x10000, dtype=np.uint32) | 0x8000).view(np.float32),
    ])
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.f64_to_bf16(v.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_bf16_decode_is_exact_for_all_finite_patterns():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = oracle.bf16_to_f64(bits)
    finite = np.isfinite(vals)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(vals[finite], ref[finite])
    # round trip of every finite pattern
    np.testing.assert_array_equal(oracle.f64_to_bf16(vals[finite]), bits[finite])


# ------------------------------------------------------------------------- logits

def test_logits_integer_hand_case():
    g = golden("logits_int.json")
    x = np.array(g["x"], dtype=np.float32)
    wg = np.array(g["wg"], dtype=np.float32)
    bias = np.array(g["bias"], dtype=np.float32)
    L, A = oracle.logits(x, wg, "f32", bias)
    np.testing.assert_array_equal(L, np.array(g["logits"]))
    np.testing.assert_array_equal(A, np.array(g["magnitude"]))
    L0, _ = oracle.logits(x, wg, "f32", None)
    np.testing.assert_array_equal(L0, np.array(g["logits"]) - bias[None, :])


def test_logits_bf16_inputs_decoded_exactly():
    g = golden("logits_int.json")
    x = torch.tensor(g["x"], dtype=torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    wg = torch.tensor(g["wg"], dtype=torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    L, _ = oracle.logits(x, wg, "bf16", np.array(g["bias"], dtype=np.float32))
    np.testing.assert_array_equal(L, np.array(g["logits"]))


def test_logits_brute_force_sum():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 7)).astype(np.float32)
    wg = rng.standard_normal((7, 3)).astype(np.float32)
    L, A = oracle.logits(x, wg, "f32")
    for s in range(5):
        for e in range(3):
            terms = [float(x[s, j]) * float(wg[j, e]) for j in range(7)]
            assert math.isclose(L[s, e], math.fsum(terms), rel_tol=0, abs_tol=1e-12)
            assert math.isclose(A[s, e], math.fsum(abs(t) for t in terms), rel_tol=0, abs_tol=1e-12)


# ---------------------------------------------------------------------- selection

def _beats(row, a, b):
    return row[a] > row[b] or (row[a] == row[b] and a < b)


def _brute_topk(row, k):
    E = len(row)
    winners = [c for c in itertools.combinations(range(E), k)
               if all(_beats(row, a, b) for a in c for b in range(E) if b not in c)]
    assert len(winners) == 1
    subset = list(winners[0])
    # rank inside the subset: how many members beat it
    return sorted(subset, key=lambda a: sum(_beats(row, b, a) for b in subset))


def test_topk_brute_force_dense_ties():
    rng = np.random.default_rng(5)
    for E in range(1, 7):
        L = rng.integers(0, 3, size=(60, E)).astype(np.float64)
        for k in range(1, E + 1):
            ids = oracle.select(L, GATE_TOPK, k)
            for s in range(L.shape[0]):
                assert list(ids[s]) == _brute_topk(L[s], k)


def test_topk_matches_stable_argsort():
    rng = np.random.default_rng(6)
    L = rng.integers(-4, 4, size=(200, 16)).astype(np.float64) * 0.5
    ids = oracle.select(L, GATE_TOPK, 4)
    ref = np.argsort(-L, axis=1, kind="stable")[:, :4]
    np.testing.assert_array_equal(ids, ref)


def test_ktop1_brute_force():
    rng = np.random.default_rng(7)
    for E, k in [(4, 2), (6, 3), (6, 2), (8, 4), (5, 1)]:
        G = E // k
        L = rng.integers(0, 3, size=(50, E)).astype(np.float64)
        ids = oracle.select(L, GATE_KTOP1, k)
        for s in range(50):
            for g in range(k):
                grp = range(g * G, (g + 1) * G)
                best = [a for a in grp if all(_beats(L[s], a, b) for b in grp if b != a)]
                assert ids[s, g] == best[0]
                assert g * G <= ids[s, g] < (g + 1) * G


def test_selection_shift_invariance_and_negative_zero():
    rng = np.random.default_rng(8)
    L = rng.standard_normal((30, 8))
    for kind, k in [(GATE_TOPK, 2), (GATE_KTOP1, 2)]:
        a = oracle.select(L, kind, k)
        b = oracle.select(L + 3.25, kind, k)
        np.testing.assert_array_equal(a, b)
    # -0.0 and +0.0 compare equal: the lower index wins
    L0 = np.array([[-0.0, 0.0, -1.0]])
    assert list(oracle.select(L0, GATE_TOPK, 2)[0]) == [0, 1]
    L1 = np.array([[0.0, -0.0, -1.0]])
    assert list(oracle.select(L1, GATE_TOPK, 2)[0]) == [0, 1]


# ------------------------------------------------------------------------ weights

def test_weights_hand_cases():
    for c in golden("softmax_hand.json")["cases"]:
        L = np.array([c["logits"]], dtype=np.float64)
        kind = GATE_TOPK if c["kind"] == "topk" else GATE_KTOP1
        ids = oracle.select(L, kind, c["k"])
        assert list(ids[0]) == c["ids"], c
        w = oracle.gate_weights(L, ids, kind, c["normalize"])
        np.testing.assert_allclose(w[0], c["weights"], rtol=1e-15, atol=0)


def test_top2_closed_form_sigmoid():
    rng = np.random.default_rng(9)
    L = rng.standard_normal((100, 6)) * 3
    ids = oracle.select(L, GATE_TOPK, 2)
    w = oracle.gate_weights(L, ids, GATE_TOPK, 1)
    delta = L[np.arange(100), ids[:, 0]] - L[np.arange(100), ids[:, 1]]
    assert (delta >= 0).all()
    sig = 1.0 / (1.0 + np.exp(-delta))
    np.testing.assert_allclose(w[:, 0], sig, rtol=1e-14)
    np.testing.assert_allclose(w[:, 1], 1 - sig, rtol=1e-12, atol=1e-15)


def test_weights_match_torch_softmax():
    rng = np.random.default_rng(10)
    L = rng.standard_normal((64, 16)) * 4
    full = torch.softmax(torch.from_numpy(L), dim=1).numpy()
    ids = oracle.select(L, GATE_TOPK, 1)
    w = oracle.gate_weights(L, ids, GATE_TOPK, 0)
    np.testing.assert_allclose(w[:, 0], full[np.arange(64), ids[:, 0]], rtol=1e-14)
    # normalized top-3: softmax over the three chosen values
    ids3 = oracle.select(L, GATE_TOPK, 3)
    w3 = oracle.gate_weights(L, ids3, GATE_TOPK, 1)
    sub = torch.softmax(torch.from_numpy(L[np.arange(64)[:, None], ids3]), dim=1).numpy()
    np.testing.assert_allclose(w3, sub, rtol=1e-14)
    # kTop1 with 4 groups of 4: softmax inside the group
    idk = oracle.select(L, GATE_KTOP1, 4)
    wk = oracle.gate_weights(L, idk, GATE_KTOP1, 0)
    for g in range(4):
        grp = torch.softmax(torch.from_numpy(L[:, 4 * g:4 * g + 4]), dim=1).numpy()
        np.testing.assert_allclose(wk[:, g], grp[np.arange(64), idk[:, g] - 4 * g], rtol=1e-14)


def test_weight_bounds_and_shift_invariance():
    rng = np.random.default_rng(12)
    L = rng.standard_normal((200, 16)) * 2
    ids = oracle.select(L, GATE_TOPK, 1)
    w = oracle.gate_weights(L, ids, GATE_TOPK, 0)
    assert (w >= 1 / 16 - 1e-15).all() and (w <= 1).all()
    w2 = oracle.gate_weights(L + 100.0, oracle.select(L + 100.0, GATE_TOPK, 1), GATE_TOPK, 0)
    np.testing.assert_allclose(w, w2, rtol=1e-12)
    idk = oracle.select(L, GATE_KTOP1, 4)
    wk = oracle.gate_weights(L, idk, GATE_KTOP1, 0)
    assert (wk >= 1 / 4 - 1e-15).all()
    ids2 = oracle.select(L, GATE_TOPK, 2)
    w2n = oracle.gate_weights(L, ids2, GATE_TOPK, 1)
    np.testing.assert_allclose(w2n.sum(axis=1), 1.0, rtol=0, atol=4e-16)
    assert (w2n[:, 0] >= w2n[:, 1]).all()


def test_hash_weights_are_one():
    w = oracle.gate_weights(None, np.zeros((5, 1), dtype=np.int32), GATE_HASH, 0)
    np.testing.assert_array_equal(w, np.ones((5, 1)))


# --------------------------------------------------------------------------- hash

def test_splitmix64_published_vector():
    g = golden("splitmix64.json")
    got = [oracle.splitmix64_output(g["seed"], n) for n in range(1, 6)]
    assert got == [int(v) for v in g["outputs"]]


def test_hash_ids_use_output_t_plus_one():
    g = golden("splitmix64.json")
    tok = np.arange(5)
    for E in (1, 7, 128):
        ids = oracle.hash_ids(tok, E, g["seed"])
        assert ids.shape == (5, 1)
        assert [int(i) for i in ids[:, 0]] == [int(v) % E for v in g["outputs"]]


def test_hash_is_roughly_uniform():
    ids = oracle.hash_ids(np.arange(20000), 16, 0)[:, 0]
    counts = np.bincount(ids, minlength=16)
    assert counts.min() > 1100 and counts.max() < 1400


# -------------------------------------------------------------------------- slots

def test_capacity_formula_at_the_five_workloads():
    assert oracle.capacity(1.0, 1, 1024, 8) == 128
    assert oracle.capacity(1.25, 2, 8192, 16) == 1280
    assert oracle.capacity(1.0, 1, 32768, 64) == 512
    assert oracle.capacity(1.25, 4, 32768, 64) == 2560
    assert oracle.capacity(2.0, 1, 65536, 128) == 1024
    assert oracle.capacity(1.0, 1, 10, 3) == 4


def test_capacity_hand_case():
    g = golden("capacity_hand.json")
    ids = np.array(g["ids"], dtype=np.int32)
    slots, counts, demand, slot_src = oracle.assign_slots(ids, g["E"], g["C"])
    np.testing.assert_array_equal(slots, g["slots"])
    np.testing.assert_array_equal(counts, g["counts"])
    np.testing.assert_array_equal(demand, g["demand"])
    np.testing.assert_array_equal(slot_src, g["slot_src"])
    x = np.array([[s, -s] for s in range(g["S"])], dtype=np.float32)
    xe = oracle.dispatch(x, slot_src, 1)
    y, _ = oracle.combine(xe, ids, slots, np.ones((g["S"], 1)), "f32")
    np.testing.assert_array_equal(y, np.array(g["y"], dtype=np.float32))


def test_rank_major_hand_case():
    g = golden("rank_major.json")
    ids = oracle.select(np.array(g["logits"]), GATE_TOPK, 2)
    np.testing.assert_array_equal(ids, g["ids"])
    slots, counts, demand, slot_src = oracle.assign_slots(ids, g["E"], g["C"])
    np.testing.assert_array_equal(slots, g["slots"])
    np.testing.assert_array_equal(slot_src, g["slot_src"])
    assert not np.array_equal(slots, np.array(g["token_major_slots_would_be"]))


def _onehot_positions(ids, E):
    # the textbook "position in expert": cumulative sum of one-hot rows over the
    # rank-major concatenation of choices, minus one
    S, k = ids.shape
    flat = ids.T.reshape(-1)                        # rank-major order
    onehot = np.zeros((flat.size, E), dtype=np.int64)
    onehot[np.arange(flat.size), flat] = 1
    pos = (np.cumsum(onehot, axis=0) - 1)[np.arange(flat.size), flat]
    return pos.reshape(k, S).T


def test_slots_match_onehot_cumsum():
    rng = np.random.default_rng(13)
    for (S, E, k, C) in [(300, 8, 1, 30), (257, 5, 2, 90), (100, 16, 4, 7), (64, 3, 3, 1)]:
        ids = rng.integers(0, E, size=(S, k)).astype(np.int32)
        slots, counts, demand, _ = oracle.assign_slots(ids, E, C)
        pos = _onehot_positions(ids, E)
        np.testing.assert_array_equal(slots, np.where(pos < C, pos, -1))
        np.testing.assert_array_equal(demand, np.bincount(ids.reshape(-1), minlength=E))
        np.testing.assert_array_equal(counts, np.minimum(demand, C))


def test_no_drop_slot_src_is_stable_counting_sort():
    rng = np.random.default_rng(14)
    S, E, k = 120, 6, 2
    ids = rng.integers(0, E, size=(S, k)).astype(np.int32)
    C = S * k
    slots, counts, demand, slot_src = oracle.assign_slots(ids, E, C)
    assert (slots >= 0).all()
    flat = ids.T.reshape(-1)                                   # rank-major
    src_rank_major = (np.arange(S)[None, :] * k + np.arange(k)[:, None]).reshape(-1)
    order = np.argsort(flat, kind="stable")
    expect = src_rank_major[order]
    got = np.concatenate([slot_src[e, :counts[e]] for e in range(E)])
    np.testing.assert_array_equal(got, expect)


def test_special_cases():
    # E = 1: the first C tokens are kept
    ids = np.zeros((10, 1), dtype=np.int32)
    slots, counts, demand, slot_src = oracle.assign_slots(ids, 1, 4)
    np.testing.assert_array_equal(slots[:, 0], [0, 1, 2, 3] + [-1] * 6)
    np.testing.assert_array_equal(slot_src, [[0, 1, 2, 3]])
    assert counts[0] == 4 and demand[0] == 10
    # all logits equal -> expert 0 (top-1) / experts 0, 1 (top-2)
    L = np.zeros((9, 5))
    np.testing.assert_array_equal(oracle.select(L, GATE_TOPK, 1)[:, 0], 0)
    np.testing.assert_array_equal(oracle.select(L, GATE_TOPK, 2), [[0, 1]] * 9)
    # C = 1
    slots, counts, _, slot_src = oracle.assign_slots(np.array([[2], [2], [0]], np.int32), 3, 1)
    np.testing.assert_array_equal(slots[:, 0], [0, -1, 0])
    np.testing.assert_array_equal(slot_src, [[2], [-1], [0]])
    # hash with E = 1
    np.testing.assert_array_equal(oracle.hash_ids(np.arange(7), 1, 0), np.zeros((7, 1)))


ids_strategy = st.tuples(st.integers(1, 40), st.integers(1, 6), st.integers(1, 3), st.integers(1, 25)).flatmap(
    lambda t: st.tuples(st.just(t), hnp.arrays(np.int32, (t[0], t[2]), elements=st.integers(0, t[1] - 1))))


@settings(max_examples=150, deadline=None)
@given(ids_strategy)
def test_slot_invariants(case):
    (S, E, k, C), ids = case
    slots, counts, demand, slot_src = oracle.assign_slots(ids, E, C)
    assert (counts <= C).all()
    assert demand.sum() == S * k
    np.testing.assert_array_equal(counts, np.minimum(demand, C))
    for e in range(E):
        assert (slot_src[e, :counts[e]] >= 0).all()
        assert (slot_src[e, counts[e]:] == -1).all()
        srcs = slot_src[e, :counts[e]]
        order = [(s % k, s // k) for s in srcs]          # (rank, token)
        assert order == sorted(order)
    kept = 0
    for s in range(S):
        for r in range(k):
            if slots[s, r] >= 0:
                kept += 1
                assert slot_src[ids[s, r], slots[s, r]] == s * k + r
    assert kept == counts.sum()
    # drops are exactly the assignments after the first C of an expert
    pos = _onehot_positions(ids, E)
    np.testing.assert_array_equal(slots == -1, pos >= C)


# ------------------------------------------------------------ dispatch / combine

def _random_route(rng, S, E, k, C, kind=GATE_TOPK):
    L = rng.standard_normal((S, E))
    ids = oracle.select(L, kind, k)
    slots, counts, demand, slot_src = oracle.assign_slots(ids, E, C)
    return L, ids, slots, slot_src


def test_dispatch_is_a_bit_copy_and_zero_fills():
    rng = np.random.default_rng(15)
    S, d, E, k, C = 50, 8, 4, 2, 20
    _, ids, slots, slot_src = _random_route(rng, S, E, k, C)
    x = rng.integers(0, 1 << 16, size=(S, d)).astype(np.uint16)      # any bit patterns
    xe = oracle.dispatch(x, slot_src, k)
    for e in range(E):
        for c in range(C):
            src = slot_src[e, c]
            if src < 0:
                assert (xe[e, c] == 0).all()
            else:
                np.testing.assert_array_equal(xe[e, c], x[src // k])


def test_combine_of_dispatch_unit_weights_counts_kept_choices():
    rng = np.random.default_rng(16)
    S, d, E, k, C = 80, 6, 5, 2, 20
    _, ids, slots, slot_src = _random_route(rng, S, E, k, C)
    x = rng.integers(-8, 8, size=(S, d)).astype(np.float32)
    xe = oracle.dispatch(x, slot_src, k)
    y, _ = oracle.combine(xe, ids, slots, np.ones((S, k)), "f32")
    nkept = (slots >= 0).sum(axis=1)
    np.testing.assert_array_equal(y, x * nkept[:, None])
    assert (nkept < k).any()          # the case exercises drops


def test_adjoint_identities_exact():
    rng = np.random.default_rng(17)
    S, d, E, k, C = 40, 5, 4, 2, 12
    _, ids, slots, slot_src = _random_route(rng, S, E, k, C)
    x = rng.integers(-5, 6, size=(S, d)).astype(np.float32)
    Z = rng.integers(-5, 6, size=(E, C, d)).astype(np.float32)
    lhs = (oracle.dispatch(x, slot_src, k).astype(np.float64) * Z).sum()
    dx, _ = oracle.dispatch_bwd(Z, ids, slots, "f32")
    rhs = (x.astype(np.float64) * dx).sum()
    assert lhs == rhs
    Y = rng.integers(-5, 6, size=(E, C, d)).astype(np.float32)
    V = rng.integers(-5, 6, size=(S, d)).astype(np.float32)
    w = rng.integers(-3, 4, size=(S, k)).astype(np.float64)
    y, _ = oracle.combine(Y, ids, slots, w, "f32")
    lhs = (y.astype(np.float64) * V).sum()
    dye, _, dw, _ = oracle.combine_bwd(V, Y, slot_src, w, k, "f32")
    rhs = (Y.astype(np.float64) * dye).sum()
    assert lhs == rhs
    # dw is the exact derivative of <combine(Y; w), V> with respect to w
    for s in range(S):
        for r in range(k):
            w2 = w.copy()
            w2[s, r] += 1.0
            y2, _ = oracle.combine(Y, ids, slots, w2, "f32")
            diff = ((y2.astype(np.float64) - y.astype(np.float64)) * V).sum()
            assert diff == dw[s, r]


def test_combine_bf16_rounds_once():
    # three bf16 terms 1, 2^-8, 2^-40: the exact sum lies just above the bf16 tie
    # 1 + 2^-8 and rounds up; rounding any partial sum first (to bf16 or to fp32)
    # lands on the tie and goes down to 1.0
    ye = oracle.f64_to_bf16(np.array([1.0, 2.0 ** -8, 2.0 ** -40])).reshape(3, 1, 1)
    assert (oracle.bf16_to_f64(ye).reshape(-1) == [1.0, 2.0 ** -8, 2.0 ** -40]).all()
    ids = np.array([[0, 1, 2]], dtype=np.int32)
    slots = np.array([[0, 0, 0]], dtype=np.int32)
    y, mag = oracle.combine(ye, ids, slots, np.ones((1, 3)), "bf16")
    assert int(y[0, 0]) == 0x3F81
    np.testing.assert_array_equal(mag, [[1.0 + 2.0 ** -8 + 2.0 ** -40]])


def test_combine_bwd_dropped_gets_zero_dw_and_empty_rows_zero():
    rng = np.random.default_rng(18)
    S, d, E, k, C = 30, 4, 3, 2, 6
    _, ids, slots, slot_src = _random_route(rng, S, E, k, C)
    dy = rng.standard_normal((S, d)).astype(np.float32)
    ye = rng.standard_normal((E, C, d)).astype(np.float32)
    w = rng.random((S, k))
    dye, _, dw, _ = oracle.combine_bwd(dy, ye, slot_src, w, k, "f32")
    assert (dw[slots < 0] == 0).all()
    assert (slots < 0).any()
    for e in range(E):
        for c in range(C):
            if slot_src[e, c] < 0:
                assert (dye[e, c] == 0).all()
            else:
                s, r = divmod(int(slot_src[e, c]), k)
                np.testing.assert_array_equal(dye[e, c], (w[s, r] * dy[s].astype(np.float64)).astype(np.float32))
                assert math.isclose(dw[s, r], math.fsum(float(a) * float(b) for a, b in zip(dy[s], ye[e, c])),
                                    rel_tol=1e-13, abs_tol=1e-13)


def test_gate_end_to_end_small():
    rng = np.random.default_rng(19)
    S, d, E = 64, 16, 8
    x = rng.standard_normal((S, d)).astype(np.float32)
    wg = (rng.standard_normal((d, E)) / 4).astype(np.float32)
    out = oracle.gate(GATE_TOPK, 2, E, 10, normalize=1, dtype="f32", x=x, wg=wg)
    ids = out["ids"]
    L = out["logits"]
    for s in range(S):
        assert L[s, ids[s, 0]] >= L[s, ids[s, 1]]
        others = [e for e in range(E) if e not in ids[s]]
        assert all(L[s, ids[s, 1]] >= L[s, e] for e in others)
    np.testing.assert_allclose(out["weights"].sum(axis=1), 1.0, atol=1e-15)
    assert out["counts"].sum() == (out["slots"] >= 0).sum()
