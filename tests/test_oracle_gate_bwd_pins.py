"""Pins of the gate-backward oracle (oracle/gate_bwd.py) against what the
mathematics fixes: central finite differences of the forward weights (which are
pinned on their own), torch's fp64 autograd, closed forms, invariants and brute
force on small integers.  CPU only."""

import math

import numpy as np
import pytest
import torch

import oracle

KINDS = [(oracle.GATE_TOPK, 1, 2), (oracle.GATE_TOPK, 0, 1), (oracle.GATE_TOPK, 0, 3), (oracle.GATE_TOPK, 1, 3),
         (oracle.GATE_KTOP1, 0, 2), (oracle.GATE_KTOP1, 0, 4)]


def _case(S, E, k, kind, seed, spread=3.0):
    rng = np.random.default_rng(seed)
    L = rng.standard_normal((S, E)) * spread
    ids = oracle.select(L, kind, k)
    dw = rng.standard_normal((S, k))
    return L, ids, dw


def _min_selection_gap(L, ids, kind):
    """Smallest logit gap between a chosen expert and one it beat."""
    S, E = L.shape
    k = ids.shape[1]
    gap = np.inf
    for s in range(S):
        if kind == oracle.GATE_TOPK:
            others = [e for e in range(E) if e not in ids[s]]
            if others:
                gap = min(gap, L[s, ids[s]].min() - L[s, others].max())
        else:
            G = E // k
            for g in range(k):
                others = [e for e in range(g * G, (g + 1) * G) if e != ids[s, g]]
                if others:
                    gap = min(gap, L[s, ids[s, g]] - L[s, others].max())
    return gap


@pytest.mark.parametrize("kind,normalize,k", KINDS)
def test_dlogits_central_differences(kind, normalize, k):
    S, E = 5, 8
    L, ids, dw = _case(S, E, k, kind, seed=10 * k + kind + normalize)
    assert _min_selection_gap(L, ids, kind) > 1e-3  # the perturbation keeps the selection
    dL, _ = oracle.gate_dlogits(L, ids, dw, kind, normalize)
    h = 1e-6
    fd = np.zeros_like(L)
    for s in range(S):
        for e in range(E):
            Lp, Lm = L.copy(), L.copy()
            Lp[s, e] += h
            Lm[s, e] -= h
            fp = (dw * oracle.gate_weights(Lp, ids, kind, normalize)).sum()
            fm = (dw * oracle.gate_weights(Lm, ids, kind, normalize)).sum()
            fd[s, e] = (fp - fm) / (2 * h)
    np.testing.assert_allclose(dL, fd, atol=1e-8, rtol=0)


def _torch_weights(Lt, ids, kind, normalize):
    idx = torch.from_numpy(ids.astype(np.int64))
    if kind == oracle.GATE_TOPK and normalize:
        return torch.softmax(Lt.gather(1, idx), dim=1)
    if kind == oracle.GATE_TOPK:
        return torch.softmax(Lt, dim=1).gather(1, idx)
    S, E = Lt.shape
    k = ids.shape[1]
    G = E // k
    cols = [torch.softmax(Lt[:, g * G:(g + 1) * G], dim=1).gather(1, idx[:, g:g + 1] - g * G) for g in range(k)]
    return torch.cat(cols, dim=1)


@pytest.mark.parametrize("kind,normalize,k", KINDS)
def test_dlogits_torch_autograd(kind, normalize, k):
    S, E = 40, 16
    L, ids, dw = _case(S, E, k, kind, seed=77 + k + 3 * normalize)
    Lt = torch.tensor(L, dtype=torch.float64, requires_grad=True)
    (torch.tensor(dw) * _torch_weights(Lt, ids, kind, normalize)).sum().backward()
    dL, M = oracle.gate_dlogits(L, ids, dw, kind, normalize)
    np.testing.assert_allclose(dL, Lt.grad.numpy(), atol=1e-13, rtol=1e-12)
    assert (np.abs(dL) <= M * (1 + 1e-12) + 1e-300).all()


def test_dlogits_closed_forms():
    # top-2 renormalised over logits [0, 1]: w = (sigma(1), 1 - sigma(1)); with
    # dw = (1, 0) the chosen logits get +-sigma'(1) = +-sigma(1)(1 - sigma(1))
    L = np.array([[0.0, 1.0]])
    ids = oracle.select(L, oracle.GATE_TOPK, 2)
    assert ids.tolist() == [[1, 0]]
    dL, _ = oracle.gate_dlogits(L, ids, np.array([[1.0, 0.0]]), oracle.GATE_TOPK, 1)
    sp = 0.19661193324148185  # sigma(1) * (1 - sigma(1))
    np.testing.assert_allclose(dL, [[-sp, sp]], rtol=1e-15)
    # Switch (k = 1, full softmax): dL[e] = dw * w * ([e == id] - p[e]); logits [2, 5, 5, 1]
    L = np.array([[2.0, 5.0, 5.0, 1.0]])
    ids = oracle.select(L, oracle.GATE_TOPK, 1)
    assert ids.tolist() == [[1]]
    den = math.exp(-3) + 2 + math.exp(-4)
    p = np.array([math.exp(-3), 1, 1, math.exp(-4)]) / den
    dL, _ = oracle.gate_dlogits(L, ids, np.array([[2.0]]), oracle.GATE_TOPK, 0)
    want = -2.0 * p[1] * p
    want[1] += 2.0 * p[1]
    np.testing.assert_allclose(dL[0], want, rtol=1e-14, atol=1e-16)
    # k = 1 renormalised over itself: the weight is constant 1, no gradient
    dL, _ = oracle.gate_dlogits(L, ids, np.array([[3.0]]), oracle.GATE_TOPK, 1)
    assert (dL == 0).all()


@pytest.mark.parametrize("kind,normalize,k", KINDS)
def test_dlogits_invariants(kind, normalize, k):
    S, E = 30, 12
    L, ids, dw = _case(S, E, k, kind, seed=5 + k)
    dL, _ = oracle.gate_dlogits(L, ids, dw, kind, normalize)
    # every softmax is shift-invariant, so each row (each group for kTop1) sums to 0
    if kind == oracle.GATE_KTOP1:
        G = E // k
        for g in range(k):
            np.testing.assert_allclose(dL[:, g * G:(g + 1) * G].sum(axis=1), 0, atol=1e-13)
    else:
        np.testing.assert_allclose(dL.sum(axis=1), 0, atol=1e-13)
    # adding a constant to a row changes nothing
    dL2, _ = oracle.gate_dlogits(L + 7.25, ids, dw, kind, normalize)
    np.testing.assert_allclose(dL2, dL, atol=1e-13)
    # linear in dw
    dL3, _ = oracle.gate_dlogits(L, ids, -2.5 * dw, kind, normalize)
    np.testing.assert_allclose(dL3, -2.5 * dL, atol=1e-13)
    # renormalised top-k: unselected logits get no gradient
    if kind == oracle.GATE_TOPK and normalize:
        mask = np.ones_like(dL, dtype=bool)
        mask[np.arange(S)[:, None], ids] = False
        assert (dL[mask] == 0).all()


def test_aux_loss_values_and_gradient():
    # balanced routing with uniform probabilities: f = P = 1/E, loss = coef
    S, E = 8, 4
    L = np.zeros((S, E))
    ids = np.array([[s % E] for s in range(S)])
    loss, dL, _, f, P = oracle.aux_loss(L, ids, 0.01)
    assert abs(loss - 0.01) < 1e-15
    np.testing.assert_allclose(f, 0.25)
    np.testing.assert_allclose(P, 0.25)
    np.testing.assert_allclose(dL, 0, atol=1e-18)
    # everything on expert 0 with certainty-like logits: loss -> coef * E
    L = np.full((S, E), -40.0)
    L[:, 0] = 40.0
    ids = np.zeros((S, 1), dtype=np.int32)
    loss, _, _, _, _ = oracle.aux_loss(L, ids, 0.5)
    assert abs(loss - 0.5 * E) < 1e-12
    # gradient: central differences with the counts held fixed, and autograd
    rng = np.random.default_rng(3)
    S, E = 7, 6
    L = rng.standard_normal((S, E))
    ids = oracle.select(L, oracle.GATE_TOPK, 2)
    coef = 0.3
    _, dL, M, f, _ = oracle.aux_loss(L, ids, coef)

    def loss_at(Lx):
        p = np.exp(Lx - Lx.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        return coef * E * float((f * p.mean(axis=0)).sum())
    h = 1e-6
    fd = np.zeros_like(L)
    for s in range(S):
        for e in range(E):
            Lp, Lm = L.copy(), L.copy()
            Lp[s, e] += h
            Lm[s, e] -= h
            fd[s, e] = (loss_at(Lp) - loss_at(Lm)) / (2 * h)
    np.testing.assert_allclose(dL, fd, atol=1e-9)
    Lt = torch.tensor(L, requires_grad=True)
    (coef * E * (torch.tensor(f) * torch.softmax(Lt, dim=1).mean(dim=0)).sum()).backward()
    np.testing.assert_allclose(dL, Lt.grad.numpy(), atol=1e-15, rtol=1e-12)
    np.testing.assert_allclose(dL.sum(axis=1), 0, atol=1e-15)
    assert (np.abs(dL) <= M + 1e-300).all()
    # f counts first choices only
    assert abs(f.sum() - 1) < 1e-15
    np.testing.assert_allclose(f * S, np.bincount(ids[:, 0], minlength=E))


def test_input_grads_integer_brute_force():
    rng = np.random.default_rng(11)
    S, d, E = 5, 4, 3
    x = rng.integers(-3, 4, (S, d)).astype(np.float32)
    w = rng.integers(-3, 4, (d, E)).astype(np.float32)
    dL = rng.integers(-5, 6, (S, E)).astype(np.float64)
    dx_in = rng.integers(-9, 10, (S, d)).astype(np.float32)
    out = oracle.gate_input_grads(x, w, dL, "f32", dx_in=dx_in)
    for j in range(d):
        for e in range(E):
            assert out["dwg"][j, e] == sum(float(x[s, j]) * dL[s, e] for s in range(S))
    for e in range(E):
        assert out["dbias"][e] == sum(dL[s, e] for s in range(S))
    for s in range(S):
        for j in range(d):
            assert out["dx"][s, j] == np.float32(dx_in[s, j] + sum(dL[s, e] * float(w[j, e]) for e in range(E)))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_input_grads_torch_autograd(dtype):
    rng = np.random.default_rng(12)
    S, d, E = 33, 20, 8
    x = oracle.encode(rng.standard_normal((S, d)), dtype)
    w = oracle.encode(rng.standard_normal((d, E)) / 4, dtype)
    b = rng.standard_normal(E)
    dL = rng.standard_normal((S, E))
    xt = torch.tensor(oracle.decode(x, dtype), requires_grad=True)
    wt = torch.tensor(oracle.decode(w, dtype), requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    ((xt @ wt + bt) * torch.tensor(dL)).sum().backward()
    out = oracle.gate_input_grads(x, w, dL, dtype)
    np.testing.assert_allclose(out["dwg"], wt.grad.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(out["dbias"], bt.grad.numpy(), rtol=1e-12, atol=1e-13)
    # dx is rounded once to the storage dtype
    assert np.array_equal(out["dx"], oracle.encode(xt.grad.numpy(), dtype))
    assert (out["dwg_mag"] >= np.abs(out["dwg"])).all() and (out["dx_mag"] >= np.abs(xt.grad.numpy()) - 1e-12).all()
