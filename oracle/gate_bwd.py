"""Oracle for the backward pass of the gate (step 1 of Algorithm 1) and for the
load-balancing loss.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper trains the MoE layer end to end (Sec. 2, Algorithm 1), so the gate of
Eq. 1 also needs its gradient.  With the loss reaching the gate only through the
gate weights w[s, r] (the combine of step 6 hands back dw = dLoss/dw), and the
selection held fixed (TopK and kTop1 are piecewise constant in the logits):

* gate_dlogits -- dL[s, e] = sum_r dw[s, r] * dw[s, r]/dL[s, e], i.e. the
                  Jacobian of the softmax of Eq. 1 (or of its readings R1 / R8)
                  applied to dw;
* gate_input_grads -- the logits are L = x . W + b (Eq. 1), so
                  dW = x^T . dL, db = sum over tokens of dL, dx = dL . W^T;
* aux_loss     -- reading R16: the load-balancing loss of the Switch gate that
                  the paper's gate list cites (Sec. 3.1), coef * E * sum_e f_e P_e,
                  with f_e the share of tokens whose first choice is e and P_e the
                  mean full-softmax probability of e; f is a count and carries no
                  gradient.

HASH gates have no logits and no gradient.  Arithmetic is fp64 on exactly
decoded inputs; each function also returns the magnitude (sum of absolute
values) of the terms of every output element, which bounds the rounding error of
any evaluation order.
"""

import numpy as np

from .bf16 import decode, encode
from .gate import GATE_HTOPK, GATE_KTOP1, GATE_TOPK


def _softmax_rows(L):
    m = L.max(axis=1, keepdims=True)
    e = np.exp(L - m)
    return e / e.sum(axis=1, keepdims=True)


def gate_dlogits(L, ids, dw, kind, normalize, temperature=0.0):
    """Gradient of sum_r dw[s, r] * w[s, r] with respect to the logits L[s, e].

    L: [S, E] logits (float32 or float64), ids: [S, k] chosen experts, dw: [S, k].
    The weights w are those of Eq. 1 and its readings:

    TOPK, normalize=1 : w = softmax over the k selected logits; only selected
                        logits receive a gradient,
                        dL[id_r] = w_r * (dw_r - sum_r' w_r' dw_r').
    TOPK, normalize=0 : w_r = p[id_r] with p the softmax over all E logits,
                        dL[e] = sum_r dw_r * w_r * ([e == id_r] - p[e]).
    KTOP1             : per group g, w_g = softmax of the group read at id_g,
                        dL[e in g] = dw_g * w_g * ([e == id_g] - p_g[e]).
    HTOPK             : as TOPK for the chosen experts (R19).
    With temperature > 0, L are Dense-To-Sparse logits (L_raw + g) / tau (R20)
    and the gradient returned is the one with respect to L_raw: dL / tau.

    Returns (dL, M) as float64 [S, E]; M sums the absolute values of the terms.
    """
    if temperature:
        dL, M = gate_dlogits(L, ids, dw, kind, normalize)
        t = float(np.float32(temperature))
        return dL / t, M / t
    if kind == GATE_HTOPK:
        kind = GATE_TOPK
    L = np.asarray(L, dtype=np.float64)
    ids = np.asarray(ids)
    dw = np.asarray(dw, dtype=np.float64)
    S, E = L.shape
    k = ids.shape[1]
    dL = np.zeros((S, E), dtype=np.float64)
    M = np.zeros((S, E), dtype=np.float64)
    rows = np.arange(S)
    if kind == GATE_TOPK and normalize:
        chosen = L[rows[:, None], ids]
        m = chosen.max(axis=1, keepdims=True)
        num = np.exp(chosen - m)
        w = num / num.sum(axis=1, keepdims=True)          # [S, k]
        wdw = w * dw
        inner = wdw.sum(axis=1)                          # sum_r' w_r' dw_r'
        inner_mag = np.abs(wdw).sum(axis=1)
        for r in range(k):
            dL[rows, ids[:, r]] = w[:, r] * (dw[:, r] - inner)
            M[rows, ids[:, r]] = np.abs(w[:, r] * dw[:, r]) + w[:, r] * inner_mag
        return dL, M
    if kind == GATE_TOPK:
        p = _softmax_rows(L)
        w = p[rows[:, None], ids]                        # [S, k]
        g = (dw * w).sum(axis=1)                         # sum_r dw_r w_r
        g_mag = np.abs(dw * w).sum(axis=1)
        dL = -p * g[:, None]
        M = p * g_mag[:, None]
        for r in range(k):
            dL[rows, ids[:, r]] += dw[:, r] * w[:, r]
            M[rows, ids[:, r]] += np.abs(dw[:, r] * w[:, r])
        return dL, M
    if kind == GATE_KTOP1:
        G = E // k
        for grp in range(k):
            lo, hi = grp * G, (grp + 1) * G
            p = _softmax_rows(L[:, lo:hi])
            wg = p[rows, ids[:, grp] - lo]
            scale = dw[:, grp] * wg
            dL[:, lo:hi] = -p * scale[:, None]
            M[:, lo:hi] = p * np.abs(scale)[:, None]
            dL[rows, ids[:, grp]] += scale
            M[rows, ids[:, grp]] += np.abs(scale)
        return dL, M
    raise ValueError("the gate gradient exists for TOPK and KTOP1 only")


def aux_loss(L, ids, coef):
    """Load-balancing loss (reading R16) and its gradient with respect to L.

    loss = coef * E * sum_e f_e * P_e, f_e = (1/S) #{s : ids[s, 0] == e},
    P_e = (1/S) sum_s p[s, e], p the softmax over all E logits.  With f held
    constant, dloss/dL[s, e] = coef * E / S * p[s, e] * (f_e - sum_e' f_e' p[s, e']).
    Returns (loss, dL_aux [S, E], M [S, E], f [E], P [E]).
    """
    L = np.asarray(L, dtype=np.float64)
    ids = np.asarray(ids)
    S, E = L.shape
    p = _softmax_rows(L)
    f = np.bincount(ids[:, 0], minlength=E).astype(np.float64) / S
    P = p.mean(axis=0)
    loss = coef * E * float((f * P).sum())
    c = coef * E / S
    fp = p @ f                                            # sum_e' f_e' p[s, e']
    dL = c * p * (f[None, :] - fp[:, None])
    M = abs(c) * p * (f[None, :] + fp[:, None])
    return loss, dL, M, f, P


def gate_input_grads(x, wg, dL, dtype, dx_in=None):
    """Backward of L = x . W + b (Eq. 1) for a given dL [S, E].

    dW[j, e] = sum_s x[s, j] * dL[s, e]       (float64, [d, E])
    db[e]    = sum_s dL[s, e]                 (float64, [E])
    dx[s, j] = dx_in[s, j] + sum_e dL[s, e] * W[j, e], rounded once to ``dtype``
               (dx_in absent: 0).
    Returns a dict with dwg, dwg_mag, dbias, dbias_mag, dx (storage dtype) and
    dx_mag.  The matrix products are the library steps.
    """
    x64 = decode(x, dtype)
    w64 = decode(wg, dtype)
    dL = np.asarray(dL, dtype=np.float64)
    out = {
        "dwg": x64.T @ dL,
        "dwg_mag": np.abs(x64).T @ np.abs(dL),
        "dbias": dL.sum(axis=0),
        "dbias_mag": np.abs(dL).sum(axis=0),
    }
    dx = dL @ w64.T
    dx_mag = np.abs(dL) @ np.abs(w64).T
    if dx_in is not None:
        d_in = decode(dx_in, dtype)
        dx = dx + d_in
        dx_mag = dx_mag + np.abs(d_in)
    out["dx"] = encode(dx, dtype)
    out["dx_mag"] = dx_mag
    return out
