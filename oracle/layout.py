"""Oracle for steps 2 and 6 of Algorithm 1 and their backward passes.

TEST INFRASTRUCTURE ONLY (see the package docstring).

* dispatch     -- Layout_Transform (Algorithm 1, step 2; Sec. 3.2, layout
                  transform): every token is copied into the
                  contiguous buffer of each expert it was kept for, here a fixed
                  [E, C, d] buffer whose empty rows are zero (reading R6).
* combine      -- Reverse_Layout_Transform (step 6) together with the
                  gate weighting of step 4 / Eq. 1's second line:
                  y_s = sum over kept choices r of w[s,r] * ye[ids[s,r], slots[s,r]]
                  (the weight is applied here rather than inside the expert,
                  which is the same sum; reading R7).
* dispatch_bwd -- adjoint of dispatch: each token sums the gradient rows of its
                  kept slots.
* combine_bwd  -- adjoint of combine with respect to ye (dye) and to the gate
                  weights (dw).

Sums are formed in fp64 on exactly decoded values and rounded once to the
storage dtype.  Each function also returns the magnitude of the terms that form
every output element (sum of absolute values), which bounds the rounding error
of any summation order.
"""

import numpy as np

from .bf16 import decode, encode


def dispatch(x, slot_src, k):
    """xe[e, c, :] = x[slot_src[e, c] // k, :], or zeros where slot_src is -1.

    A bit copy in the storage dtype of x ([S, d] float32 or bf16 bits).
    """
    x = np.asarray(x)
    slot_src = np.asarray(slot_src)
    E, C = slot_src.shape
    xe = np.zeros((E, C, x.shape[1]), dtype=x.dtype)
    full = slot_src >= 0
    xe[full] = x[slot_src[full] // k]
    return xe


def combine(ye, ids, slots, weights, dtype, with_exact=False):
    """y[s] = sum_{r: slots[s,r] >= 0} weights[s,r] * ye[ids[s,r], slots[s,r]].

    A token with no kept choice gets a zero row (reading R5).  Returns
    (y in storage dtype, magnitude sum_r |w * ye| as float64), and with
    `with_exact` also the fp64 sum before its one rounding.
    """
    ye64 = decode(ye, dtype)
    ids = np.asarray(ids)
    slots = np.asarray(slots)
    w = np.asarray(weights, dtype=np.float64)
    S, k = ids.shape
    d = ye64.shape[2]
    y = np.zeros((S, d), dtype=np.float64)
    mag = np.zeros((S, d), dtype=np.float64)
    for r in range(k):
        kept = np.nonzero(slots[:, r] >= 0)[0]
        term = w[kept, r, None] * ye64[ids[kept, r], slots[kept, r]]
        y[kept] += term
        mag[kept] += np.abs(term)
    if with_exact:
        return encode(y, dtype), mag, y
    return encode(y, dtype), mag


def dispatch_bwd(dxe, ids, slots, dtype, with_exact=False):
    """dx[s] = sum_{r kept} dxe[ids[s,r], slots[s,r]]; (dx, magnitude), and with
    `with_exact` also the fp64 sum before its one rounding."""
    dxe64 = decode(dxe, dtype)
    ids = np.asarray(ids)
    slots = np.asarray(slots)
    S, k = ids.shape
    d = dxe64.shape[2]
    dx = np.zeros((S, d), dtype=np.float64)
    mag = np.zeros((S, d), dtype=np.float64)
    for r in range(k):
        kept = np.nonzero(slots[:, r] >= 0)[0]
        term = dxe64[ids[kept, r], slots[kept, r]]
        dx[kept] += term
        mag[kept] += np.abs(term)
    if with_exact:
        return encode(dx, dtype), mag, dx
    return encode(dx, dtype), mag


def combine_bwd(dy, ye, slot_src, weights, k, dtype, want_dw=True, with_exact=False):
    """Gradients of combine.

    dye[e, c] = weights[s, r] * dy[s] for (s, r) held in slot (e, c), 0 if the
    slot is empty.  dw[s, r] = <dy[s], ye[e, c]> for the slot (e, c) holding
    (s, r); 0 for dropped choices.  Returns (dye in storage dtype, dye
    magnitude, dw float64 or None, dw magnitude or None), and with
    `with_exact` also the fp64 dye before its one rounding.
    """
    dy64 = decode(dy, dtype)
    slot_src = np.asarray(slot_src)
    w = np.asarray(weights, dtype=np.float64)
    E, C = slot_src.shape
    S, d = dy64.shape
    full = slot_src >= 0
    src = slot_src[full]
    s_of, r_of = src // k, src % k
    dye64 = np.zeros((E, C, d), dtype=np.float64)
    dye64[full] = w[s_of, r_of, None] * dy64[s_of]
    dye = encode(dye64, dtype)
    dye_mag = np.abs(dye64)
    if not want_dw:
        return (dye, dye_mag, None, None, dye64) if with_exact else (dye, dye_mag, None, None)
    ye64 = decode(ye, dtype)
    dw = np.zeros((S, k), dtype=np.float64)
    dw_mag = np.zeros((S, k), dtype=np.float64)
    rows = ye64[full]                                   # [n_kept, d]
    dw[s_of, r_of] = np.einsum("nd,nd->n", dy64[s_of], rows)
    dw_mag[s_of, r_of] = np.einsum("nd,nd->n", np.abs(dy64[s_of]), np.abs(rows))
    if with_exact:
        return dye, dye_mag, dw, dw_mag, dye64
    return dye, dye_mag, dw, dw_mag
