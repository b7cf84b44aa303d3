"""The GPU parity checkers must accept what the kernels' arithmetic produces and
reject plausible kernel mistakes.  Runs on the CPU: the "GPU" outputs are
emulated here in fp32 the way the kernels form them (fp32 products and sums,
one rounding to bf16), and each case plants one mistake in them."""

import numpy as np
import pytest

import oracle
from paper_2203_14685_amd import workloads as wl

from _fullsize import check_layout_full
from _parity import check_rounded_once, decode


def _round_f32(v):
    return np.asarray(v, dtype=np.float64).astype(np.float32)


def _emulate(dt, x, ye_s, dy, ids, slots, w, slot_src, k, partial_bf16=False, weight_bf16=False):
    """Outputs of dispatch(x), combine(ye), dispatch_bwd(ye) and
    combine_bwd(dy, ye) formed like the kernels: fp32 fused multiply-adds in
    choice order (the product of an fp32 weight and a bf16
    value is exact in fp64, so fp64 then one fp32 rounding is the fma), one
    rounding to the storage dtype.  The two flags plant mistakes: rounding each
    partial sum to bf16, or rounding the weight to bf16 first."""
    E, C = slot_src.shape
    S, d = x.shape
    xe = oracle.dispatch(x, slot_src, k)
    ye = decode(ye_s, dt)
    enc = (lambda a: oracle.encode(a, dt))
    w = np.asarray(w, dtype=np.float32)
    if weight_bf16:
        w = decode(oracle.encode(w.astype(np.float64), "bf16"), "bf16").astype(np.float32)
    y = np.zeros((S, d), np.float32)
    dx = np.zeros((S, d), np.float32)
    for r in range(k):
        kept = slots[:, r] >= 0
        rows = ye[ids[kept, r], slots[kept, r]]
        y[kept] = _round_f32(w[kept, r, None].astype(np.float64) * rows + y[kept].astype(np.float64))
        dx[kept] = _round_f32(rows + dx[kept].astype(np.float64))
        if partial_bf16:
            y = decode(enc(y.astype(np.float64)), dt).astype(np.float32)
    src = slot_src.reshape(-1)
    full = src >= 0
    dy64 = decode(dy, dt)
    dye = np.zeros((E * C, d), np.float32)
    dye[full] = _round_f32(dy64[src[full] // k] * w.reshape(-1)[src[full], None].astype(np.float64))
    dw = np.zeros((S, k), np.float32)
    dw[src[full] // k, src[full] % k] = np.einsum("nd,nd->n", dy64[src[full] // k], ye.reshape(E * C, d)[full])
    return {"xe": xe, "y": enc(y.astype(np.float64)), "dx": enc(dx.astype(np.float64)),
            "dye": enc(dye.astype(np.float64)).reshape(E, C, d), "dw": dw}


def _case(dt="bf16", S=600, d=64, E=6, k=2, C=150, seed=0):
    rng = np.random.default_rng(seed)
    L = rng.standard_normal((S, E)).astype(np.float32)
    g = oracle.gate(oracle.GATE_TOPK, k, E, C, normalize=1, sel_logits=L)
    x = wl.make_rows((S, d), dt, seed + 1)
    dy = wl.make_rows((S, d), dt, seed + 2)
    ye = wl.make_rows((E, C, d), dt, seed + 3)
    return x, ye, dy, g


def test_checker_accepts_kernel_arithmetic():
    x, ye, dy, g = _case()
    k = 2
    outs = _emulate("bf16", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], k)
    st = check_layout_full("bf16", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], k, outs,
                           chunk_tokens=128, chunk_rows=100)
    assert (g["slots"] < 0).any(), "the case should drop some choices"
    assert st["combine_err"] < 2e-2 and st["combine_bwd_dw_err"] < 1e-5


def test_checker_accepts_fp32_workload():
    x, ye, dy, g = _case(dt="f32", k=1, C=80)
    outs = _emulate("f32", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], 1)
    check_layout_full("f32", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], 1, outs, chunk_tokens=100,
                      chunk_rows=64)


@pytest.mark.parametrize("plant", ["partial_bf16", "weight_bf16"])
def test_rounding_check_catches_extra_roundings(plant):
    x, ye, dy, g = _case(seed=3)
    outs = _emulate("bf16", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], 2, **{plant: True})
    with pytest.raises(AssertionError, match="once-rounded"):
        check_layout_full("bf16", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], 2, outs)


@pytest.mark.parametrize("what", ["xe", "y", "dx", "dye", "dw", "dw_dropped"])
def test_checker_catches_one_wrong_element(what):
    x, ye, dy, g = _case(seed=5)
    outs = _emulate("bf16", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], 2)
    kept = np.argwhere(g["slots"] >= 0)
    s, r = kept[len(kept) // 2]
    if what == "xe":
        e, c = g["ids"][s, r], g["slots"][s, r]
        outs["xe"][e, c, 7] ^= np.uint16(1)
    elif what in ("y", "dx"):
        outs[what][s, 5] = np.uint16(outs[what][s, 5] + 1)  # one bf16 ulp
    elif what == "dye":
        e, c = g["ids"][s, r], g["slots"][s, r]
        outs["dye"][e, c, 3] = np.uint16(outs["dye"][e, c, 3] + 1)
    elif what == "dw":
        outs["dw"][s, r] += np.float32(0.01)  # a sum of 64 products of N(0,1) values: bound ~5e-4
    else:
        s2, r2 = np.argwhere(g["slots"] < 0)[0]
        outs["dw"][s2, r2] = np.float32(1e-30)
    with pytest.raises(AssertionError):
        check_layout_full("bf16", x, ye, dy, g["ids"], g["slots"], g["weights"], g["slot_src"], 2, outs,
                          chunk_tokens=256, chunk_rows=64)


def test_rounded_once_straddle_is_accepted_both_ways():
    # 1 + 2^-8 is the midpoint of two bf16 neighbours (1 and 1 + 2^-7); an exact
    # value just above it rounds up, but an fp32 sum one ulp below the midpoint
    # would round down: either side is accepted there, nowhere else
    ex = np.array([1 + 2.0 ** -8 + 2.0 ** -30, 1.5 + 2.0 ** -30])
    mag = np.abs(ex)
    up, down = oracle.encode(ex, "bf16"), oracle.encode(ex - 2.0 ** -20, "bf16")
    assert up[0] != down[0] and up[1] == down[1]
    assert check_rounded_once(up, ex, mag, 1, "t") == 0
    assert check_rounded_once(np.array([down[0], up[1]]), ex, mag, 1, "t") == 1
    with pytest.raises(AssertionError):
        check_rounded_once(np.array([up[0], np.uint16(up[1] + 1)]), ex, mag, 1, "t")


def test_rounded_once_cancellation_widens_the_accepted_range():
    # a result of 1.5e-6 from terms of magnitude 0.75: the fp32 bound
    # (2^-24 * 0.75 per term) spans about a dozen bf16 ulps of the result
    ex = np.array([1.495e-6])
    mag = np.array([0.76])
    want = oracle.encode(ex, "bf16")
    two_below = np.array([np.uint16(want[0] - 2)])
    assert check_rounded_once(two_below, ex, mag, 2, "t") == 1
    far = np.array([np.uint16(want[0] - 40)])
    with pytest.raises(AssertionError):
        check_rounded_once(far, ex, mag, 2, "t")
