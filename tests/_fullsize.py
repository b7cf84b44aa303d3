"""Element-by-element comparison of the layout outputs at a workload's full size
against the oracle, run in chunks so that the oracle's fp64 arrays stay small.

Each chunk of tokens (combine, dispatch backward) or of expert rows (dispatch,
combine backward) becomes a small sub-problem that holds only the rows the chunk
references; the oracle's functions run on it unchanged.  Every output element is
compared: xe bit-exact; y, dx and dye within rtol * (sum of |terms|) and, for
bf16, equal to the once-rounded exact value up to fp32-accumulation straddles;
dw within 1e-5 * (sum of |terms|), and 0 for every dropped choice.  Chunks run
on a pool of threads (numpy releases the interpreter lock in its array loops).

Needs no GPU: the GPU outputs come in as host arrays.
"""

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
from _parity import RTOL, assert_close, assert_equal, check_rounded_once, decode, kept_terms


def _threads():
    try:
        n = len(os.sched_getaffinity(0))
    except OSError:
        n = os.cpu_count() or 1
    return max(1, min(8, n))


def _compact_tokens(rows, ids, slots):
    """Sub-problem of a chunk of tokens: one expert row per (token, choice) in
    an [n*k, 1, d] buffer, so that choice (s, r) sits at expert s*k+r, slot 0."""
    n, k = ids.shape
    sub = np.zeros((n * k, 1, rows.shape[2]), dtype=rows.dtype)
    kept = slots >= 0
    sub[kept.reshape(-1), 0] = rows[ids[kept], slots[kept]]
    return sub, np.arange(n * k, dtype=np.int32).reshape(n, k), np.where(kept, 0, -1).astype(np.int32)


def _tokens_chunk(dt, ye, ids, slots, w, y_gpu, dx_gpu, s0):
    """combine and dispatch backward on one chunk of tokens"""
    rt = RTOL[dt]
    st = {}
    sub, sids, sslots = _compact_tokens(ye, ids, slots)
    nt = kept_terms(slots)
    ref, mag, ex = oracle.combine(sub, sids, sslots, w.astype(np.float64), dt, with_exact=True)
    st["combine_err"] = assert_close(decode(y_gpu, dt), decode(ref, dt), mag, rt, f"combine y, tokens {s0}..")
    if dt == "bf16":
        st["combine_straddles"] = check_rounded_once(y_gpu, ex, mag, nt, f"combine y, tokens {s0}..", ref)
    ref, mag, ex = oracle.dispatch_bwd(sub, sids, sslots, dt, with_exact=True)
    st["dispatch_bwd_err"] = assert_close(decode(dx_gpu, dt), decode(ref, dt), mag, rt,
                                          f"dispatch_bwd dx, tokens {s0}..")
    one = nt[:, 0] == 1
    assert_equal(dx_gpu[one], ref[one], f"dispatch_bwd dx of tokens {s0}.. with one kept choice (a copy)")
    if dt == "bf16":
        st["dispatch_bwd_straddles"] = check_rounded_once(dx_gpu, ex, mag, nt, f"dispatch_bwd dx, tokens {s0}..", ref)
    return st


def _rows_chunk(dt, k, dy, w, src, ye_rows, dye_gpu, dw_gpu, unit_w, r0):
    """combine backward on one chunk of expert rows; returns stats and the
    (token, choice) pairs the chunk's rows hold"""
    rt = RTOL[dt]
    st = {}
    n = len(src)
    full = src >= 0
    s_of = np.where(full, src // k, 0)
    r_of = np.where(full, src % k, 0)
    src_sub = np.where(full, np.arange(n) * k + r_of, -1)[None, :]
    w_sub = np.zeros((n, k), dtype=np.float32)
    w_sub[np.arange(n), r_of] = w.reshape(-1)[np.where(full, src, 0)]
    dye_ref, dye_mag, dw_ref, dw_mag, dye_ex = oracle.combine_bwd(dy[s_of], ye_rows[None], src_sub, w_sub, k, dt,
                                                                  with_exact=True)
    st["combine_bwd_dye_err"] = assert_close(decode(dye_gpu, dt), decode(dye_ref[0], dt), dye_mag[0], rt,
                                             f"combine_bwd dye, rows {r0}..")
    if dt == "bf16":
        st["combine_bwd_dye_straddles"] = check_rounded_once(dye_gpu, dye_ex[0], dye_mag[0], 1,
                                                             f"combine_bwd dye, rows {r0}..", dye_ref[0])
    if unit_w:  # one term with weight 1: the scaled row is the token's own row
        assert_equal(dye_gpu[full], dy[s_of[full]], f"combine_bwd dye, rows {r0}.. (unit weights: a copy)")
    i = np.nonzero(full)[0]
    st["combine_bwd_dw_err"] = assert_close(dw_gpu[s_of[i], r_of[i]], dw_ref[i, r_of[i]], dw_mag[i, r_of[i]],
                                            RTOL["f32"], f"combine_bwd dw, rows {r0}..")
    return st, s_of[i], r_of[i]


def _merge(total, st):
    for key, v in st.items():
        total[key] = (total.get(key, 0) + v) if key.endswith("straddles") else max(total.get(key, 0.0), v)


def check_layout_full(dt, x, ye, dy, ids, slots, weights, slot_src, k, outs, chunk_tokens=2048, chunk_rows=4096):
    """Compare the GPU outputs `outs` (host arrays: xe = dispatch(x), y =
    combine(ye), dx = dispatch_bwd(ye), dye and dw = combine_bwd(dy, ye)) with
    the oracle.  Returns stats."""
    E, C = slot_src.shape
    S, d = x.shape
    w = np.asarray(weights, dtype=np.float32)
    total = {}
    with ThreadPoolExecutor(max_workers=_threads()) as pool:
        # dispatch: every expert row bit-exact
        ce = max(1, chunk_rows // max(C, 1))

        def disp(e0):
            assert_equal(outs["xe"][e0:e0 + ce], oracle.dispatch(x, slot_src[e0:e0 + ce], k),
                         f"dispatch xe, experts {e0}..")
        for f in [pool.submit(disp, e0) for e0 in range(0, E, ce)]:
            f.result()

        # combine and dispatch backward, by chunks of tokens
        futs = [pool.submit(_tokens_chunk, dt, ye, ids[s0:s0 + chunk_tokens], slots[s0:s0 + chunk_tokens],
                            w[s0:s0 + chunk_tokens], outs["y"][s0:s0 + chunk_tokens], outs["dx"][s0:s0 + chunk_tokens],
                            s0) for s0 in range(0, S, chunk_tokens)]
        for f in futs:
            _merge(total, f.result())

        # combine backward, by chunks of expert rows
        src_all = slot_src.reshape(-1)
        ye_flat = ye.reshape(E * C, d)
        dye_flat = outs["dye"].reshape(E * C, d)
        dw_gpu = np.asarray(outs["dw"], dtype=np.float32)
        unit_w = bool((w == 1.0).all())
        futs = [pool.submit(_rows_chunk, dt, k, dy, w, src_all[r0:r0 + chunk_rows], ye_flat[r0:r0 + chunk_rows],
                            dye_flat[r0:r0 + chunk_rows], dw_gpu, unit_w, r0) for r0 in range(0, E * C, chunk_rows)]
        covered = np.zeros((S, k), dtype=bool)
        for f in futs:
            st, s_i, r_i = f.result()
            _merge(total, st)
            assert not covered[s_i, r_i].any(), "a choice held by two slots"
            covered[s_i, r_i] = True
    kept = slots >= 0
    assert_equal(covered, kept, "choices covered by the expert rows")
    assert (dw_gpu[~kept] == 0).all(), "dw of a dropped choice is not 0"
    return total
