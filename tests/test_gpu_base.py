"""GPU parity of the BASE layer gate (Sec. 3.1, BASE Layer; readings R22, R23)
through the C ABI against the oracle's exact balanced assignment.

The optimal total score is unique, the optimal assignment need not be, so the
checks are: every expert gets exactly S / E tokens (bit-exact counts); the
total score of the GPU's assignment is within S * eps of the oracle's optimum
(the auction's dual bound, eps reported by the call); where that total equals
the optimum up to rounding and the scores are continuous (a unique optimum with
probability 1), the ids equal the oracle's; with integer scores the total equals
the optimum exactly (S * eps < 1).  Slots are checked against the oracle's
capacity step fed the oracle's ids when those agree, else by their defining
property (token order within each expert).  Weights: sigmoid of the score,
rtol 1e-5."""

import numpy as np
import pytest
import torch

import oracle
import paper_2203_14685_amd as hm
from paper_2203_14685_amd import workloads as wl

from _parity import RTOL, announce, assert_close, assert_equal, check_layout_ops

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hm.load()
    yield


def run_base(L=None, x=None, wg=None, bias=None, E=None, C=None, dtype="f32", max_rounds=0):
    if L is not None:
        out = hm.base_gate(E, C, logits=wl.to_device(L, "f32"), logits_in=True, max_rounds=max_rounds)
    else:
        out = hm.base_gate(E, C, x=wl.to_device(x, dtype), wg=wl.to_device(wg, dtype),
                           bias=wl.to_device(bias, "f32"), want_logits=True, max_rounds=max_rounds)
    torch.cuda.synchronize()
    info = out.pop("info")
    h = {k: wl.to_host(v) for k, v in out.items()}
    h["info"] = info
    return h


def slots_by_property(ids, slots, counts, slot_src, E, C):
    """Slots of a k = 1 routing: each expert's tokens in token order take slots
    0, 1, ... and those at C or beyond are dropped."""
    S = ids.shape[0]
    exp_slots = np.full(S, -1, dtype=np.int64)
    exp_src = np.full((E, C), -1, dtype=np.int64)
    for e in range(E):
        toks = np.nonzero(ids == e)[0]
        kept = toks[:C]
        exp_slots[kept] = np.arange(len(kept))
        exp_src[e, :len(kept)] = kept
    assert_equal(slots[:, 0], exp_slots, "slots")
    assert_equal(slot_src, exp_src, "slot_src")
    assert_equal(counts, np.minimum(np.bincount(ids, minlength=E), C), "counts")


def certify(Lsel, g, E):
    """The auction's certificate on the scores it ran on (Lsel, float64): with
    its prices p, D = sum_s max_e (L - p) + (S/E) sum_e p bounds the optimum from
    above for any p, so D - total <= S * eps proves the total within S * eps of
    the optimum; and every token is within eps of its best L - p.  Holds at any
    size.  Returns D - total."""
    S = Lsel.shape[0]
    ids = g["ids"][:, 0]
    p = g["prices"].astype(np.float64)
    eps = g["info"]["eps"]
    net = Lsel - p[None, :]
    best = net.max(axis=1)
    own = net[np.arange(S), ids]
    scale = np.abs(Lsel).max(axis=1) + np.abs(p).max()
    assert (own >= best - eps - 1e-12 * scale).all(), "a token is not within eps of its best value"
    total = float(Lsel[np.arange(S), ids].sum())
    D = float(best.sum()) + S // E * float(p.sum())
    rnd = 1e-12 * float(scale.sum() + S // E * np.abs(p).sum())
    assert total <= D + rnd, f"total {total} above the dual bound {D}"
    assert D - total <= S * eps + rnd, f"dual gap {D - total} above S * eps = {S * eps}"
    return D - total


def check_base(L64, g, E, C, tol_extra=0.0, expect_ids=True, Lsel=None):
    """L64: the scores the oracle assigns on (float64); Lsel: the scores the
    auction ran on (default).  Returns stats."""
    S = L64.shape[0]
    ids = g["ids"][:, 0]
    dual_gap = certify(L64 if Lsel is None else Lsel, g, E)
    assert ((ids >= 0) & (ids < E)).all()
    assert_equal(np.bincount(ids, minlength=E), np.full(E, S // E), "tokens per expert")
    ref_ids, opt = oracle.base_assign(L64)
    rows = np.arange(S)
    total = float(L64[rows, ids].sum())
    eps = g["info"]["eps"]
    mag = float(np.abs(L64).sum())
    rnd = 1e-12 * mag
    assert total <= opt + rnd, f"total {total} above the optimum {opt}"
    assert total >= opt - S * eps - tol_extra - rnd, f"total {total} below optimum {opt} - S*eps ({S * eps}) - {tol_extra}"
    at_opt = abs(total - opt) <= rnd
    if at_opt and expect_ids:
        assert_equal(ids, ref_ids, "ids (unique optimum)")
    if np.array_equal(ids, ref_ids):
        slots, counts, _, slot_src = oracle.assign_slots(ref_ids[:, None], E, C)
        assert_equal(g["slots"], slots, "slots")
        assert_equal(g["counts"], counts, "counts")
        assert_equal(g["slot_src"], slot_src, "slot_src")
        w_ref = oracle.base_weights(L64, ref_ids)
    else:
        slots_by_property(ids, g["slots"], g["counts"], g["slot_src"], E, C)
        w_ref = 1.0 / (1.0 + np.exp(-L64[rows, ids]))
    assert_close(g["weights"][:, 0], w_ref, np.abs(w_ref), RTOL["f32"], "weights")
    return dict(gap=opt - total, dual_gap=dual_gap, bound=S * eps, same_ids=float((ids == ref_ids).mean()),
                **g["info"])


@pytest.mark.parametrize("S,E,scale,seed", [
    (2048, 64, 1.0, 0), (1024, 8, 1.0, 1), (960, 5, 3.0, 2), (4096, 128, 0.5, 3), (64, 64, 1.0, 4),
    (512, 1, 1.0, 5), (6000, 12, 2.0, 6),
])
def test_base_given_scores(S, E, scale, seed):
    announce(f"base logits_in S={S} E={E} scale={scale}")
    L = (np.random.default_rng(seed).standard_normal((S, E)) * scale).astype(np.float32)
    g = run_base(L=L, E=E)
    st = check_base(L.astype(np.float64), g, E, S // E)
    print(f"[stats] base S={S} E={E}: {st}", flush=True)


@pytest.mark.parametrize("S,E,hi,seed", [(1024, 8, 4, 0), (768, 16, 2, 1), (300, 3, 1, 2)])
def test_base_integer_scores_reach_the_optimum(S, E, hi, seed):
    """Integer scores with many ties: S * eps < 1 forces the exact optimal total."""
    announce(f"base integer scores S={S} E={E} hi={hi}")
    L = np.random.default_rng(seed).integers(0, hi + 1, (S, E)).astype(np.float32)
    g = run_base(L=L, E=E)
    L64 = L.astype(np.float64)
    _, opt = oracle.base_assign(L64)
    ids = g["ids"][:, 0]
    assert L64[np.arange(S), ids].sum() == opt
    check_base(L64, g, E, S // E, expect_ids=False)
    g2 = run_base(L=L, E=E)
    for key in ("ids", "slots", "weights", "counts", "slot_src"):
        assert_equal(g2[key], g[key], f"{key} on a second call")


def test_base_equal_scores():
    """Every score equal: one phase; the first S / E tokens take expert 0 and so on."""
    announce("base equal scores")
    S, E = 640, 10
    L = np.full((S, E), 0.25, dtype=np.float32)
    g = run_base(L=L, E=E)
    st = check_base(L.astype(np.float64), g, E, S // E, expect_ids=False)
    assert g["info"]["phases"] == 1, st


@pytest.mark.parametrize("dtype,S,d,E,bias", [("bf16", 4096, 2048, 64, True), ("f32", 1280, 260, 10, False),
                                              ("bf16", 2048, 1024, 16, False)])
def test_base_projection(dtype, S, d, E, bias):
    """End to end from x and W: logits within tolerance of the oracle's fp64
    logits, then the assignment's total on the fp64 logits within S * eps plus
    twice the logits' error bound of the fp64 optimum."""
    announce(f"base projection {dtype} S={S} d={d} E={E}")
    w = dict(kind=0, k=1, normalize=0, dtype=dtype, S=S, d=d, E=E, cf=1.0)
    if bias:
        w.update(hot_experts=4, hot_bias=0.5)
    inp = wl.make_inputs(w, seed=E + 7)
    g = run_base(x=inp["x"], wg=inp["wg"], bias=inp["bias"], E=E, dtype=dtype)
    L64, A = oracle.logits(inp["x"], inp["wg"], dtype, inp["bias"])
    assert_close(g["logits"], L64, A, RTOL["f32"], "logits")
    delta = float((RTOL["f32"] * A).max(axis=1).sum())
    st = check_base(L64, g, E, S // E, tol_extra=2 * delta, expect_ids=False, Lsel=g["logits"].astype(np.float64))
    print(f"[stats] base projection {dtype} E={E}: {st}", flush=True)


@pytest.mark.parametrize("wid", [3, 4])
def test_base_full_size(wid):
    """At the full workload shapes (S = 32768, d = 2048, E = 64, bf16; the hot
    bias of workload 3) the assignment problem is too large for the exact
    oracle; checked instead: the logits against the oracle's, exact balance,
    the auction's optimality certificate on the logits it ran on, the total on
    the oracle's fp64 logits within the certificate's bound plus the logits'
    error, slots by their definition, weights sigma(L)."""
    w = wl.WORKLOADS[wid]
    S, d, E = w["S"], w["d"], w["E"]
    announce(f"base full size workload {wid} S={S} d={d} E={E}")
    inp = wl.make_inputs(w, seed=0)
    g = run_base(x=inp["x"], wg=inp["wg"], bias=inp["bias"], E=E, dtype=w["dtype"])
    L64, A = oracle.logits(inp["x"], inp["wg"], w["dtype"], inp["bias"])
    assert_close(g["logits"], L64, A, RTOL["f32"], "logits")
    ids = g["ids"][:, 0]
    assert_equal(np.bincount(ids, minlength=E), np.full(E, S // E), "tokens per expert")
    Lg = g["logits"].astype(np.float64)
    gap = certify(Lg, g, E)
    # the same assignment scored on the fp64 logits: the certificate carried
    # through the logits' error bound (each term differs by at most rtol * A)
    delta = float((RTOL["f32"] * A).max(axis=1).sum())
    rows = np.arange(S)
    p = g["prices"].astype(np.float64)
    D64 = float((L64 - p[None, :]).max(axis=1).sum()) + S // E * float(p.sum())
    assert D64 - float(L64[rows, ids].sum()) <= S * g["info"]["eps"] + 2 * delta + 1e-9 * float(np.abs(L64).sum())
    slots_by_property(ids, g["slots"], g["counts"], g["slot_src"], E, S // E)
    # the weight is sigma of the device's logit, which is within rtol * A of the
    # fp64 one; sigma' = sigma (1 - sigma) carries that through
    w_ref = 1.0 / (1.0 + np.exp(-L64[rows, ids]))
    assert_close(g["weights"][:, 0], w_ref, w_ref + w_ref * (1 - w_ref) * A[rows, ids], RTOL["f32"], "weights")
    print(f"[stats] base full size W{wid}: dual gap {gap:.3e} bound {S * g['info']['eps']:.3e} {g['info']}", flush=True)


def test_base_many_experts_large_batch():
    """S = 65536 tokens over E = 128 experts (c = 512), scores given, a quarter
    of the experts favoured so that the auction runs long eviction chains and
    crowded rounds: exact balance, the optimality certificate on the scores,
    slots by their definition."""
    S, E = 65536, 128
    announce(f"base many experts S={S} E={E}")
    rng = np.random.default_rng(21)
    L = rng.standard_normal((S, E)).astype(np.float32)
    L[:, : E // 4] += np.float32(0.8)
    g = run_base(L=L, E=E)
    ids = g["ids"][:, 0]
    assert_equal(np.bincount(ids, minlength=E), np.full(E, S // E), "tokens per expert")
    gap = certify(L.astype(np.float64), g, E)
    slots_by_property(ids, g["slots"], g["counts"], g["slot_src"], E, S // E)
    print(f"[stats] base S={S} E={E}: dual gap {gap:.3e} bound {S * g['info']['eps']:.3e} {g['info']}", flush=True)


def test_base_capacity_and_layout():
    """Capacity below S / E drops the later tokens of each expert; dispatch and
    combine take the routing as any k = 1 gate's."""
    announce("base capacity + layout")
    S, d, E = 1536, 256, 12
    L = np.random.default_rng(9).standard_normal((S, E)).astype(np.float32)
    C = S // E - 30
    g = run_base(L=L, E=E, C=C)
    st = check_base(L.astype(np.float64), g, E, C)
    assert (g["counts"] == C).all()
    w = dict(dtype="f32")
    x = wl.make_rows((S, d), "f32", 4)
    ref_ids, _ = oracle.base_assign(L.astype(np.float64))
    slots, _, _, slot_src = oracle.assign_slots(ref_ids[:, None], E, C)
    weights = oracle.base_weights(L.astype(np.float64), ref_ids)[:, None]
    st.update(check_layout_ops(w, x, ref_ids[:, None].astype(np.int32), slots, weights, slot_src, E, C, 1, seed=5))
    print(f"[stats] base capacity: {st}", flush=True)


def test_base_zero_capacity_and_bidder_cap():
    """C = 0: the assignment is still balanced and every slot dropped.  E = 2 with
    c = 2048: the first rounds have more bidders per expert than a round takes
    (2048), so the later ones wait for the next round."""
    announce("base C = 0, E = 2 with c = 2048")
    S, E = 1024, 8
    L = np.random.default_rng(21).standard_normal((S, E)).astype(np.float32)
    g = run_base(L=L, E=E, C=0)
    assert_equal(np.bincount(g["ids"][:, 0], minlength=E), np.full(E, S // E), "tokens per expert")
    assert (g["slots"] == -1).all() and (g["counts"] == 0).all() and g["slot_src"].size == 0
    certify(L.astype(np.float64), g, E)
    S, E = 4096, 2
    L = np.random.default_rng(22).standard_normal((S, E)).astype(np.float32)
    g = run_base(L=L, E=E)
    st = check_base(L.astype(np.float64), g, E, S // E)
    print(f"[stats] base E=2 c=2048: {st}", flush=True)


def test_base_empty():
    announce("base S=0")
    out = hm.base_gate(8, 4, logits=torch.empty((0, 8), dtype=torch.float32, device="cuda"), logits_in=True)
    torch.cuda.synchronize()
    assert out["ids"].numel() == 0
    assert (wl.to_host(out["counts"]) == 0).all()
    assert (wl.to_host(out["slot_src"]) == -1).all()


def test_base_errors_found_on_the_device():
    """A round limit the auction cannot meet, and a NaN score: both are reported
    by status after the kernels finish normally."""
    announce("base round limit and NaN score")
    S, E = 2048, 64
    L = np.random.default_rng(3).standard_normal((S, E)).astype(np.float32)
    with pytest.raises(hm.MoeError) as ex:
        run_base(L=L, E=E, max_rounds=1)
    assert ex.value.status == hm.MOE_ERR_NOT_CONVERGED
    L[17, 5] = np.nan
    with pytest.raises(hm.MoeError) as ex:
        run_base(L=L, E=E)
    assert ex.value.status == 1
    L[17, 5] = np.inf
    with pytest.raises(hm.MoeError) as ex:
        run_base(L=L, E=E)
    assert ex.value.status == 1


def _base_async(E, C, launch_rounds, L=None, x=None, wg=None, bias=None, dtype="f32", max_rounds=0):
    if L is not None:
        out = hm.base_gate(E, C, logits=wl.to_device(L, "f32"), logits_in=True, max_rounds=max_rounds,
                           launch_rounds=launch_rounds)
    else:
        out = hm.base_gate(E, C, x=wl.to_device(x, dtype), wg=wl.to_device(wg, dtype),
                           bias=wl.to_device(bias, "f32"), want_logits=True, max_rounds=max_rounds,
                           launch_rounds=launch_rounds)
    torch.cuda.synchronize()
    status = hm.base_status(out.pop("status"))
    h = {k: wl.to_host(v) for k, v in out.items()}
    return h, status


_BASE_KEYS = ("ids", "slots", "weights", "counts", "slot_src", "prices")


@pytest.mark.parametrize("S,E,seed,proj", [(2048, 64, 0, False), (6000, 12, 6, False), (4096, 64, 1, True)])
def test_base_async_matches_sync(S, E, seed, proj):
    """moe_base_gate_async with enough rounds enqueued: status 0 with the
    synchronous call's phases, rounds and eps, and bitwise its outputs."""
    announce(f"base async S={S} E={E} proj={proj}")
    if proj:
        w = dict(kind=0, k=1, normalize=0, dtype="bf16", S=S, d=1024, E=E, cf=1.0, hot_experts=4, hot_bias=0.5)
        inp = wl.make_inputs(w, seed=seed)
        kw = dict(x=inp["x"], wg=inp["wg"], bias=inp["bias"], dtype="bf16")
    else:
        kw = dict(L=np.random.default_rng(seed).standard_normal((S, E)).astype(np.float32))
    g = run_base(E=E, **kw)
    info = g["info"]
    ga, st = _base_async(E, S // E, 256, **kw)
    assert st == dict(phases=info["phases"], rounds=info["rounds"], eps=info["eps"], status=0), (st, info)
    for key in _BASE_KEYS + (("logits",) if proj else ()):
        assert_equal(ga[key], g[key], f"async {key}")


def test_base_async_round_budget_too_small():
    """One round enqueued cannot finish the auction: status 1, and the outputs
    are still a valid routing (ids in range, slots by their definition).  A NaN
    score gives status 2; a phase that reaches max_rounds, status 1."""
    announce("base async, one round")
    S, E = 2048, 64
    L = np.random.default_rng(3).standard_normal((S, E)).astype(np.float32)
    g, st = _base_async(E, S // E, 1, L=L)
    assert st["status"] == 1, st
    ids = g["ids"][:, 0]
    assert ((ids >= 0) & (ids < E)).all()
    slots_by_property(ids, g["slots"], g["counts"], g["slot_src"], E, S // E)
    L[17, 5] = np.nan
    _, st = _base_async(E, S // E, 64, L=L)
    assert st["status"] == 2, st
    L[17, 5] = 0.5
    g, st = _base_async(E, S // E, 256, L=L, max_rounds=1)
    assert st["status"] == 1, st
    assert ((g["ids"] >= 0) & (g["ids"] < E)).all()


def test_base_async_empty():
    announce("base async S=0")
    out = hm.base_gate(8, 4, logits=torch.empty((0, 8), dtype=torch.float32, device="cuda"), logits_in=True,
                       launch_rounds=4)
    torch.cuda.synchronize()
    assert hm.base_status(out["status"]) == dict(phases=0, rounds=0, eps=0.0, status=0)
    assert (wl.to_host(out["counts"]) == 0).all()
    assert (wl.to_host(out["slot_src"]) == -1).all()


def test_base_async_graph_replays():
    """The asynchronous call captured in a HIP graph: each replay, on new scores
    copied into the captured input between replays, gives bitwise the eager
    synchronous call's outputs on those scores."""
    announce("base async graph capture")
    S, E = 2048, 32
    C = S // E
    dev = "cuda"
    p = hm.base_params(S, 0, E, C, 1, hm.MOE_F32)
    Lbuf = torch.empty((S, E), dtype=torch.float32, device=dev)
    out = {
        "ids": torch.empty((S, 1), dtype=torch.int32, device=dev),
        "slots": torch.empty((S, 1), dtype=torch.int32, device=dev),
        "weights": torch.empty((S, 1), dtype=torch.float32, device=dev),
        "counts": torch.empty((E,), dtype=torch.int32, device=dev),
        "slot_src": torch.empty((E, C), dtype=torch.int32, device=dev),
        "prices": torch.empty((E,), dtype=torch.float64, device=dev),
    }
    status = torch.empty((3,), dtype=torch.int64, device=dev)
    ws = torch.empty((hm.moe_base_gate_workspace_size(p),), dtype=torch.uint8, device=dev)
    args = lambda: (p, None, None, None, Lbuf, out["ids"], out["slots"], out["weights"], out["counts"],
                    out["slot_src"], out["prices"], ws, 128, status)
    Lbuf.copy_(wl.to_device(np.random.default_rng(40).standard_normal((S, E)).astype(np.float32), "f32"))
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        hm.moe_base_gate_async(*args(), stream=s)  # warm-up outside the graph
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        hm.moe_base_gate_async(*args(), stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    for rep in range(4):
        L = np.random.default_rng(41 + rep).standard_normal((S, E)).astype(np.float32) * (1 + rep)
        Lbuf.copy_(wl.to_device(L, "f32"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        st = hm.base_status(status)
        got = {k: wl.to_host(v) for k, v in out.items()}
        ref = run_base(L=L, E=E)
        assert st["status"] == 0 and st["rounds"] == ref["info"]["rounds"], (rep, st, ref["info"])
        for key in _BASE_KEYS:
            assert_equal(got[key], ref[key], f"replay {rep} {key}")


def test_base_batches_equal_paced(monkeypatch):
    """The synchronous call's two ways of enqueueing rounds (paced by the
    device's progress word, and the batches it falls back to without pinned
    memory) give bitwise the same outputs and statistics."""
    announce("base paced vs batches")
    S, E = 4096, 64
    L = np.random.default_rng(31).standard_normal((S, E)).astype(np.float32)
    L[:, :8] += np.float32(0.5)
    paced = run_base(L=L, E=E)
    monkeypatch.setenv("HETUMOE_BASE_BATCHES", "1")
    batched = run_base(L=L, E=E)
    assert paced["info"] == batched["info"]
    for key in _BASE_KEYS:
        assert_equal(batched[key], paced[key], f"batches {key}")
