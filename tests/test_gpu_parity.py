"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Integer routing and the dispatch copy are bit-exact;
floating-point outputs are within rtol * (sum of |terms|), rtol 1e-5 for fp32
and 2e-2 for bf16 outputs."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2203_14685_amd as hm
from paper_2203_14685_amd import workloads as wl

from _fullsize import check_layout_full
from _parity import (RTOL, announce, assert_close, assert_equal, check_gate, check_layout_ops, decode,
                     gpu_gate)

pytestmark = pytest.mark.gpu

W = wl.WORKLOADS


def cap(cf, k, S, E):
    return int(math.ceil(cf * k * S / E))


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hm.load()
    yield


# ------------------------------------------------------------------ reduced sizes

SMALL = [
    # (workload, S, d): several 256-token blocks plus a ragged tail
    (1, 1000, 256),
    (2, 1000, 1024),
    (3, 1000, 2048),
    (4, 1000, 2048),
    (5, 3000, 4096),
]


@pytest.mark.parametrize("wid,S,d", SMALL)
def test_small_workload_parity(wid, S, d):
    w = W[wid]
    E, k = w["E"], w["k"]
    C = cap(w["cf"], k, S, E)
    announce(f"small workload {wid} S={S} d={d} E={E} k={k} C={C}")
    inp = wl.make_inputs(w, S=S, d=d, seed=0)
    g = gpu_gate(w, inp, E, k, C, w["kind"], w["normalize"])
    ref, st = check_gate(w, inp, g, E, k, C, w["kind"], w["normalize"])
    st.update(check_layout_ops(w, inp["x"], g["ids"], g["slots"], g["weights"], g["slot_src"], E, C, k))
    print(f"[stats] workload {wid}: {st}", flush=True)


# ------------------------------------------------------------------ routing edge cases

def _logits_case(S, E, k, kind, normalize, C, L, dtype="f32"):
    w = dict(dtype=dtype)
    g = gpu_gate(w, None, E, k, C, kind, normalize, logits=L.astype(np.float32))
    check_gate(w, None, g, E, k, C, kind, normalize, logits_in=L.astype(np.float32))
    return g


@pytest.mark.parametrize("E,k,kind,normalize", [
    (5, 1, 0, 0), (5, 2, 0, 1), (12, 3, 0, 1), (16, 2, 0, 0), (64, 8, 0, 1), (1024, 8, 0, 0),
    (1024, 1, 0, 1), (12, 4, 1, 0), (64, 4, 1, 0), (1024, 8, 1, 0), (1, 1, 0, 0), (3, 3, 0, 1),
])
def test_dense_ties_logits_in(E, k, kind, normalize):
    S = 700
    announce(f"dense ties E={E} k={k} kind={kind} normalize={normalize}")
    rng = np.random.default_rng(E * 31 + k)
    L = rng.integers(0, 3, size=(S, E)).astype(np.float32)
    for C in (1, 7, cap(1.0, k, S, E), S * k):
        _logits_case(S, E, k, kind, normalize, C, L)


@pytest.mark.parametrize("S,E,k,kind,normalize", [
    # histograms (k E rows of one count per 64-token wave block) past the
    # one-launch scan-and-assign limit, so that the scan and the assignment run
    # as two kernels: ragged wave-block counts (313, 516, 625), kTop1, top-8
    # and E = 1024
    (20000, 64, 2, 0, 1), (33000, 64, 1, 0, 0), (32768, 64, 4, 1, 0), (40000, 16, 8, 0, 1),
    (9000, 1024, 2, 0, 0),
])
def test_scan_assign_histogram_sizes(S, E, k, kind, normalize):
    announce(f"scan/assign S={S} E={E} k={k} kind={kind}")
    rng = np.random.default_rng(S + E + k)
    L = rng.integers(0, 3, size=(S, E)).astype(np.float32)
    L[:, : max(1, E // 16)] += 1.0  # favoured experts overflow their capacity
    for C in (1, cap(1.0, k, S, E) // 2, cap(1.25, k, S, E), S * k):
        _logits_case(S, E, k, kind, normalize, C, L)


def test_all_equal_logits_and_zero_signs():
    S, E = 300, 8
    announce("all-equal logits")
    L = np.zeros((S, E), dtype=np.float32)
    L[::2, :] = -0.0
    g = _logits_case(S, E, 2, 0, 1, S * 2, L)
    assert (g["ids"][:, 0] == 0).all() and (g["ids"][:, 1] == 1).all()
    g = _logits_case(S, E, 1, 0, 0, 10, L)
    assert (g["counts"] == [10, 0, 0, 0, 0, 0, 0, 0]).all()


def test_capacity_zero_and_empty_batch():
    announce("C = 0 and S = 0")
    rng = np.random.default_rng(1)
    L = rng.standard_normal((100, 6)).astype(np.float32)
    g = _logits_case(100, 6, 2, 0, 1, 0, L)
    assert (g["slots"] == -1).all() and g["slot_src"].shape == (6, 0)
    g = _logits_case(0, 6, 2, 0, 1, 5, np.zeros((0, 6), np.float32))
    assert (g["slot_src"] == -1).all() and (g["counts"] == 0).all()
    w = W[5]
    tok = np.zeros(0, dtype=np.int32)
    g = gpu_gate(w, dict(token_ids=tok), 128, 1, 4, hm.MOE_GATE_HASH, 0)
    assert (g["slot_src"] == -1).all() and (g["demand"] == 0).all()


def test_hash_edge_cases():
    announce("hash E=1 and E=7")
    w = W[5]
    tok = wl.zipf_token_ids(1500, 50257, 1.1, 3)
    for E, C in ((1, 10), (7, 100), (128, 1500)):
        g = gpu_gate(w, dict(token_ids=tok), E, 1, C, hm.MOE_GATE_HASH, 0)
        check_gate(w, dict(token_ids=tok), g, E, 1, C, hm.MOE_GATE_HASH, 0)
        assert (g["weights"] == 1.0).all()


@pytest.mark.parametrize("dtype,d,E,k", [("bf16", 8, 4, 2), ("f32", 4, 3, 1), ("bf16", 520, 6, 2),
                                          ("f32", 260, 16, 4), ("bf16", 2056, 64, 1)])
def test_projection_odd_shapes(dtype, d, E, k):
    S = 517
    announce(f"projection dtype={dtype} d={d} E={E} k={k}")
    w = dict(kind=0, k=k, normalize=1, dtype=dtype, S=S, d=d, E=E, cf=1.0)
    inp = wl.make_inputs(w, seed=5)
    C = cap(1.0, k, S, E)
    g = gpu_gate(w, inp, E, k, C, 0, 1)
    check_gate(w, inp, g, E, k, C, 0, 1)
    check_layout_ops(w, inp["x"], g["ids"], g["slots"], g["weights"], g["slot_src"], E, C, k, seed=9)


@pytest.mark.parametrize("dtype,E,k,kind,normalize,d,bias,S", [
    ("f32", 8, 1, 0, 0, 2500, True, 1000), ("f32", 16, 2, 0, 1, 4096, False, 2000),
    ("f32", 32, 4, 1, 0, 1028, True, 1000), ("f32", 64, 8, 0, 1, 300, True, 130),
    ("f32", 64, 2, 1, 0, 4, False, 65), ("f32", 8, 8, 1, 0, 64, False, 64),
    ("bf16", 8, 2, 0, 1, 1032, True, 700), ("f32", 32, 3, 0, 0, 516, False, 1),
])
def test_split_projection_shapes(dtype, E, k, kind, normalize, d, bias, S):
    """Projections on the vector ALUs with 8 lanes per token (E in 8..64, d a
    whole number of 16-byte chunks): W staged in several phases with a ragged
    last one, ragged token tails, kTop1 groups down to one expert."""
    announce(f"split projection dtype={dtype} E={E} k={k} kind={kind} d={d} bias={bias} S={S}")
    w = dict(kind=kind, k=k, normalize=normalize, dtype=dtype, S=S, d=d, E=E, cf=1.0)
    if bias:
        w.update(hot_experts=2, hot_bias=0.5)
    inp = wl.make_inputs(w, seed=3 * E + k)
    C = cap(1.0, k, S, E)
    g = gpu_gate(w, inp, E, k, C, kind, normalize)
    st = check_gate(w, inp, g, E, k, C, kind, normalize)[1]
    print(f"[stats] split E={E} d={d}: {st}", flush=True)


@pytest.mark.parametrize("E,k,kind,normalize,d,bias,S", [
    # W staged through LDS (4 lanes per token select)
    (16, 1, 1, 0, 256, False, 300), (48, 1, 0, 0, 256, False, 300), (64, 4, 1, 0, 768, True, 300),
    (80, 3, 0, 1, 256, False, 300), (96, 8, 0, 0, 128, True, 300), (112, 2, 0, 0, 384, False, 300),
    (128, 8, 1, 0, 256, True, 300), (128, 2, 0, 1, 384, False, 300), (48, 3, 1, 0, 256, False, 300),
    (64, 8, 1, 0, 256, True, 300), (128, 4, 1, 0, 384, False, 300), (80, 5, 1, 0, 256, False, 300),
    # W held in registers: eight waves up to d * E = 64 K (8 lanes per token select)
    (32, 2, 0, 1, 512, True, 300), (64, 4, 1, 0, 1024, True, 300), (128, 8, 0, 1, 512, False, 300),
    (16, 2, 0, 0, 2048, False, 300), (32, 8, 1, 0, 1024, True, 300), (64, 1, 0, 0, 512, False, 300),
    (64, 2, 0, 1, 512, True, 20000),
    # ... four waves up to 128 K (4 lanes per token select); S = 20000 and 40000
    # give blocks two and three wave blocks
    (32, 2, 0, 1, 2048, True, 20000), (32, 8, 1, 0, 2048, False, 300), (64, 8, 0, 1, 2048, True, 300),
    (64, 4, 1, 0, 2048, False, 40000), (64, 1, 0, 0, 2048, True, 77), (128, 3, 0, 0, 1024, True, 700),
    (128, 8, 1, 0, 1024, False, 20000),
    # W^T staged per K phase (persistent, one block per CU); S = 40000 gives some
    # blocks three wave blocks, one of them without a partner
    (64, 2, 0, 1, 1536, True, 40000), (128, 1, 1, 0, 1024, False, 3000), (16, 4, 0, 1, 4096, True, 300),
    (64, 4, 1, 0, 3072, True, 300), (32, 8, 0, 1, 4096, False, 700),
])
def test_mfma_projection_shapes(E, k, kind, normalize, d, bias, S):
    """bf16 shapes that take the matrix-core route kernels (E a multiple of 16 up
    to 128), several wave blocks plus a ragged tail; S = 20000 makes persistent
    blocks walk more than one wave block."""
    announce(f"mfma projection E={E} k={k} kind={kind} d={d} bias={bias}")
    w = dict(kind=kind, k=k, normalize=normalize, dtype="bf16", S=S, d=d, E=E, cf=1.0)
    if bias:
        w.update(hot_experts=3, hot_bias=0.5)
    inp = wl.make_inputs(w, seed=E + k)
    C = cap(1.0, k, S, E)
    g = gpu_gate(w, inp, E, k, C, kind, normalize)
    st = check_gate(w, inp, g, E, k, C, kind, normalize)[1]
    print(f"[stats] mfma E={E}: {st}", flush=True)


@pytest.mark.parametrize("wid,S", [(3, 700), (2, 300)])
def test_projection_logits_into_unaligned_buffer(wid, S):
    """Logits written into a caller's buffer that is 4-byte but not 16-byte
    aligned match, bit for bit, those written into an aligned one, and the
    routing is the same."""
    w = W[wid]
    E, k = w["E"], w["k"]
    C = cap(w["cf"], k, S, E)
    announce(f"unaligned logits workload {wid} S={S}")
    inp = wl.make_inputs(w, S=S, seed=5)
    x, wg = wl.to_device(inp["x"], "bf16"), wl.to_device(inp["wg"], "bf16")
    bias = wl.to_device(inp["bias"], "f32")
    p = hm.gate_params(S, w["d"], E, k, C, w["kind"], w["normalize"], 0, hm.MOE_BF16, 0)
    ws = torch.empty((hm.moe_gate_workspace_size(p),), dtype=torch.uint8, device="cuda")
    runs = []
    for off in (0, 1):
        buf = torch.full((S * E + 8,), -7.0, dtype=torch.float32, device="cuda")
        lg = buf[off:off + S * E].view(S, E)
        i32 = lambda *sh: torch.full(sh, -3, dtype=torch.int32, device="cuda")
        o = dict(ids=i32(S, k), slots=i32(S, k), weights=torch.zeros((S, k), device="cuda"), counts=i32(E),
                 demand=i32(E), slot_src=i32(E, C))
        hm.moe_gate(p, x, wg, bias, None, None, None, lg, o["ids"], o["slots"], o["weights"], o["counts"],
                    o["demand"], o["slot_src"], ws)
        torch.cuda.synchronize()
        assert (buf[:off] == -7.0).all() and (buf[off + S * E:] == -7.0).all()
        runs.append({"logits": lg.clone(), **o})
    for key in runs[0]:
        assert torch.equal(runs[0][key], runs[1][key]), key


def test_ktop1_projection_with_bias():
    S, d, E, k = 600, 512, 24, 3
    announce("kTop1 projection with bias")
    w = dict(kind=1, k=k, normalize=0, dtype="bf16", S=S, d=d, E=E, cf=1.25, hot_experts=2, hot_bias=0.75)
    inp = wl.make_inputs(w, seed=8)
    C = cap(1.25, k, S, E)
    g = gpu_gate(w, inp, E, k, C, 1, 0)
    check_gate(w, inp, g, E, k, C, 1, 0)


@pytest.mark.parametrize("dtype,k,C", [("bf16", 8, 40), ("f32", 3, 5), ("bf16", 2, 600)])
def test_layout_ops_many_choices_and_drops(dtype, k, C):
    """Dispatch / combine and their backward with k > 1 (token-major scatter for
    the expert-slot outputs), heavy drops, empty slots and a ragged tail."""
    S, d, E = 555, 264 if dtype == "bf16" else 132, 12
    announce(f"layout ops dtype={dtype} k={k} C={C}")
    rng = np.random.default_rng(k * 7 + C)
    L = rng.standard_normal((S, E)).astype(np.float32)
    g = _logits_case(S, E, k, 0, 1, C, L)
    w = dict(dtype=dtype)
    x = wl.make_rows((S, d), dtype, 17)
    st = check_layout_ops(w, x, g["ids"], g["slots"], g["weights"], g["slot_src"], E, C, k, seed=21)
    assert (g["slots"] < 0).any() or C * E >= S * k
    print(f"[stats] layout k={k}: {st}", flush=True)


@pytest.mark.parametrize("dtype,d,k,S,C", [
    ("bf16", 512, 1, 517, 40), ("bf16", 1024, 2, 519, 70), ("bf16", 2048, 3, 1, 1), ("f32", 256, 1, 1023, 90),
    ("f32", 512, 2, 3, 1), ("f32", 1024, 3, 261, 50), ("bf16", 2048, 1, 2, 0),
    ("bf16", 512, 4, 301, 60), ("f32", 512, 3, 130, 30), ("bf16", 2048, 2, 97, 20),
])
def test_layout_ops_short_rows(dtype, d, k, S, C):
    """Rows of 1, 2 and 4 KiB: a wave combines several tokens at once (k >= 3, and
    every k at 4 KiB), the flat form takes k <= 2 up to 2 KiB; token counts that
    leave the last wave partly empty, drops, and C = 0."""
    E = 16
    announce(f"layout ops short rows dtype={dtype} d={d} k={k} S={S} C={C}")
    rng = np.random.default_rng(d + k + S)
    L = rng.standard_normal((S, E)).astype(np.float32)
    g = _logits_case(S, E, k, 0, 1, C, L)
    x = wl.make_rows((S, d), dtype, 31)
    st = check_layout_ops(dict(dtype=dtype), x, g["ids"], g["slots"], g["weights"], g["slot_src"], E, C, k, seed=33)
    print(f"[stats] short rows d={d}: {st}", flush=True)


@pytest.mark.parametrize("dtype,d,k,S,C", [
    ("bf16", 264, 1, 300, 30), ("f32", 100, 1, 301, 40), ("bf16", 256, 1, 130, 12), ("bf16", 8192, 1, 40, 4),
    ("f32", 8192, 1, 33, 3), ("f32", 1000, 2, 77, 11), ("bf16", 1784, 2, 65, 9),
])
def test_layout_ops_flat_row_lengths(dtype, d, k, S, C):
    """Row lengths the one-chunk-per-thread kernels treat specially: not a power
    of two (33, 25, 250, 223 chunks), a power of two below one wave (32), the
    largest row whose dw is reduced inside a block (1024 chunks) and a longer
    one (2048 chunks, rows spanning two blocks)."""
    E = 8
    announce(f"layout ops flat rows dtype={dtype} d={d} k={k} S={S} C={C}")
    rng = np.random.default_rng(d * 3 + k + S)
    L = rng.standard_normal((S, E)).astype(np.float32)
    g = _logits_case(S, E, k, 0, 1, C, L)
    x = wl.make_rows((S, d), dtype, 41)
    st = check_layout_ops(dict(dtype=dtype), x, g["ids"], g["slots"], g["weights"], g["slot_src"], E, C, k, seed=43)
    assert (g["slots"] < 0).any() and (k > 1 or (g["slot_src"] < 0).any())
    # the [E, C, d] writers leave the memory around a view alone
    pad = 64
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    buf = torch.full((E * C * d + 2 * pad,), 7.0, dtype=tdt, device="cuda")
    xe = buf[pad:pad + E * C * d].view(E, C, d)
    d_ids, d_slots = wl.to_device(g["ids"], "i32"), wl.to_device(g["slots"], "i32")
    code = hm.MOE_BF16 if dtype == "bf16" else hm.MOE_F32
    hm.moe_dispatch(hm.Layout(S, d, E, k, C, code), wl.to_device(x, dtype), d_ids, d_slots,
                    wl.to_device(g["slot_src"], "i32"), xe)
    torch.cuda.synchronize()
    assert (buf[:pad] == 7.0).all() and (buf[-pad:] == 7.0).all()
    assert_equal(wl.to_host(xe), oracle.dispatch(x, g["slot_src"], k), "dispatch into a view")
    print(f"[stats] flat rows d={d} k={k}: {st}", flush=True)


def test_determinism_and_guard_bands():
    announce("determinism and guard bands")
    w = W[2]
    S, d, E, k = 1000, 1024, 16, 2
    C = cap(1.25, k, S, E)
    inp = wl.make_inputs(w, S=S, d=d, seed=2)
    a = gpu_gate(w, inp, E, k, C, 0, 1)
    b = gpu_gate(w, inp, E, k, C, 0, 1)
    for key in a:
        if a[key] is not None:
            assert_equal(a[key], b[key], f"repeat {key}")
    # outputs written into the middle of larger buffers leave the guard bands alone
    pad = 64
    x = wl.to_device(inp["x"], "bf16")
    src = wl.to_device(a["slot_src"], "i32")
    d_ids, d_slots = wl.to_device(a["ids"], "i32"), wl.to_device(a["slots"], "i32")
    buf = torch.full((E * C * d + 2 * pad,), 7.0, dtype=torch.bfloat16, device="cuda")
    xe = buf[pad:pad + E * C * d].view(E, C, d)
    hm.moe_dispatch(hm.Layout(S, d, E, k, C, hm.MOE_BF16), x, d_ids, d_slots, src, xe)
    torch.cuda.synchronize()
    assert (buf[:pad] == 7.0).all() and (buf[-pad:] == 7.0).all()
    assert_equal(wl.to_host(xe), oracle.dispatch(inp["x"], a["slot_src"], k), "dispatch into a view")


# ------------------------------------------------------------------ full sizes, every element

@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_full_size_parity(wid):
    """Every routing integer and every element of xe, y, dx, dye and dw at the
    workload's full size, against the oracle run in chunks (the checks are in
    tests/_fullsize.py, which needs no GPU)."""
    w = W[wid]
    S, d, E, k, C, dt = w["S"], w["d"], w["E"], w["k"], w["C"], w["dtype"]
    assert C == oracle.capacity(w["cf"], k, S, E)
    announce(f"full workload {wid}: {w['name']}")
    inp = wl.make_inputs(w, seed=0)
    g = gpu_gate(w, inp, E, k, C, w["kind"], w["normalize"])
    ref, st = check_gate(w, inp, g, E, k, C, w["kind"], w["normalize"])
    del ref
    x = wl.to_device(inp["x"], dt)
    d_src = wl.to_device(g["slot_src"], "i32")
    d_ids, d_slots = wl.to_device(g["ids"], "i32"), wl.to_device(g["slots"], "i32")
    d_w = wl.to_device(g["weights"], "f32")
    dy_host = wl.make_rows((S, d), dt, 2)
    ye_host = wl.make_rows((E, C, d), dt, 3)  # random expert outputs (also the dispatch-backward input)
    ye = wl.to_device(ye_host, dt)
    xe = hm.dispatch(x, d_ids, d_slots, d_src)
    y = hm.combine(ye, d_ids, d_slots, d_w)
    dx = hm.dispatch_bwd(ye, d_ids, d_slots)
    dye, dw = hm.combine_bwd(wl.to_device(dy_host, dt), d_ids, d_slots, d_src, d_w, ye=ye, want_dw=True)
    torch.cuda.synchronize()
    outs = {"xe": wl.to_host(xe), "y": wl.to_host(y), "dx": wl.to_host(dx), "dye": wl.to_host(dye),
            "dw": wl.to_host(dw)}
    del x, xe, ye, y, dx, dye, dw
    torch.cuda.empty_cache()
    st.update(check_layout_full(dt, inp["x"], ye_host, dy_host, g["ids"], g["slots"], g["weights"], g["slot_src"], k,
                                outs))
    print(f"[stats] full workload {wid}: {st}", flush=True)
