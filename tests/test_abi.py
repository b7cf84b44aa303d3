"""CPU checks of the C-ABI library: it loads, exports every symbol the header
declares, has the struct layout the binding assumes, and rejects bad arguments
with status codes before any HIP call (so these run without a GPU)."""

import ctypes
import os
import re

import pytest

import paper_2203_14685_amd as hm
from paper_2203_14685_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hetumoe.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hm.LIB_PATH):
        pytest.fail("libhetumoe.so is not built (run `python -m paper_2203_14685_amd.build`)")
    return hm.load()


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"MOE_API\s+[\w\s\*]+?\b(moe_\w+)\s*\(", text)))


def test_header_declares_the_abi():
    names = declared_symbols()
    assert set(names) == set(b.EXPORTED), names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), f"{name} not exported"


def test_abi_version_and_struct_layout(lib):
    assert lib.moe_abi_version() == 8
    assert ctypes.sizeof(b.GateParams) == 56
    assert b.GateParams.hash_seed.offset == 40
    assert b.GateParams.temperature.offset == 48 and b.GateParams.hash_vocab.offset == 52
    assert ctypes.sizeof(b.Layout) == 24
    assert lib.moe_status_string(0) == b"MOE_OK"
    assert lib.moe_status_string(3) == b"MOE_ERR_WORKSPACE"


def _ws(params):
    n = ctypes.c_size_t(12345)
    st = hm.load().moe_gate_workspace_size(ctypes.byref(params), ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("S,E,k,kind", [(1024, 8, 1, 0), (8192, 16, 2, 0), (32768, 64, 4, 1), (65536, 128, 1, 2),
                                        (0, 8, 1, 0), (257, 5, 2, 0)])
def test_workspace_size(lib, S, E, k, kind):
    # fp32: histogram only, k x E x ceil(S / 64) int32
    p = hm.gate_params(S, 256, E, k, 10, kind)
    st, n = _ws(p)
    assert st == 0
    assert n == k * ((S + 63) // 64) * E * 4


BAD_PARAMS = [
    dict(E=0), dict(E=1025), dict(S=-1), dict(capacity=-1), dict(k=0), dict(k=9, E=16),
    dict(k=3, E=2), dict(kind=1, k=3, E=16), dict(kind=2, k=2), dict(kind=3), dict(dtype=2),
    dict(normalize=2), dict(logits_in=2), dict(kind=2, logits_in=1), dict(d=0),
    dict(E=1024, capacity=1 << 21), dict(S=1 << 30, k=2), dict(kind=4),
    dict(groups=2), dict(kind=3, groups=0), dict(kind=3, groups=3), dict(kind=3, groups=4, k=3),
    dict(temperature=-1.0), dict(temperature=float("nan")), dict(temperature=float("inf")),
    dict(kind=2, temperature=0.5), dict(hash_vocab=10), dict(kind=2, hash_vocab=-1),
]


@pytest.mark.parametrize("bad", BAD_PARAMS)
def test_bad_gate_params_rejected(lib, bad):
    base = dict(S=100, d=256, E=8, k=1, capacity=20, kind=0, normalize=0, logits_in=0, dtype=0, hash_seed=0, groups=0,
                temperature=0.0, hash_vocab=0)
    base.update(bad)
    p = hm.gate_params(**base)
    st, _ = _ws(p)
    assert st == b.MOE_ERR_INVALID_ARG, (bad, lib.moe_last_error())
    assert lib.moe_last_error() != b""


def test_null_params_and_extended_workspace(lib):
    n = ctypes.c_size_t(0)
    assert lib.moe_gate_workspace_size(None, ctypes.byref(n)) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_gate(None, *([None] * 13), None, 0, None) == b.MOE_ERR_INVALID_ARG
    # hierarchical top-k and tempered gates also hold their logits: [S, E] fp32 after the histogram
    for params in (hm.gate_params(1000, 256, 16, 2, 20, 3, groups=4), hm.gate_params(1000, 256, 16, 2, 20, 0, temperature=0.5)):
        hist = 2 * ((1000 + 63) // 64) * 16 * 4
        assert _ws(params) == (0, (hist + 255) // 256 * 256 + 1000 * 16 * 4)


def test_noalloc_validates_before_any_hip_call(lib):
    assert lib.moe_gate_noalloc(None, *([None] * 13), None) == b.MOE_ERR_INVALID_ARG
    bad = hm.gate_params(100, 256, 0, 1, 20, 0)
    assert lib.moe_gate_noalloc(ctypes.byref(bad), *([None] * 13), None) == b.MOE_ERR_INVALID_ARG
    # a histogram of 8 * 1024 * 256 int32 (8 MiB) exceeds the 4 MiB scratch:
    # refused after the pointer checks, before the scratch is looked up; the
    # stand-in addresses are never dereferenced
    p = hm.gate_params(16384, 0, 1024, 8, 4, 0, 0, 1, 0)
    fake = ctypes.c_void_p(1 << 20)
    st = lib.moe_gate_noalloc(ctypes.byref(p), None, None, None, None, None, None, fake, fake, fake, fake, fake, None,
                              fake, None)
    assert st == b.MOE_ERR_UNSUPPORTED, lib.moe_last_error()
    assert b"scratch" in lib.moe_last_error()


def test_balanced_hash_table_matches_the_oracle(lib):
    import numpy as np

    import oracle
    ranks = np.arange(1, 50258, dtype=np.float64)
    p = ranks ** -1.1
    p /= p.sum()
    for E in (128, 7, 1):
        assert np.array_equal(hm.moe_hash_balanced_table(p, E), oracle.balanced_hash_table(p, E))
    rng = np.random.default_rng(5)
    f = rng.integers(0, 4, 300).astype(np.float64)  # many equal frequencies
    assert np.array_equal(hm.moe_hash_balanced_table(f, 9), oracle.balanced_hash_table(f, 9))
    bad = np.array([1.0, -1.0])
    with pytest.raises(b.MoeError):
        hm.moe_hash_balanced_table(bad, 2)
    with pytest.raises(b.MoeError):
        hm.moe_hash_balanced_table(np.array([1.0, np.nan]), 2)
    with pytest.raises(b.MoeError):
        hm.moe_hash_balanced_table(np.ones(4), 0)


def test_row_size_must_be_16_byte_multiple(lib):
    p = hm.gate_params(100, 4, 8, 1, 20, 0, dtype=b.MOE_BF16)        # 8-byte rows
    assert _ws(p)[0] == b.MOE_ERR_UNSUPPORTED
    lay = b.Layout(100, 6, 8, 1, 20, b.MOE_F32)                         # 24-byte rows
    st = lib.moe_dispatch(ctypes.byref(lay), 16, 16, 16, 16, 16, None)
    assert st == b.MOE_ERR_UNSUPPORTED


# fake, never dereferenced device addresses: validation fails before any HIP call
A16 = 0x7f0000000000
A4 = A16 + 4


def test_gate_pointer_checks(lib):
    p = hm.gate_params(100, 256, 8, 1, 20, 0)
    call = lambda **kw: lib.moe_gate(ctypes.byref(p), kw.get("x", A16), kw.get("wg", A16), kw.get("bias"),
                                     kw.get("tok"), kw.get("noise"), kw.get("table"), kw.get("logits"),
                                     kw.get("ids", A16), kw.get("slots", A16),
                                     kw.get("w", A16), kw.get("counts", A16), kw.get("demand"),
                                     kw.get("src", A16), kw.get("ws", A16), kw.get("wsb", 1 << 20), None)
    assert call(x=None) == b.MOE_ERR_INVALID_ARG
    assert call(x=A4) == b.MOE_ERR_UNSUPPORTED                     # x must be 16-byte aligned
    assert call(ids=None) == b.MOE_ERR_INVALID_ARG
    assert call(ids=A16 + 2) == b.MOE_ERR_INVALID_ARG              # int32 arrays 4-byte aligned
    assert call(tok=A16) == b.MOE_ERR_INVALID_ARG                  # token ids only for HASH
    assert call(ws=None) == b.MOE_ERR_WORKSPACE
    assert call(wsb=16) == b.MOE_ERR_WORKSPACE
    assert call(noise=A16) == b.MOE_ERR_INVALID_ARG                # noise needs a temperature
    assert call(table=A16) == b.MOE_ERR_INVALID_ARG                # a table only for HASH
    ph = hm.gate_params(100, 0, 8, 1, 20, 2)
    assert lib.moe_gate(ctypes.byref(ph), A16, None, None, A16, None, None, None, A16, A16, A16, A16, None, A16, A16,
                        1 << 20, None) == b.MOE_ERR_INVALID_ARG  # HASH takes no x
    assert lib.moe_gate(ctypes.byref(ph), None, None, None, A16, None, A16, None, A16, A16, A16, A16, None, A16, A16,
                        1 << 20, None) == b.MOE_ERR_INVALID_ARG  # a table needs hash_vocab
    pt = hm.gate_params(100, 0, 8, 1, 20, 2, hash_vocab=50)
    assert lib.moe_gate(ctypes.byref(pt), None, None, None, A16, None, None, None, A16, A16, A16, A16, None, A16, A16,
                        1 << 20, None) == b.MOE_ERR_INVALID_ARG  # hash_vocab needs a table
    pl = hm.gate_params(100, 0, 8, 1, 20, 0, logits_in=1)
    assert lib.moe_gate(ctypes.byref(pl), None, None, None, None, None, None, None, A16, A16, A16, A16, None, A16, A16,
                        1 << 20, None) == b.MOE_ERR_INVALID_ARG  # logits required as input


def test_layout_pointer_checks(lib):
    lay = b.Layout(100, 256, 8, 2, 20, b.MOE_BF16)
    # moe_dispatch(l, x, ids, slots, slot_src, xe, stream)
    assert lib.moe_dispatch(None, A16, A16, A16, A16, A16, None) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_dispatch(ctypes.byref(lay), A16, A16, A16, A16, A16 + 8, None) == b.MOE_ERR_UNSUPPORTED
    assert lib.moe_dispatch(ctypes.byref(lay), None, A16, A16, A16, A16, None) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_dispatch(ctypes.byref(lay), A16, None, A16, A16, A16, None) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_dispatch(ctypes.byref(lay), A16, A16, A16 + 2, A16, A16, None) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_combine(ctypes.byref(lay), A16, A16, A16, None, A16, None) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_dispatch_bwd(ctypes.byref(lay), A16, None, A16, A16, None) == b.MOE_ERR_INVALID_ARG
    # moe_combine_bwd(l, dy, ye, ids, slots, slot_src, weights, dye, dw, stream): ye goes with dw
    assert lib.moe_combine_bwd(ctypes.byref(lay), A16, A16, A16, A16, A16, A16, A16, None, None) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_combine_bwd(ctypes.byref(lay), A16, None, A16, A16, A16, A16, A16, A16, None) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_combine_bwd(ctypes.byref(lay), A16, None, None, A16, A16, A16, A16, None, None) == b.MOE_ERR_INVALID_ARG
    bad = b.Layout(100, 256, 8, 9, 20, b.MOE_BF16)
    assert lib.moe_combine(ctypes.byref(bad), A16, A16, A16, A16, A16, None) == b.MOE_ERR_INVALID_ARG


def test_binding_rejects_cpu_tensors(lib):
    import torch
    x = torch.zeros(4, 8)
    with pytest.raises(ValueError):
        z = torch.zeros((4, 1), dtype=torch.int32)
        hm.dispatch(x, z, z, torch.zeros((2, 2), dtype=torch.int32))


# ------------------------------------------------------------------ gate backward

def _bwd_ws(params):
    n = ctypes.c_size_t(12345)
    st = hm.load().moe_gate_bwd_workspace_size(ctypes.byref(params), ctypes.byref(n))
    return st, n.value


def _a256(n):
    return (n + 255) // 256 * 256


def _bwd_ws_formula(S, d, E, dtype):
    nb = (S + 63) // 64
    mfma = dtype == b.MOE_BF16 and E % 16 == 0 and E <= 128 and d % 64 == 0
    per_split = -(-d // 256) if mfma else ((d + 63) // 64) * ((E + 63) // 64)
    target = 512 if mfma else 1024
    ns = -(-target // per_split)
    if mfma:
        ns = min(ns, nb // 4)
    ns = max(1, min(ns, nb))
    st = max(64, -(-(-(-S // ns)) // 64) * 64)
    nsplit = -(-S // st)
    return (_a256(S * E * 4) + (_a256(3 * nb * 64 * E * 2) if mfma else 0) + _a256((1 + -(-S // 4096)) * E * 4)
            + 2 * _a256(nb * E * 4) + _a256(E * 4) + _a256(nsplit * E * d * 4))


def test_gate_bwd_struct_and_workspace(lib):
    assert ctypes.sizeof(b.GateBwdParams) == 40
    assert b.GateBwdParams.aux_coef.offset == 32 and b.GateBwdParams.temperature.offset == 36
    for S, d, E, k, dt in [(32768, 2048, 64, 4, b.MOE_BF16), (32768, 2048, 64, 4, b.MOE_F32),
                           (1000, 256, 8, 1, b.MOE_F32), (0, 16, 3, 1, b.MOE_F32), (5000, 64, 1024, 2, b.MOE_BF16),
                           (8192, 1024, 16, 2, b.MOE_BF16), (100, 520, 48, 2, b.MOE_BF16)]:
        p = hm.gate_bwd_params(S, d, E, k, 0, dtype=dt)
        st, n = _bwd_ws(p)
        assert st == 0
        assert n == _bwd_ws_formula(S, d, E, dt), (S, d, E, k, dt)


BAD_BWD = [
    dict(kind=2), dict(kind=5), dict(E=0), dict(E=1025), dict(S=-1), dict(d=0), dict(k=0), dict(k=9, E=16),
    dict(kind=1, k=3, E=16), dict(normalize=2), dict(accumulate_dx=2), dict(dtype=2),
    dict(aux_coef=float("nan")), dict(aux_coef=float("inf")), dict(kind=1, k=2, aux_coef=0.01),
    dict(S=1 << 30, k=2), dict(temperature=-0.5), dict(temperature=float("nan")), dict(kind=4),
]


@pytest.mark.parametrize("bad", BAD_BWD)
def test_bad_gate_bwd_params_rejected(lib, bad):
    base = dict(S=100, d=256, E=8, k=1, kind=0, normalize=0, dtype=0, accumulate_dx=0, aux_coef=0.0, temperature=0.0)
    base.update(bad)
    st, _ = _bwd_ws(hm.gate_bwd_params(**base))
    assert st == b.MOE_ERR_INVALID_ARG, (bad, lib.moe_last_error())


def test_gate_bwd_pointer_checks(lib):
    p = hm.gate_bwd_params(100, 256, 8, 2, 0, 1, b.MOE_BF16, 0, 0.0)
    # moe_gate_bwd(p, x, wg, logits, ids, dw, dlogits, dx, dwg, dbias, aux_loss, ws, wsb, stream)
    call = lambda **kw: lib.moe_gate_bwd(ctypes.byref(p), kw.get("x", A16), kw.get("wg", A16),
                                         kw.get("logits", A16), kw.get("ids", A16), kw.get("dw", A16),
                                         kw.get("dl"), kw.get("dx", A16), kw.get("dwg", A16), kw.get("db"),
                                         kw.get("aux"), kw.get("ws", A16), kw.get("wsb", 1 << 30), None)
    assert lib.moe_gate_bwd(None, *([None] * 10), None, 0, None) == b.MOE_ERR_INVALID_ARG
    assert call(logits=None) == b.MOE_ERR_INVALID_ARG
    assert call(ids=None) == b.MOE_ERR_INVALID_ARG
    assert call(dw=A16 + 2) == b.MOE_ERR_INVALID_ARG
    assert call(x=None) == b.MOE_ERR_INVALID_ARG                  # dwg needs x
    assert call(x=A16 + 4) == b.MOE_ERR_UNSUPPORTED               # x 16-byte aligned
    assert call(wg=None) == b.MOE_ERR_INVALID_ARG                 # dx needs wg
    assert call(dx=A16 + 8) == b.MOE_ERR_UNSUPPORTED
    assert call(aux=A16) == b.MOE_ERR_INVALID_ARG                 # a loss value needs aux_coef
    assert call(ws=None) == b.MOE_ERR_WORKSPACE
    assert call(wsb=64) == b.MOE_ERR_WORKSPACE
    assert call(ws=A16 + 4) == b.MOE_ERR_WORKSPACE
    p6 = hm.gate_bwd_params(100, 4, 8, 2, 0, 1, b.MOE_BF16)     # 8-byte rows of x / dx
    assert lib.moe_gate_bwd(ctypes.byref(p6), A16, A16, A16, A16, A16, None, A16, None, None, None, A16,
                            1 << 30, None) == b.MOE_ERR_UNSUPPORTED


# ---------------------------------------------------------------- BASE layer gate

def _base_ws(params):
    n = ctypes.c_size_t(12345)
    st = hm.load().moe_base_gate_workspace_size(ctypes.byref(params), ctypes.byref(n))
    return st, n.value


def _base_ws_formula(S, E, logits_in):
    nb = (S + 63) // 64
    return (_a256(nb * E * 4) + (0 if logits_in else _a256(S * E * 4)) + _a256(E * 8) + _a256(S * 8)
            + _a256(S * 4) + _a256(E * 4) + 2 * _a256(S * 4) + _a256(S * 8) + _a256(E * 4) + _a256(S * 4)
            + 256 + 256 + 3072)


def test_base_struct_and_workspace(lib):
    assert ctypes.sizeof(b.BaseParams) == 28 and b.BaseParams.max_rounds.offset == 24
    assert ctypes.sizeof(b.BaseInfo) == 16 and b.BaseInfo.eps.offset == 8
    assert lib.moe_status_string(b.MOE_ERR_NOT_CONVERGED) == b"MOE_ERR_NOT_CONVERGED"
    for S, d, E, li in [(32768, 2048, 64, 0), (32768, 0, 64, 1), (0, 16, 8, 0), (4096, 256, 1024, 0), (2048, 8, 1, 0)]:
        st, n = _base_ws(hm.base_params(S, d, E, max(1, S // E), li, b.MOE_BF16))
        assert st == 0, lib.moe_last_error()
        assert n == _base_ws_formula(S, E, li), (S, E, li)


BAD_BASE = [
    (dict(S=100, E=8), b.MOE_ERR_INVALID_ARG), (dict(E=0), b.MOE_ERR_INVALID_ARG),
    (dict(E=1025), b.MOE_ERR_INVALID_ARG), (dict(S=-64), b.MOE_ERR_INVALID_ARG),
    (dict(capacity=-1), b.MOE_ERR_INVALID_ARG), (dict(logits_in=2), b.MOE_ERR_INVALID_ARG),
    (dict(dtype=2), b.MOE_ERR_INVALID_ARG), (dict(max_rounds=-1), b.MOE_ERR_INVALID_ARG),
    (dict(d=0), b.MOE_ERR_INVALID_ARG), (dict(E=1024, capacity=1 << 21), b.MOE_ERR_INVALID_ARG),
    (dict(S=8 * 2049), b.MOE_ERR_UNSUPPORTED), (dict(d=6), b.MOE_ERR_UNSUPPORTED),
]


@pytest.mark.parametrize("bad,status", BAD_BASE)
def test_bad_base_params_rejected(lib, bad, status):
    base = dict(S=128, d=256, E=8, capacity=16, logits_in=0, dtype=0, max_rounds=0)
    base.update(bad)
    st, _ = _base_ws(hm.base_params(**base))
    assert st == status, (bad, lib.moe_last_error())
    assert lib.moe_last_error() != b""


def test_base_pointer_checks(lib):
    p = hm.base_params(128, 256, 8, 16, 0, b.MOE_F32)
    # moe_base_gate(p, x, wg, bias, logits, ids, slots, weights, counts, slot_src, prices, ws, wsb, info, stream)
    call = lambda prm=p, **kw: lib.moe_base_gate(
        ctypes.byref(prm), kw.get("x", A16), kw.get("wg", A16), kw.get("bias"), kw.get("logits"),
        kw.get("ids", A16), kw.get("slots", A16), kw.get("weights", A16), kw.get("counts", A16),
        kw.get("slot_src", A16), kw.get("prices"), kw.get("ws", A16), kw.get("wsb", 1 << 30), None, None)
    n = ctypes.c_size_t(0)
    assert lib.moe_base_gate_workspace_size(None, ctypes.byref(n)) == b.MOE_ERR_INVALID_ARG
    assert lib.moe_base_gate(None, *([None] * 11), 0, None, None) == b.MOE_ERR_INVALID_ARG
    assert call(prices=A16 + 4) == b.MOE_ERR_INVALID_ARG
    assert call(x=None) == b.MOE_ERR_INVALID_ARG
    assert call(x=A16 + 4) == b.MOE_ERR_UNSUPPORTED
    assert call(wg=None) == b.MOE_ERR_INVALID_ARG
    assert call(ids=None) == b.MOE_ERR_INVALID_ARG
    assert call(slot_src=None) == b.MOE_ERR_INVALID_ARG
    assert call(weights=A16 + 2) == b.MOE_ERR_INVALID_ARG
    assert call(ws=None) == b.MOE_ERR_WORKSPACE
    assert call(wsb=64) == b.MOE_ERR_WORKSPACE
    assert call(ws=A16 + 4) == b.MOE_ERR_WORKSPACE
    pl = hm.base_params(128, 0, 8, 16, 1, b.MOE_F32)
    assert call(pl, x=None, wg=None) == b.MOE_ERR_INVALID_ARG          # logits_in needs logits
    assert call(pl, logits=A16) == b.MOE_ERR_INVALID_ARG               # ... and no x / wg


def test_base_async_argument_checks(lib):
    """moe_base_gate_async: launch_rounds within [1, MOE_BASE_MAX_LAUNCH_ROUNDS]
    and an 8-byte aligned status are required; everything else is checked as
    for moe_base_gate.  All refused before any HIP call."""
    p = hm.base_params(128, 256, 8, 16, 0, b.MOE_F32)
    call = lambda prm=p, **kw: lib.moe_base_gate_async(
        ctypes.byref(prm), kw.get("x", A16), kw.get("wg", A16), None, None, A16, A16, A16, A16, A16, None,
        kw.get("ws", A16), kw.get("wsb", 1 << 30), kw.get("rounds", 64), kw.get("status", A16), None)
    for r in (0, -1, b.MOE_BASE_MAX_LAUNCH_ROUNDS + 1):
        assert call(rounds=r) == b.MOE_ERR_INVALID_ARG, r
        assert b"launch_rounds" in lib.moe_last_error()
    assert call(status=None) == b.MOE_ERR_INVALID_ARG
    assert call(status=A16 + 4) == b.MOE_ERR_INVALID_ARG
    assert call(x=None) == b.MOE_ERR_INVALID_ARG
    assert call(x=A16 + 4) == b.MOE_ERR_UNSUPPORTED
    assert call(ws=None) == b.MOE_ERR_WORKSPACE
    assert call(wsb=64) == b.MOE_ERR_WORKSPACE
    assert call(hm.base_params(100, 256, 8, 16, 0, b.MOE_F32)) == b.MOE_ERR_INVALID_ARG  # S not a multiple of E
    assert lib.moe_base_gate_async(None, *([None] * 10), None, 0, 64, A16, None) == b.MOE_ERR_INVALID_ARG
    # the header's limit is the binding's
    text = open(HEADER).read()
    assert f"#define MOE_BASE_MAX_LAUNCH_ROUNDS {b.MOE_BASE_MAX_LAUNCH_ROUNDS}" in text


# (call, argument names after the params struct, elements each needs) at
# S=100, d=64, E=8, k=2, C=30 (hash_vocab=5 for the gate; BASE: S=96, C=12)
_S, _d, _E, _k, _C = 100, 64, 8, 2, 30
_SIZES = {
    "moe_gate": (["x", "wg", "bias", "token_ids", "noise", "hash_table", "logits", "ids", "slots", "weights",
                  "counts", "demand", "slot_src", "workspace"],
                 [_S * _d, _d * _E, _E, _S, _S * _E, 5, _S * _E, _S * _k, _S * _k, _S * _k, _E, _E, _E * _C, 0]),
    "moe_dispatch": (["x", "ids", "slots", "slot_src", "xe"], [_S * _d, _S * _k, _S * _k, _E * _C, _E * _C * _d]),
    "moe_combine": (["ye", "ids", "slots", "weights", "y"], [_E * _C * _d, _S * _k, _S * _k, _S * _k, _S * _d]),
    "moe_dispatch_bwd": (["dxe", "ids", "slots", "dx"], [_E * _C * _d, _S * _k, _S * _k, _S * _d]),
    "moe_combine_bwd": (["dy", "ye", "ids", "slots", "slot_src", "weights", "dye", "dw"],
                        [_S * _d, _E * _C * _d, _S * _k, _S * _k, _E * _C, _S * _k, _E * _C * _d, _S * _k]),
    "moe_gate_bwd": (["x", "wg", "logits", "ids", "dw", "dlogits", "dx", "dwg", "dbias", "aux_loss", "workspace"],
                     [_S * _d, _d * _E, _S * _E, _S * _k, _S * _k, _S * _E, _S * _d, _d * _E, _E, 1, 0]),
    "moe_base_gate": (["x", "wg", "bias", "logits", "ids", "slots", "weights", "counts", "slot_src", "prices",
                       "workspace"], [96 * _d, _d * _E, _E, 96 * _E, 96, 96, 96, _E, _E * 12, _E, 0]),
}


def _params(call):
    if call == "moe_gate":
        return b.gate_params(_S, _d, _E, _k, _C, b.MOE_GATE_TOPK, hash_vocab=5)
    if call == "moe_gate_bwd":
        return b.gate_bwd_params(_S, _d, _E, _k, b.MOE_GATE_TOPK)
    if call == "moe_base_gate":
        return b.base_params(96, _d, _E, 12)
    return b.Layout(_S, _d, _E, _k, _C, b.MOE_F32)


@pytest.mark.parametrize("call", sorted(_SIZES))
def test_binding_rejects_short_buffers(call):
    """Every tensor argument of every call: one element short of the call's
    sizes is refused before any device work (the other arguments are None, so
    the check runs on a CPU tensor here); the right size passes the size check
    and is then refused for being on the CPU."""
    import torch
    names, sizes = _SIZES[call]
    fn = getattr(b, call)
    for pos, (name, n) in enumerate(zip(names, sizes)):
        if n == 0:
            continue
        args = [None] * len(names)
        args[pos] = torch.zeros(n - 1)
        with pytest.raises(ValueError, match=f"^{name} holds {n - 1} elements"):
            fn(_params(call), *args)
        args[pos] = torch.zeros(n)
        with pytest.raises(ValueError, match=f"^{name} must be on the GPU"):
            fn(_params(call), *args)
