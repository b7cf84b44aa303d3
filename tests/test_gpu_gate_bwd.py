"""GPU parity of the gate backward (moe_gate_bwd, through the C ABI) against
the CPU oracle (oracle/gate_bwd.py).

Stage by stage, as for the forward gate: dL is compared with the oracle's dL
from the same fp32 logits; dW, db and dx are compared with the oracle fed the
GPU's own dL (so each stage's arithmetic is checked on its own); an end-to-end
bound then checks dW and dx against the oracle's dL as well.  Floats:
|gpu - oracle| <= rtol * M with M the sum of |terms|, rtol 1e-5 for fp32 outputs
and 2e-2 for bf16 outputs."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2203_14685_amd as hm
from paper_2203_14685_amd import workloads as wl

from _parity import RTOL, announce, assert_close, assert_equal, decode

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hm.load()
    yield


def _inputs(S, d, E, k, kind, dtype, seed, drop=0.2):
    rng = np.random.default_rng(seed)
    L = (rng.standard_normal((S, E)) * 1.5).astype(np.float32)
    ids = oracle.select(L, kind, k) if S > 0 else np.zeros((0, k), dtype=np.int32)
    dw = rng.standard_normal((S, k)).astype(np.float32)
    dw[rng.random((S, k)) < drop] = 0.0   # dropped choices carry no gradient
    x = wl.f32_to_storage(rng.standard_normal((S, d)).astype(np.float32), dtype)
    wg = wl.f32_to_storage((rng.standard_normal((d, E)) / math.sqrt(d)).astype(np.float32), dtype)
    dx_in = wl.f32_to_storage(rng.standard_normal((S, d)).astype(np.float32), dtype)
    return L, ids, dw, x, wg, dx_in


def run_case(S, d, E, k, kind, normalize, dtype, aux=0.0, accumulate=False, seed=0, end_to_end=True):
    L, ids, dw, x, wg, dx_in = _inputs(S, d, E, k, kind, dtype, seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dx_dev = wl.to_device(dx_in, dtype) if accumulate else None
    out = hm.gate_bwd(kind, wl.to_device(L, "f32"), wl.to_device(ids, "i32"), wl.to_device(dw, "f32"),
                      x=wl.to_device(x, dtype), wg=wl.to_device(wg, dtype), normalize=normalize, dx=dx_dev,
                      accumulate_dx=accumulate, aux_coef=aux)
    torch.cuda.synchronize()
    g = {key: (wl.to_host(v) if v is not None else None) for key, v in out.items()}
    assert out["dx"].dtype == tdt
    stats = {}
    # stage 1: dL
    dL_ref, M = oracle.gate_dlogits(L, ids, dw, kind, normalize)
    if aux:
        loss_ref, dLa, Ma, _, _ = oracle.aux_loss(L, ids, aux)
        dL_ref, M = dL_ref + dLa, M + Ma
        stats["aux_err"] = assert_close(g["aux_loss"], np.array([loss_ref]), np.array([abs(loss_ref)]), RTOL["f32"], "aux loss")
    stats["dl_err"] = assert_close(g["dlogits"], dL_ref, M, RTOL["f32"], "dlogits")
    # stage 2: dW, db, dx from the GPU's dL
    ref = oracle.gate_input_grads(x, wg, g["dlogits"], dtype, dx_in=dx_in if accumulate else None)
    stats["dwg_err"] = assert_close(g["dwg"], ref["dwg"], ref["dwg_mag"], RTOL["f32"], "dwg")
    stats["dbias_err"] = assert_close(g["dbias"], ref["dbias"], ref["dbias_mag"], RTOL["f32"], "dbias")
    rt = RTOL[dtype]
    stats["dx_err"] = assert_close(decode(g["dx"], dtype), decode(ref["dx"], dtype), ref["dx_mag"], rt, "dx")
    if end_to_end and S > 0:
        # the oracle's own dL: the GPU's dL differs by at most rtol * M per element
        e2e = oracle.gate_input_grads(x, wg, dL_ref, dtype, dx_in=dx_in if accumulate else None)
        xa = np.abs(decode(x, dtype))
        wa = np.abs(decode(wg, dtype))
        dwg_bound = RTOL["f32"] * (e2e["dwg_mag"] + xa.T @ M)
        assert (np.abs(g["dwg"] - e2e["dwg"]) <= dwg_bound).all(), "dwg end to end"
        dx_bound = rt * e2e["dx_mag"] + RTOL["f32"] * (M @ wa.T)
        assert (np.abs(decode(g["dx"], dtype) - decode(e2e["dx"], dtype)) <= dx_bound).all(), "dx end to end"
    return stats


CASES = [
    # (S, d, E, k, kind, normalize, dtype, aux, accumulate)
    (1000, 256, 8, 1, 0, 0, "f32", 0.01, False),        # Switch, fp32
    (3000, 1024, 16, 2, 0, 1, "bf16", 0.0, True),       # GShard top-2, dx accumulated
    (1000, 2048, 64, 4, 1, 0, "bf16", 0.0, False),      # kTop1 4 x 16
    (2500, 2048, 64, 1, 0, 0, "bf16", 0.01, True),      # Switch + balance loss
    (130, 132, 5, 3, 0, 1, "f32", 0.0, False),          # odd E and d
    (200, 64, 1024, 8, 0, 0, "f32", 0.05, False),       # 16 experts per lane
    (333, 128, 200, 2, 0, 1, "bf16", 0.0, True),        # E not a power of two
    (77, 512, 24, 3, 1, 0, "bf16", 0.0, False),         # kTop1 3 x 8
    (500, 256, 16, 4, 1, 0, "f32", 0.0, False),         # kTop1 4 x 4: groups of one lane set (P = 4)
    (600, 128, 32, 4, 1, 0, "bf16", 0.0, True),         # kTop1 4 x 8: groups of one lane set (P = 8)
    (1, 256, 8, 2, 0, 1, "f32", 0.0, True),
    (4100, 512, 32, 1, 0, 0, "f32", 0.1, False),        # several token ranges for dW
    # matrix-core dW: blocks of 256 columns with waves past d, 2..8 expert tiles
    (700, 320, 32, 2, 0, 1, "bf16", 0.0, True),         # d = 320: second block has one live wave
    (130, 448, 48, 1, 0, 0, "bf16", 0.01, False),       # 3 tiles, fewer than 4 chunks per range
    (900, 64, 80, 3, 0, 1, "bf16", 0.0, True),          # d = 64: one live wave per block
    (1500, 192, 128, 2, 0, 1, "bf16", 0.0, False),      # E = 128, one wave per SIMD
    # first-choice counts past one block's batch (several count blocks), and a
    # balance loss over more experts than one block of column sums holds
    (70000, 64, 16, 1, 0, 0, "bf16", 0.02, False),
    (66000, 128, 96, 2, 0, 1, "bf16", 0.03, True),
    # matrix-core dW over 47 token ranges with a ragged batch, and over 64
    # ranges at E = 32
    (12000, 1024, 16, 2, 0, 1, "bf16", 0.0, True),
    (16400, 512, 32, 1, 0, 0, "bf16", 0.01, True),
]


@pytest.mark.parametrize("S,d,E,k,kind,normalize,dtype,aux,acc", CASES)
def test_gate_bwd_parity(S, d, E, k, kind, normalize, dtype, aux, acc):
    announce(f"gate bwd S={S} d={d} E={E} k={k} kind={kind} normalize={normalize} {dtype} aux={aux} acc={acc}")
    st = run_case(S, d, E, k, kind, normalize, dtype, aux, acc, seed=S + E + k)
    print(f"[stats] gate bwd S={S} E={E}: {st}", flush=True)


@pytest.mark.parametrize("wid", [2, 3, 4])
def test_gate_bwd_full_size(wid):
    w = wl.WORKLOADS[wid]
    announce(f"gate bwd full size workload {wid}")
    aux = 0.01 if w["kind"] == 0 else 0.0
    st = run_case(w["S"], w["d"], w["E"], w["k"], w["kind"], w["normalize"], w["dtype"], aux, True, seed=wid,
                  end_to_end=False)
    print(f"[stats] gate bwd workload {wid}: {st}", flush=True)


def test_gate_bwd_empty_batch_and_partial_outputs():
    announce("gate bwd S=0 and partial outputs")
    E, d = 8, 64
    z = torch.zeros((0, E), dtype=torch.float32, device="cuda")
    zi = torch.zeros((0, 2), dtype=torch.int32, device="cuda")
    zw = torch.zeros((0, 2), dtype=torch.float32, device="cuda")
    x = torch.zeros((0, d), dtype=torch.float32, device="cuda")
    wg = torch.ones((d, E), dtype=torch.float32, device="cuda")
    out = hm.gate_bwd(0, z, zi, zw, x=x, wg=wg, normalize=0, aux_coef=0.5)
    torch.cuda.synchronize()
    assert (out["dwg"] == 0).all() and (out["dbias"] == 0).all() and out["aux_loss"].item() == 0.0
    # only dbias: x may be absent; dL kept in the workspace
    L, ids, dw, x, wg, _ = _inputs(300, 64, 8, 2, 0, "f32", 3)
    out = hm.gate_bwd(0, wl.to_device(L, "f32"), wl.to_device(ids, "i32"), wl.to_device(dw, "f32"), normalize=1,
                      want_dlogits=False, want_dwg=False, want_dx=False)
    torch.cuda.synchronize()
    dL, M = oracle.gate_dlogits(L, ids, dw, 0, 1)
    assert out["dwg"] is None and out["dx"] is None
    assert_close(wl.to_host(out["dbias"]), dL.sum(axis=0), np.abs(M).sum(axis=0) + np.abs(dL).sum(axis=0),
                 RTOL["f32"], "dbias only")


def test_gate_bwd_bitwise_repeatable():
    announce("gate bwd determinism")
    L, ids, dw, x, wg, dx_in = _inputs(5000, 512, 64, 2, 0, "bf16", 9)
    args = (0, wl.to_device(L, "f32"), wl.to_device(ids, "i32"), wl.to_device(dw, "f32"))
    kw = dict(x=wl.to_device(x, "bf16"), wg=wl.to_device(wg, "bf16"), normalize=1, aux_coef=0.02)
    a = hm.gate_bwd(*args, **kw)
    b = hm.gate_bwd(*args, **kw)
    torch.cuda.synchronize()
    for key in ("dlogits", "dwg", "dbias", "dx", "aux_loss"):
        assert_equal(wl.to_host(a[key]), wl.to_host(b[key]), key)
