"""GPU parity of the further gates of Sec. 3.1 (through the C ABI) against the
oracle: hierarchical top-k (R19), Dense-To-Sparse noisy tempered logits (R20)
and the Hash Layer's balanced table (R21), their routing through the capacity
and layout steps, and the gate gradient for them.  Integer routing bit-exact;
floats within rtol * (sum of |terms|)."""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2203_14685_amd as hm
from paper_2203_14685_amd import workloads as wl

from _parity import RTOL, announce, assert_close, assert_equal, check_gate, check_layout_ops, gpu_gate

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hm.load()
    yield


def cap(cf, k, S, E):
    return int(math.ceil(cf * k * S / E))


def gumbel(shape, seed):
    u = np.random.default_rng(seed).random(shape)
    return (-np.log(-np.log(u))).astype(np.float32)


@pytest.mark.parametrize("dtype,S,d,E,groups,k,normalize,bias", [
    ("bf16", 1000, 2048, 64, 4, 2, 1, True), ("bf16", 700, 1024, 64, 8, 4, 0, False),
    ("f32", 517, 256, 16, 2, 3, 1, False), ("bf16", 300, 512, 48, 3, 8, 0, True),
    ("f32", 130, 132, 6, 3, 2, 1, False), ("bf16", 65, 256, 128, 16, 8, 1, False), ("f32", 64, 64, 12, 1, 4, 0, False),
    # selection inside the register-resident projection (four waves)
    ("bf16", 3000, 2048, 64, 4, 1, 0, True), ("bf16", 20000, 1024, 128, 8, 4, 1, False),
    ("bf16", 333, 2048, 32, 2, 8, 0, True),
])
def test_htopk_projection(dtype, S, d, E, groups, k, normalize, bias):
    announce(f"htopk dtype={dtype} S={S} d={d} E={E} groups={groups} k={k} normalize={normalize}")
    w = dict(kind=0, k=k, normalize=normalize, dtype=dtype, S=S, d=d, E=E, cf=1.0)
    if bias:
        w.update(hot_experts=3, hot_bias=0.75)
    inp = wl.make_inputs(w, seed=E + groups + k)
    C = cap(1.0, k, S, E)
    g = gpu_gate(w, inp, E, k, C, hm.MOE_GATE_HTOPK, normalize, groups=groups)
    ref, st = check_gate(w, inp, g, E, k, C, hm.MOE_GATE_HTOPK, normalize, groups=groups)
    Gs = E // groups
    assert (g["ids"] // Gs == g["ids"][:, :1] // Gs).all()
    st.update(check_layout_ops(w, inp["x"], g["ids"], g["slots"], g["weights"], g["slot_src"], E, C, k, seed=3))
    print(f"[stats] htopk E={E} groups={groups}: {st}", flush=True)


@pytest.mark.parametrize("E,groups,k,normalize", [(8, 2, 2, 1), (12, 4, 3, 0), (64, 8, 4, 1), (6, 3, 1, 0)])
def test_htopk_dense_ties(E, groups, k, normalize):
    announce(f"htopk ties E={E} groups={groups} k={k}")
    S = 777
    L = np.random.default_rng(E + k).integers(0, 3, (S, E)).astype(np.float32)
    C = cap(1.25, k, S, E)
    w = dict(dtype="f32")
    g = gpu_gate(w, None, E, k, C, hm.MOE_GATE_HTOPK, normalize, logits=L, groups=groups)
    check_gate(w, None, g, E, k, C, hm.MOE_GATE_HTOPK, normalize, logits_in=L, groups=groups)


@pytest.mark.parametrize("kind,k,normalize,groups,tau,dtype,E", [
    (0, 2, 0, 0, 0.5, "bf16", 64), (0, 1, 0, 0, 2.0, "f32", 16), (1, 4, 0, 0, 0.7, "bf16", 64),
    (3, 2, 1, 4, 0.3, "bf16", 32), (0, 3, 1, 0, 1.0, "f32", 5),
])
def test_dense_to_sparse_projection(kind, k, normalize, groups, tau, dtype, E):
    announce(f"dense-to-sparse kind={kind} k={k} tau={tau} {dtype} E={E}")
    S, d = 600, 512 if dtype == "bf16" else 260
    w = dict(kind=kind, k=k, normalize=normalize, dtype=dtype, S=S, d=d, E=E, cf=1.25)
    inp = wl.make_inputs(w, seed=11 + k)
    noise = gumbel((S, E), 21 + k)
    C = cap(1.25, k, S, E)
    g = gpu_gate(w, inp, E, k, C, kind, normalize, groups=groups, noise=noise, temperature=tau)
    _, st = check_gate(w, inp, g, E, k, C, kind, normalize, groups=groups, noise=noise, temperature=tau)
    print(f"[stats] dense-to-sparse kind={kind}: {st}", flush=True)


@pytest.mark.parametrize("kind,k,normalize,groups,tau,E,d,S", [
    (1, 4, 0, 0, 0.5, 64, 2048, 5000), (0, 1, 0, 0, 0.5, 64, 2048, 20000), (3, 2, 1, 4, 0.3, 128, 1024, 700),
    (0, 8, 1, 0, 1.5, 32, 2048, 257),
])
def test_dense_to_sparse_register_kernel(kind, k, normalize, groups, tau, E, d, S):
    """Shapes whose projection keeps W in registers (four waves): noise,
    temperature and selection run in the projection kernel's epilogue."""
    announce(f"dense-to-sparse in the projection kind={kind} k={k} tau={tau} E={E} d={d} S={S}")
    w = dict(kind=kind, k=k, normalize=normalize, dtype="bf16", S=S, d=d, E=E, cf=1.25)
    inp = wl.make_inputs(w, seed=5 + k + E)
    noise = gumbel((S, E), 31 + k)
    C = cap(1.25, k, S, E)
    g = gpu_gate(w, inp, E, k, C, kind, normalize, groups=groups, noise=noise, temperature=tau)
    _, st = check_gate(w, inp, g, E, k, C, kind, normalize, groups=groups, noise=noise, temperature=tau)
    print(f"[stats] dense-to-sparse in the projection kind={kind} E={E}: {st}", flush=True)


@pytest.mark.parametrize("kind,k,groups", [(0, 2, 0), (3, 3, 2), (1, 2, 0)])
def test_dense_to_sparse_given_logits(kind, k, groups):
    """With the raw logits given, the selection sees (L + g) / tau in fp32."""
    announce(f"dense-to-sparse logits_in kind={kind}")
    S, E, tau = 999, 16, 0.25
    L = (np.random.default_rng(5).standard_normal((S, E)) * 2).astype(np.float32)
    noise = gumbel((S, E), 6)
    C = cap(1.0, k, S, E)
    w = dict(dtype="f32")
    g = gpu_gate(w, None, E, k, C, kind, 0, logits=L, groups=groups, noise=noise, temperature=tau)
    check_gate(w, None, g, E, k, C, kind, 0, logits_in=oracle.noisy_logits_f32(L, noise, tau), groups=groups)


@pytest.mark.parametrize("S,E", [(3000, 128), (65536, 128), (5000, 7)])
def test_balanced_hash_table(S, E):
    announce(f"balanced hash S={S} E={E}")
    w = wl.WORKLOADS[5]
    ranks = np.arange(1, w["vocab"] + 1, dtype=np.float64)
    p = ranks ** -w["zipf_a"]
    p /= p.sum()
    table = hm.moe_hash_balanced_table(p, E)
    tok = wl.zipf_token_ids(S, w["vocab"], w["zipf_a"], seed=2)
    C = cap(2.0, 1, S, E)
    inp = dict(token_ids=tok)
    g = gpu_gate(dict(dtype="bf16"), inp, E, 1, C, hm.MOE_GATE_HASH, 0, hash_table=table)
    assert_equal(g["ids"][:, 0], table[tok], "ids = table[token]")
    check_gate(dict(dtype="bf16"), inp, g, E, 1, C, hm.MOE_GATE_HASH, 0, hash_table=table)
    # the balanced table spreads this batch better than the random hash does
    gr = gpu_gate(dict(dtype="bf16"), inp, E, 1, C, hm.MOE_GATE_HASH, 0)
    if E > 8:
        assert g["demand"].max() <= gr["demand"].max()


@pytest.mark.parametrize("kind,k,normalize,groups,tau,aux", [
    (3, 2, 1, 4, 0.0, 0.01), (3, 3, 0, 2, 0.0, 0.0), (0, 2, 0, 0, 0.5, 0.02), (1, 4, 0, 0, 0.7, 0.0),
])
def test_gate_bwd_htopk_and_temperature(kind, k, normalize, groups, tau, aux):
    announce(f"gate bwd kind={kind} groups={groups} tau={tau} aux={aux}")
    S, d, E = 2000, 1024, 64
    rng = np.random.default_rng(k + groups)
    L = (rng.standard_normal((S, E)) * 1.5).astype(np.float32)
    ids = oracle.select(L.astype(np.float64), kind, k, groups)
    dw = rng.standard_normal((S, k)).astype(np.float32)
    x = wl.f32_to_storage(rng.standard_normal((S, d)).astype(np.float32), "bf16")
    wg = wl.f32_to_storage((rng.standard_normal((d, E)) / 32).astype(np.float32), "bf16")
    out = hm.gate_bwd(kind, wl.to_device(L, "f32"), wl.to_device(ids, "i32"), wl.to_device(dw, "f32"),
                      x=wl.to_device(x, "bf16"), wg=wl.to_device(wg, "bf16"), normalize=normalize, aux_coef=aux,
                      temperature=tau)
    torch.cuda.synchronize()
    dL_ref, M = oracle.gate_dlogits(L, ids, dw, kind, normalize, temperature=tau)
    if aux:
        _, dLa, Ma, _, _ = oracle.aux_loss(L, ids, aux)
        t = float(np.float32(tau)) if tau else 1.0
        dL_ref, M = dL_ref + dLa / t, M + Ma / t
    assert_close(wl.to_host(out["dlogits"]), dL_ref, M, RTOL["f32"], "dlogits")
    gi = oracle.gate_input_grads(x, wg, wl.to_host(out["dlogits"]), "bf16")
    assert_close(wl.to_host(out["dwg"]), gi["dwg"], gi["dwg_mag"], RTOL["f32"], "dwg")
    assert_close(oracle.decode(wl.to_host(out["dx"]), "bf16"), oracle.decode(gi["dx"], "bf16"), gi["dx_mag"],
                 RTOL["bf16"], "dx")
