"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic.  The same arrays feed the HIP library and the CPU oracle.

The paper's end-to-end runs use sequences of 1024 tokens, embedding width 2048,
16 experts and batches up to 32 (Sec. 4, overall performance).  The five
workloads below follow those shapes; the hash workload's token ids are drawn
from a Zipf(1.1) law over a 50257-entry BPE vocabulary as a stand-in for
natural-text token frequencies.  No dataset is used.

Host arrays use "storage" form: float32 arrays for fp32, uint16 bit patterns
for bf16 (rounded from float32 draws to nearest-even by torch's CPU cast).
"""

import numpy as np
import torch

TOPK, KTOP1, HASH = 0, 1, 2

# Capacities follow C = ceil(cf * k * S / E); they are listed, not computed here.
WORKLOADS = {
    1: dict(name="switch_top1_fp32_S1024_d256_E8_cf1.0", kind=TOPK, k=1, normalize=0, dtype="f32",
            S=1024, d=256, E=8, cf=1.0, C=128),
    2: dict(name="gshard_top2_bf16_S8192_d1024_E16_cf1.25", kind=TOPK, k=2, normalize=1, dtype="bf16",
            S=8192, d=1024, E=16, cf=1.25, C=1280),
    3: dict(name="switch_top1_hotbias_bf16_S32768_d2048_E64_cf1.0", kind=TOPK, k=1, normalize=0, dtype="bf16",
            S=32768, d=2048, E=64, cf=1.0, C=512, hot_experts=4, hot_bias=1.10),
    4: dict(name="ktop1_4x16_bf16_S32768_d2048_E64_cf1.25", kind=KTOP1, k=4, normalize=0, dtype="bf16",
            S=32768, d=2048, E=64, cf=1.25, C=2560),
    5: dict(name="hash_zipf1.1_bf16_S65536_d4096_E128_cf2.0", kind=HASH, k=1, normalize=0, dtype="bf16",
            S=65536, d=4096, E=128, cf=2.0, C=1024, vocab=50257, zipf_a=1.1),
}


def f32_to_storage(a, dtype):
    """float32 array -> storage form (bf16 via torch's round-to-nearest-even cast)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    return torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def zipf_token_ids(S, vocab, a, seed):
    """S token ids with P(id = r - 1) proportional to r^-a, r = 1..vocab."""
    ranks = np.arange(1, vocab + 1, dtype=np.float64)
    p = ranks ** (-a)
    p /= p.sum()
    return np.random.default_rng(seed).choice(vocab, size=S, p=p).astype(np.int32)


def make_inputs(w, S=None, d=None, E=None, seed=0):
    """Forward inputs of workload dict `w` (optionally resized).  Returns a dict
    of host arrays: x, wg, bias, token_ids (absent entries are None)."""
    S = w["S"] if S is None else S
    d = w["d"] if d is None else d
    E = w["E"] if E is None else E
    dt = w["dtype"]
    out = dict(x=None, wg=None, bias=None, token_ids=None)
    if w["kind"] == HASH:
        out["token_ids"] = zipf_token_ids(S, w["vocab"], w["zipf_a"], seed)
        x = np.random.default_rng(seed + 1).standard_normal((S, d), dtype=np.float32)
        out["x"] = f32_to_storage(x, dt)
        return out
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((S, d), dtype=np.float32)
    wg = rng.standard_normal((d, E), dtype=np.float32) / np.float32(np.sqrt(d))
    out["x"] = f32_to_storage(x, dt)
    out["wg"] = f32_to_storage(wg, dt)
    if w.get("hot_experts"):
        bias = np.zeros(E, dtype=np.float32)
        bias[: w["hot_experts"]] = np.float32(w["hot_bias"])
        out["bias"] = bias
    return out


def make_rows(shape, dtype, seed):
    """N(0, 1) rows in storage form (gradients, expert outputs)."""
    a = np.random.default_rng(seed).standard_normal(shape, dtype=np.float32)
    return f32_to_storage(a, dtype)


def to_device(a, dtype, device="cuda"):
    """Host storage array -> contiguous torch tensor on `device`."""
    if a is None:
        return None
    if a.dtype == np.uint16:
        assert dtype == "bf16"
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device).contiguous()
    return torch.from_numpy(np.ascontiguousarray(a)).to(device).contiguous()


def to_host(t):
    """torch tensor -> host storage array (bf16 as uint16 bits)."""
    if t is None:
        return None
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
