"""Oracle for step 1 of Algorithm 1: the gate, and the capacity slot assignment.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Steps, each in the paper's order:

* logits      -- x . W of Eq. 1 (Sec. 3.1), plus an optional per-expert bias.
* select      -- which experts each token goes to: TopK of Eq. 1, kTop1
                 (Sec. 3.1, expert prototyping), or a hash (Sec. 3.1, Hash Layer).
* gate_weights-- the softmax of Eq. 1 (and its readings for Switch and kTop1).
* assign_slots-- the expert capacity of Sec. 3.1 (GShard/Switch capacity factor):
                 each expert keeps at most C tokens; the rest are dropped.

Readings taken where the paper is silent (numbered as in the rest of the oracle):

R1  Eq. 1 normalises over the K selected logits (``normalize=1``).  For the
    Switch gate (K=1) that would make every weight 1, so ``normalize=0`` gives
    the full-softmax probability of the chosen expert instead.  Selection is on
    the logits either way.
R2  capacity C = ceil(cf * k * S / E).
R3  slots are handed out rank-major: every token's first choice, in token
    order, then every token's second choice, and so on.
R4  ties: the larger logit wins; on equal logits the lower expert index wins.
R5  a dropped assignment contributes nothing; weights are not renormalised.
R8  kTop1 groups are contiguous, [g*E/k, (g+1)*E/k); softmax within each group.
R9  hash: H(t) is output number t+1 of a SplitMix64 generator seeded with
    ``seed`` (Steele, Lea & Flood, OOPSLA 2014); expert = H(t) mod E; weight 1.
R19 hierarchical top-k (Sec. 3.1, H Topk / SAM): experts form G contiguous
    groups; the switch step picks the group holding the best expert, the
    mixture step the k best experts inside that group; weights as for TopK.
R20 Dense-To-Sparse (Sec. 3.1): the gate acts on (L + g) / tau, g a Gumbel
    sample given as input and tau the temperature, evaluated in fp32 (one
    rounded addition, one rounded division) so that selection on it is exact.
R21 balanced hash (Sec. 3.1, Hash Layer, balanced assignment): tokens in order
    of decreasing frequency (ties: lower id) each go to the expert with the
    smallest load so far (ties: lower index); the load is the summed frequency.
"""

import math

import numpy as np

from .bf16 import decode

GATE_TOPK = 0
GATE_KTOP1 = 1
GATE_HASH = 2
GATE_HTOPK = 3

_MASK64 = (1 << 64) - 1
# SplitMix64 constants as published by Steele, Lea & Flood (OOPSLA 2014) and in
# Vigna's public-domain reference: the odd "golden gamma" increment and the two
# multipliers of the output mixing function (David Stafford's "Mix13" variant).
_SM64_GAMMA = 0x9E3779B97F4A7C15
_SM64_M1 = 0xBF58476D1CE4E5B9
_SM64_M2 = 0x94D049BB133111EB


def capacity(cf, k, S, E):
    """Expert capacity (reading R2 of the capacity-factor sentence, Sec. 3.1)."""
    return int(math.ceil(cf * k * S / E))


def logits(x, wg, dtype, bias=None):
    """Gate logits L = x . W (+ bias), Eq. 1, in fp64.

    x: [S, d] and wg: [d, E] in storage ``dtype`` ("f32" float32 or "bf16" uint16
    bits); bias: [E] float32 or None.  Returns (L, A) where A[s, e] =
    sum_j |x[s, j] * wg[j, e]| is the magnitude of the terms of each dot product
    (used for error bounds).  The matrix product is the library step.
    """
    x64 = decode(x, dtype)
    w64 = decode(wg, dtype)
    L = x64 @ w64
    A = np.abs(x64) @ np.abs(w64)
    if bias is not None:
        b64 = np.asarray(bias, dtype=np.float32).astype(np.float64)
        L = L + b64[None, :]
        A = A + np.abs(b64)[None, :]
    return L, A


def _key(row, e):
    # Order of experts for one token (reading R4): larger logit first, then
    # lower expert index.
    return (-row[e], e)


def select(L, kind, k, groups=0):
    """Chosen experts per token: ids[S, k] int32 (TopK of Eq. 1, kTop1 or H Topk).

    TOPK : ids[s, r] is the r-th expert in key order (rank 0 is the best).
    KTOP1: ids[s, g] is the best expert of group g = [g*E/k, (g+1)*E/k)
           (Sec. 3.1, kTop1: experts split into k prototypes, top-1 in each).
    HTOPK: with ``groups`` contiguous groups of E/groups experts, the group of
           the best expert, then its k best experts in key order (R19).
    """
    L = np.asarray(L, dtype=np.float64)
    S, E = L.shape
    ids = np.empty((S, k), dtype=np.int32)
    if kind == GATE_TOPK:
        if not 1 <= k <= E:
            raise ValueError("TOPK needs 1 <= k <= E")
        for s in range(S):
            row = L[s]
            order = sorted(range(E), key=lambda e: _key(row, e))
            ids[s, :] = order[:k]
    elif kind == GATE_HTOPK:
        if groups < 1 or E % groups != 0 or not 1 <= k <= E // groups:
            raise ValueError("HTOPK needs E % groups == 0 and 1 <= k <= E / groups")
        Gs = E // groups
        for s in range(S):
            row = L[s]
            best = min(range(E), key=lambda e: _key(row, e))
            g = best // Gs
            order = sorted(range(g * Gs, (g + 1) * Gs), key=lambda e: _key(row, e))
            ids[s, :] = order[:k]
    elif kind == GATE_KTOP1:
        if E % k != 0:
            raise ValueError("KTOP1 needs E % k == 0")
        G = E // k
        for s in range(S):
            row = L[s]
            for g in range(k):
                ids[s, g] = min(range(g * G, (g + 1) * G), key=lambda e: _key(row, e))
    else:
        raise ValueError("select() handles TOPK and KTOP1; use hash_ids() for HASH")
    return ids


def gate_weights(L, ids, kind, normalize):
    """Gate weight of each chosen expert, float64 [S, k] (softmax of Eq. 1).

    TOPK, normalize=1: softmax over the k selected logits (Eq. 1 as printed).
    TOPK, normalize=0: full softmax over all E experts, read at the chosen one
                       (reading R1, the Switch gate).
    HTOPK            : as TOPK (the chosen experts come from one group, R19).
    KTOP1            : softmax within the chosen expert's group (reading R8).
    HASH             : 1.
    Every softmax subtracts the maximum of the logits it normalises over; the
    result is the same function, evaluated without overflow.
    """
    ids = np.asarray(ids)
    S, k = ids.shape
    if kind == GATE_HASH:
        return np.ones((S, k), dtype=np.float64)
    L = np.asarray(L, dtype=np.float64)
    E = L.shape[1]
    rows = np.arange(S)[:, None]
    chosen = L[rows, ids]                      # [S, k]
    if kind == GATE_HTOPK:
        kind = GATE_TOPK
    if kind == GATE_TOPK and normalize:
        m = chosen.max(axis=1, keepdims=True)
        num = np.exp(chosen - m)
        return num / num.sum(axis=1, keepdims=True)
    if kind == GATE_TOPK:
        m = L.max(axis=1, keepdims=True)
        den = np.exp(L - m).sum(axis=1, keepdims=True)
        return np.exp(chosen - m) / den
    if kind == GATE_KTOP1:
        G = E // k
        w = np.empty((S, k), dtype=np.float64)
        for g in range(k):
            grp = L[:, g * G:(g + 1) * G]
            m = grp.max(axis=1)
            den = np.exp(grp - m[:, None]).sum(axis=1)
            w[:, g] = np.exp(chosen[:, g] - m) / den
        return w
    raise ValueError(f"unknown gate kind {kind}")


def splitmix64_output(seed, n):
    """Output number n (n >= 1) of SplitMix64 seeded with ``seed``.

    The generator adds the gamma constant to its 64-bit state and returns the
    mixed state; after n steps the state is seed + n * gamma (mod 2^64).  The
    mixing function is two xor-shift-multiply rounds and a final xor-shift.
    """
    z = (seed + n * _SM64_GAMMA) & _MASK64
    z = ((z ^ (z >> 30)) * _SM64_M1) & _MASK64
    z = ((z ^ (z >> 27)) * _SM64_M2) & _MASK64
    return z ^ (z >> 31)


def hash_ids(token_ids, E, seed):
    """Hash gate (Sec. 3.1, Hash Layer, random hash; reading R9): ids[S, 1].

    Token t goes to bucket H(t) mod E, H(t) = SplitMix64 output number t+1.
    """
    token_ids = np.asarray(token_ids)
    out = np.empty((token_ids.shape[0], 1), dtype=np.int32)
    for s, t in enumerate(token_ids.tolist()):
        out[s, 0] = splitmix64_output(int(seed), int(t) + 1) % E
    return out


def noisy_logits_f32(L, noise, temperature):
    """Dense-To-Sparse logits (R20): (L + g) / tau in fp32, each operation rounded
    to nearest; L, noise float32 [S, E] (noise may be None), tau > 0."""
    L = np.asarray(L, dtype=np.float32)
    v = L if noise is None else (L + np.asarray(noise, dtype=np.float32)).astype(np.float32)
    return (v / np.float32(temperature)).astype(np.float32)


def balanced_hash_table(freq, E):
    """Balanced assignment of token ids to E experts (R21): table[vocab] int32."""
    freq = [float(f) for f in freq]
    order = sorted(range(len(freq)), key=lambda t: (-freq[t], t))
    load = [0.0] * E
    table = np.empty(len(freq), dtype=np.int32)
    for t in order:
        e = min(range(E), key=lambda i: (load[i], i))
        table[t] = e
        load[e] += freq[t]
    return table


def table_hash_ids(token_ids, table):
    """Hash gate with a lookup table (Sec. 3.1, Hash Layer): ids[S, 1] = table[t]."""
    table = np.asarray(table)
    return table[np.asarray(token_ids)].astype(np.int32).reshape(-1, 1)


def assign_slots(ids, E, C):
    """Capacity-limited position of every (token, rank) in its expert's buffer.

    Expert capacity (Sec. 3.1, next to Eq. 1) caps how many tokens an expert
    receives; the layout transform (Algorithm 1, step 2) then needs each kept
    token's position inside its expert's contiguous buffer.  Order (R3, R4):
    rank-major, then token order.  Returns
      slots[S, k]    int32: position in the expert's buffer, -1 if dropped;
      counts[E]      int32: tokens kept per expert (<= C);
      demand[E]      int32: tokens routed to each expert before the cap;
      slot_src[E, C] int32: s*k + r of the assignment held in each slot, -1 if empty.
    """
    ids = np.asarray(ids)
    S, k = ids.shape
    slots = np.full((S, k), -1, dtype=np.int32)
    slot_src = np.full((E, C), -1, dtype=np.int32)
    cnt = [0] * E
    for r in range(k):
        for s in range(S):
            e = int(ids[s, r])
            if cnt[e] < C:
                slots[s, r] = cnt[e]
                slot_src[e, cnt[e]] = s * k + r
            cnt[e] += 1
    demand = np.array(cnt, dtype=np.int32)
    counts = np.minimum(demand, C).astype(np.int32)
    return slots, counts, demand, slot_src


def gate(kind, k, E, C, normalize=0, dtype="f32", x=None, wg=None, bias=None,
         token_ids=None, hash_seed=0, sel_logits=None, groups=0, noise=None, temperature=0.0,
         hash_table=None):
    """Step 1 of Algorithm 1 end to end: logits -> selection -> weights -> slots.

    ``sel_logits`` (float array [S, E]) overrides the logits used for selection
    and weights; the parity tests pass the device's own fp32 logits here so that
    integer routing can be compared bit for bit.  With ``temperature`` > 0 the
    computed logits are made Dense-To-Sparse logits (R20; in fp64 here, for the
    tolerance check of the device's values).  Returns a dict.
    """
    out = {}
    if kind == GATE_HASH:
        if hash_table is not None:
            ids = table_hash_ids(token_ids, hash_table)
        else:
            ids = hash_ids(token_ids, E, hash_seed)
        w = gate_weights(None, ids, GATE_HASH, 0)
    else:
        if sel_logits is None:
            L, A = logits(x, wg, dtype, bias)
            if temperature > 0:
                g = 0.0 if noise is None else np.asarray(noise, dtype=np.float32).astype(np.float64)
                L, A = (L + g) / float(np.float32(temperature)), (A + np.abs(g)) / float(np.float32(temperature))
            out["logits"], out["logits_mag"] = L, A
            sel = L
        else:
            sel = np.asarray(sel_logits, dtype=np.float64)
        ids = select(sel, kind, k, groups)
        w = gate_weights(sel, ids, kind, normalize)
    slots, counts, demand, slot_src = assign_slots(ids, E, C)
    out.update(ids=ids, weights=w, slots=slots, counts=counts, demand=demand,
               slot_src=slot_src)
    return out
