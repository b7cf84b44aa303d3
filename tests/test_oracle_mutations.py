"""The oracle's pins must catch plausible mistakes.  Each case plants one mistake
in a copy of the oracle (on the CPU, in a temporary directory) and runs the pin
tests against that copy; every mutant must make them fail."""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = [
    ("gate.py", "return (-row[e], e)", "return (row[e], e)", "selection order reversed"),
    ("gate.py", "return (-row[e], e)", "return (-row[e], -e)", "tie-break on the higher index"),
    ("gate.py", "den = np.exp(L - m).sum(axis=1, keepdims=True)", "den = np.exp(L - m).sum(axis=0, keepdims=True)",
     "softmax normalised over the wrong axis"),
    ("gate.py", "    for r in range(k):\n        for s in range(S):", "    for s in range(S):\n        for r in range(k):",
     "token-major instead of rank-major slots"),
    ("gate.py", "if cnt[e] < C:", "if cnt[e] <= C:", "capacity off by one"),
    ("gate.py", "slot_src[e, cnt[e]] = s * k + r", "slot_src[e, cnt[e]] = r * S + s", "slot source encoding"),
    ("gate.py", "splitmix64_output(int(seed), int(t) + 1)", "splitmix64_output(int(seed), int(t))", "hash output index"),
    ("gate.py", "grp = L[:, g * G:(g + 1) * G]", "grp = L", "kTop1 softmax over all experts"),
    ("gate.py", "z = ((z ^ (z >> 27)) * _SM64_M2) & _MASK64", "z = ((z ^ (z >> 29)) * _SM64_M2) & _MASK64",
     "hash mixing shift"),
    ("gate.py", "A = np.abs(x64) @ np.abs(w64)", "A = np.abs(x64 @ w64)", "magnitude without cancellation"),
    ("gate.py", "L = L + b64[None, :]", "L = L - b64[None, :]", "bias sign"),
    ("gate.py", "ids[s, g] = min(range(g * G, (g + 1) * G), key=lambda e: _key(row, e))",
     "ids[s, g] = min(range(g, E, k), key=lambda e: _key(row, e))", "strided kTop1 groups"),
    ("gate.py", "counts = np.minimum(demand, C)", "counts = demand", "counts not capped"),
    ("layout.py", "xe[full] = x[slot_src[full] // k]", "xe[full] = x[slot_src[full] % k]", "dispatch source row"),
    ("layout.py", "term = w[kept, r, None] * ye64[ids[kept, r], slots[kept, r]]",
     "term = ye64[ids[kept, r], slots[kept, r]]", "combine without the gate weight"),
    ("layout.py", "dye64[full] = w[s_of, r_of, None] * dy64[s_of]", "dye64[full] = dy64[s_of]",
     "combine backward without the weight"),
    ("layout.py", 'dw[s_of, r_of] = np.einsum("nd,nd->n", dy64[s_of], rows)',
     'dw[s_of, r_of] = np.einsum("nd,nd->n", dy64[s_of], rows) * w[s_of, r_of]', "dw scaled by the weight"),
    ("layout.py", "kept = np.nonzero(slots[:, r] >= 0)[0]\n        term = dxe64",
     "kept = np.nonzero(slots[:, r] >= -1)[0]\n        term = dxe64", "dropped choices counted in dispatch backward"),
    ("layout.py", "        y[kept] += term\n", "        y[kept] = decode(encode(y[kept] + term, dtype), dtype)\n",
     "combine rounding every partial sum"),
    ("bf16.py", "ulp_exp = np.maximum(ex.astype(np.int64) - 8, -133)", "ulp_exp = np.maximum(ex.astype(np.int64) - 8, -126)",
     "bf16 subnormal spacing"),
    ("bf16.py", "q = np.rint(v / ulp) * ulp", "q = np.floor(v / ulp + 0.5) * ulp", "bf16 ties away from zero"),
    ("gate_bwd.py", "w[:, r] * (dw[:, r] - inner)", "w[:, r] * (dw[:, r] + inner)", "renormalised softmax Jacobian sign"),
    ("gate_bwd.py", "dL = -p * g[:, None]", "dL = p * g[:, None]", "full softmax Jacobian sign"),
    ("gate_bwd.py", "dL[rows, ids[:, r]] += dw[:, r] * w[:, r]", "dL[rows, ids[:, r]] += dw[:, r]",
     "Switch gradient without the weight"),
    ("gate_bwd.py", "scale = dw[:, grp] * wg", "scale = dw[:, grp]", "kTop1 gradient without the weight"),
    ("gate_bwd.py", "p = _softmax_rows(L[:, lo:hi])", "p = _softmax_rows(L)[:, lo:hi]", "kTop1 softmax over all experts"),
    ("gate_bwd.py", "dL = c * p * (f[None, :] - fp[:, None])", "dL = c * p * f[None, :]", "aux gradient without the mean term"),
    ("gate_bwd.py", "np.bincount(ids[:, 0]", "np.bincount(ids[:, -1]", "aux counts on the last choice"),
    ("gate_bwd.py", '"dwg": x64.T @ dL', '"dwg": x64.T @ np.abs(dL)', "dW from |dL|"),
    ("gate_bwd.py", "dx = dx + d_in", "dx = dx - d_in", "incoming dx subtracted"),
    ("gate_bwd.py", '"dbias": dL.sum(axis=0)', '"dbias": dL.mean(axis=0)', "bias gradient averaged"),
    ("gate.py", "            g = best // Gs\n", "            g = best % groups\n", "H Topk group index"),
    ("gate.py", "order = sorted(range(g * Gs, (g + 1) * Gs), key=lambda e: _key(row, e))",
     "order = sorted(range(g * Gs, (g + 1) * Gs), key=lambda e: (row[e], e))", "H Topk inner order"),
    ("gate.py", "v = L if noise is None else (L + np.asarray(noise, dtype=np.float32)).astype(np.float32)",
     "v = L if noise is None else (L - np.asarray(noise, dtype=np.float32)).astype(np.float32)", "noise subtracted"),
    ("gate.py", "order = sorted(range(len(freq)), key=lambda t: (-freq[t], t))",
     "order = sorted(range(len(freq)), key=lambda t: (freq[t], t))", "balanced hash in increasing frequency"),
    ("gate.py", "e = min(range(E), key=lambda i: (load[i], i))", "e = min(range(E), key=lambda i: (load[i], -i))",
     "balanced hash ties to the higher expert"),
    ("gate_bwd.py", "        return dL / t, M / t", "        return dL * t, M * t", "temperature chain rule"),
    ("base.py", "ids[rows] = cols // c", "ids[rows] = cols % E", "BASE slot-to-expert map"),
    ("base.py", "linear_sum_assignment(cost, maximize=True)", "linear_sum_assignment(cost, maximize=False)",
     "BASE minimises"),
    ("base.py", "return 1.0 / (1.0 + np.exp(-v))", "return 1.0 / (1.0 + np.exp(v))", "BASE weight sign"),
]


@pytest.mark.parametrize("fname,old,new,what", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, fname, old, new, what):
    shutil.copytree(os.path.join(ROOT, "oracle"), tmp_path / "oracle")
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tmp_path / "tests" / "golden")
    for f in ("conftest.py", "test_oracle_pins.py", "test_oracle_gate_bwd_pins.py", "test_oracle_gate_more_pins.py",
              "test_oracle_base_pins.py"):
        shutil.copy(os.path.join(ROOT, "tests", f), tmp_path / "tests" / f)
    path = tmp_path / "oracle" / fname
    src = path.read_text()
    assert old in src, f"mutation site for '{what}' not found"
    path.write_text(src.replace(old, new, 1))
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          "tests/test_oracle_pins.py", "tests/test_oracle_gate_bwd_pins.py",
                          "tests/test_oracle_gate_more_pins.py", "tests/test_oracle_base_pins.py"], cwd=tmp_path, capture_output=True, text=True, timeout=300)
    assert res.returncode != 0, f"pins did not catch: {what}\n{res.stdout[-2000:]}"
