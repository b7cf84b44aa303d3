"""The whole pass (gate, dispatch, combine and both backward ops) captured into a
HIP graph and replayed: every replay must reproduce the eager results bit for
bit, with eager work and synchronisations between replays, and a replay after
the input buffers are refilled must match an eager pass on the new inputs.  (The
eager pass itself is checked against the oracle by the parity tests.)"""

import numpy as np
import pytest
import torch

import paper_2203_14685_amd as hm
from paper_2203_14685_amd import workloads as wl

from _parity import announce

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hm.load()
    yield


def _buffers(S, d, E, k, C, tdt, dev, learned):
    i32, f32 = torch.int32, torch.float32
    return dict(
        ids=torch.empty((S, k), dtype=i32, device=dev), slots=torch.empty((S, k), dtype=i32, device=dev),
        weights=torch.empty((S, k), dtype=f32, device=dev), counts=torch.empty((E,), dtype=i32, device=dev),
        demand=torch.empty((E,), dtype=i32, device=dev), slot_src=torch.empty((E, C), dtype=i32, device=dev),
        xe=torch.empty((E, C, d), dtype=tdt, device=dev), y=torch.empty((S, d), dtype=tdt, device=dev),
        dye=torch.empty((E, C, d), dtype=tdt, device=dev),
        dw=torch.empty((S, k), dtype=f32, device=dev) if learned else None,
        dx=torch.empty((S, d), dtype=tdt, device=dev))


@pytest.mark.parametrize("wid,S,d", [(2, 3000, 1024), (5, 2500, 512), (1, 1000, 256)])
def test_graph_replay_matches_eager(wid, S, d):
    w = dict(wl.WORKLOADS[wid])
    E, k, dt = w["E"], w["k"], w["dtype"]
    C = int(np.ceil(w["cf"] * k * S / E))
    announce(f"graph replay workload {wid} S={S} d={d} E={E} k={k} C={C}")
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    dcode = hm.MOE_BF16 if dt == "bf16" else hm.MOE_F32
    learned = w["kind"] != hm.MOE_GATE_HASH
    inp = wl.make_inputs(w, S=S, d=d, seed=1)
    x = wl.to_device(inp["x"], dt)
    wg = wl.to_device(inp["wg"], dt)
    bias = wl.to_device(inp["bias"], "f32")
    tok = wl.to_device(inp["token_ids"], "i32")
    dy = wl.to_device(wl.make_rows((S, d), dt, 5), dt)
    params = hm.gate_params(S, d if learned else 0, E, k, C, w["kind"], w["normalize"], 0, dcode, 0)
    ws = torch.empty((hm.moe_gate_workspace_size(params),), dtype=torch.uint8, device=dev)
    lay = hm.Layout(S, d, E, k, C, dcode)
    b = _buffers(S, d, E, k, C, tdt, dev, learned)
    outs = [key for key in ("ids", "slots", "weights", "counts", "demand", "slot_src", "xe", "y", "dye", "dw", "dx")
            if b[key] is not None]

    def step(st):
        hm.moe_gate(params, x if learned else None, wg, bias, tok if not learned else None, None, None, None, b["ids"],
                    b["slots"], b["weights"], b["counts"], b["demand"], b["slot_src"], ws, st)
        hm.moe_dispatch(lay, x, b["ids"], b["slots"], b["slot_src"], b["xe"], st)
        hm.moe_combine(lay, b["xe"], b["ids"], b["slots"], b["weights"], b["y"], st)
        hm.moe_combine_bwd(lay, dy, b["xe"] if learned else None, b["ids"], b["slots"], b["slot_src"],
                           b["weights"], b["dye"], b["dw"], st)
        hm.moe_dispatch_bwd(lay, b["dye"], b["ids"], b["slots"], b["dx"], st)

    def scramble():
        for key in outs:
            b[key].fill_(-3)

    # eager reference on the side stream used for capture warm-up
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref = {key: b[key].clone() for key in outs}
    graph = torch.cuda.CUDAGraph()
    scramble()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step(torch.cuda.current_stream())
    torch.cuda.synchronize()

    for rep in range(4):
        scramble()               # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for key in outs:
            assert torch.equal(b[key], ref[key]), f"replay {rep}: {key} differs from the eager pass"

    # refill the captured inputs in place: the replay must follow the new values
    inp2 = wl.make_inputs(w, S=S, d=d, seed=7)
    x.copy_(wl.to_device(inp2["x"], dt))
    if not learned:
        tok.copy_(wl.to_device(inp2["token_ids"], "i32"))
    torch.cuda.synchronize()
    scramble()
    with torch.cuda.stream(side):
        step(side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref2 = {key: b[key].clone() for key in outs}
    for rep in range(2):
        scramble()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for key in outs:
            assert torch.equal(b[key], ref2[key]), f"replay {rep} on new inputs: {key} differs"
    assert not torch.equal(ref2["y"], ref["y"])
    del graph
    torch.cuda.synchronize()
