#!/usr/bin/env python3
"""Benchmark of the MoE gate / layout-transform hot path on one MI355X.

A step is one pass of the whole path over one batch: gate (projection,
softmax, selection, capacity slots) -> dispatch -> combine (identity experts:
ye = xe) -> combine backward -> dispatch backward (identity expert backward:
dxe = dye).  Inputs are synthetic, seeded, and resident in HBM before timing.

Prints ONE JSON line (metric, value = tokens/s, roofline of the dominant
kernel, CPU-oracle baseline).  Default workload: the hash-gate workload
(S=65536 tokens, d=4096, E=128, bf16), the largest of the five.
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak, GB/s
METRIC = "tokens/s through gate+dispatch+combine; achieved HBM GB/s vs MI355X peak"
OPS = ("gate", "dispatch", "combine", "combine_bwd", "dispatch_bwd")
# sources each op's kernel is compiled from; "file:Struct" stands for that
# struct's definition alone (the argument block the kernel reads)
_LAYOUT_SRC = ("layout.hip", "common.hpp", "kernels.hpp:RowArgs")
_GATE_SRC = ("gate.hip", "route_mfma.hip", "route_mfma_rs.hip", "route_mfma_ph.hip", "route_valu.hpp", "route_valu_f32.hip",
             "route_valu_bf16.hip", "select.hpp", "common.hpp", "kernels.hpp:RouteArgs")
OPS_KERNELS = ("dispatch", "combine", "combine_bwd", "dispatch_bwd", "gate")


def kernel_of_op(op, w):
    """(kernel symbol fragment in traces, sources that kernel is compiled from) of
    the one kernel an op launches for workload dict `w`, following the launch
    rules of the layout library: with one choice per token, dispatch and combine
    backward run the slot-row kernel (its compile-time form on rows of 64 to 512
    chunks, a power of two; combine backward with dw only there, else one wave
    per row); with
    several, the token-major forms; combine and dispatch backward always run the
    token-row kernel, its choice list sized 1, 2, 4 or 8."""
    elt = "hetumoe::bf16_t" if w["dtype"] == "bf16" else "float"
    k = w["k"]
    nch = w["d"] * (2 if w["dtype"] == "bf16" else 4) // 16
    pow2 = nch > 0 and (nch & (nch - 1)) == 0
    p2 = "true" if pow2 else "false"
    dw = w["kind"] != 2  # learned gates have weights to differentiate (hash: none)
    kmax = 1 if k == 1 else 2 if k == 2 else 4 if k <= 4 else 8
    lg = nch.bit_length() - 1
    fast = pow2 and 64 <= nch <= 512 and w["E"] * w["C"] > 0  # the compile-time row length form
    slot = (lambda t, sc, d: f"slot_rows_pow2_kernel<{t}, {sc}, {d}, {lg}") if fast else \
        (lambda t, sc, d: f"slot_rows_kernel<{t}, {sc}, {d}, {p2}")
    if k > 1:
        cbwd = f"combine_bwd_scatter_kernel<{elt}, {'true' if dw else 'false'}>"
    elif dw and not (pow2 and 64 <= nch <= 512):
        cbwd = f"combine_bwd_wave_kernel<{elt}>"
    else:
        cbwd = slot(elt, "true", "true" if dw else "false")
    return {"dispatch": ("dispatch_scatter_kernel" if k > 1 else slot("float", "false", "false"), _LAYOUT_SRC),
            "combine": (f"token_rows_kernel<{elt}, true, {kmax},", _LAYOUT_SRC),
            "combine_bwd": (cbwd, _LAYOUT_SRC),
            "dispatch_bwd": (f"token_rows_kernel<{elt}, false, {kmax},", _LAYOUT_SRC),
            "gate": ("route_", _GATE_SRC)}[op]


def summarize_pmc(args):
    """Turn two rocprofv3 --pmc runs of this benchmark (FETCH_SIZE, WRITE_SIZE; KiB
    per dispatch) into profiles/traffic_<op>_<workload>.txt.  Each run must have
    used --calib-copy-mib: the counter is scaled by the ratio of the known bytes of
    that plain device copy to what the counter read for it."""
    import csv
    import glob
    w = None
    from paper_2203_14685_amd import workloads as wl
    w = wl.WORKLOADS[args.workload]
    calib_bytes = args.calib_copy_mib * (1 << 20)

    def load(d, counter):
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(f) as fh:
                rows += [r for r in csv.DictReader(fh) if r.get("Counter_Name") == counter]
        if not rows:
            raise SystemExit(f"no {counter} rows under {d}")
        return rows

    out = {}
    for counter, d in (("FETCH_SIZE", args.summarize_pmc[0]), ("WRITE_SIZE", args.summarize_pmc[1])):
        rows = load(d, counter)
        copy = [float(r["Counter_Value"]) for r in rows if "elementwise" in r["Kernel_Name"] or "copy" in r["Kernel_Name"].lower()]
        if not copy:
            raise SystemExit(f"{counter}: no calibration copy kernel found")
        scale = calib_bytes / (max(copy) * 1024.0)
        for op in OPS_KERNELS:
            frag = kernel_of_op(op, w)[0]
            vals = [float(r["Counter_Value"]) for r in rows if frag in r["Kernel_Name"]]
            if vals:
                out.setdefault(op, {})[counter] = (sum(vals) / len(vals), len(vals), scale, max(copy))
    for op, cs in out.items():
        if set(cs) != {"FETCH_SIZE", "WRITE_SIZE"}:
            continue
        fk, fn, fs, fc = cs["FETCH_SIZE"]
        wk, wn, ws, wc = cs["WRITE_SIZE"]
        total = fk * 1024 * fs + wk * 1024 * ws
        frag, src = kernel_of_op(op, w)
        with open(traffic_path(w["name"], op), "w") as f:
            f.write(f"# HBM traffic per launch of {frag} ({op}), workload {w['name']}\n")
            f.write("# from two rocprofv3 counter runs (TMPDIR=/tmp, from /tmp, repo at $R):\n")
            f.write(f"#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d <dir> -- python3 $R/bench.py --workload "
                    f"{args.workload} --steps 3 --warmup 1 --no-cpu-baseline --no-base --no-workloads --cold-iters 0 "
                    f"--calib-copy-mib {args.calib_copy_mib}\n")
            f.write("#   (the same with --pmc WRITE_SIZE)\n")
            f.write(f"# calibration: one {args.calib_copy_mib} MiB device copy read FETCH {fc:.0f} KiB, WRITE {wc:.0f} KiB\n")
            f.write(f"fetch_kib_per_launch: {fk:.1f}\nwrite_kib_per_launch: {wk:.1f}\n")
            f.write(f"fetch_scale: {fs:.4f}\nwrite_scale: {ws:.4f}\nlaunches: {fn}\n")
            f.write(f"hbm_bytes_per_launch: {total:.0f}\nsource_sha: {source_sha(src)}\n")
        print(f"{op}: {total / 1e6:.1f} MB per launch -> {traffic_path(w['name'], op)}")


MFMA_KERNELS = (("route_mfma", "projection x.W", 1), ("dwg_mfma_kernel", "gate backward dW = x^T.dL", 3),
                ("dx_mfma_kernel", "gate backward dx = dL.W^T", 3))


def summarize_mfma(args):
    """Matrix-core evidence from one rocprofv3 --pmc run (MfmaUtil, MfmaFlopsBF16,
    GRBM_GUI_ACTIVE per dispatch): for each matrix-core kernel of this workload,
    the busy share of the matrix units and the bf16 MFMA flops counted per launch
    against the algorithmic 2*S*d*E (the gate backward runs three bf16 planes of
    dL, so three times that)."""
    import csv
    import glob
    from paper_2203_14685_amd import workloads as wl
    w = wl.WORKLOADS[args.workload]
    rows = []
    for f in glob.glob(os.path.join(args.summarize_mfma, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    if not rows:
        raise SystemExit(f"no counter rows under {args.summarize_mfma}")
    alg = 2 * w["S"] * w["d"] * w["E"]
    path = os.path.join(ROOT, "profiles", f"mfma_{w['name']}.txt")
    lines = [f"# matrix-core use per launch, workload {w['name']}",
             "# from one rocprofv3 counter run (TMPDIR=/tmp, from /tmp, repo at $R):",
             f"#   rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 GRBM_GUI_ACTIVE --output-format csv -d <dir> -- python3 "
             f"$R/bench.py --workload {args.workload} --steps 3 --warmup 1 --no-cpu-baseline --no-base --no-workloads "
             "--cold-iters 0",
             "# MfmaUtil = matrix-unit busy cycles summed over SIMDs / (GPU active cycles x SIMDs) x 100;",
             "# MfmaFlopsBF16 = bf16 MFMA operations x 512 (flops counted by the hardware)",
             f"# algorithmic flops of one projection 2*S*d*E = {alg}",
             "%-34s %-28s %8s %10s %16s %12s" % ("kernel", "computes", "launches", "mfma_util%", "mfma_flops",
                                                 "flops/alg")]
    found = 0
    for frag, what, mult in MFMA_KERNELS:
        sel = [r for r in rows if frag in r["Kernel_Name"]]
        if not sel:
            continue
        by = {}
        for r in sel:
            by.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
        util = by.get("MfmaUtil", [float("nan")])
        flops = by.get("MfmaFlopsBF16", [float("nan")])
        name = sel[0]["Kernel_Name"].split("(")[0].replace("hetumoe::", "").replace("void ", "")
        fl = sum(flops) / len(flops)
        lines.append("%-34s %-28s %8d %10.2f %16.0f %12.4f" % (name[:34], what[:28], len(util), sum(util) / len(util),
                                                               fl, fl / (alg * mult)))
        found += 1
    if not found:
        raise SystemExit("no matrix-core kernel in the counter rows")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_route(args):
    """profiles/route_choice_<workload>.txt from two rocprofv3 --kernel-trace
    --stats runs of this benchmark on one workload: the library as built (matrix
    cores where the shape allows) and a build with HETUMOE_ROUTE_VALU_ONLY (the
    vector-ALU projection).  Lists the gate's kernels of each run, average
    duration per launch and calls."""
    import csv
    import glob
    from paper_2203_14685_amd import workloads as wl
    w = wl.WORKLOADS[args.workload]

    def gate_rows(d):
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True):
            with open(f) as fh:
                rows += list(csv.DictReader(fh))
        out = []
        for r in rows:
            name = r["Name"].replace("void ", "").replace("hetumoe::", "").split("(")[0]
            if name.startswith(("route_", "scan_", "assign_", "scan_assign", "select_ext")):
                out.append((name, int(r["Calls"]), float(r["AverageNs"])))
        if not out:
            raise SystemExit(f"no gate kernels in {d}")
        return out
    runs = {"matrix cores (as built)": gate_rows(args.summarize_route[0]),
            "vector ALUs (HETUMOE_ROUTE_VALU_ONLY)": gate_rows(args.summarize_route[1])}
    alg = w["S"] * w["d"] * (2 if w["dtype"] == "bf16" else 4) + w["d"] * w["E"] * 2
    lines = [f"# gate projection route, matrix cores against vector ALUs, workload {w['name']}",
             "# two rocprofv3 kernel traces (TMPDIR=/tmp, from /tmp, repo at $R):",
             f"#   rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -- python3 $R/bench.py --workload "
             f"{args.workload} --steps 20 --warmup 5 --no-cpu-baseline --no-base --no-workloads --cold-iters 0",
             "#   the same with HETUMOE_LIBRARY=<lib> after `python -m paper_2203_14685_amd.build --out <lib> "
             "-D HETUMOE_ROUTE_VALU_ONLY`",
             f"# x + W bytes the projection must read: {alg}",
             "%-40s %-60s %7s %10s %9s" % ("build", "kernel", "calls", "avg_us", "GB/s")]
    for label, rows in runs.items():
        for name, calls, ns in sorted(rows, key=lambda r: -r[2]):
            gbs = alg / ns if name.startswith("route_") else float("nan")
            lines.append("%-40s %-60s %7d %10.2f %9.1f" % (label, name[:60], calls, ns / 1e3, gbs))
    path = os.path.join(ROOT, "profiles", f"route_choice_{w['name']}.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_trace(args):
    """profiles/kernels_<workload>.txt from one rocprofv3 --kernel-trace --stats
    run of this benchmark on one workload (its kernel_stats.csv)."""
    import csv
    import glob
    from paper_2203_14685_amd import workloads as wl
    w = wl.WORKLOADS[args.workload]
    rows = []
    for f in glob.glob(os.path.join(args.summarize_trace, "**", "*kernel_stats.csv"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    if not rows:
        raise SystemExit(f"no kernel_stats.csv under {args.summarize_trace}")
    lines = [f"# rocprofv3 kernel trace: workload {w['name']}, one fwd+bwd step per call",
             "# command (from /tmp, TMPDIR=/tmp; repo at $R):",
             f"#   rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -- python3 $R/bench.py --workload "
             f"{args.workload} --steps 20 --warmup 5 --no-cpu-baseline --no-workloads",
             "# kernel_stats.csv of that run, MI355X (gfx950).  The step's kernels run warmup + steps + cold-cache",
             "# launches; the timings after the timed step (gate backward, further gates, BASE layer, copy",
             "# ceiling) add their own launches, hence the other call counts.",
             "%-74s %6s %12s %12s %12s %7s" % ("kernel", "calls", "avg_ns", "min_ns", "max_ns", "pct")]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = r["Name"].replace("void ", "").replace("hetumoe::", "").split("(")[0]
        lines.append("%-74s %6d %12.0f %12d %12d %7.2f" % (name[:74], int(r["Calls"]), float(r["AverageNs"]),
                                                           int(r["MinNs"]), int(r["MaxNs"]), float(r["Percentage"])))
    path = os.path.join(ROOT, "profiles", f"kernels_{w['name']}.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines[:20]))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=5, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the step captured into a HIP graph (per-op times then come from an "
                         "eager pass with events)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write profiles/traffic_*.txt from two rocprofv3 --pmc output folders and exit")
    ap.add_argument("--summarize-mfma", metavar="DIR",
                    help="write profiles/mfma_<workload>.txt from a rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 "
                         "GRBM_GUI_ACTIVE output folder and exit")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="write profiles/kernels_<workload>.txt from a rocprofv3 --kernel-trace --stats folder and exit")
    ap.add_argument("--summarize-route", nargs=2, metavar=("MFMA_DIR", "VALU_DIR"),
                    help="write profiles/route_choice_<workload>.txt from two rocprofv3 --kernel-trace --stats "
                         "folders (library as built, and built with HETUMOE_ROUTE_VALU_ONLY) and exit")
    ap.add_argument("--no-base", action="store_true",
                    help="skip the BASE-layer timing (thousands of small launches; for counter runs)")
    ap.add_argument("--cold-iters", type=int, default=10,
                    help="per-op timings from a cold cache: launches of each op, each after reading a 1 GiB "
                         "buffer (0 = skip)")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the compact figures of the other four workloads (for counter and trace runs of one "
                         "workload)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before the timed region, run one device copy of this many MiB (counter calibration)")
    return ap.parse_args()


def alg_bytes(w, S, d, E, k, C, elt, n_kept, tok_kept, dw):
    """Bytes each op must move at minimum: every input read once, every output
    written once (zero rows of the expert buffers included)."""
    row = d * elt
    if w["kind"] == 2:
        gate_in = S * 4
    else:
        gate_in = S * row + d * E * elt + (E * 4 if w.get("hot_experts") else 0)
    b = {
        "gate": gate_in + S * k * 12 + E * C * 4 + 2 * E * 4,
        "dispatch": tok_kept * row + E * C * row + E * C * 4,
        "combine": n_kept * row + S * row + S * k * 12,
        "dispatch_bwd": n_kept * row + S * row + S * k * 8,
        "combine_bwd": tok_kept * row + E * C * row + E * C * 4 + S * k * 4
                       + ((n_kept * row + S * k * 8) if dw else 0),
    }
    return b


def source_sha(names):
    h = hashlib.sha256()
    for name in names:
        fname, _, struct = name.partition(":")
        with open(os.path.join(ROOT, "paper_2203_14685_amd", "csrc", fname), "rb") as f:
            text = f.read()
        if struct:
            i = text.index(f"struct {struct} {{".encode())
            text = text[i:text.index(b"};", i) + 2]
        h.update(text)
    return h.hexdigest()[:16]


def traffic_path(workload_name, op):
    return os.path.join(ROOT, "profiles", f"traffic_{op}_{workload_name}.txt")


def measured_traffic(workload_name, op, sha):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    when there is none for this op's kernel and workload or its source changed."""
    path = traffic_path(workload_name, op)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for ln in f:
            if ":" in ln and not ln.startswith("#"):
                key, _, v = ln.partition(":")
                vals[key.strip()] = v.strip()
    if vals.get("source_sha") != sha:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, target_s=8.0):
    """The oracle, untuned, on a bounded sample of the same workload (its first
    S_s tokens, capacity scaled the same way), timed on this host, stage by
    stage; the sample doubles until a pass takes about target_s / 2, then the
    pass runs three times and each stage reports its median (one run when a
    pass exceeds 30 s).  For learned gates the fp64 projection (a numpy BLAS
    product) is also timed with the whole BLAS pool and with one thread, median
    of three."""
    import math

    import oracle
    from paper_2203_14685_amd import workloads as wl
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # threadpoolctl missing: report the host's count
        threadpool_limits = None
        blas_threads = os.cpu_count() or 1
    k, E, d, dt = w["k"], w["E"], w["d"], w["dtype"]
    learned = w["kind"] != 2

    def run(S_s, data=None):
        C_s = int(math.ceil(w["cf"] * k * S_s / E))
        inp, dy = data if data is not None else (wl.make_inputs(w, S=S_s, seed=0), wl.make_rows((S_s, d), dt, 2))
        t0 = time.perf_counter()
        g = oracle.gate(w["kind"], k, E, C_s, normalize=w["normalize"], dtype=dt, x=inp["x"], wg=inp["wg"],
                        bias=inp["bias"], token_ids=inp["token_ids"], hash_seed=0)
        t1 = time.perf_counter()
        xe = oracle.dispatch(inp["x"], g["slot_src"], k)
        t2 = time.perf_counter()
        oracle.combine(xe, g["ids"], g["slots"], g["weights"], dt)
        t3 = time.perf_counter()
        dye, _, _, _ = oracle.combine_bwd(dy, xe, g["slot_src"], g["weights"], k, dt, want_dw=learned)
        t4 = time.perf_counter()
        oracle.dispatch_bwd(dye, g["ids"], g["slots"], dt)
        t5 = time.perf_counter()
        st = {"gate": t1 - t0, "dispatch": t2 - t1, "combine": t3 - t2, "combine_bwd": t4 - t3, "dispatch_bwd": t5 - t4}
        return t5 - t0, st, (inp, dy)

    S_s = 512
    t, st, data = run(S_s)
    while t < target_s / 2 and S_s * 2 <= w["S"]:
        S_s *= 2
        t, st, data = run(S_s)
    runs = [(t, st)]
    if t <= 30.0:
        runs += [run(S_s, data)[:2] for _ in range(2)]

    def med(v):
        return sorted(v)[len(v) // 2]
    t = med([r[0] for r in runs])
    stage = {key: med([r[1][key] for r in runs]) for key in runs[0][1]}
    out = {"value": round(S_s / t, 1), "unit": "tokens/s", "cores": int(blas_threads if learned else 1),
           "kind": "oracle",
           "sample": f"first {S_s} of {w['S']} tokens of the same workload (capacity scaled alike), "
                     f"full pass gate+dispatch+combine+combine_bwd+dispatch_bwd, median of {len(runs)} "
                     f"passes {t:.2f} s, fp64 numpy",
           "stage_s": {key: round(v, 3) for key, v in stage.items()}, "passes": len(runs)}
    if learned:
        # the projection alone (numpy BLAS, fp64) with the whole pool and with one thread
        inp = data[0]
        pt = {}
        for n in sorted({blas_threads, 1}, reverse=True):
            if threadpool_limits is None and n != blas_threads:
                continue
            ts = []
            for _ in range(3):
                t0 = time.perf_counter()
                if threadpool_limits is not None:
                    with threadpool_limits(limits=n, user_api="blas"):
                        oracle.logits(inp["x"], inp["wg"], dt, inp["bias"])
                else:
                    oracle.logits(inp["x"], inp["wg"], dt, inp["bias"])
                ts.append(time.perf_counter() - t0)
            pt[str(n)] = round(med(ts), 3)
        out["projection_s_by_threads"] = pt
    try:
        out["host"] = {"cpus_allowed": len(os.sched_getaffinity(0)),
                       "model": next((ln.split(":", 1)[1].strip() for ln in open("/proc/cpuinfo")
                                      if ln.startswith("model name")), "unknown")}
    except OSError:
        pass
    return out


def build_pass(w, dev):
    """Device inputs, outputs and the five op calls of one step of workload `w`
    (identity experts: ye = xe, dxe = dye)."""
    import types

    import torch
    import paper_2203_14685_amd as hm
    from paper_2203_14685_amd import workloads as wl
    S, d, E, k, C, dt = w["S"], w["d"], w["E"], w["k"], w["C"], w["dtype"]
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    dcode = hm.MOE_BF16 if dt == "bf16" else hm.MOE_F32
    learned = w["kind"] != 2
    P = types.SimpleNamespace()
    P.inp = inp = wl.make_inputs(w, seed=0)
    P.x = x = wl.to_device(inp["x"], dt)
    P.wg = wg = wl.to_device(inp["wg"], dt)
    P.bias = bias = wl.to_device(inp["bias"], "f32")
    P.tok = tok = wl.to_device(inp["token_ids"], "i32")
    P.dy = dy = wl.to_device(wl.make_rows((S, d), dt, 2), dt)
    P.params = params = hm.gate_params(S, d if learned else 0, E, k, C, w["kind"], w["normalize"], 0, dcode, 0)
    i32, f32 = torch.int32, torch.float32
    P.ids = ids = torch.empty((S, k), dtype=i32, device=dev)
    P.slots = slots = torch.empty((S, k), dtype=i32, device=dev)
    P.weights = weights = torch.empty((S, k), dtype=f32, device=dev)
    P.counts = counts = torch.empty((E,), dtype=i32, device=dev)
    P.demand = demand = torch.empty((E,), dtype=i32, device=dev)
    P.slot_src = slot_src = torch.empty((E, C), dtype=i32, device=dev)
    P.ws = ws = torch.empty((hm.moe_gate_workspace_size(params),), dtype=torch.uint8, device=dev)
    P.xe = xe = torch.empty((E, C, d), dtype=tdt, device=dev)
    P.y = y = torch.empty((S, d), dtype=tdt, device=dev)
    P.dye = dye = torch.empty((E, C, d), dtype=tdt, device=dev)
    P.dw = dw = torch.empty((S, k), dtype=f32, device=dev) if learned else None
    P.dx = dx = torch.empty((S, d), dtype=tdt, device=dev)
    lay = hm.Layout(S, d, E, k, C, dcode)
    P.op_calls = {
        "gate": lambda st: hm.moe_gate(params, x if learned else None, wg, bias, tok if not learned else None, None,
                                       None, None, ids, slots, weights, counts, demand, slot_src, ws, st),
        "dispatch": lambda st: hm.moe_dispatch(lay, x, ids, slots, slot_src, xe, st),
        "combine": lambda st: hm.moe_combine(lay, xe, ids, slots, weights, y, st),
        "combine_bwd": lambda st: hm.moe_combine_bwd(lay, dy, xe if learned else None, ids, slots, slot_src, weights,
                                                     dye, dw, st),
        "dispatch_bwd": lambda st: hm.moe_dispatch_bwd(lay, dye, ids, slots, dx, st),
    }
    return P


def workload_summary(wid, steps, warmup):
    """Compact figures of one workload, measured in the same run as the headline:
    step time eager (per-op HIP events on the library's stream) and as a HIP
    graph replay, tokens/s, the step's and each op's share of the HBM peak, the
    dominant op's kernel, and the gate's time."""
    import torch
    from paper_2203_14685_amd import workloads as wl
    w = wl.WORKLOADS[wid]
    dev = torch.device("cuda:0")
    S, d, E, k, C = w["S"], w["d"], w["E"], w["k"], w["C"]
    elt = 2 if w["dtype"] == "bf16" else 4
    P = build_pass(w, dev)
    stream = torch.cuda.current_stream()

    def step(evs=None, st=None):
        st = stream if st is None else st
        for i, op in enumerate(OPS):
            if evs is not None:
                evs[i].record(st)
            P.op_calls[op](st)
        if evs is not None:
            evs[len(OPS)].record(st)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(OPS) + 1)] for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    eager_ms = (time.perf_counter() - t0) * 1e3 / steps
    op_ms = {op: sum(e[j].elapsed_time(e[j + 1]) for e in evs) / steps for j, op in enumerate(OPS)}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(None, torch.cuda.current_stream())  # the capture stream
    torch.cuda.synchronize()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    graph_ms = (time.perf_counter() - t0) * 1e3 / steps
    sl = P.slots.cpu().numpy()
    n_kept = int((sl >= 0).sum())
    tok_kept = int((sl >= 0).any(axis=1).sum())
    ab = alg_bytes(w, S, d, E, k, C, elt, n_kept, tok_kept, w["kind"] != 2)
    step_bytes = sum(ab.values())
    fwd_ms = op_ms["gate"] + op_ms["dispatch"] + op_ms["combine"]
    fwd_bytes = ab["gate"] + ab["dispatch"] + ab["combine"]
    dom = max(OPS, key=lambda o: op_ms[o])

    def frac(b, ms):
        return round(b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    del graph, P
    torch.cuda.empty_cache()
    return {"step_ms": {"eager": round(eager_ms, 4), "graph": round(graph_ms, 4)},
            "tokens/s": {"eager": round(S / (eager_ms * 1e-3), 1), "graph": round(S / (graph_ms * 1e-3), 1)},
            "step_frac": {"eager": frac(step_bytes, eager_ms), "graph": frac(step_bytes, graph_ms)},
            "fwd": {"ms": round(fwd_ms, 5), "frac": frac(fwd_bytes, fwd_ms)},
            "ops_frac": {op: frac(ab[op], op_ms[op]) for op in OPS},
            "ops_us": {op: round(op_ms[op] * 1e3, 2) for op in OPS},
            "dominant": {"op": dom, "kernel": kernel_of_op(dom, w)[0].split("<")[0], "frac": frac(ab[dom], op_ms[dom])},
            "gate_us": round(op_ms["gate"] * 1e3, 2)}


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args)
        return
    if args.summarize_mfma:
        summarize_mfma(args)
        return
    if args.summarize_route:
        summarize_route(args)
        return
    if args.summarize_trace:
        summarize_trace(args)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this library runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)

    import torch
    import paper_2203_14685_amd as hm
    from paper_2203_14685_amd import workloads as wl

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        sys.exit(3)
    hm.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = wl.WORKLOADS[args.workload]
    S, d, E, k, C, dt = w["S"], w["d"], w["E"], w["k"], w["C"], w["dtype"]
    elt = 2 if dt == "bf16" else 4
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    dcode = hm.MOE_BF16 if dt == "bf16" else hm.MOE_F32
    learned = w["kind"] != 2
    want_dw = learned

    P = build_pass(w, dev)
    x, wg, bias, tok, dy, inp = P.x, P.wg, P.bias, P.tok, P.dy, P.inp
    params, ids, slots, weights, counts, demand, slot_src, ws = (P.params, P.ids, P.slots, P.weights, P.counts,
                                                                 P.demand, P.slot_src, P.ws)
    xe, dw, dx = P.xe, P.dw, P.dx
    stream = torch.cuda.current_stream()
    op_calls = P.op_calls

    def step(evs=None, st=None):
        st = stream if st is None else st
        for i, op in enumerate(OPS):
            if evs is not None:
                evs[i].record(st)
            op_calls[op](st)
        if evs is not None:
            evs[len(OPS)].record(st)

    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        bcp = torch.empty_like(a)
        torch.cuda.synchronize()
        bcp.copy_(a)
        torch.cuda.synchronize()
        del a, bcp

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] workload {args.workload} {w['name']}: warmup done", file=sys.stderr, flush=True)

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(OPS) + 1)] for _ in range(args.steps)]
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step(None, torch.cuda.current_stream())
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for i in range(args.steps):  # per-op events: an eager pass after the timed region
            step(evs[i])
        torch.cuda.synchronize()
    else:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            step(evs[i])
        torch.cuda.synchronize()
        t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    op_ms = {op: sum(e[j].elapsed_time(e[j + 1]) for e in evs) / args.steps for j, op in enumerate(OPS)}
    step_ev = sorted(e[0].elapsed_time(e[len(OPS)]) for e in evs)

    def pct(v, q):
        return v[min(len(v) - 1, int(q * len(v)))]

    # gradient of the gate (learned gates), outside the timed step: moe_gate_bwd
    # with dx accumulated into the dispatch-backward output, dW, db and, for
    # top-k gates, the load-balancing loss
    gate_bwd = None
    if learned:
        aux = 0.01 if w["kind"] == hm.MOE_GATE_TOPK else 0.0
        lg = torch.empty((S, E), dtype=torch.float32, device=dev)
        hm.moe_gate(params, x, wg, bias, None, None, None, lg, ids, slots, weights, counts, demand, slot_src, ws,
                    stream)
        bp = hm.gate_bwd_params(S, d, E, k, w["kind"], w["normalize"], dcode, 1, aux)
        bws = torch.empty((hm.moe_gate_bwd_workspace_size(bp),), dtype=torch.uint8, device=dev)
        dwg_out = torch.empty((d, E), dtype=torch.float32, device=dev)
        db_out = torch.empty((E,), dtype=torch.float32, device=dev)
        loss_out = torch.empty((1,), dtype=torch.float32, device=dev) if aux else None

        def gbwd():
            hm.moe_gate_bwd(bp, x, wg, lg, ids, dw, None, dx, dwg_out, db_out, loss_out, bws, stream)
        for _ in range(3):
            gbwd()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        g0.record(stream)
        for _ in range(args.steps):
            gbwd()
        g1.record(stream)
        torch.cuda.synchronize()
        gms = g0.elapsed_time(g1) / args.steps
        gbytes = S * E * 4 + S * k * 8 + S * d * elt + d * E * elt + 2 * S * d * elt + d * E * 4 + E * 4
        gflop = 4 * S * d * E
        gate_bwd = {"ms": round(gms, 5), "alg_bytes": gbytes, "GB/s": round(gbytes / (gms * 1e-3) / 1e9, 1),
                    "hbm_frac": round(gbytes / (gms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                    "flop": gflop, "TFLOP/s": round(gflop / (gms * 1e-3) / 1e12, 2),
                    "what": "moe_gate_bwd: dL, dW = x^T dL, db, dx += dL W^T" + (", balance loss" if aux else "")}
        del bws, lg

    # routing statistics of this batch (outside the timed region)
    sl = slots.cpu().numpy()
    n_kept = int((sl >= 0).sum())
    tok_kept = int((sl >= 0).any(axis=1).sum())
    ab = alg_bytes(w, S, d, E, k, C, elt, n_kept, tok_kept, want_dw)
    step_bytes = sum(ab.values())

    # the further gates of Sec. 3.1 on this workload's shape, outside the timed
    # step: hierarchical top-k (groups of 16 experts) and Dense-To-Sparse
    # (Gumbel noise, temperature 0.5) for learned gates, the balanced table for
    # the hash gate; each timed over `steps` calls of moe_gate
    def time_gate(gp, **kw):
        gws = torch.empty((hm.moe_gate_workspace_size(gp),), dtype=torch.uint8, device=dev)

        def call():
            hm.moe_gate(gp, kw.get("x"), kw.get("wg"), kw.get("bias"), kw.get("tok"), kw.get("noise"),
                        kw.get("table"), None, ids, slots, weights, counts, demand, slot_src, gws, stream)
        for _ in range(3):
            call()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    gates = {}
    if learned:
        G = max(1, E // 16)
        kh = min(k, E // G, 8)
        gp = hm.gate_params(S, d, E, kh, C, hm.MOE_GATE_HTOPK, w["normalize"], 0, dcode, 0, groups=G)
        ms = time_gate(gp, x=x, wg=wg, bias=bias)
        b = ab["gate"] - S * k * 12 + S * kh * 12  # the same bytes as the top-k gate, for kh choices
        gates["htopk"] = {"ms": round(ms, 5), "groups": G, "k": kh, "alg_bytes": b,
                          "GB/s": round(b / (ms * 1e-3) / 1e9, 1)}
        noise = torch.from_numpy(
            (-np.log(-np.log(np.random.default_rng(3).random((S, E))))).astype(np.float32)).to(dev)
        gp = hm.gate_params(S, d, E, k, C, w["kind"], w["normalize"], 0, dcode, 0, temperature=0.5)
        ms = time_gate(gp, x=x, wg=wg, bias=bias, noise=noise)
        b = ab["gate"] + S * E * 4  # + the noise read
        gates["dense_to_sparse"] = {"ms": round(ms, 5), "temperature": 0.5, "alg_bytes": b,
                                    "GB/s": round(b / (ms * 1e-3) / 1e9, 1)}
        del noise
        if S % E == 0 and S // E <= 2048 and not args.no_base:
            # BASE layer: balanced assignment by the auction (each call
            # synchronizes its stream); bound by the latency of its rounds
            cb_ = S // E
            bpp = hm.base_params(S, d, E, cb_, 0, dcode)
            bws = torch.empty((hm.moe_base_gate_workspace_size(bpp),), dtype=torch.uint8, device=dev)
            bo = [torch.empty((S,), dtype=torch.int32, device=dev), torch.empty((S,), dtype=torch.int32, device=dev),
                  torch.empty((S,), dtype=torch.float32, device=dev), torch.empty((E,), dtype=torch.int32, device=dev),
                  torch.empty((E, cb_), dtype=torch.int32, device=dev)]
            info = hm.BaseInfo()

            def bcall():
                hm.moe_base_gate(bpp, x, wg, bias, None, bo[0], bo[1], bo[2], bo[3], bo[4], None, bws, info, stream)
            bcall()
            nb_calls = max(1, min(args.steps, 10))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(nb_calls):
                bcall()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / nb_calls
            gates["base"] = {"ms": round(ms, 4), "phases": info.phases, "rounds": info.rounds,
                             "us_per_round": round(ms * 1e3 / max(1, info.rounds), 2), "eps": info.eps,
                             "optimality_bound": S * info.eps, "bound": "latency",
                             "what": "moe_base_gate: projection, eps-scaling auction, slots"}
            del bws, bo
    else:
        ranks = np.arange(1, w["vocab"] + 1, dtype=np.float64)
        pz = ranks ** -w["zipf_a"]
        pz /= pz.sum()
        table = torch.from_numpy(hm.moe_hash_balanced_table(pz, E)).to(dev)
        gp = hm.gate_params(S, 0, E, 1, C, hm.MOE_GATE_HASH, 0, 0, dcode, 0, hash_vocab=int(table.shape[0]))
        ms = time_gate(gp, tok=tok, table=table)
        gates["balanced_hash"] = {"ms": round(ms, 5), "alg_bytes": ab["gate"] + S * 4,
                                  "GB/s": round((ab["gate"] + S * 4) / (ms * 1e-3) / 1e9, 1)}

    # per op from a cold cache, outside the timed region: before each launch read
    # a 1 GiB buffer (more than the L2s and the 256 MB Infinity Cache, and it
    # leaves clean lines behind); median of the launches
    cold = None
    if args.cold_iters > 0:
        flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        cold = {}
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for op in OPS:
            ts = []
            for _ in range(args.cold_iters):
                flush.sum()
                c0.record(stream)
                op_calls[op](stream)
                c1.record(stream)
                torch.cuda.synchronize()
                ts.append(c0.elapsed_time(c1))
            ts.sort()
            med = ts[len(ts) // 2]
            cold[op] = {"ms_p50": round(med, 5), "GB/s": round(ab[op] / (med * 1e-3) / 1e9, 1),
                        "frac": round(ab[op] / (med * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        del flush

    dom = max(("dispatch", "combine", "combine_bwd", "dispatch_bwd", "gate"), key=lambda o: op_ms[o])
    achieved = ab[dom] / (op_ms[dom] * 1e-3) / 1e9
    kern, ksrc = kernel_of_op(dom, w)
    traffic = measured_traffic(w["name"], dom, source_sha(ksrc))
    dom_ev = sorted(e[j].elapsed_time(e[j + 1]) for e in evs for j in [OPS.index(dom)])

    # context, outside the timed region: a plain device-to-device copy moving the
    # dominant kernel's algorithmic bytes (half read, half written)
    n_copy = max(1, ab[dom] // 2)
    ca = torch.empty(n_copy, dtype=torch.uint8, device=dev)
    cb = torch.empty_like(ca)
    for _ in range(3):
        cb.copy_(ca)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(10):
        cb.copy_(ca)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * n_copy / (c0.elapsed_time(c1) / 10 * 1e-3) / 1e9
    del ca, cb

    out = {
        "metric": METRIC,
        "value": round(S / (ms_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if dt == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w["name"], "S": S, "d": d, "E": E, "k": k, "capacity": C,
                   "gate": ["topk", "ktop1", "hash"][w["kind"]], "passes": "fwd+bwd",
                   "parallelism": "single-gpu", "launch": "hip-graph" if args.graph else "eager"},
        "roofline": {"bound": "hbm", "kernel": kern.split("<")[0], "op": dom, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "alg_bytes_per_launch": ab[dom],
                     "avg_launch_ms": round(op_ms[dom], 5),
                     "launch_ms_p10_p50_p90": [round(pct(dom_ev, q), 5) for q in (0.1, 0.5, 0.9)],
                     "copy_ceiling": {"GB/s": round(copy_gbs, 1), "frac": round(copy_gbs / HBM_PEAK_GBS, 4),
                                      "kernel_vs_copy": round(achieved / copy_gbs, 4),
                                      "what": "device-to-device copy of the same byte count"}},
        "step_ms_p10_p50_p90": [round(pct(step_ev, q), 5) for q in (0.1, 0.5, 0.9)],
        "step_hbm": {"alg_bytes": step_bytes, "GB/s": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
                     "frac": round(step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "ops": {op: {"ms": round(op_ms[op], 5), "alg_bytes": ab[op],
                     "GB/s": round(ab[op] / (op_ms[op] * 1e-3) / 1e9, 1)} for op in OPS},
        "routing": {"kept_assignments": n_kept, "tokens_with_kept": tok_kept, "assignments": S * k},
        "gate_bwd": gate_bwd,
        "gates": gates,
        "cold": cold,
    }
    fwd_ms = op_ms["gate"] + op_ms["dispatch"] + op_ms["combine"]
    out["fwd"] = {"ms": round(fwd_ms, 5), "tokens/s": round(S / (fwd_ms * 1e-3), 1),
                  "frac": round((ab["gate"] + ab["dispatch"] + ab["combine"]) / (fwd_ms * 1e-3) / 1e9
                                / HBM_PEAK_GBS, 4)}
    if not args.no_workloads:
        # the other workloads, compact, in the same run (no CPU baseline, no BASE)
        out["workloads"] = {}
        for wid in sorted(wl.WORKLOADS):
            if wid == args.workload:
                continue
            print(f"[bench] workload {wid} {wl.WORKLOADS[wid]['name']}: compact figures", file=sys.stderr, flush=True)
            out["workloads"][wl.WORKLOADS[wid]["name"]] = workload_summary(wid, min(args.steps, 20),
                                                                           max(1, min(args.warmup, 5)))
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
