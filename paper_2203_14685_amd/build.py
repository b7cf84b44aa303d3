"""Build libhetumoe.so (the C-ABI library) for gfx950 with hipcc, in-tree.

Usage: python -m paper_2203_14685_amd.build   (or call build()).
"""

import os
import shutil
import subprocess
import sys
import time

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libhetumoe.so")

SOURCES = ["base.hip", "gate_bwd.hip", "route_valu_f32.hip", "route_valu_bf16.hip", "route_mfma_rs.hip", "route_mfma_ph.hip", "route_mfma.hip",
           "gate.hip", "layout.hip", "capi.hip"]

# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in generated code.
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fvisibility=hidden",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    return res.returncode, res.stdout + res.stderr


def prune_stale_objects(objdir, sources=SOURCES):
    """Delete the objects in `objdir` that no source of `sources` produces.  Such
    objects (left by a source since removed or renamed) could otherwise be linked
    in and their weak kernel symbols win over the current ones."""
    current = {src.replace(".hip", ".o") for src in sources}
    removed = []
    for name in sorted(os.listdir(objdir)):
        if name.endswith(".o") and name not in current:
            os.remove(os.path.join(objdir, name))
            removed.append(name)
    return removed


def link_command(cc, objdir, out, sources=SOURCES):
    """The link line: exactly the objects of `sources`, never a glob of `objdir`."""
    objs = [os.path.join(objdir, src.replace(".hip", ".o")) for src in sources]
    return [cc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", out]


def build(verbose=True, out=None, defines=()):
    """Compile every HIP source (in parallel) and link paper_2203_14685_amd/libhetumoe.so
    (or `out`, from objects in a folder of its own, with the macros `defines`:
    HETUMOE_ROUTE_VALU_ONLY builds a library whose gate projects on the vector
    ALUs only, to time those routes against the matrix-core ones)."""
    from concurrent.futures import ThreadPoolExecutor
    cc = hipcc()
    t0 = time.time()
    lib = LIB if out is None else os.path.abspath(out)
    objdir = os.path.join(PKG, "_build") if out is None else lib + ".objs"
    os.makedirs(objdir, exist_ok=True)
    prune_stale_objects(objdir)
    jobs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        flags = [f for f in HIPCC_FLAGS if f != "-shared"] + [f"-D{d}" for d in defines]
        jobs.append((obj, [cc, *flags, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]))
    if verbose:
        print(f"[build] {cc} {' '.join(HIPCC_FLAGS)} ... ({len(jobs)} sources)", flush=True)
    workers = min(len(jobs), max(1, int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        results = list(ex.map(lambda j: _run(j[1]), jobs))
    logs = []
    for (obj, cmd), (rc, out) in zip(jobs, results):
        if rc != 0:
            sys.stderr.write(" ".join(cmd) + "\n" + out)
            raise RuntimeError(f"hipcc failed on {cmd[-3]} with exit code {rc}")
        logs.append(out)
    tmp = lib + ".tmp"
    rc, log = _run(link_command(cc, objdir, tmp))
    if rc != 0:
        sys.stderr.write(log)
        raise RuntimeError(f"link failed with exit code {rc}")
    os.replace(tmp, lib)
    if verbose:
        warn = [ln for out in logs for ln in out.splitlines() if "packed-fp32-ops" not in ln and ln.strip()]
        if warn:
            sys.stderr.write("\n".join(warn) + "\n")
        print(f"[build] {lib} in {time.time() - t0:.1f}s", flush=True)
    return lib


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", help="write the library here instead of the package")
    ap.add_argument("-D", dest="defines", action="append", default=[], help="macro for every source")
    args = ap.parse_args()
    build(out=args.out, defines=args.defines)
