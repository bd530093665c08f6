"""Build libmaddness.so for gfx950 in-tree with hipcc (always recompiles).

Each source is compiled to an object in its own hipcc process (in parallel),
then the objects are linked into the shared library.  Kernels are launched
only from the translation unit that defines them, so no relocatable device
code is needed.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["csrc/kernels.hip", "csrc/fused_gather.hip", "csrc/fused_rows.hip", "csrc/tiled_accum.hip",
           "csrc/row_lanes.hip", "csrc/onehot_mfma.hip", "csrc/lut_build.hip", "csrc/lut_fit.hip", "csrc/api.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # every multiply-add is written explicitly; nothing is contracted
    "-ffp-contract=off",
    # no packed fp32 instructions anywhere
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]
NOISE = "packed-fp32-ops"


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in r.stderr.splitlines() if NOISE not in l)
    return r.returncode, errs


def build(verbose: bool = False, jobs: int = 0) -> str:
    out = os.path.join(HERE, "libmaddness.so")
    tmp = out + ".tmp"
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
    jobs = jobs or min(len(SOURCES), max(1, os.cpu_count() or 1))
    with tempfile.TemporaryDirectory(prefix="mdn_build_") as tdir:
        objs, cmds = [], []
        for s in SOURCES:
            obj = os.path.join(tdir, os.path.basename(s) + ".o")
            objs.append(obj)
            cmds.append([HIPCC, *FLAGS, *inc, "-c", os.path.join(HERE, s), "-o", obj])
        if verbose:
            for c in cmds:
                print(" ".join(c), flush=True)
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            results = list(ex.map(_run, cmds))
        for (rc, errs), c in zip(results, cmds):
            if rc != 0:
                raise RuntimeError(f"hipcc failed ({rc}) on {c[-3]}:\n{errs}")
            if verbose and errs.strip():
                print(errs, file=sys.stderr)
        link = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(link), flush=True)
        rc, errs = _run(link)
        if rc != 0:
            raise RuntimeError(f"link failed ({rc}):\n{errs}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
