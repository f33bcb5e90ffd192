"""Build libw4a8.so (all HIP sources, gfx950 only) in-tree with hipcc.

Each source compiles to its own object in parallel (the kernels of one file
never call device code of another), then one hipcc line links the shared
library.  Objects are rebuilt only when their source or a header is newer.
"""
from __future__ import annotations

import glob
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libw4a8.so")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")

# -ffp-contract=off: the quantizers must round every fp32 step on its own;
# fused multiply-adds are written explicitly (fmaf) where they are wanted.
# The target-feature flag keeps the compiler from emitting packed fp32 math.
# -amdgpu-mfma-vgpr-form: matrix products write ordinary VGPRs, so the fp32
# scaling reads their results without a copy out of the accumulator file.
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-mfma-vgpr-form", "-Wall",
]
# the host pass does not know the packed-fp32 feature name: harmless
_NOISE = "packed-fp32-ops' is not a recognized feature"


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _headers():
    return glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(INCLUDE, "*.h"))


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (res.stdout + res.stderr).splitlines() if _NOISE not in l]
    return res.returncode, msgs


def build(verbose: bool = False, force: bool = True) -> str:
    """Compile every source (all of them when `force`, else only the stale
    ones) and link libw4a8.so."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJ, exist_ok=True)
    newest_header = max((os.path.getmtime(h) for h in _headers()), default=0.0)
    jobs = []
    objs = []
    for src in sources():
        obj = os.path.join(OBJ, os.path.basename(src)[:-4] + ".o")
        objs.append(obj)
        stale = (force or not os.path.exists(obj) or
                 os.path.getmtime(obj) < max(os.path.getmtime(src), newest_header))
        if stale:
            jobs.append((src, obj))
    errors, notes = [], []

    def compile_one(job):
        src, obj = job
        rc, msgs = _run([hipcc, *HIPCC_FLAGS, "-c", "-o", obj + ".tmp", src])
        return src, obj, rc, msgs

    with ThreadPoolExecutor(max_workers=min(8, max(1, len(jobs)))) as ex:
        for src, obj, rc, msgs in ex.map(compile_one, jobs):
            if rc != 0:
                errors.append(f"{os.path.basename(src)}:\n" + "\n".join(msgs))
            else:
                os.replace(obj + ".tmp", obj)
                notes.extend(msgs)
    if errors:
        raise RuntimeError("hipcc failed:\n" + "\n".join(errors))
    rc, msgs = _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", LIB + ".tmp",
                     *objs])
    if rc != 0:
        raise RuntimeError("link failed:\n" + "\n".join(msgs))
    if verbose and (notes or msgs):
        print("\n".join(notes + msgs))
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    import sys
    print(build(verbose=True, force="--incremental" not in sys.argv))
