"""Build libdvs.so (the C-ABI library) for gfx950 with hipcc, in-tree.

    python -m paper_2609_26638_amd.build        # or: from ... import build; build.build()

Every HIP translation unit under csrc/ is compiled to an object in _build/
(in parallel), then linked into paper_2609_26638_amd/libdvs.so.  Always
recompiles: this is the "does it build" check as well as the build.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build", "dvs")
LIB = os.path.join(PKG, "libdvs.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # never emit packed fp32 VALU ops (v_pk_fma_f32 and friends)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result", "-Wno-unused-command-line-argument",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    return p.returncode, out


def build(verbose: bool = False, jobs: int = 8) -> str:
    if not os.path.exists(HIPCC) and shutil.which("hipcc") is None:
        raise RuntimeError("hipcc not found; cannot build libdvs.so")
    hipcc = HIPCC if os.path.exists(HIPCC) else shutil.which("hipcc")
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    objs = []
    cmds = []
    for s in srcs:
        o = os.path.join(BUILD_DIR, os.path.basename(s)[:-4] + ".o")
        objs.append(o)
        cmds.append([hipcc, *COMMON_FLAGS, "-c", s, "-o", o])
    with cf.ThreadPoolExecutor(max_workers=min(jobs, len(cmds))) as ex:
        results = list(ex.map(_run, cmds))
    for cmd, (rc, out) in zip(cmds, results):
        if verbose or rc != 0:
            sys.stderr.write(" ".join(cmd) + "\n" + out + "\n")
        if rc != 0:
            raise RuntimeError(f"hipcc failed for {cmd[-3]}")
    tmp = LIB + ".tmp"
    rc, out = _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    if rc != 0:
        sys.stderr.write(out + "\n")
        raise RuntimeError("link of libdvs.so failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
