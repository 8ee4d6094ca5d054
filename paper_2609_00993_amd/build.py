"""Build libmoepd.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2609_00993_amd.build

Each source under csrc/ is compiled to an object in _build/ (at the repo
root, git-ignored), then linked into paper_2609_00993_amd/libmoepd.so.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libmoepd.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    # hipcc -O3 forms packed fp32 instructions on its own; keep them off.
    "-Xclang",
    "-target-feature",
    "-Xclang",
    "-packed-fp32-ops",
    f"-I{INCLUDE}",
    f"-I{CSRC}",
]


# Host-only sources (the turnstile and the P-epoch runner) take the host
# compiler: they include the HIP runtime API but hold no device code.
CXX = os.environ.get("CXX", "g++")
HOST_CFLAGS = [
    "-O2",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-pthread",
    "-D__HIP_PLATFORM_AMD__",
    f"-I{os.environ.get('ROCM_PATH', '/opt/rocm')}/include",
    f"-I{INCLUDE}",
    f"-I{CSRC}",
]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def _compile_cmd(src, obj):
    if src.endswith(".cpp"):
        return [CXX, *HOST_CFLAGS, "-c", src, "-o", obj]
    return [HIPCC, *CFLAGS, "-c", src, "-o", obj]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    return p.returncode, out


def build(verbose: bool = False, jobs: int = 8) -> str:
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(BUILD, os.path.splitext(os.path.basename(s))[0] + ".o") for s in srcs]
    cmds = [_compile_cmd(s, o) for s, o in zip(srcs, objs)]
    with cf.ThreadPoolExecutor(max_workers=min(jobs, len(cmds))) as ex:
        results = list(ex.map(_run, cmds))
    for cmd, (rc, out) in zip(cmds, results):
        if verbose or rc:
            print(" ".join(cmd))
            if out.strip():
                print(out)
        if rc:
            raise RuntimeError(f"compile failed: {cmd[-3]}")
    tmp = LIB + ".tmp"
    rc, out = _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-pthread", "-o", tmp, *objs])
    if rc:
        print(out)
        raise RuntimeError("link failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
