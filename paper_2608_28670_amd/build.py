"""Build libbarycache.so in-tree for gfx950.

HIP sources are compiled with hipcc (device code for gfx950 only); the host
plan library (plain C++17) with g++; everything is linked into one shared
library next to this file.  Object files go to _build/.
"""
from __future__ import annotations

import hashlib
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libbarycache.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-munsafe-fp-atomics",
    # Packed fp32 instructions stay off: hipcc would otherwise form them from
    # ordinary float code.  (The host pass warns that it does not know the
    # feature; that is harmless.)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]


def _hipcc() -> str:
    p = os.path.join(ROCM, "bin", "hipcc")
    return p if os.path.exists(p) else "hipcc"


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def sources():
    hip = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    cpp = sorted(f for f in os.listdir(CSRC) if f.endswith(".cpp"))
    return hip, cpp


INCLUDE = os.path.join(os.path.dirname(HERE), "include")


def source_hash() -> str:
    """Hash of everything the library is built from: every source and header
    under csrc/ and include/, and the compiler flags.  The built library
    returns the value it was built with from bc_build_id()."""
    h = hashlib.sha256()
    files = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".h", ".cpp"))]
    files += [os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h")]
    for path in sorted(files, key=os.path.basename):
        h.update(os.path.basename(path).encode() + b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    h.update(" ".join(HIP_FLAGS + CXX_FLAGS).encode())
    return h.hexdigest()[:20]


def build(jobs: int | None = None, verbose: bool = False) -> str:
    """Compile every source and link libbarycache.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    hip, cpp = sources()
    inc = ["-I", CSRC, "-I", os.path.join(os.path.dirname(HERE), "include")]
    cmds = []
    for f in hip:
        cmds.append([_hipcc(), *HIP_FLAGS, *inc, "-c", os.path.join(CSRC, f),
                     "-o", os.path.join(BUILD, f + ".o")])
    for f in cpp:
        cmds.append(["g++", *CXX_FLAGS, *inc, "-c", os.path.join(CSRC, f),
                     "-o", os.path.join(BUILD, f + ".o")])
    jobs = jobs or min(16, os.cpu_count() or 4)
    with ThreadPoolExecutor(jobs) as ex:
        outs = list(ex.map(_run, cmds))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    # the build id: the source hash, exported as bc_build_id()
    bid_src = os.path.join(BUILD, "build_id.cpp")
    with open(bid_src, "w") as f:
        f.write('extern "C" const char* bc_build_id(void) { return "%s"; }\n' % source_hash())
    _run(["g++", *CXX_FLAGS, "-c", bid_src, "-o", bid_src + ".o"])
    objs = [os.path.join(BUILD, f + ".o") for f in hip + cpp] + [bid_src + ".o"]
    tmp = LIB + ".tmp"
    _run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs,
          f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib"])
    os.replace(tmp, LIB)
    return LIB


def clean():
    shutil.rmtree(BUILD, ignore_errors=True)
    if os.path.exists(LIB):
        os.remove(LIB)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
