"""Build the gfx950 HIP library ``libgrkv.so`` in-tree.

``python -m paper_2605_31105_amd.build`` compiles every source under ``csrc/``
with hipcc for gfx950 and links them into ``paper_2605_31105_amd/libgrkv.so``.
Objects go to ``_build/`` at the repository root.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libgrkv.so")
SOURCES = ["attention.hip", "stream.hip", "selection.hip", "merge.hip", "solve_big.hip", "merge_generic.hip", "key.hip", "key_ring.hip", "carrier.hip", "frontend.hip",
           "h2o.hip", "noalloc.hip", "api.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions are kept out of generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    noise = ("packed-fp32-ops", "is not a recognized feature")
    msg = "\n".join(l for l in r.stdout.splitlines() if not any(s in l for s in noise))
    if r.returncode != 0:
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), msg))
    return msg


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile all sources (always) and link libgrkv.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    objs = [os.path.join(BUILD, s.replace(".hip", ".o")) for s in SOURCES]

    def compile_one(pair):
        src, obj = pair
        return _run([HIPCC, *FLAGS, *extra_flags, "-c", os.path.join(CSRC, src), "-o", obj])

    with ThreadPoolExecutor(len(SOURCES)) as ex:
        for msg in ex.map(compile_one, zip(SOURCES, objs)):
            if verbose and msg.strip():
                print(msg)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
