"""Build liblram.so for gfx950 with hipcc (in-tree, under paper_2107_03474_amd/_build)."""
from __future__ import annotations

import glob
import hashlib
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(BUILD, "liblram.so")
SOURCES = [os.path.join(CSRC, "lram.hip")]
DEPS = SOURCES + sorted(glob.glob(os.path.join(CSRC, "*.h"))) + [
    os.path.join(CSRC, "e8_candidates.inc"), os.path.join(ROOT, "include", "lram.h")]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # the fp32 distance recipe must not be fused into FMAs; FMAs are written out where wanted
    "-ffp-contract=off",
    # hardware fp32 atomic add for the value-gradient scatter
    "-munsafe-fp-atomics",
    # no packed-fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


def _code_text(path: str) -> bytes:
    """A source file with its comments dropped and whitespace collapsed: edits
    that cannot change the compiled code leave it unchanged."""
    with open(path, encoding="utf-8") as f:
        txt = f.read()
    txt = re.sub(r"/\*.*?\*/", " ", txt, flags=re.S)
    txt = re.sub(r"//[^\n]*", " ", txt)
    return " ".join(txt.split()).encode()


def source_digest() -> str:
    """sha256 over the code of every file the library is compiled from (names
    and comment-free text, in a fixed order)."""
    h = hashlib.sha256()
    for d in DEPS:
        h.update(os.path.relpath(d, ROOT).encode() + b"\0")
        h.update(_code_text(d) + b"\0")
    return h.hexdigest()


def build(force: bool = True, verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    if not force and os.path.exists(LIB) and all(os.path.getmtime(LIB) >= os.path.getmtime(d) for d in DEPS):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + ["-I", os.path.join(ROOT, "include")] + SOURCES + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(force=True, verbose="-v" in sys.argv))
