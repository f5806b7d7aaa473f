"""Build the gfx950 sampling library ``libalbireo.so`` in-tree with hipcc (one object per source,
compiled in parallel, then linked)."""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", n) for n in ("albireo.hip", "stream.hip", "state.hip")]
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libalbireo.so")

HIPCC_FLAGS = [
    "-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC",
    # bit-exact processed logits: no contraction of the canonical fp32 multiplies and adds
    "-ffp-contract=off",
    # a host function whose every path calls itself fails the build (clang leaves this warning off)
    "-Werror=infinite-recursion",
    # no packed fp32 instructions (v_pk_*_f32) anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def build(out: str = LIB, extra=()) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    with tempfile.TemporaryDirectory(prefix="albireo_build_") as tmpd:
        objs = [os.path.join(tmpd, os.path.basename(src) + ".o") for src in SRCS]

        def compile_one(pair):
            src, obj = pair
            subprocess.check_call([hipcc, *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-c", src, "-o", obj])

        with concurrent.futures.ThreadPoolExecutor(max_workers=len(SRCS)) as ex:
            list(ex.map(compile_one, zip(SRCS, objs)))
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(extra=sys.argv[1:]))
