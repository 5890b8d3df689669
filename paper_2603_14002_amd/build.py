"""Builds liblightbeam.so (hipcc, gfx950) in-tree.

    python -m paper_2603_14002_amd.build
"""

from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "liblightbeam.so")
SOURCES = ["lb_kernels.hip", "lb_api.cpp"]
# k_decode loops over frames: machine-level hoisting of loop-invariant values
# out of that loop keeps them live across it and makes the kernel spill
EXTRA = {"lb_kernels.hip": ["-mllvm", "-disable-machine-licm"]}
ARCH = os.environ.get("LB_OFFLOAD_ARCH", "gfx950")

COMMON = [
    "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"--offload-arch={ARCH}",
]


# every file whose text goes into the library, for its build id
HASHED = [os.path.join(CSRC, f) for f in ("lb_kernels.hip", "lb_device.h", "lb_launch.h", "lb_api.cpp")] + \
    [os.path.join(os.path.dirname(HERE), "include", "lightbeam.h")]


def source_hash() -> str:
    """sha256 over the library's sources with comments and spacing removed, and
    over the build flags: the build id compiled into liblightbeam.so, and the
    id that the binding expects of a library built from this tree."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in HASHED:
        with open(f) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(os.path.basename(f).encode() + b"\0" + " ".join(text.split()).encode() + b"\0")
    h.update(" ".join(COMMON + [f"{k}:{' '.join(v)}" for k, v in sorted(EXTRA.items())]).encode())
    return h.hexdigest()


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    cc = hipcc()
    build_id = [f'-DLB_BUILD_ID="{source_hash()}"']
    with tempfile.TemporaryDirectory(prefix="lb_build_") as tmp:
        objs, procs = [], []
        for src in SOURCES:  # the sources compile concurrently
            obj = os.path.join(tmp, os.path.splitext(src)[0] + ".o")
            cmd = [cc, *COMMON, *EXTRA.get(src, []), *build_id, "-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
        failed = []
        for src, pr in procs:
            out, _ = pr.communicate()
            if pr.returncode != 0:
                sys.stderr.write(out)
                failed.append(src)
        if failed:
            raise RuntimeError(f"hipcc failed on {', '.join(failed)}")
        out_tmp = LIB + ".tmp"
        cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out_tmp, *objs]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            sys.stderr.write(r.stdout + r.stderr)
            raise RuntimeError("link failed")
        os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
