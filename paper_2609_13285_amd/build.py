"""Build libgva.so (HIP, gfx950) in-tree with hipcc.

``python -m paper_2609_13285_amd.build`` compiles the kernel sources under
``csrc/`` (decode path, ordinary-RoPE contrast path, causal prefill, and the
read-bandwidth probe) to objects in parallel and links them into
``paper_2609_13285_amd/libgva.so``.  Packed-FP32 instructions are disabled for
the device code (``-packed-fp32-ops``); hipcc's host pass warns that it does
not know that feature, which is harmless.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SRCS = [os.path.join(CSRC, f) for f in ("gva_decode.hip", "gva_rope.hip", "gva_prefill.hip", "probe.hip")]
LIB = os.path.join(HERE, "libgva.so")
ARCH = "gfx950"
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument", "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libgva.so)")


def build(verbose: bool = False) -> str:
    cc = hipcc()
    with tempfile.TemporaryDirectory(prefix="gva_build_") as tmpdir:
        objs, procs = [], []
        for src in SRCS:
            obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
            objs.append(obj)
            procs.append(subprocess.Popen([cc, *FLAGS, "-c", src, "-o", obj],
                                          stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
        failed = False
        for src, pr in zip(SRCS, procs):
            out, err = pr.communicate()
            if pr.returncode != 0:
                failed = True
                sys.stderr.write(f"--- {os.path.basename(src)}\n{out}{err}")
            elif verbose:
                sys.stderr.write(err)
        if failed:
            raise RuntimeError("hipcc failed")
        tmp = LIB + ".tmp"
        res = subprocess.run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp],
                             capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc link failed ({res.returncode})")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
