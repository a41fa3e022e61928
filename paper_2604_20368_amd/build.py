"""Build the gfx950 HIP library ``liblapattn.so`` in-tree with hipcc.

Run ``python -m paper_2604_20368_amd.build`` (or call ``build()``); the library is
placed next to this file, where the binding loads it from.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "liblapattn.so")
SOURCES = ["fwd.hip", "fast.hip", "nsbig.hip", "bwd.hip", "dwc.hip", "noalloc.hip", "host.cpp"]
ARCH = "gfx950"

# Packed fp32 VALU instructions are disabled for every device pass (the compiler would
# otherwise form them from plain float code).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(verbose=False, jobs=4):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objs = []
    procs = []
    for src in SOURCES:
        path = os.path.join(CSRC, src)
        obj = os.path.join(CSRC, "_build_" + os.path.splitext(src)[0] + ".o")
        cmd = [hipcc, "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
               "-I", os.path.join(HERE, "..", "include"), "-c", path, "-o", obj] + DEVICE_FLAGS
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((subprocess.Popen(cmd, stderr=subprocess.PIPE, text=True), src))
        objs.append(obj)
    failed = []
    for p, src in procs:
        _, err = p.communicate()
        if p.returncode != 0:
            failed.append((src, err))
        elif err and verbose:
            sys.stderr.write(err)
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join("%s:\n%s" % f for f in failed))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    for o in objs:
        os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
