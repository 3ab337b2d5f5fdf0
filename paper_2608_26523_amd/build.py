"""Build the native libraries in-tree: the HIP attention library (hipcc for gfx950) into
paper_2608_26523_amd/libvpp_chunk_attn.so, and the host-only schedule model (g++) into
paper_2608_26523_amd/libvpp_sched.so."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "vpp_chunk_attn.hip")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libvpp_chunk_attn.so")
SCHED_SRC = os.path.join(PKG, "csrc", "vpp_sched.cpp")
SCHED_LIB = os.path.join(PKG, "libvpp_sched.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++20", "-fPIC", "-shared",
    # no packed fp32 instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


PARTS = (0, 1, 2)  # VPP_PART values: host code + contiguous-cache kernels, paged, split-key


def build(extra_flags=(), out: str = LIB, quiet: bool = True, src: str = None) -> str:
    """Compile the parts of the HIP source in parallel (one hipcc each), then link."""
    src = src or SRC
    base = [hipcc()] + HIPCC_FLAGS + list(extra_flags) + ["-I", INCLUDE]
    objs = [out + ".part%d.o" % part for part in PARTS]
    procs = []
    for part, obj in zip(PARTS, objs):
        cmd = [c for c in base if c != "-shared"] + ["-c", "-DVPP_PART=%d" % part, "-o", obj, src]
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    outs = [pr.communicate()[0] for pr in procs]
    msgs = [ln for o in outs for ln in o.splitlines() if "packed-fp32-ops" not in ln and ln.strip()]
    if any(pr.returncode != 0 for pr in procs):
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    tmp = out + ".tmp"
    res = subprocess.run(base + ["-o", tmp] + objs, capture_output=True, text=True)
    msgs += [ln for ln in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in ln and ln.strip()]
    for obj in objs:
        if os.path.exists(obj):
            os.remove(obj)
    if res.returncode != 0:
        raise RuntimeError("hipcc link failed:\n" + "\n".join(msgs))
    if msgs and not quiet:
        print("\n".join(msgs), file=sys.stderr)
    os.replace(tmp, out)
    return out


def build_sched(out: str = SCHED_LIB) -> str:
    """The schedule model is plain host C++: no HIP, so it loads on any machine."""
    tmp = out + ".tmp"
    cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-I", INCLUDE, "-o", tmp, SCHED_SRC]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("g++ failed:\n" + res.stdout + res.stderr)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(quiet=False))
    print(build_sched())
