"""Build the native libraries in-tree.

libpagedweight.so : HIP kernels (gfx950) + C ABI (include/pw.h); hipcc.
libpw_hosttest.so : the host-side page-table protocol alone, built with g++,
                    for CPU tests of the allocator and commit/reclaim logic.
"""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INC = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libpagedweight.so")
HOSTLIB = os.path.join(HERE, "libpw_hosttest.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 instructions are disabled for all device code.
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-I" + INC, "-I" + CSRC,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-function"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops' is not a recognized" not in l)
    if r.returncode != 0:
        sys.stderr.write(out + "\n")
        raise RuntimeError("build failed: " + " ".join(cmd[:3]) + " ...")
    return out


# Per-file device flags. The decode GEMMs keep their MFMA accumulators in
# architectural VGPRs: each group's partial product is read back by VALU code
# right after its last MFMA, and VGPR destinations avoid the AGPR moves.
SOURCES = {
    "pw_kernels.hip": [],
    "pw_decode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "pw_tgemm.hip": [],
    "pw_probe.hip": [],
    "pw_scratch.hip": [],
    "pw_api.cpp": [],
    "pw_state.cpp": [],
    "pw_plan.cpp": [],
}


def build_hip(verbose=False):
    """Compile every source (in parallel) and link libpagedweight.so."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    procs, objs = [], []
    for src, flags in SOURCES.items():
        obj = os.path.join(objdir, src + ".o")
        extra = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [HIPCC] + HIP_FLAGS + flags + extra + ["-c", os.path.join(CSRC, src), "-o", obj]
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
        objs.append(obj)
    failed = []
    for cmd, p in procs:
        out = "\n".join(l for l in p.communicate()[0].splitlines() if "packed-fp32-ops' is not a recognized" not in l)
        if p.returncode != 0:
            sys.stderr.write(out + "\n")
            failed.append(os.path.basename(cmd[-3]))
        elif verbose and out:
            print(out)
    if failed:
        raise RuntimeError("build failed: " + ", ".join(failed))
    tmp = LIB + ".tmp%d" % os.getpid()
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs)
    os.replace(tmp, LIB)
    return LIB


def build_hosttest():
    tmp = HOSTLIB + ".tmp%d" % os.getpid()
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-Wall", "-I" + INC, "-I" + CSRC,
          os.path.join(CSRC, "pw_state.cpp"), os.path.join(CSRC, "pw_hosttest.cpp"), "-o", tmp])
    os.replace(tmp, HOSTLIB)
    return HOSTLIB


def build_all(verbose=False):
    build_hosttest()
    return build_hip(verbose)


if __name__ == "__main__":
    print(build_all(verbose=True))
