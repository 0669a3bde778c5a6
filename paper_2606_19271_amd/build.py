"""Builds, in-tree: libts_attn.so (the HIP kernels and their C ABI) for gfx950 with hipcc, and
libts_sched.so (the closed-loop session scheduler, host code only) with g++."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libts_attn.so")
SOURCES = [os.path.join(CSRC, "attn_kernels.hip"), os.path.join(CSRC, "state_copy.hip"),
           os.path.join(CSRC, "attn_plan.cpp"), os.path.join(CSRC, "ts_attn.cpp")]

SCHED_LIB = os.path.join(HERE, "libts_sched.so")
SCHED_SOURCES = [os.path.join(CSRC, "sched.cpp")]
# no contraction into fused multiply-adds: the scheduler's comparisons of latency gains are
# specified in plain IEEE double arithmetic
# only the C ABI is exported from either library
EXPORTS = ["-Wl,--version-script=" + os.path.join(CSRC, "exports.map")]
GXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off", "-Wall", "-Wextra",
             "-I" + INCLUDE] + EXPORTS

# Packed fp32 VALU instructions are kept out of the generated code on purpose.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Wall", "-Wno-unused-function", "-I" + INCLUDE, "-I" + CSRC] + EXPORTS


def hipcc():
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(out=LIB, extra_flags=()):
    """Compile every source into the shared library `out` (always recompiles); returns out."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + list(extra_flags) + SOURCES + ["-o", tmp]
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + proc.stdout)
    os.replace(tmp, out)
    return out


def build_sched(out=SCHED_LIB):
    """Compile the scheduler library `out` with g++ (always recompiles); returns out."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [os.environ.get("CXX", "g++")] + GXX_FLAGS + SCHED_SOURCES + ["-o", tmp]
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if proc.returncode != 0:
        raise RuntimeError("g++ failed:\n" + proc.stdout)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
    print(build_sched())
