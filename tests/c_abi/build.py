"""Compiles tests/c_abi/caller.c, a plain C client of libts_attn.so, with gcc against the HIP
runtime.  Test infrastructure: only tests/test_gpu_c_abi.py runs the program."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "caller.c")
EXE = os.path.join(HERE, "caller")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(out=EXE):
    """Compile caller.c into out; the library is found next to the package ($ORIGIN-relative)."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I" + os.path.join(ROCM, "include"), "-I" + os.path.join(ROOT, "include"), SRC,
           "-o", tmp, "-L" + os.path.join(ROOT, "paper_2606_19271_amd"), "-lts_attn",
           "-L" + os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2606_19271_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
