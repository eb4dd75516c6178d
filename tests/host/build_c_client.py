"""Builds tests/host/c_client (a C program using only include/pcs.h and the
HIP runtime API) against the in-tree libpcs.so.  Called by the build entry
point, so the client exists before any GPU run, and by its test if missing."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "c_client.c")
EXE = os.path.join(HERE, "c_client")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    pkg = os.path.join(ROOT, "paper_2607_21686_amd")
    tmp = EXE + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", tmp,
           "-L", pkg, "-lpcs", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2607_21686_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build())
