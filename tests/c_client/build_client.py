"""Build tests/c_client/rlsim_client: plain C11 (gcc) against include/rlsim.h,
librlsim.so and the HIP runtime's C API.  Called by __graft_entry__.build()."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "rlsim_client.c")
EXE = os.path.join(HERE, "rlsim_client")
PKG = os.path.join(ROOT, "paper_2207_07736_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    tmp = EXE + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), "-o", tmp, SRC,
           "-L", PKG, "-lrlsim", "-Wl,-rpath,$ORIGIN/../../paper_2207_07736_amd", "-L", os.path.join(ROCM, "lib"),
           "-lamdhip64",
           "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build())
