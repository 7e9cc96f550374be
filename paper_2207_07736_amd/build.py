"""Build librlsim.so (the HIP kernels and the C ABI) and librlsim_probe.so (the
store-only probe the bench measures the store ceiling with, and the error probe
of the policy kernel's elementwise functions) for gfx950 with hipcc.

Floating-point flags matter for the results: no contraction of a*b+c into an
FMA unless written, IEEE single-precision division, denormals kept, and no
packed-FP32 instructions.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "rlsim.hip")
LIB = os.path.join(HERE, "librlsim.so")
PROBE_SRCS = [os.path.join(HERE, "csrc", "store_probe.hip")]      # includes math_probe.hip.h
PROBE_LIB = os.path.join(HERE, "librlsim_probe.so")
INCLUDE = os.path.join(ROOT, "include")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-ffp-contract=off",
    "-fno-fast-math",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",   # MFMA accumulators in VGPRs: no AGPR copies before tanh
    "-Wall",
    "-Wno-unused-command-line-argument",
]


def sources():
    csrc = os.path.join(HERE, "csrc")
    return [os.path.join(csrc, f) for f in sorted(os.listdir(csrc))] + [os.path.join(INCLUDE, "rlsim.h")]


def build(verbose: bool = False) -> str:
    """Compile csrc/rlsim.hip into librlsim.so and the probe sources into
    librlsim_probe.so next to this file (always).  Returns the main library."""
    _compile([SRC], LIB, verbose)
    _compile(PROBE_SRCS, PROBE_LIB, verbose)
    return LIB


def _compile(srcs: list, lib: str, verbose: bool) -> None:
    tmp = lib + ".tmp"
    cmd = [HIPCC, *FLAGS, "-I", INCLUDE, "-o", tmp, *srcs]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature: drop that warning
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l and "(ignoring feature)" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, lib)


def asm(out_path: str, src: str = SRC) -> str:
    """Write the gfx950 assembly of a source's device code (for inspection)."""
    cmd = [HIPCC, *[f for f in FLAGS if f not in ("-shared", "-fPIC")], "-I", INCLUDE,
           "--cuda-device-only", "-S", "-o", out_path, src]
    subprocess.run(cmd, check=True)
    return out_path


def device_object(out_path: str, src: str = SRC) -> str:
    """Write the gfx950 code object of a source's device code (for inspection
    with llvm-objdump)."""
    bundled = out_path + ".bundle"
    cmd = [HIPCC, *[f for f in FLAGS if f not in ("-shared", "-fPIC")], "-I", INCLUDE,
           "--cuda-device-only", "-c", "-o", bundled, src]
    subprocess.run(cmd, check=True)
    bundler = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "bin", "clang-offload-bundler")
    subprocess.run([bundler, "--unbundle", "--type=o", f"--input={bundled}",
                    "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--output={out_path}"], check=True)
    return out_path


if __name__ == "__main__":
    print(build(verbose=True))
