"""Builds the plain-C check of the ABI (tests/c/abi_step_check.c) against the
built libonebit.so and the oracle library."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
BIN = os.path.join(HERE, "_build", "abi_step_check")


def build(verbose=False):
    os.makedirs(os.path.dirname(BIN), exist_ok=True)
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I" + os.path.join(ROOT, "include"), os.path.join(HERE, "abi_step_check.c"),
           "-o", BIN,
           "-L" + os.path.join(ROOT, "paper_2102_02888_amd", "lib"), "-lonebit",
           "-L" + os.path.join(ROOT, "oracle", "_build"), "-loracle",
           "-L/opt/rocm/lib", "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../../paper_2102_02888_amd/lib",
           "-Wl,-rpath,$ORIGIN/../../../oracle/_build", "-Wl,-rpath,/opt/rocm/lib"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return BIN


if __name__ == "__main__":
    print(build(verbose=True))
