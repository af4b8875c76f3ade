"""Builds libonebit.so (the gfx950 HIP kernels and the C ABI) in-tree, and
the HBM streaming probe's own library lib/libhbmprobe.so."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("onebit_kernels.hip", "onebit_abi.hip")]
LIB = os.path.join(HERE, "lib", "libonebit.so")
PROBE_SOURCE = os.path.join(HERE, "csrc", "hbm_probe.hip")
PROBE = os.path.join(HERE, "lib", "libhbmprobe.so")

# -ffp-contract=off: every fp32 operation is rounded once, as the method's
# arithmetic is specified (no fused multiply-add contraction).
# -packed-fp32-ops: keep the compiler from emitting packed fp32 instructions.
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc(flags, sources, target, verbose):
    os.makedirs(os.path.dirname(target), exist_ok=True)
    tmp = target + ".tmp%d" % os.getpid()
    cmd = ["hipcc"] + flags + ["-o", tmp] + sources
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l and "unused during compilation" not in l)
    if r.returncode != 0:
        sys.stderr.write(out + "\n")
        raise RuntimeError("hipcc failed building " + os.path.basename(target))
    if verbose and out.strip():
        print(out)
    os.replace(tmp, target)
    return target


def build(verbose: bool = False) -> str:
    _hipcc(HIPCC_FLAGS, SOURCES, LIB, verbose)
    _hipcc(HIPCC_FLAGS, [PROBE_SOURCE], PROBE, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
