"""Builds the two libraries in-tree with hipcc for gfx950:

* libnmspmm.so -- the method (C ABI in include/nmspmm.h and include/nmsearch.h),
  from csrc/*.cpp and csrc/*.hip;
* libnmprobe.so -- measurement and test aids (include/nmprobe.h), from
  csrc/probe/*.hip, linked against libnmspmm.so for the GEMM kernels its
  store-only probe launches.
"""
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libnmspmm.so")
PROBE_LIB = os.path.join(HERE, "libnmprobe.so")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
    # packed fp32 instructions are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
_NOISE = "is not a recognized feature for this target"


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.cpp")) + glob.glob(os.path.join(CSRC, "*.hip")))


def probe_sources():
    return sorted(glob.glob(os.path.join(CSRC, "probe", "*.hip")))


def _hipcc(cmd, out, verbose):
    tmp = out + ".tmp"
    cmd = cmd + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in proc.stderr.splitlines() if _NOISE not in l)
    if proc.returncode != 0:
        raise RuntimeError(f"hipcc failed ({proc.returncode}):\n{err}")
    if verbose and err.strip():
        print(err)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    _hipcc(["hipcc", *FLAGS, f"-I{INCLUDE}", *sources()], LIB, verbose)
    _hipcc(["hipcc", *FLAGS, f"-I{INCLUDE}", *probe_sources(), f"-L{HERE}", "-lnmspmm",
            "-Wl,-rpath,$ORIGIN"], PROBE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
