"""Build ``libtlc.so`` (gfx950 HIP kernels + C ABI) in-tree with hipcc."""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libtlc.so")
# The stress build of the look-back scans: every status-word publish sleeps
# a pseudo-random while first (TLC_DELAY_INJECT); used only by
# tests/test_gpu_lookback_delays.py.
LIB_DELAY = os.path.join(PKG, "libtlc_delay.so")
SOURCES = ["encode.hip", "decode.hip", "int8.hip", "tlc_api.hip", "noalloc.hip"]
HEADERS = ["tlc_internal.h", "device_common.hpp", "lookback.hpp", "wave_scan.hpp", "zre_scan.hpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    "-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-shared",
    "-fvisibility=hidden",
    # fp32 results must be the IEEE operations of the method, bit for bit
    "-ffp-contract=off", "-fno-fast-math",
    # no packed-fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def sources():
    return [os.path.join(CSRC, s) for s in SOURCES]


def deps():
    return sources() + [os.path.join(CSRC, h) for h in HEADERS] + [
        os.path.join(ROOT, "include", "tlc.h")]


def stale():
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(d) > t for d in deps())


def build(verbose=False, delay=False):
    """Compile libtlc.so (delay=True: the stress build libtlc_delay.so)."""
    out = LIB_DELAY if delay else LIB
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *(["-DTLC_DELAY_INJECT"] if delay else []),
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-o", tmp, *sources()]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv, delay="--delay" in sys.argv))
