"""Build the gfx950 shared library of the CPDP path (and the synthetic-input
library the tests and benchmark use) with hipcc, in-tree."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

LIB_CPDP = os.path.join(PKG, "libcpdp.so")
# the same sources with 64-thread blocks: a different launch shape for the
# tests that check results do not depend on it
LIB_CPDP_BLOCK64 = os.path.join(PKG, "libcpdp_block64.so")
LIB_SYNTH = os.path.join(ROOT, "synth", "libsynth.so")

# -ffp-contract=off: only the explicit fmaf calls fuse, so the arithmetic is
# exactly what the source says.  Packed fp32 instructions are disabled.
HIP_FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
             "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-Wall", "-Wno-unused-command-line-argument"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)


def build_cpdp(out: str = LIB_CPDP, extra=()) -> str:
    csrc = os.path.join(PKG, "csrc")
    tmp = out + ".tmp"
    _run([HIPCC, *HIP_FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-I", csrc,
          "-o", tmp, os.path.join(csrc, "cpdp_kernels.hip"),
          os.path.join(csrc, "cpdp_api.cpp")])
    os.replace(tmp, out)
    return out


def build_synth(out: str = LIB_SYNTH) -> str:
    tmp = out + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-o", tmp, os.path.join(ROOT, "synth", "synth.hip")])
    os.replace(tmp, out)
    return out


CONSUMER = os.path.join(ROOT, "tests", "consumer", "abi_consumer")


def build_consumer(out: str = CONSUMER) -> str:
    """The torch-free host program of the ABI tests, linked to libcpdp.so."""
    tmp = out + ".tmp"
    _run([HIPCC, "-O2", "-std=c++17", "-Wall", "-I", os.path.join(ROOT, "include"),
          "-o", tmp, out + ".cpp", "-L", PKG, "-lcpdp",
          "-Wl,-rpath,$ORIGIN/../../paper_2607_21224_amd"])
    os.replace(tmp, out)
    return out


def build_all() -> None:
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(3) as ex:
        jobs = [ex.submit(build_cpdp), ex.submit(build_synth),
                ex.submit(build_cpdp, LIB_CPDP_BLOCK64, ("-DCPDP_BLOCK=64",))]
        for j in jobs:
            j.result()
    build_consumer()


if __name__ == "__main__":
    build_all()
    print("built", LIB_CPDP, LIB_SYNTH)
