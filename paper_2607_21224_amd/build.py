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
# the same sources with 256-thread blocks: a different launch shape for the
# tests that check results do not depend on it
LIB_CPDP_BLOCK256 = os.path.join(PKG, "libcpdp_block256.so")
LIB_SYNTH = os.path.join(ROOT, "synth", "libsynth.so")

# -ffp-contract=off: only the explicit fmaf calls fuse, so the arithmetic is
# exactly what the source says.  Packed fp32 instructions are disabled.
COMPILE_FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
                 "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang",
                 "-packed-fp32-ops", "-Wall", "-Wno-unused-command-line-argument"]
HIP_FLAGS = COMPILE_FLAGS + ["-shared"]

# the kernel translation units of libcpdp.so (compiled in parallel) and the
# host validation layer
KERNEL_SOURCES = ("kernels_flat.hip", "kernels_sync_cpdp.hip", "kernels_sync_localsgd.hip",
                  "kernels_sync_ddp.hip", "kernels_plan.hip", "kernels_plan_table.hip",
                  "kernels_table.hip", "kernels_check.hip")
# headers the kernel sources include (part of what the recorded traffic is for)
KERNEL_HEADERS = ("cpdp_device.h", "cpdp_sync_impl.h", "cpdp_plan_impl.h", "cpdp_launch.h")
HOST_SOURCES = ("cpdp_api.cpp",)
# the library's own device memory (no kernels): the static plan table
SCRATCH_SOURCES = ("plan_scratch.hip",)
OBJ_ROOT = os.path.join(ROOT, "_build")


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)


def build_cpdp(out: str = LIB_CPDP, extra=()) -> str:
    from concurrent.futures import ThreadPoolExecutor
    csrc = os.path.join(PKG, "csrc")
    objdir = os.path.join(OBJ_ROOT, os.path.basename(out) + ".objs")
    os.makedirs(objdir, exist_ok=True)
    sources = KERNEL_SOURCES + HOST_SOURCES + SCRATCH_SOURCES

    def compile_one(name):
        obj = os.path.join(objdir, name + ".o")
        _run([HIPCC, *COMPILE_FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-I", csrc,
              "-c", "-o", obj, os.path.join(csrc, name)])
        return obj

    with ThreadPoolExecutor(len(sources)) as ex:
        objs = list(ex.map(compile_one, sources))
    tmp = out + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
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
                ex.submit(build_cpdp, LIB_CPDP_BLOCK256, ("-DCPDP_BLOCK=256",))]
        for j in jobs:
            j.result()
    build_consumer()


if __name__ == "__main__":
    build_all()
    print("built", LIB_CPDP, LIB_SYNTH)
