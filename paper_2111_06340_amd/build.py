"""Build the HIP library libhmmgpu.so in-tree for gfx950 (hipcc).

Every call compiles from source.  The packed-FP32 target feature is turned
off for all device code: the compiler must not form packed fp32 ops."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libhmmgpu.so")
SOURCES = ["hmm_host.cpp", "hmm_kernels.hip", "hmm_decode.hip", "hmm_coop.hip", "hmm_probe.hip"]
ARCH = os.environ.get("HMM_OFFLOAD_ARCH", "gfx950")

DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    return os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def build(verbose: bool = False, save_temps: str | None = None) -> str:
    """Compile every source (concurrently) and link the shared library."""
    cmds, objs = [], []
    for src in SOURCES:
        obj = os.path.join(CSRC, src + ".o")
        cmd = [hipcc(), "-x", "hip", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
               "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
               *DEVICE_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        if save_temps:
            cmd.insert(1, f"-save-temps={save_temps}")
        if verbose:
            print(" ".join(cmd), flush=True)
        cmds.append(cmd)
        objs.append(obj)
    jobs = max(1, min(len(cmds), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
    with ThreadPoolExecutor(jobs) as ex:
        for f in [ex.submit(subprocess.check_call, c, cwd=save_temps or CSRC) for c in cmds]:
            f.result()
    tmp = LIB + ".tmp"
    subprocess.check_call([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    for o in objs:
        os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
