"""Build libmoe.so (the C-ABI library of gfx950 HIP kernels) in-tree with hipcc."""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
PROBE = os.path.join(HERE, "probe")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(HERE, "libmoe.so")
# measurement probes (not part of the MoE path or its C ABI), a library of their own
PROBE_LIB_PATH = os.path.join(HERE, "libmoe_probe.so")
ARCH = "gfx950"

# -packed-fp32-ops: keep the compiler from emitting packed fp32 arithmetic.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the gfx950 library cannot be built")
    return path


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [hipcc(), *HIP_FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def _link(objs, path: str):
    tmp = path + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, path)


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libmoe.so next to this file, and the
    measurement probes into libmoe_probe.so."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources()
    probes = sorted(glob.glob(os.path.join(PROBE, "*.hip")))
    with ThreadPoolExecutor(min(8, len(srcs) + len(probes))) as ex:
        objs = list(ex.map(_compile, srcs + probes))
    _link(objs[:len(srcs)], LIB_PATH)
    if probes:
        _link(objs[len(srcs):], PROBE_LIB_PATH)
    if verbose:
        print(f"built {LIB_PATH}" + (f" and {PROBE_LIB_PATH}" if probes else ""))
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
