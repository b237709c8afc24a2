"""Build libhxf.so (host scheduler + HIP kernels for gfx950) in-tree.

    python -m paper_2505_05286_amd.build

Every call recompiles every source.  Objects go to ``_build/`` next to this
file; the shared library is written next to this file.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libhxf.so")
BUILD = os.path.join(PKG, "_build")

SOURCES = [
    "sched.cpp",
    "decode_plan.cpp",
    "coord.cpp",
    "api.cpp",
    "ops.cpp",
    "noalloc.hip",
    "executor.hip",
    "kernels/gemm.hip",
    "kernels/norm.hip",
    "kernels/rope_kv.hip",
    "kernels/attention.hip",
    "kernels/misc.hip",
]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]
# Packed fp32 VALU ops (v_pk_*_f32) are disabled for device code: some of their forms have given
# wrong results on this part now and then, without an error.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# The attention kernels rescale their MFMA accumulators with VALU every tile: with
# accumulators in VGPRs the compiler stops copying them to and from AGPRs.
EXTRA = {"kernels/attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def _compile(src, build_dir=BUILD, host_flags=()):
    path = os.path.join(CSRC, src)
    obj = os.path.join(build_dir, src.replace("/", "_") + ".o")
    cmd = [HIPCC] + COMMON + DEVICE + EXTRA.get(src, []) + list(host_flags) + ["-c", path, "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose=False, out=OUT, build_dir=BUILD, host_flags=(), link_flags=()):
    """Compile every source and link the shared library.  host_flags / link_flags: extra
    options for the compile and link lines (e.g. instrumentation of the host code)."""
    os.makedirs(build_dir, exist_ok=True)
    jobs = max(1, min(len(SOURCES), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4))))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, host_flags), SOURCES))
    tmp = out + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}"] + list(link_flags) + ["-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
