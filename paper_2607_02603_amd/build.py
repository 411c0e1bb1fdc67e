"""Build step of the gfx950 library and of the input generators.

    python -m paper_2607_02603_amd.build

compiles, in-tree:
  paper_2607_02603_amd/libwl.so                 (hipcc, the C ABI of include/wl.h)
  paper_2607_02603_amd/inputs/libwlgen_cpu.so   (gcc, seeded graph samplers)
  paper_2607_02603_amd/inputs/libwlgen_gpu.so   (hipcc, the same samplers on the GPU)
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = os.environ.get("WL_OFFLOAD_ARCH", "gfx950")
# Packed-FP32 instructions are disabled for every HIP translation unit.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

LIB_WL = os.path.join(HERE, "libwl.so")
LIB_GEN_CPU = os.path.join(HERE, "inputs", "libwlgen_cpu.so")
LIB_GEN_GPU = os.path.join(HERE, "inputs", "libwlgen_gpu.so")


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("build failed: " + " ".join(cmd))
    return r


def _atomic_build(cmd, out):
    tmp = out + ".tmp"
    _run(cmd + ["-o", tmp])
    os.replace(tmp, out)


def build_wl():
    src = os.path.join(HERE, "csrc", "wl_lib.hip")
    _atomic_build([HIPCC] + HIP_FLAGS + ["-I", os.path.join(ROOT, "include"), src],
                  LIB_WL)
    return LIB_WL


def build_inputs():
    d = os.path.join(HERE, "inputs")
    _atomic_build(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                   os.path.join(d, "gen_cpu.c"), "-lm"], LIB_GEN_CPU)
    _atomic_build([HIPCC] + HIP_FLAGS + [os.path.join(d, "gen_gpu.hip")], LIB_GEN_GPU)
    return LIB_GEN_CPU, LIB_GEN_GPU


def build_all():
    build_wl()
    build_inputs()


if __name__ == "__main__":
    build_all()
    print("built", LIB_WL, LIB_GEN_CPU, LIB_GEN_GPU)
