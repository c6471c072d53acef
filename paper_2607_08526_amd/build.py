"""Build libqlinear.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2607_08526_amd.build
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libqlinear.so")
SOURCES = ["qlinear.hip", "quantize.hip", "qgemm.hip", "qgemm_wide.hip", "qgemm_skinny.hip", "xprep.hip", "qgemm_stream.hip", "qgemv.hip",
           "qgemm_w8a8.hip", "steer.hip", "attention.hip", "qgemm_mid.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# -packed-fp32-ops: keep the compiler from emitting packed fp32 VALU ops.
# Denormals are kept (the quantizer's exactness needs fp32/fp64 subnormals).
DEVICE_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-gpu-flush-denormals-to-zero", "-fno-fast-math",
    "-Wall", "-Wno-unused-command-line-argument",
    f"-I{INCLUDE}",
]
# MFMA results straight into VGPRs: the per-block scale FMAs of these kernels
# read them without v_accvgpr_read copies.  The large-M fp16 kernel keeps its
# 256 accumulators per lane in AGPRs instead.
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
SOURCE_FLAGS = {"qgemm.hip": VGPR_FORM, "qgemm_skinny.hip": VGPR_FORM,
                "qgemm_stream.hip": VGPR_FORM, "qgemm_w8a8.hip": VGPR_FORM,
                "attention.hip": VGPR_FORM, "qgemm_mid.hip": VGPR_FORM}


def _compile(src):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *DEVICE_FLAGS, *SOURCE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src),
           "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


BENCH_SRC = os.path.join(HERE, "bench_csrc", "read_ceiling.hip")
BENCH_LIB = os.path.join(HERE, "libqlbench.so")


def build_bench_helper():
    """The benchmark's read-ceiling kernel (libqlbench.so, not the product)."""
    tmp = BENCH_LIB + ".tmp"
    cmd = [HIPCC, *DEVICE_FLAGS, "-shared", BENCH_SRC, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for the bench helper:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, BENCH_LIB)
    return BENCH_LIB


def build(verbose=True):
    """Compile every HIP source for gfx950 and link libqlinear.so (and the
    benchmark's helper library); returns the library's path."""
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    build_bench_helper()
    if verbose:
        print(f"built {LIB} and {BENCH_LIB}")
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
