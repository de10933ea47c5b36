"""Build the gfx950 library (libmcpu.so) and the input generator (libmcpu_synth.so)."""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
BUILD = os.path.join(HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall",
    # no packed-fp32 instructions in any kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]
SOURCES = ["attention.hip", "gemm.hip", "gemm_tiled.hip", "gemm_pipe.hip", "gemm_slab.hip", "gemm_mx.hip", "moe.hip",
           "lm_head.hip", "mcpu_host.hip"]
# per-source code generation: the tiled GEMM and the attention kernels keep
# their matrix-core accumulators in ordinary VGPRs (the AGPR form shuffles them
# between loop iterations and needs more registers in all)
_VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
SOURCE_FLAGS = {"gemm_tiled.hip": _VGPR_FORM, "gemm_pipe.hip": _VGPR_FORM, "gemm_slab.hip": _VGPR_FORM,
                "gemm_mx.hip": _VGPR_FORM, "attention.hip": _VGPR_FORM}


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r


def build_synth() -> str:
    out = os.path.join(HERE, "libmcpu_synth.so")
    _run(["gcc", "-O3", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-Wall", "-o", out + ".tmp",
          os.path.join(CSRC, "synth.c")])
    os.replace(out + ".tmp", out)
    return out


def build_hip(jobs: int = 4) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []

    def one(src):
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        _run([HIPCC, *HIP_FLAGS, *SOURCE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj])
        return obj

    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(one, SOURCES))
    out = os.path.join(HERE, "libmcpu.so")
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", out + ".tmp", *objs])
    os.replace(out + ".tmp", out)
    return out


def build_synth_device() -> str:
    """Device twin of the input generator (bench and tests only; no layer arithmetic)."""
    out = os.path.join(HERE, "libmcpu_synth_dev.so")
    _run([HIPCC, *HIP_FLAGS, "-shared", "-o", out + ".tmp", os.path.join(CSRC, "synth_fill.hip")])
    os.replace(out + ".tmp", out)
    return out


def build() -> None:
    build_synth()
    build_synth_device()
    build_hip()


if __name__ == "__main__":
    build()
    print("built", os.path.join(HERE, "libmcpu.so"))
