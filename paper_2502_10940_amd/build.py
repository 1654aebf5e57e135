"""Build libcola.so (the gfx950 HIP kernels + C ABI) in-tree.

hipcc cross-compiles for gfx950 without a GPU.  Every source is compiled with
packed-fp32 instructions disabled (the compiler would otherwise form
v_pk_*_f32 from plain float code) and linked into
``paper_2502_10940_amd/libcola.so``.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libcola.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["gemm_dispatch.hip", "gemm_stream.hip", "gemm_pp.hip", "gemm_f32.hip", "cola_abi.hip",
           "attention.hip", "block_ops.hip", "block_abi.hip"]
# Per-source extra flags.  The 256 x 256 kernel's epilogues run over 256
# accumulators per lane: past the default limit the unroller stops and the
# accumulators go to scratch memory.
EXTRA = {"gemm_pp.hip": ["-mllvm", "-pragma-unroll-threshold=500000"],
         # MFMA accumulators in ordinary VGPRs: the attention kernels scale and read
         # theirs with VALU code between MFMAs (no copies to and from AGPRs)
         "attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}
FLAGS = ["-std=c++17", "-O3", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function"]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass warns that it does not know the packed-fp32 feature: harmless
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip() and verbose:
        print(err, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", LIB + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
