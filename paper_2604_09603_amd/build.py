"""Compile the HIP sources into the in-tree shared library ``libecho.so`` (gfx950)."""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libecho.so")

ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # keep hipcc from emitting packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


# Per-file flags for the attention kernel:
# * its MFMA accumulators stay in VGPRs: left to its heuristics the compiler
#   holds them in AGPRs and copies all of them to VGPRs and back on every tile
#   (a v_accvgpr read and write per register), which costs as many VALU cycles
#   as the tile's MFMAs;
# * no NaN semantics: with them every fmaxf over MFMA results (the softmax row
#   maxima) is preceded by a v_max_f32 x, x, x that quiets signalling NaNs,
#   about 50 extra VALU instructions per 64-row tile.  Infinities (masked keys
#   are -inf) keep their meaning; NaN inputs give unspecified outputs.
# The fused step's tail kernel holds the attention's combine and is built the
# same way, so that its merges are the combine launch's to the bit.
FILE_FLAGS = {
    "attn.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form=1", "-fno-honor-nans"],
    "tail.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form=1", "-fno-honor-nans"],
}


def _hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return path


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))

    def compile_one(name):
        obj = os.path.join(BUILD, name[:-4] + ".o")
        cmd = [hipcc, *FLAGS, *FILE_FLAGS.get(name, []), "-c", os.path.join(CSRC, name), "-o", obj]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc failed for {name}:\n{res.stderr}")
        if verbose and res.stderr:
            print(res.stderr, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max(1, min(8, len(srcs)))) as ex:
        objs = list(ex.map(compile_one, srcs))
    tmp = LIB + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
