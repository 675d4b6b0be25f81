"""Build the okvq HIP library (libokvq.so) in-tree for gfx950 with hipcc."""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libokvq.so")
SOURCES = ["api.hip", "codec_kernels.hip", "codec_fused.hip", "decode_kernels.hip", "calib_kernels.hip",
           "dense_decode.hip", "ladder_codec.hip", "ladder_decode.hip", "append_window.hip"]

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    # bit-exact codecs: no fused multiply-add contraction (fmaf is spelled out where wanted)
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-fast-math",
    # no packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs (no AGPR copies around the softmax rescale)
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# per-source additions: the decode kernels (packed and dense) never see NaN (finite inputs; -inf is the only special
# value they use), so min / max need no NaN quieting
EXTRA = {"decode_kernels.hip": ["-fno-honor-nans"], "dense_decode.hip": ["-fno-honor-nans"],
         "ladder_decode.hip": ["-fno-honor-nans"],
         # the codecs take window minima and maxima of finite directions (finite inputs are part of the device data
         # contract): no NaN quieting around them
         "append_window.hip": ["-fno-honor-nans"], "codec_fused.hip": ["-fno-honor-nans"]}


def build(verbose: bool = False, jobs: int = 4) -> str:
    """Compile every source and link libokvq.so next to this file. Always rebuilds."""
    obj_dir = os.path.join(PKG, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    cc = hipcc()

    def compile_one(src: str) -> str:
        obj = os.path.join(obj_dir, src.replace(".hip", ".o"))
        cmd = [cc, *FLAGS, *EXTRA.get(src, []), "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
        if verbose and r.stderr.strip():
            print(r.stderr)
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    r = subprocess.run([cc, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
