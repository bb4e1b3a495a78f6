"""Build libippd.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2609_05707_amd.build   (or call build())
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(HERE, "libippd.so")

SOURCES = ["ippd_api.hip", "rope_append.hip", "decode_step.hip", "prefill.hip", "dense_mask.hip"]
# standalone measurement programs, built next to the library
TOOLS = {"stream_ceiling.hip": os.path.join(HERE, "stream_ceiling"), "l2_handoff.hip": os.path.join(HERE, "l2_handoff")}
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
    f"-I{INCLUDE}", f"-I{CSRC}",
]

# Per-source additions.  The decode kernels never rely on NaN propagation
# (their marks are +-inf and negative sums), so fmax needs no quieting of
# its MFMA/permlane inputs: without this every max costs two instructions.
SOURCE_FLAGS = {
    "decode_step.hip": ["-fno-honor-nans"],
    "prefill.hip": ["-fno-honor-nans"],
    "dense_mask.hip": ["-fno-honor-nans"],
}


def flags_for(src: str):
    """hipcc flags of one source file (without -c/-o)."""
    return [*HIPCC_FLAGS, *SOURCE_FLAGS.get(src, [])]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def _compile(src: str, extra) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *flags_for(src), *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def _tool(src: str, exe: str) -> str:
    cmd = [hipcc(), *flags_for(src), os.path.join(CSRC, src), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return exe


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile every HIP source for gfx950 and link libippd.so next to this file
    (and the standalone measurement programs beside it)."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES) + len(TOOLS)) as ex:
        tools = [ex.submit(_tool, src, exe) for src, exe in TOOLS.items()]
        objs = list(ex.map(lambda s: _compile(s, list(extra_flags)), SOURCES))
        for f in tools:
            f.result()
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB_PATH)
    if verbose:
        print(f"built {LIB_PATH}")
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
