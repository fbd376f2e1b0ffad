"""Build libasv.so in-tree for gfx950 with hipcc (no GPU needed to compile)."""

from __future__ import annotations

import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(_HERE)
SOURCES = [os.path.join(_HERE, "csrc", "asv_api.hip")]
HEADERS = [os.path.join(ROOT, "include", "asv.h")] + [
    os.path.join(_HERE, "csrc", f) for f in ("k_common.h", "k_lmhead.h", "k_reduce.h",
                                               "k_accept.h", "k_draft.h", "k_tree.h")]
OUT = os.path.join(_HERE, "libasv.so")
# measurement-only library (achievable-peak microbenchmarks), separate from libasv
MICROBENCH_SOURCES = [os.path.join(_HERE, "csrc", "microbench.hip")]
MICROBENCH_OUT = os.path.join(_HERE, "libasv_microbench.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # code objects every ROCm 7.x runtime loads (torch may bring an older runtime than hipcc)
    "-mcode-object-version=5",
    # keep the compiler from forming packed fp32 (v_pk_*_f32) instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    cand = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def build_library(out: str = OUT, verbose: bool = False, sources=None) -> str:
    """Compile the HIP sources (libasv's by default) into ``out`` (written atomically)."""
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-o", tmp,
           *(sources or SOURCES)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{msgs}")
    if verbose and msgs.strip():
        print(msgs)
    os.replace(tmp, out)
    return out


def build_microbench(verbose: bool = False) -> str:
    return build_library(MICROBENCH_OUT, verbose, MICROBENCH_SOURCES)


def is_built(out: str = OUT) -> bool:
    return os.path.exists(out)
