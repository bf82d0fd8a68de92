"""Build ``libtmamba.so`` (gfx950 only) in-tree with hipcc.

    python -m paper_2606_18114_amd.build          # or __graft_entry__.build()

Every translation unit under ``csrc/`` is compiled in parallel to an object
file under ``_build/`` and the objects are linked into
``paper_2606_18114_amd/libtmamba.so`` next to the Python binding.  The
roofline probes of ``csrc/micro.hip`` (an MFMA loop and an HBM read stream,
used by ``bench.py --micro``) go into a separate ``libtm_micro.so``.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import time

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libtmamba.so")
MICRO_OUT = os.path.join(PKG, "libtm_micro.so")
MICRO_SOURCES = ["micro.hip"]
OBJ = os.path.join(ROOT, "_build")

SOURCES = [
    "abi.cpp",
    "ternarize_pack.hip",
    "tgemm_fwd.hip",
    "tgemm_bwd_dx.hip",
    "tgemm_bwd_dx_f16.hip",
    "tgemm_bwd_dw.hip",
    "tgemv.hip",
    "tgemv_b16.hip",
    "dgemv.hip",
    "mixer.hip",
    "decode_stack.hip",
    "group_code_dot.hip",
]

ARCH = "gfx950"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    if os.path.exists(path):
        return path
    found = shutil.which("hipcc")
    if not found:
        raise RuntimeError("hipcc not found (ROCm is required to build libtmamba.so)")
    return found


COMMON_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-Werror",
    f"--offload-arch={ARCH}",
    # packed float32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # hardware float32 atomic add for the split-K reduction of dW
    "-munsafe-fp-atomics",
    "-I", os.path.join(ROOT, "include"),
]


# per-source additions
EXTRA_FLAGS = {}


def _compile(src: str) -> str:
    os.makedirs(OBJ, exist_ok=True)
    obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc(), *lang, *COMMON_FLAGS, *EXTRA_FLAGS.get(src, []), "-c",
           os.path.join(CSRC, src), "-o", obj]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{proc.stderr}")
    return obj


def _link(objs, out: str) -> None:
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError(f"link failed:\n{proc.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = True) -> str:
    """Compile every source and link the shared libraries; returns the path
    of libtmamba.so."""
    t0 = time.time()
    srcs = SOURCES + MICRO_SOURCES
    with cf.ThreadPoolExecutor(max_workers=min(len(srcs), os.cpu_count() or 4)) as ex:
        objs = dict(zip(srcs, ex.map(_compile, srcs)))
    _link([objs[s] for s in SOURCES], OUT)
    _link([objs[s] for s in MICRO_SOURCES], MICRO_OUT)
    if verbose:
        print(f"built {OUT} and {os.path.basename(MICRO_OUT)} in {time.time() - t0:.1f}s",
              file=sys.stderr)
    return OUT


if __name__ == "__main__":
    build()
