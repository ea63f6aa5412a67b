"""Build ``libflashkmeans.so`` (gfx950 only) from the HIP sources in ``csrc/``.

``python -m paper_2608_12629_amd.build`` or ``build()``; the library is written
next to this file, where ``paper_2608_12629_amd.kmeans`` loads it.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libflashkmeans.so")
# the benchmark's in-run ceilings (include/fkm_calib.h), a library of its own
CALIB_LIB = os.path.join(HERE, "libfkm_calib.so")
CALIB_SOURCES = ["calib.hip"]
SOURCES = ["api.hip", "assign.hip", "assign_pipe_bf16.hip", "assign_pipe_f16.hip",
           "assign_smallk_bf16.hip", "assign_smallk_f16.hip", "assign_tiled.hip", "update.hip",
           "knn_bf16.hip", "knn_f16.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions are not emitted (see the design notes)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


# Per-source flags.  The KNN search is defined for finite inputs only, so its
# sources may assume no NaNs: the compiler then drops the quieting of each
# operand before a float maximum and turns compare-and-select pairs in the
# list insertion into single instructions.
SOURCE_FLAGS = {"knn_bf16.hip": ["-fno-honor-nans"], "knn_f16.hip": ["-fno-honor-nans"]}


def build(out: str = LIB, extra=(), sources=None) -> str:
    """Compile each source to an object (in parallel), then link the library."""
    sources = SOURCES if sources is None else sources
    import tempfile
    from concurrent.futures import ThreadPoolExecutor

    with tempfile.TemporaryDirectory(prefix="fkm_build_") as tmpdir:
        def compile_one(src):
            obj = os.path.join(tmpdir, os.path.splitext(src)[0] + ".o")
            cmd = [HIPCC, *FLAGS, *SOURCE_FLAGS.get(src, []), *extra, "-c", os.path.join(CSRC, src),
                   "-o", obj]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed on {src} ({r.returncode}):\n{r.stderr[-6000:]}")
            return obj

        with ThreadPoolExecutor(max_workers=len(sources)) as pool:
            objs = list(pool.map(compile_one, sources))
        tmp = out + f".tmp{os.getpid()}"
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc link failed ({r.returncode}):\n{r.stderr[-6000:]}")
        os.replace(tmp, out)
    return out


def build_calib(out: str = CALIB_LIB) -> str:
    return build(out, sources=CALIB_SOURCES)


if __name__ == "__main__":
    print(build(*sys.argv[1:2]))
    print(build_calib())
