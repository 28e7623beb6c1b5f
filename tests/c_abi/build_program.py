"""Builds the plain-C drivers of the pipeline (window_pipeline: grouping, alignment,
collate and loss weights of a window; stream_pipeline: one streaming iteration, its
collate and loss weights), through include/odb.h, with gcc against the in-tree libodb.so
and the HIP runtime.  Test infrastructure: the GPU tests run the binaries this writes
next to their sources."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PROGRAMS = ["window_pipeline", "stream_pipeline"]
PKG = os.path.join(ROOT, "paper_2606_19989_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def command(src: str, out: str) -> list:
    # the library is found next to the package relative to the binary, so the tree can
    # move; strict C11 with warnings as errors checks that the header is plain C
    return ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
            "-I", os.path.join(ROCM, "include"), src, "-o", out,
            "-L", PKG, "-l:libodb.so", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
            "-Wl,-rpath,$ORIGIN/" + os.path.relpath(PKG, os.path.dirname(os.path.abspath(out))),
            "-Wl,-rpath," + os.path.join(ROCM, "lib")]


def build(out_dir: str = HERE) -> list:
    """Compile every driver into out_dir; returns the binaries' paths."""
    outs = []
    for name in PROGRAMS:
        src, out = os.path.join(HERE, name + ".c"), os.path.join(out_dir, name)
        r = subprocess.run(command(src, out), capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"gcc failed for {src}:\n{r.stdout}\n{r.stderr}")
        outs.append(out)
    return outs


if __name__ == "__main__":
    print(build())
