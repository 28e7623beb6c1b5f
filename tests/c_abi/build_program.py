"""Builds window_pipeline (the window pipeline driven from plain C through include/odb.h)
with gcc against the in-tree libodb.so and the HIP runtime.  Test infrastructure: the GPU
test runs the binary this writes next to its source."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "window_pipeline.c")
BIN = os.path.join(HERE, "window_pipeline")
PKG = os.path.join(ROOT, "paper_2606_19989_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def command(out: str) -> list:
    # the library is found next to the package relative to the binary, so the tree can
    # move; strict C11 with warnings as errors checks that the header is plain C
    return ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
            "-I", os.path.join(ROCM, "include"), SRC, "-o", out,
            "-L", PKG, "-l:libodb.so", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
            "-Wl,-rpath,$ORIGIN/" + os.path.relpath(PKG, os.path.dirname(os.path.abspath(out))),
            "-Wl,-rpath," + os.path.join(ROCM, "lib")]


def build(out: str = BIN) -> str:
    r = subprocess.run(command(out), capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gcc failed for {SRC}:\n{r.stdout}\n{r.stderr}")
    return out


if __name__ == "__main__":
    print(build())
