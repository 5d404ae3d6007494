"""Compile the plain C consumer of the C ABI (layer_fwd_c.c) with gcc, linked
against the in-tree libmoe.so and the HIP runtime.  Test infrastructure: the
binary only exercises the boundary from C."""
from __future__ import annotations

import subprocess
from pathlib import Path

HERE = Path(__file__).resolve().parent
ROOT = HERE.parents[1]
SRC = HERE / "layer_fwd_c.c"
BIN = HERE / "layer_fwd_c"
ROCM = Path("/opt/rocm")


def build(verbose: bool = False) -> Path:
    pkg = ROOT / "paper_2608_28511_amd"
    if not (pkg / "libmoe.so").exists():
        raise RuntimeError("libmoe.so is not built")
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", str(ROOT / "include"), "-I", str(ROCM / "include"), str(SRC), "-o", str(BIN),
           "-L", str(pkg), "-lmoe", "-L", str(ROCM / "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2608_28511_amd", f"-Wl,-rpath,{ROCM / 'lib'}"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"gcc failed for {SRC.name}:\n{r.stdout}\n{r.stderr}")
    return BIN


def ensure_built() -> Path:
    """The consumer binary, compiled first if it is missing."""
    return BIN if BIN.exists() else build()
