"""Builds liblynx.so (the HIP kernels and the C ABI) for gfx950, in-tree.

hipcc flags: -O3, gfx950 only, no fast-math; packed-fp32 instructions are
disabled (-packed-fp32-ops) so the compiler never emits v_pk_{add,mul,fma}_f32.
"""
import os
import subprocess
import sys
from pathlib import Path

HERE = Path(__file__).resolve().parent
CSRC = HERE / "csrc"
ROOT = HERE.parent
LIBRARY = HERE / "liblynx.so"
SOURCES = ["codec.hip", "hier.hip", "attention.hip", "anchor_decode.hip", "anchor_split.hip", "verify.hip", "spec.hip",
           "abi.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-fast-math", "-Wall", "-Wno-unused-function",
    f"-I{ROOT / 'include'}", f"-I{CSRC}",
]


def build(verbose: bool = False) -> Path:
    """Compile every HIP source into liblynx.so; always recompiles."""
    tmp = LIBRARY.with_name(LIBRARY.name + f".tmp{os.getpid()}")
    cmd = [HIPCC, *FLAGS, *[str(CSRC / s) for s in SOURCES], "-o", str(tmp)]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
