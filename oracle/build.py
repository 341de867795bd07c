"""Builds the Lynx CPU oracle (test infrastructure only) into oracle/liblynx_oracle.so.

Plain gcc, no fast-math, no floating-point contraction: the oracle's fp32
codec arithmetic must be exactly the IEEE operations its source spells out.
"""
import os
import subprocess
import sys
from pathlib import Path

HERE = Path(__file__).resolve().parent
SOURCE = HERE / "lynx_oracle.c"
LIBRARY = HERE / "liblynx_oracle.so"

CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra", "-shared", "-fPIC", "-pthread"]


def build(verbose: bool = False) -> Path:
    """Compile the oracle; always recompiles.  Returns the library path."""
    tmp = LIBRARY.with_name(LIBRARY.name + f".tmp{os.getpid()}")
    cmd = ["gcc", *CFLAGS, str(SOURCE), "-o", str(tmp), "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
