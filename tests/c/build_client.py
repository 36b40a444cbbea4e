"""Builds tests/c/abi_client (the plain-C client of libiefwd the tests run)
with gcc, linked against paper_2503_05130_amd/libiefwd.so with the library's
directory as its run path.  Called by __graft_entry__.build()."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_client.c")
OUT = os.path.join(HERE, "abi_client")
PKG = os.path.join(ROOT, "paper_2503_05130_amd")
INCLUDE = os.path.join(ROOT, "include")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Werror", f"-I{INCLUDE}", SRC, "-o", OUT,
           f"-L{PKG}", "-liefwd", f"-Wl,-rpath,{PKG}"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"C client build failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
