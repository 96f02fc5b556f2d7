"""Compile oracle/mfma8.c into oracle/libmfma8.so (gcc, OpenMP).  Test infrastructure only.

Run by __graft_entry__.build() and usable as `python -m oracle.build_mfma8`.
"""

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mfma8.c")
LIB = os.path.join(HERE, "libmfma8.so")


def build():
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        raise RuntimeError("no C compiler for the oracle's mfma8.c")
    tmp = LIB + ".tmp"
    r = subprocess.run([cc, "-O2", "-fopenmp", "-fPIC", "-shared", SRC, "-o", tmp, "-lm"], capture_output=True,
                       text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building {SRC} failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
