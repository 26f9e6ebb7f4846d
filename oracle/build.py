"""Build the CPU oracle shared library (test infrastructure only).

The oracle is plain C compiled with gcc; it shares no source with the GPU
library.  ``mutant`` builds a copy with one planted mistake (see the
ORACLE_MUTANT switch in glide_oracle.c) for the mutation tests.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "glide_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(out=LIB, mutant=0, quiet=True):
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           f"-DORACLE_MUTANT={int(mutant)}", "-o", out + ".tmp", SRC, "-lm"]
    subprocess.run(cmd, check=True, capture_output=quiet)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(quiet=False))
