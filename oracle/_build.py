"""Build the CPU oracle (plain C++, no OpenMP, no GPU) in-tree."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SO = os.path.join(HERE, "liboracle.so")


def build(out=SO, flags=("-O2",)):
    """Compiles the oracle into `out`; `flags` replaces the optimisation
    flags (the sanitizer tests build an instrumented copy elsewhere)."""
    cmd = ["g++", *flags, "-fPIC", "-shared", "-std=c++17", "-Wall", "-o", out + ".tmp",
           os.path.join(HERE, "oracle.cpp"), os.path.join(HERE, "head.cpp"),
           os.path.join(HERE, "ngram.cpp")]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("oracle build failed:\n" + r.stdout)
    os.replace(out + ".tmp", out)


if __name__ == "__main__":
    build()
