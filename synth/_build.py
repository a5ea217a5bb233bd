"""Build the seeded input generator's native parts (host OpenMP library and
the gfx950 device filler) in-tree."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
HOST_SO = os.path.join(HERE, "libsynth_host.so")
DEV_SO = os.path.join(HERE, "libsynth_dev.so")

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed: %s\n%s" % (" ".join(cmd), r.stdout))


def build():
    _run(["g++", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c++17", "-Wall",
          "-o", HOST_SO + ".tmp", os.path.join(CSRC, "synth_host.cpp")])
    os.replace(HOST_SO + ".tmp", HOST_SO)
    _run(["hipcc"] + HIP_FLAGS + ["-o", DEV_SO + ".tmp", os.path.join(CSRC, "synth_dev.hip")])
    os.replace(DEV_SO + ".tmp", DEV_SO)


if __name__ == "__main__":
    build()
