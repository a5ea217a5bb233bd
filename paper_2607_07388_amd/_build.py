"""Build libtfe.so (HIP kernels for gfx950 + host runtime + C ABI) in-tree."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
SO = os.path.join(HERE, "libtfe.so")
ROCM_INC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")

SOURCES = ["tfe_api.cpp", "tfe_head_api.cpp", "tfe_host.cpp", "tfe_stage.cpp", "tfe_build.hip", "tfe_head.hip",
           "tfe_head_noalloc.hip", "tfe_lookup.hip", "tfe_multi.hip", "tfe_tiered.hip"]

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
             # Packed-FP32 instructions stay off: ordinary float code only.
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include")]


def build(verbose=False):
    objs = []
    for src in SOURCES:
        path = os.path.join(CSRC, src)
        obj = os.path.join(CSRC, "_" + src + ".o")
        cmd = ["hipcc"] + HIP_FLAGS + ["-c", path, "-o", obj]
        if src.endswith(".cpp"):
            # Host-only translation units.
            cmd = ["hipcc", "-x", "c++", "-O3", "-std=c++17", "-fPIC", "-Wall",
                   "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INC, "-I", os.path.join(ROOT, "include"),
                   "-c", path, "-o", obj]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
        if r.returncode != 0:
            raise RuntimeError("libtfe build failed: %s\n%s" % (" ".join(cmd), out))
        if verbose and out.strip():
            print(out)
        objs.append(obj)
    # -z defs: a symbol left undefined fails the link here, not the library load at run time.
    cmd = ["hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", "-pthread", "-Wl,-z,defs",
           "-o", SO + ".tmp"] + objs
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("libtfe link failed:\n" + r.stdout)
    os.replace(SO + ".tmp", SO)
    for o in objs:
        os.remove(o)


if __name__ == "__main__":
    build(verbose=True)
