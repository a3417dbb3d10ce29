"""Build the HIP library (libemo.so) in-tree for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libemo.so")
SOURCES = ["emo_host.cpp", "emo_jit.cpp", "emo_pack.cpp", "emo_model.cpp", "emo_kernels.hip", "emo_chains.hip", "emo_dp.hip"]
ARCH = os.environ.get("EMO_OFFLOAD_ARCH", "gfx950")

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    f"--offload-arch={ARCH}",
    # packed fp32 VALU forms stay off (hipcc's host pass warns that it does not know the
    # feature; that warning is harmless)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def embed_select_source(build_dir: str) -> None:
    """Embeds the text of csrc/emo_select.h into the library for the run-time compiler."""
    with open(os.path.join(CSRC, "emo_select.h")) as f:
        text = f.read()
    assert ")EMO_SRC\"" not in text
    with open(os.path.join(build_dir, "emo_select_src.inc"), "w") as f:
        f.write("// generated from emo_select.h by build.py\n")
        f.write('static const char kEmoSelectSource[] = R"EMO_SRC(\n' + text + '\n)EMO_SRC";\n')


def build(verbose: bool = False) -> str:
    """Compile every source and link libemo.so.  Always rebuilds."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objs = []
    build_dir = os.path.join(PKG, "_build")
    os.makedirs(build_dir, exist_ok=True)
    embed_select_source(build_dir)
    for src in SOURCES:
        obj = os.path.join(build_dir, src + ".o")
        cmd = [hipcc, *HIPCC_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        if src.endswith(".cpp"):
            cmd = [hipcc, "-O2", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC,
                   "-I", build_dir, "-D__HIP_PLATFORM_AMD__", "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc failed on {src}")
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp, "-lhiprtc"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("link failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
