"""Build libtq.so, the HIP library of this package, for gfx950.

    python -m paper_2003_02989_amd.build

compiles every source under csrc/ with hipcc into libtq.so next to this file.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libtq.so")
SOURCES = ["kernels.hip", "program.cpp", "tq_abi.cpp", "jit.cpp"]
# device code the run-time specialised kernels are compiled with, in order
JIT_HEADERS = ["tq_internal.h", "kernel_args.h", "device_ops.h"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed FP32 instructions are disabled for all device code: they are avoided
# on this target.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def write_prelude(path):
    """The shared device headers as one C++ string literal (local includes
    dropped: the headers are concatenated in dependency order)."""
    text = []
    for h in JIT_HEADERS:
        with open(os.path.join(CSRC, h)) as f:
            text += [line for line in f.read().split("\n")
                     if not line.startswith('#include "') and line.strip() != "#pragma once"]
    body = "\n".join(text)
    delim = "TQJIT"
    assert ")" + delim + '"' not in body
    out = 'R"' + delim + "(" + body + ")" + delim + '"\n'
    if os.path.exists(path):
        with open(path) as f:
            if f.read() == out:
                return
    with open(path, "w") as f:
        f.write(out)


def build(verbose=True):
    objs = []
    os.makedirs(os.path.join(HERE, "_build"), exist_ok=True)
    write_prelude(os.path.join(HERE, "_build", "jit_prelude.inc"))
    for src in SOURCES:
        obj = os.path.join(HERE, "_build", src + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [HIPCC] + FLAGS + lang + ["-I", os.path.join(HERE, "..", "include"), "-I", os.path.join(HERE, "_build"),
                                        "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        objs.append(obj)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs + ["-lhiprtc", "-pthread", "-Wl,--no-undefined"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
