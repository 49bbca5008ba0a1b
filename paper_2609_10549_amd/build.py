"""Build libcompass.so (HIP kernels for gfx950 + host runtime + C ABI) in-tree.

    python -m paper_2609_10549_amd.build [--sanitize]

Every HIP/C++ source is compiled with hipcc for gfx950 only; packed fp32
instructions are disabled in device code.

--sanitize builds libcompass_san.so instead: the host code of every source
instrumented with AddressSanitizer and UndefinedBehaviorSanitizer (device
code is built as usual), for CPU-only test runs of the host paths
(validation, model, calibration, partition layout, the runtime up to its
first GPU call):

    COMPASS_LIBRARY=paper_2609_10549_amd/libcompass_san.so \
    LD_PRELOAD=$(python -m paper_2609_10549_amd.build --asan-runtime) \
    ASAN_OPTIONS=detect_leaks=0 python -m pytest tests -m "not gpu"
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libcompass.so")
SAN_LIB = os.path.join(HERE, "libcompass_san.so")
SOURCES = ["kernels.hip", "noalloc.hip", "runtime.cpp", "model.cpp", "abi.cpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Werror=shadow", "-Wno-unused-function", f"-I{INCLUDE}", f"-I{CSRC}"]
# host-only instrumentation: each sanitizer flag applies to the host pass
SANITIZE = ["-g", "-fno-omit-frame-pointer",
            "-Xarch_host", "-fsanitize=address",
            "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(ln for ln in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in ln)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def asan_runtime() -> str:
    """Path of the compiler's AddressSanitizer runtime (to preload into a
    Python process that loads the sanitizer build)."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], stdout=subprocess.PIPE, text=True)
    return r.stdout.strip()


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile every source and link libcompass.so (libcompass_san.so with
    sanitize=True); returns its path."""
    objdir = os.path.join(HERE, "_build_san" if sanitize else "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = []
    for src in SOURCES:
        path = os.path.join(CSRC, src)
        obj = os.path.join(objdir, src + ".o")
        lang = ["-x", "hip"]
        cmd = [HIPCC] + lang + DEVICE_FLAGS + COMMON + (SANITIZE if sanitize else []) + ["-c", path, "-o", obj]
        out = _run(cmd)
        if verbose and out.strip():
            print(out)
        objs.append(obj)
    out = SAN_LIB if sanitize else LIB
    tmp = out + ".tmp"
    cmd = [HIPCC] + DEVICE_FLAGS + ["-shared", "-fPIC", "-o", tmp] + objs + \
        ["-L/opt/rocm/lib", "-lhsa-runtime64", "-lamdhip64", "-lpthread", "-rdynamic", "-Wl,-rpath,/opt/rocm/lib"]
    if sanitize:   # the runtimes come from the preloaded ASan library
        cmd += ["-Wl,--unresolved-symbols=ignore-in-shared-libs", "-Wl,-z,undefs"]
    _run(cmd)
    os.replace(tmp, out)
    shutil.rmtree(objdir, ignore_errors=True)
    return out


if __name__ == "__main__":
    if "--asan-runtime" in sys.argv:
        print(asan_runtime())
    else:
        print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
