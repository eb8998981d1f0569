"""Build libstepkv.so (C ABI + HIP kernels for gfx950) in-tree with hipcc.

    python -m paper_2609_22158_amd.build          # compile every source, link
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libstepkv.so")
C_DEMO_SRC = os.path.join(ROOT, "tests", "c_abi", "compress_demo.c")
C_DEMO = os.path.join(ROOT, "tests", "c_abi", "compress_demo")

SOURCES = ["api.cpp", "step_text.cpp", "saliency.hip", "fuse.hip", "select.hip", "compact.hip",
           "decode.hip", "scratch.hip", "probe.hip"]
ARCH = "gfx950"


def _hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _flags():
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Werror=return-type",
        # gfx950 packed-FP32 ops are kept out of every kernel
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        f"-I{INCLUDE}", f"-I{CSRC}",
    ]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = (r.stdout + r.stderr).splitlines()
    noise = "is not a recognized feature for this target"
    msg = "\n".join(line for line in out if noise not in line)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{msg}")
    return msg


def build(verbose: bool = False, extra_flags=(), lib_path: str = LIB) -> str:
    """Compile every source and link libstepkv.so; returns the library path.

    extra_flags (e.g. -D tuning macros) and lib_path allow building variants
    side by side with the default library.
    """
    tag = "" if lib_path == LIB else "_" + os.path.basename(lib_path).replace(".", "_")
    bdir = BUILD + tag
    os.makedirs(bdir, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(bdir, src.rsplit(".", 1)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmds.append([_hipcc(), *lang, *_flags(), *extra_flags, "-c", os.path.join(CSRC, src),
                     "-o", obj])
        objs.append(obj)
    with ThreadPoolExecutor(min(8, len(cmds))) as ex:
        for msg in ex.map(_run, cmds):
            if verbose and msg:
                print(msg)
    tmp = lib_path + ".tmp"
    _run([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,-z,defs", "-o", tmp, *objs])
    os.replace(tmp, lib_path)
    if lib_path == LIB and os.path.exists(C_DEMO_SRC):
        build_c_demo()
    return lib_path


HOST_SOURCES = ["api.cpp", "step_text.cpp"]
ASAN_LIB = os.path.join(BUILD + "_asan", "libstepkv_asan.so")


def build_host_sanitized() -> str:
    """libstepkv with its host C++ (argument validation, workspace planning, the step
    utility and the text engine) built with AddressSanitizer and UndefinedBehaviorSanitizer
    by g++, linked with the unsanitized HIP objects of the default build (device code is
    not sanitized). Load it with the sanitizer runtime preloaded (see sanitizer_env)."""
    if not all(os.path.exists(os.path.join(BUILD, src.rsplit(".", 1)[0] + ".o"))
               for src in SOURCES):
        build()
    bdir = os.path.dirname(ASAN_LIB)
    os.makedirs(bdir, exist_ok=True)
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(_hipcc())))
    san = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=all"]
    objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(bdir, src.rsplit(".", 1)[0] + ".o")
        _run(["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-Wall", "-D__HIP_PLATFORM_AMD__",
              *san, f"-I{rocm}/include", f"-I{INCLUDE}", f"-I{CSRC}", "-c",
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    hip_objs = [os.path.join(BUILD, src.rsplit(".", 1)[0] + ".o") for src in SOURCES
                if src not in HOST_SOURCES]
    tmp = ASAN_LIB + ".tmp"
    _run(["g++", "-shared", "-fPIC", *san, "-o", tmp, *objs, *hip_objs, f"-L{rocm}/lib",
          "-lamdhip64", f"-Wl,-rpath,{rocm}/lib"])
    os.replace(tmp, ASAN_LIB)
    return ASAN_LIB


def sanitizer_env() -> dict:
    """Environment for a Python process that loads the sanitized library."""
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    env = dict(os.environ)
    env.update({"LD_PRELOAD": asan, "STEPKV_LIB": ASAN_LIB, "PYTHONMALLOC": "malloc",
                "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0:exitcode=86",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1:exitcode=87"})
    return env


def build_c_demo() -> str:
    """Compile the plain-C consumer of the ABI (tests/c_abi) against the in-tree library."""
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(_hipcc())))
    _run(["gcc", "-std=c11", "-O2", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
          f"-I{rocm}/include", f"-I{INCLUDE}", C_DEMO_SRC, "-o", C_DEMO, f"-L{PKG}", "-lstepkv",
          f"-L{rocm}/lib", "-lamdhip64", "-lm", "-Wl,-rpath,$ORIGIN/../../paper_2609_22158_amd",
          f"-Wl,-rpath,{rocm}/lib"])
    return C_DEMO


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
