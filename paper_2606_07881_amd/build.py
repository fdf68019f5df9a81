"""Builds libpaci_stage.so (the HIP stage library) for gfx950 with hipcc.

Every translation unit of the library under csrc/ is compiled in parallel into
_build/ and linked in place next to this file, where the binding loads it.
stage_bench (a native driver used for profiling) is linked against it. Run as
``python -m paper_2606_07881_amd.build`` or call ``build()``.
"""
import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libpaci_stage.so")
EXE = os.path.join(HERE, "stage_bench")
SOURCES = ["gemm.hip", "attention.hip", "rowwise.hip", "optim.hip", "stage.hip", "planner.cpp"]
TOOLS = ["stage_bench.hip"]

ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-I", CSRC, "-I", INCLUDE,
    # keep the compiler from forming packed fp32 VALU ops from scalar float code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc():
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found; the HIP toolchain is required to build libpaci_stage.so")
    return exe


def _compile(src):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc()] + FLAGS + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    return obj, err


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(SOURCES) + len(TOOLS))) as ex:
        results = list(ex.map(_compile, SOURCES + TOOLS))
    for obj, err in results:
        if verbose and err.strip():
            print(err, file=sys.stderr)
    tools = results[len(SOURCES):]
    results = results[:len(SOURCES)]
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + [o for o, _ in results]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    tmp = EXE + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-o", tmp, tools[0][0], "-L", HERE, "-lpaci_stage",
           "-Wl,-rpath,$ORIGIN"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link of stage_bench failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, EXE)
    return LIB


SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer"]


def build_host_sanitized(out_dir):
    """The library with AddressSanitizer and UBSan on its host code only (device
    code is built as usual), for the host-only tests:
    LD_PRELOAD=<clang asan runtime> ASAN_OPTIONS=detect_leaks=0 PACI_STAGE_LIB=<out_dir>/libpaci_stage.so
    python -m pytest tests/test_abi_host.py tests/test_planner_host.py"""
    os.makedirs(out_dir, exist_ok=True)
    flags = [f for f in FLAGS if f != "-O3"] + ["-O1", "-g"] + SANITIZE

    def one(src):
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        r = subprocess.run([hipcc()] + flags + ["-c", os.path.join(CSRC, src), "-o", obj], capture_output=True,
                           text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(one, SOURCES))
    lib = os.path.join(out_dir, "libpaci_stage.so")
    r = subprocess.run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC"] + SANITIZE[:4] + ["-o", lib] + objs,
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    return lib


if __name__ == "__main__":
    if len(sys.argv) == 3 and sys.argv[1] == "--host-sanitize":
        print(build_host_sanitized(sys.argv[2]))
    else:
        print(build(verbose=True))
