"""Build libmoesplit.so (HIP for gfx950) in-tree with hipcc.

python paper_2509_08342_amd/build.py              the library
python paper_2509_08342_amd/build.py --sanitize   a second copy whose host code is
    built with AddressSanitizer and UndefinedBehaviorSanitizer (device code
    unchanged), in paper_2509_08342_amd/_san/, and the CPU tests of the host
    logic (ABI, planner, oracle pins) run against it and against an equally
    instrumented oracle, each in its own process with the sanitizer runtime
    preloaded.  Needs no GPU.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmoesplit.so")
SAN_DIR = os.path.join(PKG, "_san")
SOURCES = ["kernels.hip", "runtime.hip", "planner.cpp", "decoder.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    # no packed-fp32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]
# host code only: every sanitizer flag is scoped to the host compilation
SAN_FLAGS = ["-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile every HIP source and link libmoesplit.so; returns its path."""
    objs = []
    out_lib = os.path.join(SAN_DIR, "libmoesplit.so") if sanitize else LIB
    build_dir = os.path.join(PKG, "_build_san" if sanitize else "_build")
    os.makedirs(build_dir, exist_ok=True)
    os.makedirs(os.path.dirname(out_lib), exist_ok=True)
    flags = [f for f in FLAGS if f != "-O3"] + SAN_FLAGS if sanitize else FLAGS
    for src in SOURCES:
        obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC, *flags, "-I" + INCLUDE, "-I" + CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        objs.append(obj)
    tmp = out_lib + ".tmp%d" % os.getpid()
    link = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"] if sanitize else []
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *link, *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out_lib)
    return out_lib


def _runtime(pattern):
    hits = sorted(glob.glob(pattern))
    if not hits:
        raise SystemExit("sanitizer runtime not found: %s" % pattern)
    return hits[-1]


def sanitize_check() -> int:
    """The CPU tests of the host logic under ASan + UBSan: the library's
    host code (sizes, split plan, argument checks, the planner) with clang's
    runtime preloaded, and the oracle built with gcc's sanitizers with gcc's
    runtime preloaded.  Returns the first non-zero pytest status, else 0."""
    lib = build(sanitize=True)
    sys.path.insert(0, ROOT)
    import oracle
    orc = oracle.build_oracle(force=True, sanitize=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    runs = [
        (dict(env, MOESPLIT_LIB=lib,
              LD_PRELOAD=_runtime("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")),
         ["tests/test_abi.py", "tests/test_planner.py"]),
        (dict(env, MOE_ORACLE_LIB=orc,
              LD_PRELOAD=subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip() + ":" +
              subprocess.check_output(["gcc", "-print-file-name=libubsan.so"], text=True).strip()),
         ["tests/test_oracle.py", "tests/test_quant_oracle.py", "tests/test_planner_oracle.py",
          "tests/test_replacement_oracle.py"]),
    ]
    for e, tests in runs:
        print("sanitized run: %s (%s)" % (" ".join(tests), e["LD_PRELOAD"]), flush=True)
        rc = subprocess.call([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider", *tests],
                             cwd=ROOT, env=e)
        if rc != 0:
            return rc
    return 0


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        sys.exit(sanitize_check())
    print(build(verbose="-v" in sys.argv))
