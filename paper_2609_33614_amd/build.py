"""Build libeat.so (gfx950) in-tree with hipcc.

    python -m paper_2609_33614_amd.build [--jobs N]

Every source under csrc/ is compiled to an object under _build/, then
linked into paper_2609_33614_amd/libeat.so next to this file.  Compiles
every time it is called.

    python -m paper_2609_33614_amd.build --sanitize --out PATH

builds a variant whose host code (the C ABI's validation, planning and
launch sequencing) carries AddressSanitizer and UndefinedBehaviorSanitizer
checks; device code is built as usual.  Load it with the sanitizer runtime
preloaded (``sanitizer_runtime()``), e.g. for the CPU tests of the ABI.
"""
from __future__ import annotations

import argparse
import hashlib
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libeat.so")

ARCH = "gfx950"
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    "-Wall", "-Wno-unused-result",
    # keep hipcc from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]
# host-only instrumentation: each -fsanitize= is applied to the host pass alone
SAN_CFLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
SAN_LDFLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan"]
SOURCES = ["api.cpp", "route.hip", "permute.hip", "expert.hip", "wide.hip", "combine.hip", "ppl.hip", "pack.hip",
           "noalloc.hip"]


def _compile(src: str, extra=(), tag: str = "") -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + tag + ".o")
    cmd = [HIPCC, *CFLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def sanitizer_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (it carries the
    UndefinedBehaviorSanitizer handlers too), for LD_PRELOAD."""
    clang = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = shutil.which("clang") or "/opt/rocm/llvm/bin/clang"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("no shared AddressSanitizer runtime found next to the compiler")
    return path


def build(jobs: int = 8, verbose: bool = False, defines=(), out: str = LIB, sanitize: bool = False) -> str:
    """Compile and link.  ``defines`` are extra -D flags (tuning variants);
    ``out`` is the library path (default: the package's libeat.so);
    ``sanitize`` instruments the host code (see the module docstring)."""
    os.makedirs(BUILD, exist_ok=True)
    tag = "" if not defines else "_" + hashlib.sha1(" ".join(defines).encode()).hexdigest()[:10]
    extra = [f"-D{d}" for d in defines]
    if sanitize:
        tag += "_san"
        extra += SAN_CFLAGS
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(lambda s: _compile(s, extra, tag), SOURCES))
    LIBOUT = out
    tmp = LIBOUT + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, *(SAN_LDFLAGS if sanitize else [])]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIBOUT)
    if verbose:
        print(f"built {LIBOUT}")
    return LIBOUT


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=min(8, os.cpu_count() or 1))
    ap.add_argument("-D", dest="defines", action="append", default=[], help="extra preprocessor define")
    ap.add_argument("--out", default=LIB)
    ap.add_argument("--sanitize", action="store_true", help="host code with ASan and UBSan (needs --out)")
    args = ap.parse_args(argv)
    if args.sanitize and os.path.abspath(args.out) == LIB:
        ap.error("--sanitize builds a separate library: give --out")
    build(args.jobs, verbose=True, defines=args.defines, out=args.out, sanitize=args.sanitize)
    return 0


if __name__ == "__main__":
    sys.exit(main())
