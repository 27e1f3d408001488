"""Builds libapack.so for gfx950 in-tree with hipcc.

Every HIP source under csrc/ is compiled to an object in parallel, then
linked into paper_2608_08794_amd/libapack.so.  Packed fp32 instructions are
disabled for all device code.
"""

import concurrent.futures
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libapack.so")
ARCH = os.environ.get("APACK_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{msgs}")
    return obj, msgs


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(_compile, srcs))
    for _, msgs in results:
        if verbose and msgs.strip():
            print(msgs, file=sys.stderr)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp,
           *[o for o, _ in results]]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


ASAN_BUILD = os.path.join(HERE, "_build_asan")
ASAN_LIB = os.path.join(ASAN_BUILD, "libapack_asan.so")
# Host code only: every -fsanitize= follows -Xarch_host, so the device code
# is compiled exactly as in the product build.
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
              "-Xarch_host", "-g", "-shared-libasan"]


def asan_runtime():
    """The shared AddressSanitizer runtime the sanitized library needs
    preloaded into a host process that was not built with it."""
    out = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = out.stdout.strip()
    if os.path.isabs(path) and os.path.exists(path):
        return path
    cands = sorted(glob.glob(os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "lib", "clang",
                                          "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
    if not cands:
        raise RuntimeError("libclang_rt.asan-x86_64.so not found")
    return os.path.realpath(cands[-1])


def build_sanitized(verbose=False):
    """libapack with its host code (validation, planning, staging, launch
    set-up) built with AddressSanitizer and UndefinedBehaviorSanitizer, for
    CPU-only runs of the ABI tests; the device code is unchanged."""
    os.makedirs(ASAN_BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))

    def comp(src):
        obj = os.path.join(ASAN_BUILD, os.path.basename(src) + ".o")
        r = subprocess.run([HIPCC, *FLAGS, *ASAN_FLAGS, "-c", src, "-o", obj], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc (sanitized) failed on {src}:\n{r.stdout}{r.stderr}")
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(comp, srcs))
    r = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *ASAN_FLAGS, "-o", ASAN_LIB, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("sanitized link failed:\n" + r.stdout + r.stderr)
    return ASAN_LIB


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "asan":
        print(build_sanitized(verbose=True))
    else:
        print(build(verbose=True))
