"""Build the HIP library libpk.so for gfx950, in-tree.

Each source under csrc/ is compiled by hipcc in parallel, then linked into a
shared library next to this file.  Run as ``python -m paper_1904_05347_amd.build``.

``python -m paper_1904_05347_amd.build --sanitized`` builds a second copy,
``_build_san/libpk_san.so``, whose HOST code (argument checks, shape
derivation, selection, workspace planning) is instrumented with
AddressSanitizer and UndefinedBehaviorSanitizer; the device code is built as
usual.  It is for CPU-only checks of that host logic (load it with the clang
ASan runtime preloaded); it never replaces libpk.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.environ.get("PK_BUILD_DIR") or os.path.join(HERE, "_build")
LIB = os.environ.get("PK_LIBRARY") or os.path.join(HERE, "libpk.so")
ARCH = os.environ.get("PK_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++20", "-fPIC",
    # code object v5: loadable by the HIP runtime that PyTorch ships as well
    "-mcode-object-version=5",
    "-Wall", "-Wno-unused-result", "-Rpass-analysis=kernel-resource-usage",
    # no packed fp32 instructions: hipcc would otherwise form v_pk_* fp32
    # ops from ordinary float code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(os.path.dirname(HERE), "include"),
] + os.environ.get("PK_EXTRA_CFLAGS", "").split()


RESOURCE_LOG = os.path.join(BUILD, "resource_usage.log")


SAN_BUILD = os.path.join(HERE, "_build_san")
SAN_LIB = os.path.join(SAN_BUILD, "libpk_san.so")
# host-side sanitizers only (each -fsanitize= behind -Xarch_host)
SAN_FLAGS = ["-g", "-fno-omit-frame-pointer",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all"]


def _compile(src: str, build_dir: str = BUILD, extra=()):
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC] + CFLAGS + list(extra) + ["-c", src, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    lines = [l for l in res.stderr.splitlines() if noise not in l]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s" % (src, "\n".join(lines)))
    # the per-kernel register / LDS / occupancy remarks go to the resource log;
    # anything else the compiler says is shown
    remarks = [l for l in lines if "[-Rpass-analysis=kernel-resource-usage]" in l]
    other = [l for l in lines if "[-Rpass-analysis=kernel-resource-usage]" not in l and
             not l.lstrip().startswith(("|", "^")) and not l.strip().isdigit() and "| {" not in l]
    if any(l.strip() for l in other):
        sys.stderr.write("\n".join(other) + "\n")
    return obj, remarks


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(_compile, srcs))
    objs = [o for o, _ in results]
    with open(RESOURCE_LOG, "w") as fh:
        for _, remarks in results:
            fh.write("\n".join(remarks) + "\n")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


def build_sanitized(verbose: bool = True) -> str:
    """The library with host-side ASan + UBSan, for CPU checks of the host logic."""
    os.makedirs(SAN_BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(lambda src: _compile(src, SAN_BUILD, SAN_FLAGS), srcs))
    objs = [o for o, _ in results]
    tmp = SAN_LIB + ".tmp%d" % os.getpid()
    # the sanitizer runtimes stay undefined in the library and come from the
    # preloaded clang ASan runtime (which carries the UBSan handlers too)
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-shared-libsan",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-o", tmp] + objs
    subprocess.run(cmd, check=True, capture_output=True)
    os.replace(tmp, SAN_LIB)
    if verbose:
        print("built", SAN_LIB)
    return SAN_LIB


def asan_runtime() -> str:
    """Path of the clang ASan runtime that the sanitized library links against."""
    res = subprocess.run([HIPCC, "--print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = res.stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        cands = sorted(glob.glob(os.path.join(os.path.dirname(os.path.dirname(HIPCC)), "lib", "llvm", "lib", "clang",
                                              "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
        path = cands[-1] if cands else ""
    return path


if __name__ == "__main__":
    if "--sanitized" in sys.argv[1:]:
        build_sanitized()
    else:
        build()
