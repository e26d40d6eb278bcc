"""The oracle and the library's host logic under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU.

  - oracle.c is built with gcc's ASan + UBSan and every pin runs against
    that copy in a child process with the sanitizer runtimes preloaded;
  - a copy of the HIP library whose host code (argument checks, shape
    derivation, selection, workspace planning) is instrumented with clang's
    ASan + UBSan runs the C-ABI tests, which reach no GPU;
  - a planted out-of-bounds read in an oracle copy must be reported, so the
    instrumentation is known to be live.
Any sanitizer report ends the child process with a non-zero status (UBSan
does not recover; ASan aborts on its first error).
"""
import glob
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:alloc_dealloc_mismatch=0:detect_odr_violation=0:abort_on_error=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _gcc_runtimes():
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        path = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
        if not os.path.isabs(path) or not os.path.exists(path):
            pytest.skip("gcc sanitizer runtime %s not found" % name)
        libs.append(path)
    return ":".join(libs)


def _build_oracle(src_text, out):
    src = out + ".c"
    with open(src, "w") as fh:
        fh.write(src_text)
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", out, src, "-lm"], check=True)
    return out


def _run_child(code, preload, extra_env=None):
    env = dict(os.environ)
    env.update(SAN_ENV)
    env["LD_PRELOAD"] = preload
    env.update(extra_env or {})
    return subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=600)


_PINS = """
import oracle
from tests import pins
o = oracle.Oracle(%r)
for p in pins.ALL_PINS:
    if p.__name__ in %r:
        continue
    p(o)
    print("ok", p.__name__, flush=True)
"""


def test_oracle_pins_under_asan_ubsan(tmp_path):
    lib = _build_oracle(oracle.source(), str(tmp_path / "liboracle_san.so"))
    # torch's own libraries are not instrumented and are not what is checked here
    proc = _run_child(_PINS % (lib, ("pin_torch_float64",)), _gcc_runtimes())
    assert proc.returncode == 0, proc.stderr[-4000:]
    assert "AddressSanitizer" not in proc.stderr and "runtime error" not in proc.stderr, proc.stderr[-4000:]
    assert proc.stdout.count("ok ") >= 14


def test_sanitizer_reports_a_planted_overflow(tmp_path):
    src = oracle.source()
    old = "for (int64_t k = 0; k < K; ++k)"
    assert src.count(old) == 1
    lib = _build_oracle(src.replace(old, "for (int64_t k = 0; k <= K; ++k)"), str(tmp_path / "liboracle_bad.so"))
    code = ("import numpy as np, oracle\n"
            "o = oracle.Oracle(%r)\n"
            "a = np.ones((5, 7), np.float32); b = np.ones((7, 3), np.float32)\n"
            "o.sgemm('N', 'N', 5, 3, 7, 1.0, a, 7, b, 3, 0.0, None, 3)\n") % lib
    proc = _run_child(code, _gcc_runtimes())
    assert proc.returncode != 0
    assert "AddressSanitizer" in proc.stderr, proc.stderr[-2000:]


def _sanitized_library():
    from paper_1904_05347_amd import build
    srcs = glob.glob(os.path.join(build.CSRC, "*"))
    if not os.path.exists(build.SAN_LIB) or \
            os.path.getmtime(build.SAN_LIB) < max(os.path.getmtime(s) for s in srcs):
        build.build_sanitized(verbose=False)
    rt = build.asan_runtime()
    if not rt:
        pytest.skip("clang ASan runtime not found")
    return build.SAN_LIB, rt


def test_host_logic_under_asan_ubsan():
    lib, rt = _sanitized_library()
    code = ("import sys, pytest\n"
            "sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', 'tests/test_abi_cpu.py']))\n")
    proc = _run_child(code, rt, {"PK_LIBRARY": lib})
    out = proc.stdout + proc.stderr
    assert proc.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in proc.stdout
