"""Host-side sanitizer job (CPU only): the oracle and the library's host code
under AddressSanitizer and UndefinedBehaviorSanitizer.

1. The oracle's C source is compiled with gcc -fsanitize=address,undefined and
   the oracle test files run against that build (ORACLE_LIB), with gcc's ASan
   runtime preloaded into the Python process.
2. The HIP library is compiled with both sanitizers on its host code only
   (the device code is built but never launched here) and the boundary tests
   run against that build (DYNCONV_TEST_LIB): argument validation, workspace
   sizing, launch planning, the static-scratch checks and every error path,
   all of which index the plan and shape arrays that a mistake would overrun.

Any sanitizer report fails the test; a negative control checks that a
planted overrun and a planted undefined shift are reported.  The
instrumented builds are cached under paper_1912_03203_amd/_build/sanitize,
keyed by a hash of their sources and flags, so only the first run after a
change pays for the compile.  The index maps of Sec. 3.2 (dilation, gather
and scatter lists) are where an overrun would hide, in the oracle's C loops
and in the library's host-side plans alike."""
import glob
import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_1912_03203_amd")
OUT = os.path.join(PKG, "_build", "sanitize")
ORACLE_SRC = os.path.join(ROOT, "oracle", "dynconv_oracle.c")
ORACLE_TESTS = sorted(glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
BOUNDARY_TEST = os.path.join(ROOT, "tests", "test_boundary.py")

# one sanitizer flag per host-side argument: hipcc compiles device code too,
# and the sanitizers must stay out of it
HIP_HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address",
                     "-Xarch_host", "-fsanitize=undefined",
                     "-Xarch_host", "-fno-sanitize-recover=undefined",
                     "-Xarch_host", "-fno-omit-frame-pointer",
                     "-Xarch_host", "-g",
                     "-Xarch_device", "-O0"]
GCC_SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                "-fno-omit-frame-pointer", "-g", "-O1"]
REPORT_MARKERS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer",
                  "SUMMARY: AddressSanitizer", "SUMMARY: UndefinedBehaviorSanitizer")


def _digest(paths, flags):
    h = hashlib.sha1()
    for p in sorted(paths):
        with open(p, "rb") as f:
            h.update(p.encode() + b"\0" + f.read())
    h.update("\0".join(flags).encode())
    return h.hexdigest()[:16]


def _cached_build(name, sources, flags, cmd_for):
    """Build once per source hash; returns the library path."""
    os.makedirs(OUT, exist_ok=True)
    lib = os.path.join(OUT, "%s_%s.so" % (name, _digest(sources, flags)))
    if not os.path.exists(lib):
        tmp = lib + ".tmp%d" % os.getpid()
        r = subprocess.run(cmd_for(tmp), capture_output=True, text=True, timeout=900)
        assert r.returncode == 0, "sanitizer build of %s failed:\n%s%s" % (name, r.stdout, r.stderr[-4000:])
        os.replace(tmp, lib)
    return lib


def _runtime(compiler, name):
    path = subprocess.run([compiler, "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip("%s has no %s here" % (compiler, name))
    return path


def _run_pytest(files, extra_env):
    env = dict(os.environ)
    env.update(extra_env)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1:exitcode=86"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["PYTHONDONTWRITEBYTECODE"] = "1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider"] + files
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    out = r.stdout + r.stderr
    reports = [ln for ln in out.splitlines() if any(m in ln for m in REPORT_MARKERS)]
    assert not reports, "sanitizer reports:\n" + "\n".join(reports[:20]) + "\n" + out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out, out[-2000:]
    return out


def test_oracle_under_asan_ubsan():
    flags = ["-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"] + GCC_SANITIZE
    lib = _cached_build("liboracle", [ORACLE_SRC], flags,
                        lambda tmp: ["gcc"] + flags + ["-o", tmp, ORACLE_SRC, "-lm"])
    asan = _runtime("gcc", "libasan.so")
    _run_pytest(ORACLE_TESTS, {"ORACLE_LIB": lib, "LD_PRELOAD": asan})


@pytest.mark.slow
def test_library_host_code_under_asan_ubsan():
    from paper_1912_03203_amd import build

    srcs = glob.glob(os.path.join(PKG, "csrc", "*")) + [os.path.join(ROOT, "include", "dynconv.h")]
    flags = [f for f in build.HIPCC_FLAGS if f != "-O3"] + ["-O1"] + HIP_HOST_SANITIZE
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]
    lib = _cached_build("libdynconv", srcs, flags,
                        lambda tmp: [build.hipcc()] + flags + inc + ["-o", tmp, build.SRC])
    clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
    asan = _runtime(clang, "libclang_rt.asan-x86_64.so")
    _run_pytest([BOUNDARY_TEST], {"DYNCONV_TEST_LIB": lib, "LD_PRELOAD": asan})


PLANTED = r"""
#include <stdlib.h>
int planted_overrun(int n) { int *a = malloc(n * sizeof(int)); for (int i = 0; i < n; ++i) a[i] = i;
                             int v = a[n]; free(a); return v; }
int planted_shift(int s) { return 1 << s; }
"""


@pytest.mark.parametrize("call", ["planted_overrun(8)", "planted_shift(40)"])
def test_harness_reports_a_planted_error(call):
    """The job's own negative control: the same flags, runtime and report
    markers catch a heap overrun and an undefined shift planted on the CPU."""
    src = os.path.join(OUT, "planted.c")
    os.makedirs(OUT, exist_ok=True)
    with open(src, "w") as f:
        f.write(PLANTED)
    flags = ["-std=c11", "-fPIC", "-shared"] + GCC_SANITIZE
    lib = _cached_build("libplanted", [src], flags, lambda tmp: ["gcc"] + flags + ["-o", tmp, src])
    env = dict(os.environ, LD_PRELOAD=_runtime("gcc", "libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:exitcode=86",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    code = "import ctypes; print(ctypes.CDLL(%r).%s)" % (lib, call)
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=120)
    out = r.stdout + r.stderr
    assert r.returncode != 0
    assert any(m in out for m in REPORT_MARKERS), out[-2000:]
