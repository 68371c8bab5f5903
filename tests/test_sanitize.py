"""CPU sanitizer tier (no GPU): AddressSanitizer and UndefinedBehaviorSanitizer
over the fp64 oracle and over the host code of the HIP library (argument
validation, workspace plans, dispatch).

* The oracle is rebuilt with gcc -fsanitize=address,undefined
  (-fno-sanitize-recover=all: any report aborts) and its pins
  (tests/test_oracle.py, tests/test_oracle_dropout.py) run against that
  build in a child process with gcc's ASan runtime preloaded.
* The library is rebuilt with the sanitizers on its host code only
  (hipcc -Xarch_host ...; GPU code unchanged) and the host ABI tests
  (tests/test_abi_host.py: every error path of every entry point, the
  workspace sizing) run against it with clang's ASan runtime preloaded.
* A planted out-of-bounds read in a call of the sanitized oracle must be
  reported, which shows the runtime is really active.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gcc_asan():
    path = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip("gcc's libasan is not installed")
    return path


def _clang_asan():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        pytest.skip("clang's ASan runtime is not installed")
    return hits[-1]


def _child(cmd, env_extra, timeout=900):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:verify_asan_link_order=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    return subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


@pytest.fixture(scope="module")
def oracle_asan():
    import oracle
    return oracle.build_sanitized()


def test_oracle_pins_under_asan_ubsan(oracle_asan):
    r = _child([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                "-m", "not gpu", "tests/test_oracle.py", "tests/test_oracle_dropout.py"],
               {"LD_PRELOAD": _gcc_asan(), "FASTMAX_ORACLE_LIB": oracle_asan})
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "Sanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out


def test_sanitized_oracle_reports_a_planted_overflow(oracle_asan):
    """Standardise 5 rows of a 4-row array: the last row is read past the
    end of the allocation, which the sanitized build must report."""
    prog = (
        "import ctypes, numpy as np, oracle\n"
        "assert oracle._LIB.endswith('_asan.so'), oracle._LIB\n"
        "L = oracle._load()\n"
        "dp = ctypes.POINTER(ctypes.c_double)\n"
        "x = np.ones((4, 512)); x[:, 0] = 2.0\n"
        "o = np.empty((5, 512)); m = np.empty(5); s = np.empty(5)\n"
        "p = lambda a: a.ctypes.data_as(dp)\n"
        "L.fmo_standardize(p(x), 5, 512, p(o), p(m), p(s))\n"
        "print('no report')\n")
    r = _child([sys.executable, "-c", prog],
               {"LD_PRELOAD": _gcc_asan(), "FASTMAX_ORACLE_LIB": oracle_asan}, timeout=120)
    out = r.stdout + r.stderr
    assert r.returncode != 0 and "heap-buffer-overflow" in out, out[-3000:]


def _newer_than_sources(lib, srcdir):
    if not os.path.exists(lib):
        return False
    t = os.path.getmtime(lib)
    srcs = glob.glob(os.path.join(srcdir, "*")) + [os.path.join(ROOT, "include", "fastmax.h")]
    return all(os.path.getmtime(f) <= t for f in srcs)


def test_library_host_code_under_asan_ubsan():
    from paper_2402_07901_amd import build
    if not _newer_than_sources(build.LIB_ASAN, build.CSRC):
        build.build(sanitize=True)
    r = _child([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                "tests/test_abi_host.py"],
               {"LD_PRELOAD": _clang_asan(), "FASTMAX_LIB": build.LIB_ASAN})
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "Sanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
