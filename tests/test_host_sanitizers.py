"""CPU sanitizer builds of the host code (no GPU).

- The host half of libtfe (error messages, the allocation-failure hook, the
  held-memory count, phrase validation and the lock-free multi-threaded index
  build) runs a driver under AddressSanitizer + UndefinedBehaviorSanitizer and
  under ThreadSanitizer.
- The oracle's pins run against an ASan + UBSan build of the oracle library
  (the Python process preloads the ASan runtime).
- A canary with a planted out-of-bounds read proves the toolchain's sanitizer
  reports on this machine, so a silent pass means something.

Compilers are started only inside the tests, never at import: a GPU test run
collects this module too, and a process that has loaded the HIP runtime
loses its device if it starts another program.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_07388_amd", "csrc")
DRIVER = os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp")
ASAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _runtime(name):
    """Path of g++'s sanitizer runtime `name`; skips the test without one."""
    if not shutil.which("g++"):
        pytest.skip("no g++")
    p = subprocess.run(["g++", "-print-file-name=" + name], stdout=subprocess.PIPE,
                       text=True).stdout.strip()
    if not (os.path.isabs(p) and os.path.exists(p)):
        pytest.skip("no g++ runtime " + name)
    return p


def _compile(out, flags, sources):
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-Wall", "-pthread", *flags,
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, *sources, "-o", out]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout


def _run(exe, env=None, timeout=300):
    e = dict(os.environ)
    e.pop("TFE_FAIL_ALLOC", None)
    e.update(env or {})
    return subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
                          env=e, timeout=timeout)


def test_sanitizer_reports_a_planted_overflow(tmp_path):
    _runtime("libasan.so")
    src = tmp_path / "canary.cpp"
    src.write_text("#include <vector>\nint main(int c, char**) {\n"
                   "  std::vector<int> v(4);\n  return v.data()[3 + c];\n}\n")
    exe = str(tmp_path / "canary")
    _compile(exe, ASAN, [str(src)])
    r = _run(exe)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr


def test_host_index_build_under_asan_ubsan(tmp_path):
    _runtime("libasan.so")
    exe = str(tmp_path / "host_asan")
    _compile(exe, ASAN, [DRIVER, os.path.join(CSRC, "tfe_host.cpp")])
    r = _run(exe, {"ASAN_OPTIONS": "detect_leaks=1:halt_on_error=1",
                   "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"})
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
    assert "runtime error" not in r.stderr


def test_host_index_build_under_tsan(tmp_path):
    _runtime("libtsan.so")
    exe = str(tmp_path / "host_tsan")
    _compile(exe, ["-fsanitize=thread"], [DRIVER, os.path.join(CSRC, "tfe_host.cpp")])
    r = _run(exe, {"TSAN_OPTIONS": "halt_on_error=1:second_deadlock_stack=1"})
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
    assert "WARNING: ThreadSanitizer" not in r.stderr


def test_oracle_pins_under_asan_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    sys.path.insert(0, ROOT)
    from oracle import _build
    so = str(tmp_path / "liboracle_asan.so")
    _build.build(so, ("-O1", "-g", *ASAN))
    env = dict(os.environ)
    env.update({"LD_PRELOAD": asan, "ORACLE_SO": so,
                # The Python interpreter and numpy are not instrumented; only
                # the oracle's own accesses are checked.
                "ASAN_OPTIONS": "detect_leaks=0:alloc_dealloc_mismatch=0:halt_on_error=1",
                "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"})
    probe = subprocess.run(
        [sys.executable, "-c", "import oracle; oracle.lib(); "
         "print(open('/proc/self/maps').read().count('liboracle_asan.so') > 0)"],
        cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, timeout=120)
    assert probe.stdout.strip() == "True", probe.stderr
    pins = ["tests/test_oracle_pins.py", "tests/test_oracle_multi_pins.py",
            "tests/test_oracle_head_pins.py", "tests/test_oracle_ngram_pins.py"]
    # The workload-3 hit-rate pin builds a 2^22-phrase table: minutes under
    # ASan, and no code path the smaller pins miss.
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", "-k", "not workload3", *pins],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-4000:]
    assert "runtime error" not in r.stdout and "AddressSanitizer" not in r.stdout
