"""Host-side memory and undefined-behaviour checks (CPU only, no GPU).

The oracle's C sources, built with AddressSanitizer and UndefinedBehaviorSanitizer, run
the oracle's pin suites; the library, built with the same sanitizers on its host code (its
device code unchanged), runs the C ABI suite, whose calls exercise every host-side
argument check, workspace layout and error path.  Each suite runs in a child process with
the sanitizer runtime preloaded; any report aborts it."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SUITES = ["tests/test_oracle_pins.py", "tests/test_lp_oracle.py",
                 "tests/test_sample_oracle.py", "tests/test_feature_oracle.py"]


def _run(env_extra, files):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", *files], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout


def test_oracle_under_address_and_ub_sanitizers():
    gcc_asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                              text=True, check=True).stdout.strip()
    if not os.path.isabs(gcc_asan):
        pytest.skip("gcc's ASan runtime is not installed")
    env = {"ORACLE_SANITIZE": "1", "LD_PRELOAD": gcc_asan}
    subprocess.run([sys.executable, "-c", "import oracle; oracle.build(force=True)"],
                   cwd=ROOT, env=dict(os.environ, ORACLE_SANITIZE="1"), check=True)
    _run(env, ORACLE_SUITES)


def test_library_host_code_under_address_and_ub_sanitizers():
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt:
        pytest.skip("clang's ASan runtime is not installed")
    sys.path.insert(0, ROOT)
    from paper_2406_06022_amd import build

    build.build(sanitize=True)
    _run({"RGCN_LIB_SANITIZE": "1", "LD_PRELOAD": rt[-1]}, ["tests/test_abi.py"])
