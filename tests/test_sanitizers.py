"""CPU builds of the host code and of the oracle with AddressSanitizer and
UndefinedBehaviorSanitizer (every report fatal):

* the library's host code (argument checks, launch planning, workspace layout) with stub
  launchers that check every planned launch against the call's buffers and the 32-bit launch
  limits, driven by a seeded sweep of ordinary and extreme dims through every entry point;
* the oracle, driven by seeded random small workloads with exactly sized buffers;
* the ABI checks (test_library_abi.py) against the sanitized host code built as a shared
  library, and the oracle pins (test_oracle_pins.py) against the sanitized oracle, each in a
  child process with the sanitizer runtimes preloaded.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, os.path.join(ROOT, "tests", "c"))
import build as c_build  # noqa: E402  (tests/c/build.py)


@pytest.fixture(scope="module")
def builds(tmp_path_factory):
    return c_build.build_sanitized(str(tmp_path_factory.mktemp("sanitized")))


def _env(**extra):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1",
               OMP_NUM_THREADS="4")
    env.update(extra)
    return env


def test_host_code_sweep_under_sanitizers(builds):
    r = subprocess.run([builds["host"], "20000"], capture_output=True, text=True, timeout=600, env=_env())
    assert r.returncode == 0, r.stdout + r.stderr
    assert "launches checked" in r.stdout


def test_oracle_sweep_under_sanitizers(builds):
    r = subprocess.run([builds["oracle"], "300"], capture_output=True, text=True, timeout=600, env=_env())
    assert r.returncode == 0, r.stdout + r.stderr


@pytest.mark.parametrize("suite,var,key", [("test_library_abi.py", "BANA_LIBRARY", "host_lib"),
                                           ("test_oracle_pins.py", "ORACLE_LIB", "oracle_lib")])
def test_suite_against_sanitized_library(builds, suite, var, key):
    env = _env(**{var: builds[key], "LD_PRELOAD": c_build.sanitizer_preload()})
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", suite)], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=900)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
