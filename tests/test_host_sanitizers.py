"""The host code (C ABI, block manager, planner) under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: the library's host sources are
built with both sanitizers by g++ (tests/host_sanitizer.py), and the CPU
tests of the host side run against that build in a fresh interpreter with
the sanitizer runtimes preloaded. They include the hypothesis comparison of
the block manager with the oracle manager (single and batched appends),
error codes, every coverage proof of the planner (the full-size plans at 256
compute units included) and the refusals of spork_plan_advance. Any
sanitizer report aborts the run. Two tests are left out: their last calls
have nothing to do and reach the kernel launchers, which this build
replaces with stubs that fail."""
import os
import subprocess
import sys

import host_sanitizer

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_code_is_clean_under_asan_and_ubsan():
    lib = host_sanitizer.build()
    env = dict(os.environ)
    env.update(LD_PRELOAD=host_sanitizer.runtime_preload(), SPORK_HOST_SANITIZER_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_host.py"), "-q",
                        "-p", "no:cacheprovider", "-k", "not confidence_error_codes and not ngram_error_codes"],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=1500)
    tail = r.stdout[-3000:]
    assert "AddressSanitizer" not in r.stdout and "runtime error" not in r.stdout, tail
    assert r.returncode == 0, tail
    assert " passed" in tail and "failed" not in tail, tail
