"""The CPU tests of the C ABI and the host schedulers, re-run against a build whose host
code carries AddressSanitizer and UndefinedBehaviorSanitizer (device code untouched).

Any out-of-bounds access, use after free or undefined behaviour in the validation,
the create-time dry pass, the greedy simulations or the actor-critic agent aborts the
child run; the test passes only if every child test passes with no sanitizer report.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CHILD_TESTS = ["tests/test_abi_cpu.py", "tests/test_abi_layout.py", "tests/test_sched_cpu.py", "tests/test_rl_cpu.py"]


@pytest.mark.timeout(600)
def test_cpu_abi_and_schedulers_under_host_sanitizers():
    from paper_1804_06087_amd import build_sanitized as bs
    lib = bs.build_sanitized()
    env = bs.env_for(lib)
    # the child loads the instrumented build, with the ASan runtime in the process
    probe = ("import ctypes, paper_1804_06087_amd as p; L = p.load_library(); "
             "ctypes.CDLL(None).__asan_address_is_poisoned; print(L._name)")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == lib, r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"] + CHILD_TESTS,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=540)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out
