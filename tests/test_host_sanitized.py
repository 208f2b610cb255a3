"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

build.build(sanitize=True) compiles a copy of the library whose host code (argument validation,
the active-cell plan, buffer layouts and launch sequences of every entry point) carries both
sanitizers; device code is built as usual.  The host-side ABI tests then run against that copy
in a child process that preloads the sanitizer runtime (the binding loads the copy named by
TFM_LIB).  Any report (an out-of-bounds or freed access, an overflow, a misaligned or
out-of-range conversion) ends the child with an error.

A positive control shows that the checks are live: a caller that passes fewer n_train entries
than datasets makes the plan read past the end of that host array, which AddressSanitizer must
report as a heap-buffer-overflow inside the library."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def san_env():
    from paper_2606_03681_amd import build
    lib = build.build(sanitize=True)
    env = dict(os.environ)
    env.update(LD_PRELOAD=build.san_runtime(), TFM_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return env


def _run(env, args, timeout=600):
    p = subprocess.run([sys.executable] + args, env=env, cwd=ROOT, capture_output=True,
                       text=True, timeout=timeout)
    return p.returncode, p.stdout + p.stderr


def test_abi_tests_clean_under_sanitizers(san_env):
    rc, out = _run(san_env, ["-m", "pytest", "-q", "-p", "no:cacheprovider",
                             os.path.join("tests", "test_abi_cpu.py")])
    assert rc == 0, out[-6000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-6000:]
    assert " passed" in out


_SHORT_NTRAIN = """
import ctypes, sys
import numpy as np
sys.path.insert(0, {root!r})
from paper_2606_03681_amd import tfm
assert tfm._LIB_PATH.endswith("libtfmlayer_san.so"), tfm._LIB_PATH
d = tfm.make_dims(B=4, R=64, C=8, E=64, heads=4, H=128, dtype="f32")
nt = np.full(1, 5, np.int32)          # one entry for four datasets
cm = np.ones((4, 9), np.uint8)
p = 1 << 20
tfm.lib().tfm_layer_fwd(ctypes.byref(d), nt.ctypes.data, cm.ctypes.data, p, p, p, p, 1 << 40,
                        p, 1 << 40, None)
print("NOT DETECTED")
"""


def test_sanitizer_reports_a_host_overread(san_env):
    rc, out = _run(san_env, ["-c", _SHORT_NTRAIN.format(root=ROOT)], timeout=120)
    assert rc != 0 and "NOT DETECTED" not in out, out[-4000:]
    assert "heap-buffer-overflow" in out and "make_plan" in out, out[-4000:]
