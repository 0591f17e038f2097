"""CPU sanitizers: the single-lane replay of the kernel's per-wave logic
(kvr_core.h) and the oracle, built with AddressSanitizer and
UndefinedBehaviorSanitizer (errors abort), run on cases that reach every
path of both; the replay's results are also compared with the oracle's.
Runs in a child process that preloads the ASan runtime (the interpreter
itself is not instrumented)."""
import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _runtime(name: str) -> str:
    cc = shutil.which("gcc") or shutil.which("g++")
    if cc is None:
        return ""
    p = subprocess.run([cc, f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else ""


@pytest.mark.slow
def test_kernel_logic_and_oracle_under_asan_and_ubsan():
    asan = _runtime("libasan.so")
    if not asan:
        pytest.skip("no AddressSanitizer runtime")
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, os.path.join(HERE, "sanitized_replay.py")], env=env, capture_output=True,
                       text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "sanitized replay ok" in r.stdout
