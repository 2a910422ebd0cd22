"""The host-side ABI tests (tests/test_abi_host.py) again, against libmkor
built with AddressSanitizer and UndefinedBehaviorSanitizer on its host code
(tests/sanitize/build_asan.py), in a subprocess with clang's ASan runtime
preloaded.  CPU only: no call reaches the device."""
import os
import subprocess
import sys

import pytest

from tests.sanitize import build_asan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_host_under_asan_and_ubsan():
    try:
        rt = build_asan.asan_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    lib = build_asan.build()
    env = dict(os.environ, MKOR_LIBRARY=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    # the instrumented library and the runtime are what the process maps
    probe = ("import paper_2306_01685_amd as M; M.load_library(); m = open('/proc/self/maps').read(); "
             "print('libmkor_asan.so' in m, 'libclang_rt.asan' in m)")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0 and r.stdout.split() == ["True", "True"], r.stdout + r.stderr[-2000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_abi_host.py", "-x", "-q",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
