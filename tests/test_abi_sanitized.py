"""The C-ABI tests (tests/test_abi.py) against a copy of the library whose host
code is built with AddressSanitizer and UndefinedBehaviorSanitizer
(paper_2502_05370_amd/build_sanitized.py), in a child process with the
sanitizer runtime preloaded.  CPU only: the ABI tests make no compute call.

Any sanitizer report fails the test (halt_on_error); leak detection is off
because the Python interpreter itself is not built for it."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2502_05370_amd")
sys.path.insert(0, PKG)


def _sanitized_library():
    import build_sanitized as S
    sources = glob.glob(os.path.join(PKG, "csrc", "*")) + glob.glob(os.path.join(ROOT, "include", "*.h"))
    if not os.path.exists(S.OUT) or os.path.getmtime(S.OUT) < max(os.path.getmtime(f) for f in sources):
        S.build()
    return S.OUT, S.sanitizer_runtime()


def test_abi_under_address_and_undefined_behaviour_sanitizers():
    try:
        lib, runtime = _sanitized_library()
    except RuntimeError as e:   # no hipcc / no clang sanitizer runtime in this image
        pytest.skip(str(e))
    env = dict(os.environ)
    env["FM_LIBRARY"] = lib
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = runtime + (":" + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
