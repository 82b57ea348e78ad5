"""The C-ABI tests (tests/test_abi.py) again, against a build of the library
whose host code carries AddressSanitizer and UndefinedBehaviorSanitizer
checks (argument validation, workspace carving, launch set-up).  No GPU:
the valid calls end in NAMOH_ERR_HIP without a device.  Runs in a
subprocess with the ASan runtime preloaded; any sanitizer report fails it."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2609_38832_amd import build as B  # noqa: E402


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def _stale(lib):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    srcs = [os.path.join(B.CSRC, f) for f in os.listdir(B.CSRC)]
    srcs.append(os.path.join(ROOT, "include", "namoh.h"))
    return any(os.path.getmtime(f) > t for f in srcs)


def test_abi_under_host_sanitizers():
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("no ASan runtime in this toolchain")
    try:
        B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    if _stale(B.SAN_LIB):
        B.build_library(verbose=False, sanitize=True)
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": rt,
        "ASAN_OPTIONS": "detect_leaks=0:verify_asan_link_order=0:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "NAMOH_LIB": B.SAN_LIB,
        "HIP_VISIBLE_DEVICES": "",      # the host paths only, also on a GPU machine
    })
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"),
                        "-q", "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in r.stdout
