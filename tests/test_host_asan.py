"""The library's host code under AddressSanitizer (CPU only).

A second build of the library instruments its host pass (argument validation, planning, workspace
sizing and carving) with AddressSanitizer; its device code is the release build's. The host-side
ABI checks of test_abi.py then run against that build in a child process that preloads the
sanitizer's runtime, so any heap or stack overrun on those paths ends the child with a report.
"""
import glob
import os
import subprocess
import sys

import pytest

from paper_2608_02691_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

_CHILD = r"""
import ctypes, sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
assert hasattr(ctypes.CDLL(None), "__asan_init"), "sanitizer runtime not loaded"
from paper_2608_02691_amd import int2kv as K
lib = K.load_library({lib!r})
import test_abi
names = sorted(n for n in dir(test_abi) if n.startswith("test_"))
for n in names:
    getattr(test_abi, n)()
print("host checks under the sanitizer:", len(names), flush=True)
"""


def _stale(lib):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    srcs = B.sources() + glob.glob(os.path.join(B.PKG, "csrc", "*.h")) + glob.glob(os.path.join(ROOT, "include", "*.h"))
    return any(os.path.getmtime(s) > t for s in srcs)


def test_host_code_is_clean_under_address_sanitizer():
    if not os.path.exists(B.HIPCC):
        pytest.skip("hipcc is not installed")
    rt = B.asan_runtime()
    if not rt:
        pytest.skip("the compiler's shared AddressSanitizer runtime is not installed")
    if _stale(B.ASAN_LIB):
        B.build_host_asan()
    env = dict(os.environ)
    # the sanitizer's runtime goes first; anything already preloaded stays
    env["LD_PRELOAD"] = " ".join(p for p in (rt, os.environ.get("LD_PRELOAD", "")) if p)
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:verify_asan_link_order=0"
    code = _CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=B.ASAN_LIB)
    r = subprocess.run([sys.executable, "-c", code], env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       timeout=600)
    out = r.stdout.decode(errors="replace")
    assert "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "host checks under the sanitizer:" in out, out[-2000:]
