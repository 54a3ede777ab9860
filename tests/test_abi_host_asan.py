"""The host half of the C ABI under AddressSanitizer: libkvgov built with
host-side ASan (device code as usual), loaded into a process that preloads
the ASan runtime, runs the host ABI tests (every export, argument
validation before any launch, error strings).  Without a GPU every call
stays on the host, so this covers the validation and bookkeeping code."""
import os
import subprocess
import sys

import pytest

from paper_2608_09225_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

RUNNER = """
import sys
sys.path.insert(0, {root!r})
import paper_2608_09225_amd.kvgov as K
K.LIB_PATH = {lib!r}
with open('/proc/self/maps') as f:
    assert 'libclang_rt.asan' in f.read(), 'ASan runtime not loaded'
import pytest
rc = pytest.main(['-q', '-s', '-p', 'no:cacheprovider', {tests!r}])
import ctypes
assert ctypes.CDLL({lib!r})._handle  # the instrumented library itself
sys.exit(rc)
"""


def test_host_abi_under_address_sanitizer(tmp_path):
    rt = B.asan_runtime()
    if not rt:
        pytest.skip("no ASan runtime next to hipcc's clang")
    lib = B.build_host_asan(str(tmp_path))
    nm = subprocess.run(["nm", "-D", lib], capture_output=True, text=True)
    assert "__asan_" in nm.stdout, "library not instrumented"
    script = tmp_path / "run.py"
    script.write_text(RUNNER.format(root=ROOT, lib=lib,
                                    tests=os.path.join(ROOT, "tests", "test_abi_host.py")))
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1")
    res = subprocess.run([sys.executable, str(script)], env=env, capture_output=True, text=True,
                         timeout=600)
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    assert " passed" in res.stdout
