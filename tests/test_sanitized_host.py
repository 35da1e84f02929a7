"""The library's host code and the CPU oracle under sanitizers, on the CPU.

AddressSanitizer + UndefinedBehaviorSanitizer: the host-side tests (LRU
resolve against the oracle, working sets and batch control, the C ABI's
argument checks, the oracle's pins) run in a child process on the
sanitized builds of the library and of the oracle.  ThreadSanitizer: the
tests that drive the resolve pool and the working-set tracker's workers.
The builds come from paper_2509_24626_amd/build_sanitized.py (host code
instrumented, the gfx950 kernels built as usual).  The FlashD2H saver's
threads wait on HIP copies, so they need a GPU and are not covered here."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# the child checks that the sanitized builds are the ones mapped
PROBE = r"""
import oracle
from paper_2509_24626_amd import binding
binding.lib(); oracle.lib()
maps = open("/proc/self/maps").read()
libs = sorted({line.split()[-1] for line in maps.splitlines() if "libsparseserve" in line or "liboracle" in line})
print("mapped:", libs)
assert any(l.endswith("libsparseserve_%s.so") for l in libs) and not any(l.endswith("libsparseserve.so") for l in libs)
"""

REPORTS = ("ERROR: AddressSanitizer", "runtime error:", "WARNING: ThreadSanitizer", "ERROR: ThreadSanitizer")


def _run(kind, tests, oracle_too):
    from paper_2509_24626_amd import build_sanitized as S
    try:
        S.runtime(kind)
    except FileNotFoundError as e:
        pytest.skip(str(e))
    S.build(kind)
    env = S.env(kind)
    probe = PROBE % kind
    if oracle_too:
        probe += "\nassert any(l.endswith('liboracle_asan.so') for l in libs)\n"
    r = subprocess.run([sys.executable, "-c", probe], env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:xdist", "-p", "no:cacheprovider",
                        *tests], env=env, cwd=ROOT, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0 and " passed" in out, out[-4000:]
    for rep in REPORTS:
        assert rep not in out, out[-4000:]


def test_host_code_and_oracle_under_asan_ubsan():
    _run("asan", ["tests/test_cache_parity.py", "tests/test_ws_parity.py", "tests/test_abi_host.py",
                  "tests/test_oracle_pins.py"], oracle_too=True)


def test_threaded_host_code_under_tsan():
    _run("tsan", ["tests/test_cache_parity.py", "tests/test_ws_parity.py"], oracle_too=False)
