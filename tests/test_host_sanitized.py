"""The C-ABI host layer under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

kashin_api.cpp (argument validation, sign masks, plan tables, grouped-call tables) is rebuilt with
host-only sanitizers and linked with the regular kernel objects; a subprocess with the sanitizer
runtime preloaded runs the host ABI tests and builds the plan tables of every supported length
(kashin_plan computes them on the host before it needs a device).  Any sanitizer report fails."""
import os
import subprocess
import sys

import pytest

from paper_2609_11687_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r'''
import ctypes, sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
from paper_2609_11687_amd import kashin as K
K.LIB_PATH = {lib!r}; K._lib = None
L = K.lib()
assert hasattr(ctypes.CDLL(None), "__asan_init"), "the sanitizer runtime is not loaded"
# plan tables of every supported length (host work), then the device step fails or succeeds
for n in range(2, 20001, 2):
    if L.kashin_supported_n(n):
        h = ctypes.c_void_p()
        st = L.kashin_plan(ctypes.byref(h), n, 12345, 3)
        assert st in (K.KASHIN_OK, K.KASHIN_E_HIP), (n, st)
        if st == K.KASHIN_OK:
            assert L.kashin_plan_destroy(h) == K.KASHIN_OK
import pytest
sys.exit(pytest.main(["-q", "-x", "-p", "no:cacheprovider", {host_tests!r}]))
'''


def test_host_layer_clean_under_asan_ubsan():
    try:
        lib = B.build_host_sanitized()
        runtime = B.asan_runtime()
    except (RuntimeError, FileNotFoundError) as e:  # pragma: no cover - no hipcc
        pytest.skip(f"no sanitizer build: {e}")
    if not os.path.exists(runtime):
        pytest.skip("no AddressSanitizer runtime")
    code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib,
                        host_tests=os.path.join(ROOT, "tests", "test_abi_host.py"))
    env = dict(os.environ, LD_PRELOAD=runtime, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=600)
    out = res.stdout + res.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
