"""Host-only checks of the C-ABI library: it loads, exports every declared entry point,
computes the sign mask like the oracle, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle.kashin_ref as ref
from paper_2609_11687_amd import kashin as K

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kashin.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kashin_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = K.lib()
    names = _declared()
    assert len(names) >= 13
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(K.EXPORTS)


@pytest.mark.parametrize("n", [64, 96, 172, 512, 768, 1024, 3072, 4096, 11008, 16384])
def test_supported_sizes(n):
    assert K.kashin_supported_n(n)


@pytest.mark.parametrize("n", [0, 1, 2, 7, 100, 4095, 4097, 32768])
def test_unsupported_sizes(n):
    assert not K.kashin_supported_n(n)


@pytest.mark.parametrize("n,seed", [(64, 0), (512, 1), (4096, 123456789), (11008, 2**64 - 1)])
def test_signs_match_oracle(n, seed):
    np.testing.assert_array_equal(K.kashin_signs(n, seed), ref.sign_mask(n, seed))


def test_signs_published_top_bits():
    # splitmix64 from state 0 starts 0xe220..., 0x6e78..., 0x06c4...: top bits 1, 0, 0
    np.testing.assert_array_equal(K.kashin_signs(3, 0), [-1, 1, 1])


def test_plan_validation_before_device():
    L = K.lib()
    h = ctypes.c_void_p()
    assert L.kashin_plan(None, 512, 0, 20) == K.KASHIN_E_INVALID
    assert L.kashin_plan(ctypes.byref(h), 512, 0, 0) == K.KASHIN_E_INVALID
    assert "iters" in L.kashin_last_error().decode()
    assert L.kashin_plan(ctypes.byref(h), 511, 0, 20) == K.KASHIN_E_UNSUPPORTED_N
    assert L.kashin_plan(ctypes.byref(h), 100, 0, 20) == K.KASHIN_E_UNSUPPORTED_N
    assert not h.value


def test_calls_reject_dead_plan():
    L = K.lib()
    fake = ctypes.c_void_p(0x1234)
    buf = ctypes.c_void_p(0x1000)
    assert L.kashin_decompose(None, buf, 0, 4, 512, buf, buf, None, None, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_decompose(fake, buf, 0, 4, 512, buf, buf, None, None, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_quantize(fake, buf, 0, 4, 512, 0, buf, buf, buf, None) == K.KASHIN_E_INVALID
    assert L.kashin_apply_p(None, buf, buf, 4, None) == K.KASHIN_E_INVALID
    assert L.kashin_plan_destroy(fake) == K.KASHIN_E_INVALID
    assert L.kashin_plan_signs(None, buf) == K.KASHIN_E_INVALID
    assert "plan" in L.kashin_last_error().decode()


def test_status_strings():
    L = K.lib()
    for st in (0, -1, -2, -3, -4):
        assert L.kashin_status_string(st)
    assert L.kashin_status_string(0) == b"ok"


def test_plan_needs_a_device_or_succeeds():
    """With no GPU the plan's table upload fails with KASHIN_E_HIP (after host validation)."""
    L = K.lib()
    h = ctypes.c_void_p()
    st = L.kashin_plan(ctypes.byref(h), 512, 0, 20)
    if st == K.KASHIN_OK:
        assert L.kashin_plan_destroy(h) == K.KASHIN_OK
    else:
        assert st == K.KASHIN_E_HIP


def test_rotate_validation_before_device():
    """kashin_rotate rejects bad sizes, dtypes, strides and overlapping buffers on the host;
    m = 0 is a no-op (pointers are never dereferenced)."""
    L = K.lib()
    x = ctypes.c_void_p(0x10000)
    y = ctypes.c_void_p(0x90000)
    assert L.kashin_rotate(320, 0, 0, x, 0, 4, 320, y, 320, None) == K.KASHIN_E_UNSUPPORTED_N  # odd part 5
    assert L.kashin_rotate(32768, 0, 0, x, 0, 4, 32768, y, 32768, None) == K.KASHIN_E_UNSUPPORTED_N
    assert L.kashin_rotate(512, 0, 2, x, 0, 4, 512, y, 512, None) == K.KASHIN_E_INVALID
    assert L.kashin_rotate(512, 0, 0, x, 7, 4, 512, y, 512, None) == K.KASHIN_E_INVALID
    assert L.kashin_rotate(512, 0, 0, x, 0, -1, 512, y, 512, None) == K.KASHIN_E_INVALID
    assert L.kashin_rotate(512, 0, 0, x, 0, 4, 511, y, 512, None) == K.KASHIN_E_INVALID
    assert L.kashin_rotate(512, 0, 0, x, 0, 4, 512, y, 500, None) == K.KASHIN_E_INVALID
    assert L.kashin_rotate(512, 0, 0, None, 0, 4, 512, y, 512, None) == K.KASHIN_E_INVALID
    # y starts inside x's rows without being the same rows
    assert L.kashin_rotate(512, 0, 0, x, 0, 4, 512, ctypes.c_void_p(0x10000 + 64), 512, None) == K.KASHIN_E_INVALID
    # in place is allowed only for fp32 rows with equal strides
    assert L.kashin_rotate(512, 0, 0, x, 1, 4, 512, x, 512, None) == K.KASHIN_E_INVALID
    assert "overlap" in L.kashin_last_error().decode()
    assert L.kashin_rotate(11008, 0, 1, x, 0, 0, 11008, y, 11008, None) == K.KASHIN_OK


def test_schedule_validation_before_device():
    L = K.lib()
    fake = ctypes.c_void_p(0x1234)
    buf = ctypes.c_void_p(0x1000)
    f = ctypes.c_float
    # dead plan first, then the schedule arguments
    assert L.kashin_decompose_schedule(fake, 0, f(0.0), buf, 0, 4, 512, buf, buf, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_trace_schedule(None, 2, f(0.0), buf, 0, 4, 512, buf, 1, buf, buf, buf, buf, buf, buf,
                                   None) == K.KASHIN_E_INVALID
    assert "plan" in L.kashin_last_error().decode()


def test_rotated_entry_points_reject_dead_plan():
    """The fused-rotation entry points validate the plan like their unrotated forms (the
    rotation itself needs no argument beyond the seed: every plan length has odd part 1, 3 or 43)."""
    L = K.lib()
    fake = ctypes.c_void_p(0x1234)
    buf = ctypes.c_void_p(0x1000)
    assert L.kashin_quantize_rotated(None, 7, buf, 0, 4, 512, 0, buf, buf, buf, None) == K.KASHIN_E_INVALID
    assert L.kashin_quantize_rotated(fake, 7, buf, 0, 4, 512, 0, buf, buf, buf, None) == K.KASHIN_E_INVALID
    assert L.kashin_reconstruct_rotated(fake, 7, buf, buf, buf, 4, buf, 512, None) == K.KASHIN_E_INVALID
    assert "plan" in L.kashin_last_error().decode()


@pytest.mark.parametrize("n", [64, 96, 172, 256, 512, 768, 1024, 2048, 3072, 4096, 8192, 11008, 16384])
def test_every_plan_length_is_rotatable(n):
    assert K.kashin_supported_n(n)
    assert n // (n & -n) in (1, 3, 43)


def test_grouped_quantize_validation_before_device():
    """kashin_quantize_grouped checks its item table on the host: an empty table is a no-op, and a
    null table, a bad count or dtype, or an item with a dead plan is rejected before any launch."""
    L = K.lib()
    fake = ctypes.c_void_p(0x1234)
    buf = 0x1000
    items = (K.QuantizeItem * 2)()
    items[0] = K.QuantizeItem(fake, buf, 4, 512, buf, buf, buf)
    items[1] = K.QuantizeItem(None, buf, 4, 512, buf, buf, buf)
    table = ctypes.cast(items, ctypes.c_void_p)
    assert L.kashin_quantize_grouped(table, 0, 0, 0, None, None) == K.KASHIN_OK
    assert L.kashin_quantize_grouped(None, 0, 0, 0, None, None) == K.KASHIN_OK
    assert L.kashin_quantize_grouped(None, 1, 0, 0, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_quantize_grouped(table, -1, 0, 0, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_quantize_grouped(table, 1, 5, 0, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_quantize_grouped(table, 1, 0, -1, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_quantize_grouped(table, 2, 0, 0, None, None) == K.KASHIN_E_INVALID
    assert "item 0" in L.kashin_last_error().decode()
    # the Python binding builds the same table from tensors
    assert ctypes.sizeof(K.QuantizeItem) == 56


def test_grouped_reconstruct_validation_before_device():
    """kashin_reconstruct_grouped checks its item table on the host: an empty table is a no-op, and
    a null table, a negative count or an item with a dead plan is rejected before any launch."""
    L = K.lib()
    fake = ctypes.c_void_p(0x1234)
    buf = 0x1000
    items = (K.ReconstructItem * 2)()
    items[0] = K.ReconstructItem(fake, buf, buf, buf, 4, buf, 512)
    items[1] = K.ReconstructItem(None, buf, buf, buf, 4, buf, 512)
    table = ctypes.cast(items, ctypes.c_void_p)
    assert L.kashin_reconstruct_grouped(table, 0, None) == K.KASHIN_OK
    assert L.kashin_reconstruct_grouped(None, 0, None) == K.KASHIN_OK
    assert L.kashin_reconstruct_grouped(None, 1, None) == K.KASHIN_E_INVALID
    assert L.kashin_reconstruct_grouped(table, -1, None) == K.KASHIN_E_INVALID
    assert L.kashin_reconstruct_grouped(table, 1, None) == K.KASHIN_E_INVALID
    assert "item 0" in L.kashin_last_error().decode()
    # the Python binding builds the same table from tensors
    assert ctypes.sizeof(K.ReconstructItem) == 56
