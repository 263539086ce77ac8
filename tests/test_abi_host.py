"""Host-only checks of the C-ABI library: it loads, exports every declared entry point,
computes the sign mask like the oracle, and rejects bad arguments before touching a device."""
import ctypes
import os
import re
import subprocess

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


def _documented_lengths():
    """The supported set as the header states it (the comment of kashin_supported_n)."""
    text = open(HEADER).read()
    block = text[text.index("The supported lengths are exactly"):text.index("int kashin_supported_n")]
    block = block[:block.index("(")]
    return sorted(int(v) for v in re.findall(r"\b\d+\b", block))


def test_supported_lengths_are_exactly_the_documented_set():
    """The length contract: kashin_supported_n is 1 exactly on the set the header lists (every
    integer up to 40000 is asked), and that set holds the widths of the paper's models and its
    N = 10^4 convergence set-up."""
    doc = _documented_lengths()
    got = [n for n in range(0, 40001) if K.kashin_supported_n(n)]
    assert got == doc
    for n in (768, 3072, 4096, 11008, 5120, 13824, 14336, 16384, 2048, 8192, 10000):
        assert n in got


@pytest.mark.parametrize("n", [64, 96, 172, 512, 768, 1024, 3072, 4096, 5120, 6144, 10000, 11008, 13824, 14336,
                               16384])
def test_supported_sizes(n):
    assert K.kashin_supported_n(n)


@pytest.mark.parametrize("n", [-4, 0, 1, 2, 7, 100, 4095, 4097, 12288, 20000, 28672, 32768])
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
    """The fused-rotation entry points validate the plan like their unrotated forms (dead plans
    first; the plan's length is checked against the rotation's after that, which needs a live
    plan, hence a device: see the GPU tests)."""
    L = K.lib()
    fake = ctypes.c_void_p(0x1234)
    buf = ctypes.c_void_p(0x1000)
    assert L.kashin_quantize_rotated(None, 7, buf, 0, 4, 512, 0, buf, buf, buf, None) == K.KASHIN_E_INVALID
    assert L.kashin_quantize_rotated(fake, 7, buf, 0, 4, 512, 0, buf, buf, buf, None) == K.KASHIN_E_INVALID
    assert L.kashin_reconstruct_rotated(fake, 7, buf, buf, buf, 4, buf, 512, None) == K.KASHIN_E_INVALID
    assert "plan" in L.kashin_last_error().decode()


@pytest.mark.parametrize("n", [64, 96, 172, 256, 512, 768, 1024, 2048, 3072, 4096, 5120, 6144, 8192, 10000, 11008,
                               13824, 14336, 16384])
def test_rotation_lengths(n):
    """The rotation takes the plan lengths whose odd part is 1, 3 or 43; the others (odd parts 5,
    625, 27 and 7) are rejected on the host with KASHIN_E_UNSUPPORTED_N."""
    L = K.lib()
    x = ctypes.c_void_p(0x10000)
    y = ctypes.c_void_p(0x10000000)
    st = L.kashin_rotate(n, 0, 0, x, 0, 0, n, y, n, None)  # m = 0: validated, nothing launched
    if n // (n & -n) in (1, 3, 43):
        assert st == K.KASHIN_OK
    else:
        assert st == K.KASHIN_E_UNSUPPORTED_N


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


def test_binding_checks_buffers_before_calling():
    """The binding rejects output buffers of the wrong shape, dtype or layout, and tensors off the
    plan's device, before calling into the library (the C side trusts the layouts it documents).
    Zero-row tensors reach the shape checks without a device."""
    import torch

    plan = K.Plan(None, 512, 0, 4, 0)
    w0 = torch.zeros((0, 512), dtype=torch.float32)
    cu, cv, ce = torch.zeros((0, 128), dtype=torch.uint8), torch.zeros((0, 128), dtype=torch.uint8), \
        torch.zeros((0, 2, 4), dtype=torch.float32)
    with pytest.raises(ValueError, match="shape"):
        K.kashin_quantize(plan, w0, 0, torch.zeros((0, 127), dtype=torch.uint8), cv, ce)
    with pytest.raises(TypeError, match="uint8"):
        K.kashin_quantize(plan, w0, 0, torch.zeros((0, 128), dtype=torch.int8), cv, ce)
    with pytest.raises(ValueError, match="shape"):
        K.kashin_quantize(plan, w0, 0, cu, cv, torch.zeros((0, 8), dtype=torch.float32))
    with pytest.raises(ValueError, match="entries"):
        K.kashin_quantize(plan, torch.zeros((0, 256), dtype=torch.float32), 0, cu, cv, ce)
    with pytest.raises(ValueError, match="shape"):
        K.kashin_decompose(plan, w0, w0, torch.zeros((0, 511), dtype=torch.float32))
    with pytest.raises(ValueError, match="required"):
        K.kashin_decompose(plan, w0, w0, None)
    with pytest.raises(ValueError, match="shape"):
        K.kashin_trace(plan, w0, torch.zeros(0, dtype=torch.int64), torch.zeros((0, 16, 512), dtype=torch.int8),
                       torch.zeros((0, 15), dtype=torch.float32), torch.zeros((0, 512)), torch.zeros((0, 512)))
    # a non-contiguous output and a host tensor with rows: rejected before any call
    with pytest.raises(ValueError, match="contiguous"):
        K.kashin_apply_p(plan, torch.zeros((512, 2), dtype=torch.float32).t(), torch.zeros((2, 512)))
    with pytest.raises(ValueError, match="cuda"):
        K.kashin_quantize(plan, torch.zeros((2, 512), dtype=torch.float32), 0, cu, cv, ce)
    # all layouts right: the call reaches the library, which rejects the null plan
    with pytest.raises(K.KashinError):
        K.kashin_quantize(plan, w0, 0, cu, cv, ce, stream=0)


def test_optq_entry_points_validate_before_device():
    """The compensation entry points check sizes, factors, chunk, workspace and the plan on the host."""
    L = K.lib()
    buf = ctypes.c_void_p(0x1000)
    f = ctypes.c_double
    assert L.kashin_optq_factor(buf, 0, 0, f(0.01), buf, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_optq_factor(buf, 4, 3, f(0.01), buf, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_optq_factor(buf, 4, 4, f(-1.0), buf, None, None) == K.KASHIN_E_INVALID
    assert L.kashin_optq_factor(None, 4, 4, f(0.01), buf, None, None) == K.KASHIN_E_INVALID
    assert K.kashin_optq_workspace_bytes(-1, 512, 8) == -1
    assert K.kashin_optq_workspace_bytes(100, 512, 8) == ((8 * 512 * 4 + 255) // 256) * 256 + 8 * 100 * 4
    fake = ctypes.c_void_p(0x1234)
    args = (buf, 4, 512, buf, buf, 4, 4, 8, 0, 0, buf, buf, buf, buf, buf, 1 << 20, None)
    assert L.kashin_optq_quantize(fake, *args) == K.KASHIN_E_INVALID
    assert "plan" in L.kashin_last_error().decode()


def _abi_check_binary():
    from paper_2609_11687_amd import build as B

    if not os.path.exists(B.ABI_CHECK) or os.path.getmtime(B.ABI_CHECK) < os.path.getmtime(B.ABI_CHECK_SRC):
        B.build_abi_check()
    return B.ABI_CHECK


def test_c_program_uses_the_abi_host_side():
    """A C program linked against libkashin.so with include/kashin.h alone: the supported-length
    set, the sign mask against published splitmix64 outputs, validation and error messages."""
    res = subprocess.run([_abi_check_binary(), "host"], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().endswith("ok")


def test_input_dtype_codes():
    """F32, F16 and BF16 are the input element types; any other code is rejected before a launch
    with a message naming the three (the pointers are never dereferenced)."""
    L = K.lib()
    assert (K.KASHIN_F32, K.KASHIN_F16, K.KASHIN_BF16) == (0, 1, 2)
    p = ctypes.c_void_p(0x1000)
    assert L.kashin_rotate(512, 0, 0, p, 3, 4, 512, p, 512, None) == K.KASHIN_E_INVALID
    assert "BF16" in L.kashin_last_error().decode()
    import torch

    assert K._dtype_code(torch.zeros(1, dtype=torch.bfloat16)) == K.KASHIN_BF16
    with pytest.raises(TypeError):
        K._dtype_code(torch.zeros(1, dtype=torch.float64))
