"""Thin ctypes binding of libkashin.so (argument marshalling only).

Every function has the name of the C entry point it calls (see include/kashin.h)
and takes torch tensors that already live on the GPU; all work runs in the HIP
kernels.  A non-OK status raises ``KashinError`` carrying the library's message.
There is no CPU fallback: if the library is not built, ``lib()`` raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkashin.so")

KASHIN_OK = 0
KASHIN_E_INVALID = -1
KASHIN_E_UNSUPPORTED_N = -2
KASHIN_E_NOMEM = -3
KASHIN_E_HIP = -4
KASHIN_F32 = 0
KASHIN_F16 = 1
KASHIN_BF16 = 2

EXPORTS = (
    "kashin_supported_n", "kashin_signs", "kashin_plan", "kashin_plan_destroy", "kashin_plan_signs",
    "kashin_plan_info", "kashin_decompose", "kashin_cluster2bit", "kashin_reconstruct",
    "kashin_quantize", "kashin_quantize_grouped", "kashin_reconstruct_grouped", "kashin_apply_p", "kashin_rotate", "kashin_trace", "kashin_decompose_schedule",
    "kashin_trace_schedule", "kashin_quantize_rotated", "kashin_reconstruct_rotated", "kashin_optq_factor",
    "kashin_optq_workspace_bytes", "kashin_optq_quantize", "kashin_optq_quantize_noalloc", "kashin_status_string",
    "kashin_last_error",
)
SCHEDULES = {"alternating": 0, "reverse": 1, "adaptive": 2, "original": 3}

_lib = None


class KashinError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libkashin.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2609_11687_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    sig = {
        "kashin_supported_n": [i32],
        "kashin_signs": [i32, u64, vp],
        "kashin_plan": [ctypes.POINTER(vp), i32, u64, i32],
        "kashin_plan_destroy": [vp],
        "kashin_plan_signs": [vp, vp],
        "kashin_plan_info": [vp, vp, vp, vp],
        "kashin_decompose": [vp, vp, i32, i64, i64, vp, vp, vp, vp, vp, vp],
        "kashin_cluster2bit": [vp, vp, vp, vp, i64, i32, vp, vp, vp, vp],
        "kashin_reconstruct": [vp, vp, vp, vp, i64, vp, i64, vp],
        "kashin_quantize": [vp, vp, i32, i64, i64, i32, vp, vp, vp, vp],
        "kashin_quantize_grouped": [vp, i32, i32, i32, vp, vp],
        "kashin_reconstruct_grouped": [vp, i32, vp],
        "kashin_apply_p": [vp, vp, vp, i64, vp],
        "kashin_rotate": [i32, u64, i32, vp, i32, i64, i64, vp, i64, vp],
        "kashin_quantize_rotated": [vp, u64, vp, i32, i64, i64, i32, vp, vp, vp, vp],
        "kashin_reconstruct_rotated": [vp, u64, vp, vp, vp, i64, vp, i64, vp],
        "kashin_decompose_schedule": [vp, i32, ctypes.c_float, vp, i32, i64, i64, vp, vp, vp, vp],
        "kashin_trace_schedule": [vp, i32, ctypes.c_float, vp, i32, i64, i64, vp, i64, vp, vp, vp, vp, vp, vp, vp],
        "kashin_trace": [vp, vp, i32, i64, i64, vp, i64, vp, vp, vp, vp, vp],
        "kashin_optq_factor": [vp, i32, i64, ctypes.c_double, vp, vp, vp],
        "kashin_optq_quantize": [vp, vp, i64, i64, vp, vp, i64, i64, i32, i32, i32, vp, vp, vp, vp, vp, i64, vp],
        "kashin_optq_quantize_noalloc": [vp, vp, i64, i64, vp, vp, i64, i64, i32, i32, i32, vp, vp, vp, vp, vp],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.kashin_optq_workspace_bytes.argtypes = [i64, i32, i32]
    L.kashin_optq_workspace_bytes.restype = i64
    L.kashin_status_string.argtypes = [ctypes.c_int]
    L.kashin_status_string.restype = ctypes.c_char_p
    L.kashin_last_error.argtypes = []
    L.kashin_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int) -> None:
    if status != KASHIN_OK:
        raise KashinError(status, lib().kashin_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return KASHIN_F32
    if t.dtype == torch.float16:
        return KASHIN_F16
    if t.dtype == torch.bfloat16:
        return KASHIN_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _rows(w):
    """(m, ldw) of a row-major 2-D tensor whose rows are unit-stride."""
    if w.dim() == 2 and w.shape[0] == 0:  # no rows: strides are arbitrary (torch gives 0 for empty arrays)
        return 0, w.shape[1]
    if w.dim() != 2 or (w.stride(1) != 1 and w.shape[1] > 1):
        raise ValueError("expected a 2-D tensor with unit-stride rows")
    if w.shape[0] == 1:  # one row: its stride is never used (numpy and torch may report 0)
        return 1, w.shape[1]
    return w.shape[0], w.stride(0)


def _on_plan_device(plan, t, name):
    if t.device.type != "cuda" or (plan is not None and t.device.index != plan.device):
        where = "cuda" if plan is None else f"cuda:{plan.device}"
        raise ValueError(f"{name} must live on {where} (got {t.device})")


def _need(plan, t, shape, dtype, name, nullable=False):
    """Check an output or side input the library reads or writes with a fixed layout: exact shape,
    dtype, contiguous, on the plan's device.  The C side trusts these (a wrong buffer would be a
    device out-of-bounds access), so they are checked before every call."""
    import torch

    if t is None:
        if nullable:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if t.numel():
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        _on_plan_device(plan, t, name)


def _need_rows(plan, w, n, name, dtypes=None):
    """A row-major input or output of m rows of n entries (unit-stride rows, any ld >= n)."""
    import torch

    m, ld = _rows(w)
    if w.shape[1] != n:
        raise ValueError(f"{name} rows must have {n} entries (got {w.shape[1]})")
    if dtypes is not None and w.dtype not in dtypes:
        raise TypeError(f"{name} must be one of {dtypes} (got {w.dtype})")
    if m:
        _on_plan_device(plan, w, name)
    return m, ld


def _f32():
    import torch
    return torch.float32


def _codes_shapes(plan, m):
    import torch
    nb = (plan.n + 3) // 4
    return (m, nb), torch.uint8, (m, 2, 4), torch.float32


def _need_codes(plan, m, codes_u, codes_v, centers):
    cs, cdt, ces, cedt = _codes_shapes(plan, m)
    _need(plan, codes_u, cs, cdt, "codes_u")
    _need(plan, codes_v, cs, cdt, "codes_v")
    _need(plan, centers, ces, cedt, "centers")


class Plan:
    """Owns a kashin_plan_t; destroyed explicitly (``destroy``) or on garbage collection."""

    def __init__(self, handle: ctypes.c_void_p, n: int, seed: int, iters: int, device: int = 0):
        self.handle = handle
        self.n = n
        self.seed = seed
        self.iters = iters
        self.device = device  # the HIP device the plan's tables live on (current at creation)

    def destroy(self) -> None:
        if self.handle:
            _check(lib().kashin_plan_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            if self.handle:
                lib().kashin_plan_destroy(self.handle)
        except Exception:
            pass


# ----------------------------------------------------------------------------- host-only
def kashin_supported_n(n: int) -> bool:
    return bool(lib().kashin_supported_n(n))


def kashin_signs(n: int, seed: int):
    import numpy as np
    out = np.empty(n, dtype=np.int8)
    _check(lib().kashin_signs(n, seed, out.ctypes.data_as(ctypes.c_void_p)))
    return out


# ----------------------------------------------------------------------------- plan
def kashin_plan(n: int, seed: int, iters: int) -> Plan:
    import torch
    h = ctypes.c_void_p()
    _check(lib().kashin_plan(ctypes.byref(h), n, seed, iters))
    return Plan(h, n, seed, iters, torch.cuda.current_device())


def kashin_plan_destroy(plan: Plan) -> None:
    plan.destroy()


def kashin_plan_signs(plan: Plan):
    import numpy as np
    out = np.empty(plan.n, dtype=np.int8)
    _check(lib().kashin_plan_signs(plan.handle, out.ctypes.data_as(ctypes.c_void_p)))
    return out


def kashin_plan_info(plan: Plan):
    n, it, sd = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_uint64()
    _check(lib().kashin_plan_info(plan.handle, ctypes.byref(n), ctypes.byref(it), ctypes.byref(sd)))
    return n.value, it.value, sd.value


# ----------------------------------------------------------------------------- device calls
def kashin_decompose(plan, w, u, vhat, r=None, cstep=None, bounds=None, stream=None):
    import torch
    m, ldw = _need_rows(plan, w, plan.n, "w", (torch.float32, torch.float16, torch.bfloat16))
    for name, t, nl in (("u", u, False), ("vhat", vhat, False), ("r", r, True)):
        _need(plan, t, (m, plan.n), torch.float32, name, nullable=nl)
    _need(plan, cstep, (m, 4), torch.float32, "cstep", nullable=True)
    _need(plan, bounds, (m, 4), torch.float32, "bounds", nullable=True)
    _check(lib().kashin_decompose(plan.handle, _ptr(w), _dtype_code(w), m, ldw, _ptr(u), _ptr(vhat), _ptr(r),
                                  _ptr(cstep), _ptr(bounds), _stream(stream)))


def kashin_cluster2bit(plan, u, vhat, cstep, lloyd_iters, codes_u, codes_v, centers, stream=None):
    import torch
    m = u.shape[0]
    _need(plan, u, (m, plan.n), torch.float32, "u")
    _need(plan, vhat, (m, plan.n), torch.float32, "vhat")
    _need(plan, cstep, (m, 4), torch.float32, "cstep")
    cs, cdt, ces, cedt = _codes_shapes(plan, m)
    _need(plan, codes_u, cs, cdt, "codes_u")
    _need(plan, codes_v, cs, cdt, "codes_v")
    _need(plan, centers, ces, cedt, "centers")
    _check(lib().kashin_cluster2bit(plan.handle, _ptr(u), _ptr(vhat), _ptr(cstep), m, lloyd_iters, _ptr(codes_u),
                                    _ptr(codes_v), _ptr(centers), _stream(stream)))


def kashin_reconstruct(plan, codes_u, codes_v, centers, w_hat, stream=None):
    m, ldw = _need_rows(plan, w_hat, plan.n, "w_hat", (_f32(),))
    _need_codes(plan, m, codes_u, codes_v, centers)
    _check(lib().kashin_reconstruct(plan.handle, _ptr(codes_u), _ptr(codes_v), _ptr(centers), m, _ptr(w_hat), ldw,
                                    _stream(stream)))


def kashin_quantize(plan, w, lloyd_iters, codes_u, codes_v, centers, stream=None):
    m, ldw = _need_rows(plan, w, plan.n, "w")
    _need_codes(plan, m, codes_u, codes_v, centers)
    _check(lib().kashin_quantize(plan.handle, _ptr(w), _dtype_code(w), m, ldw, lloyd_iters, _ptr(codes_u),
                                 _ptr(codes_v), _ptr(centers), _stream(stream)))


class QuantizeItem(ctypes.Structure):
    """kashin_quantize_item of include/kashin.h."""
    _fields_ = [("plan", ctypes.c_void_p), ("w", ctypes.c_void_p), ("m", ctypes.c_int64), ("ldw", ctypes.c_int64),
                ("codes_u", ctypes.c_void_p), ("codes_v", ctypes.c_void_p), ("centers", ctypes.c_void_p)]


def kashin_quantize_grouped(items, lloyd_iters, stream=None, rot_seed=None):
    """items: sequence of (plan, w, codes_u, codes_v, centers), one per matrix, all of one dtype;
    rot_seed: None, or the seed of the incoherence rotation applied to every matrix's rows."""
    arr = (QuantizeItem * max(1, len(items)))()
    dtype = KASHIN_F32
    for i, (plan, w, cu, cv, ce) in enumerate(items):
        m, ldw = _need_rows(plan, w, plan.n, f"items[{i}].w")
        _need_codes(plan, m, cu, cv, ce)
        dtype = _dtype_code(w)
        arr[i] = QuantizeItem(plan.handle, w.data_ptr(), m, ldw, cu.data_ptr(), cv.data_ptr(), ce.data_ptr())
    if any(_dtype_code(it[1]) != dtype for it in items):
        raise TypeError("every matrix of a grouped call has the same dtype")
    seed = None if rot_seed is None else ctypes.byref(ctypes.c_uint64(rot_seed))
    _check(lib().kashin_quantize_grouped(ctypes.cast(arr, ctypes.c_void_p), len(items), dtype, lloyd_iters, seed,
                                         _stream(stream)))


class ReconstructItem(ctypes.Structure):
    """kashin_reconstruct_item of include/kashin.h."""
    _fields_ = [("plan", ctypes.c_void_p), ("codes_u", ctypes.c_void_p), ("codes_v", ctypes.c_void_p),
                ("centers", ctypes.c_void_p), ("m", ctypes.c_int64), ("w_hat", ctypes.c_void_p),
                ("ldw", ctypes.c_int64)]


def kashin_reconstruct_grouped(items, stream=None):
    """items: sequence of (plan, codes_u, codes_v, centers, w_hat), one per matrix."""
    arr = (ReconstructItem * max(1, len(items)))()
    for i, (plan, cu, cv, ce, wh) in enumerate(items):
        m, ldw = _need_rows(plan, wh, plan.n, f"items[{i}].w_hat", (_f32(),))
        _need_codes(plan, m, cu, cv, ce)
        arr[i] = ReconstructItem(plan.handle, cu.data_ptr(), cv.data_ptr(), ce.data_ptr(), m, wh.data_ptr(), ldw)
    _check(lib().kashin_reconstruct_grouped(ctypes.cast(arr, ctypes.c_void_p), len(items), _stream(stream)))


def kashin_apply_p(plan, x, y, stream=None):
    m = x.shape[0]
    _need(plan, x, (m, plan.n), _f32(), "x")
    _need(plan, y, (m, plan.n), _f32(), "y")
    _check(lib().kashin_apply_p(plan.handle, _ptr(x), _ptr(y), m, _stream(stream)))


def kashin_decompose_schedule(plan, schedule, w, u, vhat, r=None, tol=0.0, stream=None):
    m, ldw = _need_rows(plan, w, plan.n, "w")
    for name, t, nl in (("u", u, False), ("vhat", vhat, False), ("r", r, True)):
        _need(plan, t, (m, plan.n), _f32(), name, nullable=nl)
    _check(lib().kashin_decompose_schedule(plan.handle, SCHEDULES[schedule], tol, _ptr(w), _dtype_code(w), m, ldw,
                                           _ptr(u), _ptr(vhat), _ptr(r), _stream(stream)))


def kashin_trace_schedule(plan, schedule, w, rows, sign_trace, c_trace, choice_trace, r2_trace, u, vhat, tol=0.0,
                          stream=None):
    import torch
    m, ldw = _need_rows(plan, w, plan.n, "w")
    nr, st = rows.numel(), 4 * plan.iters
    _need(plan, rows, (nr,), torch.int64, "rows")
    _need(plan, sign_trace, (nr, st, plan.n), torch.int8, "sign_trace")
    _need(plan, c_trace, (nr, st), torch.float32, "c_trace")
    _need(plan, choice_trace, (nr, st), torch.int8, "choice_trace")
    _need(plan, r2_trace, (nr, st), torch.float32, "r2_trace")
    _need(plan, u, (nr, plan.n), torch.float32, "u")
    _need(plan, vhat, (nr, plan.n), torch.float32, "vhat")
    _check(lib().kashin_trace_schedule(plan.handle, SCHEDULES[schedule], tol, _ptr(w), _dtype_code(w), m, ldw,
                                       _ptr(rows), rows.numel(), _ptr(sign_trace), _ptr(c_trace), _ptr(choice_trace),
                                       _ptr(r2_trace), _ptr(u), _ptr(vhat), _stream(stream)))


def kashin_quantize_rotated(plan, rot_seed, w, lloyd_iters, codes_u, codes_v, centers, stream=None):
    m, ldw = _need_rows(plan, w, plan.n, "w")
    _need_codes(plan, m, codes_u, codes_v, centers)
    _check(lib().kashin_quantize_rotated(plan.handle, rot_seed, _ptr(w), _dtype_code(w), m, ldw, lloyd_iters,
                                         _ptr(codes_u), _ptr(codes_v), _ptr(centers), _stream(stream)))


def kashin_reconstruct_rotated(plan, rot_seed, codes_u, codes_v, centers, w_hat, stream=None):
    m, ldw = _need_rows(plan, w_hat, plan.n, "w_hat", (_f32(),))
    _need_codes(plan, m, codes_u, codes_v, centers)
    _check(lib().kashin_reconstruct_rotated(plan.handle, rot_seed, _ptr(codes_u), _ptr(codes_v), _ptr(centers), m,
                                            _ptr(w_hat), ldw, _stream(stream)))


def kashin_rotate(n, seed, x, y, inverse=False, stream=None):
    """y = R x (or R^T x) row-wise; x fp32, fp16 or bf16 rows, y fp32 rows (y may be x, fp32)."""
    m, ldx = _need_rows(None, x, n, "x")
    my, ldy = _need_rows(None, y, n, "y", (_f32(),))
    if my != m:
        raise ValueError("x and y must have the same number of rows")
    _check(lib().kashin_rotate(n, seed, 1 if inverse else 0, _ptr(x), _dtype_code(x), m, ldx, _ptr(y), ldy,
                               _stream(stream)))


def kashin_trace(plan, w, rows, sign_trace, c_trace, u, vhat, stream=None):
    import torch
    m, ldw = _need_rows(plan, w, plan.n, "w")
    nr, st = rows.numel(), 4 * plan.iters
    _need(plan, rows, (nr,), torch.int64, "rows")
    _need(plan, sign_trace, (nr, st, plan.n), torch.int8, "sign_trace")
    _need(plan, c_trace, (nr, st), torch.float32, "c_trace")
    _need(plan, u, (nr, plan.n), torch.float32, "u")
    _need(plan, vhat, (nr, plan.n), torch.float32, "vhat")
    _check(lib().kashin_trace(plan.handle, _ptr(w), _dtype_code(w), m, ldw, _ptr(rows), rows.numel(),
                              _ptr(sign_trace), _ptr(c_trace), _ptr(u), _ptr(vhat), _stream(stream)))


def kashin_optq_factor(h, u, v=None, damp=0.01, stream=None):
    """U (upper, U^T U = (H + damp mean(diag H) I)^-1) and V = U^-1 into u, v (d x d float64,
    contiguous, on H's device); H is d x d fp32 with unit-stride rows."""
    import torch
    d, ldh = _rows(h)
    if h.shape[1] != d or h.dtype != torch.float32:
        raise ValueError("h must be a square fp32 matrix")
    _need(None, u, (d, d), torch.float64, "u")
    _need(None, v, (d, d), torch.float64, "v", nullable=True)
    _on_plan_device(None, h, "h")
    _check(lib().kashin_optq_factor(_ptr(h), d, ldh, damp, _ptr(u), _ptr(v), _stream(stream)))


def kashin_optq_workspace_bytes(d_in: int, n: int, chunk: int) -> int:
    return int(lib().kashin_optq_workspace_bytes(d_in, n, chunk))


def _need_square_rows(plan, t, d, name, nullable=False):
    """A d x d float64 matrix (or a d x d block of a larger one) with unit-stride rows."""
    import torch
    if t is None:
        if nullable:
            return None
        raise ValueError(f"{name} is required")
    if t.dtype != torch.float64 or t.dim() != 2 or tuple(t.shape) != (d, d) or (d > 1 and t.stride(1) != 1):
        raise ValueError(f"{name} must be a {d} x {d} float64 matrix with unit-stride rows")
    if d:
        _on_plan_device(plan, t, name)
    return t.stride(0) if d > 1 else max(d, 1)


def kashin_optq_quantize(plan, w_t, u, v, chunk, exact, lloyd_iters, codes_u, codes_v, centers, q_t, work,
                         quantize_rows=None, stream=None):
    """Error-compensated quantisation of the rows of w_t (d_in x n fp32, updated in place) with the
    factor (u, v) of kashin_optq_factor (or trailing blocks of it: any leading dimension); the first
    `quantize_rows` rows (default all) are quantised.  work: a uint8 device buffer of at least
    kashin_optq_workspace_bytes(d_in, n, chunk) bytes."""
    import torch
    d_in, ldw = _need_rows(plan, w_t, plan.n, "w_t", (torch.float32,))
    qr = d_in if quantize_rows is None else quantize_rows
    ldu = _need_square_rows(plan, u, d_in, "u")
    ldv = _need_square_rows(plan, v, d_in, "v", nullable=bool(exact))
    if ldv is not None and ldv != ldu:
        raise ValueError("u and v must have the same leading dimension")
    _need_codes(plan, qr, codes_u, codes_v, centers)
    _need(plan, q_t, (qr, plan.n), torch.float32, "q_t")
    if work.dtype != torch.uint8 or work.dim() != 1 or (work.numel() and not work.is_contiguous()):
        raise ValueError("work must be a contiguous 1-D uint8 tensor")
    if work.numel():
        _on_plan_device(plan, work, "work")
    _check(lib().kashin_optq_quantize(plan.handle, _ptr(w_t), d_in, ldw, _ptr(u), _ptr(v), ldu, qr, chunk,
                                      1 if exact else 0, lloyd_iters, _ptr(codes_u), _ptr(codes_v), _ptr(centers),
                                      _ptr(q_t), _ptr(work), work.numel(), _stream(stream)))


def kashin_optq_quantize_noalloc(plan, w_t, u, v, chunk, exact, lloyd_iters, codes_u, codes_v, centers, q_t,
                                 quantize_rows=None, stream=None):
    """kashin_optq_quantize with the library's static device workspace (no workspace argument)."""
    import torch
    d_in, ldw = _need_rows(plan, w_t, plan.n, "w_t", (torch.float32,))
    qr = d_in if quantize_rows is None else quantize_rows
    ldu = _need_square_rows(plan, u, d_in, "u")
    ldv = _need_square_rows(plan, v, d_in, "v", nullable=bool(exact))
    if ldv is not None and ldv != ldu:
        raise ValueError("u and v must have the same leading dimension")
    _need_codes(plan, qr, codes_u, codes_v, centers)
    _need(plan, q_t, (qr, plan.n), torch.float32, "q_t")
    _check(lib().kashin_optq_quantize_noalloc(plan.handle, _ptr(w_t), d_in, ldw, _ptr(u), _ptr(v), ldu, qr, chunk,
                                              1 if exact else 0, lloyd_iters, _ptr(codes_u), _ptr(codes_v),
                                              _ptr(centers), _ptr(q_t), _stream(stream)))


# ----------------------------------------------------------------------------- allocating helpers
def quantize_alloc(plan, w, lloyd_iters=0, stream=None):
    """Allocate outputs (torch, on w's device) and run kashin_quantize."""
    import torch
    m = w.shape[0]
    nb = (plan.n + 3) // 4
    cu = torch.empty((m, nb), dtype=torch.uint8, device=w.device)
    cv = torch.empty((m, nb), dtype=torch.uint8, device=w.device)
    ce = torch.empty((m, 2, 4), dtype=torch.float32, device=w.device)
    kashin_quantize(plan, w, lloyd_iters, cu, cv, ce, stream)
    return cu, cv, ce


def decompose_alloc(plan, w, want_r=False, stream=None):
    import torch
    m, n = w.shape[0], plan.n
    f = dict(dtype=torch.float32, device=w.device)
    u = torch.empty((m, n), **f)
    vh = torch.empty((m, n), **f)
    r = torch.empty((m, n), **f) if want_r else None
    cs = torch.empty((m, 4), **f)
    bd = torch.empty((m, 4), **f)
    kashin_decompose(plan, w, u, vh, r, cs, bd, stream)
    return u, vh, r, cs, bd
