"""Error-compensated quantisation of a weight matrix (Sec. 5, Fig. 1; eq. optq_update).

The columns of W (d_out x d_in) are the vectors quantised here; the matrix is held transposed,
w_t = W^T (d_in x d_out), so that each column is a row of length d_out for the library kernels.
Argument marshalling only: the factor of the damped inverse Hessian comes from kashin_optq_factor
and the quantisation with the error carry from kashin_optq_quantize (both in libkashin); torch
only allocates the device buffers.

Chunk form (exact=False): chunks of `chunk` columns are quantised at once, dequantised, and their
error Delta = W_c - Q_c is carried into the columns not yet quantised through the upper Cholesky
factor U of (H + damp mean(diag H) I)^-1:

    W_r <- W_r - Delta U_cc^-1 U_cr        (held transposed: w_t[r] -= (U_cc^-1 U_cr)^T Delta^T)

which is eq. optq_update column by column at chunk = 1.  Exact form (exact=True): the columns of
a chunk are quantised one at a time, each one's error reaching the chunk's later columns before
they are quantised (err_i = Delta_i / U_ii, w_j -= err_i U_ij inside the chunk) and the remaining
columns in one product at the chunk's end (W_r -= E U_cr): OPTQ's lazy block update, equal to
eq. optq_update column by column for any chunk size.
"""
from __future__ import annotations

from . import kashin as K


def compensation_factor(h, damp: float = 0.01, want_v: bool = True):
    """(U, V) of kashin_optq_factor: U the upper Cholesky factor of Hd^-1, Hd = H + damp
    mean(diag H) I, and V = U^-1 (float64 device tensors; V None unless want_v)."""
    import torch

    h32 = h.to(torch.float32).contiguous()
    d = h32.shape[0]
    u = torch.empty((d, d), dtype=torch.float64, device=h32.device)
    v = torch.empty_like(u) if want_v else None
    K.kashin_optq_factor(h32, u, v, damp)
    return u, v


def optq_quantize(plan, w_t, h, chunk: int = 128, damp: float = 0.01, lloyd_iters: int = 0, record=None,
                  stream=None, exact: bool = False, factor=None):
    """Quantise the rows of w_t (d_in x d_out fp32, CUDA; the columns of W) with error
    compensation; w_t is updated in place to the compensated weights.  Returns
    (codes_u, codes_v, centers, q_t) for all d_in rows (q_t = the dequantised rows).
    `factor`: (U, V) from compensation_factor, computed from h when None.  `record`, if a list,
    receives per chunk (per column with exact) a dict of snapshots, the chunks being run by
    separate calls that resume on the tail (for tests).  Everything is queued on `stream` (a
    torch stream; default: the current one), so matrices given different streams are quantised
    concurrently; the factorisation synchronises its stream."""
    import torch

    d_in, d_out = w_t.shape
    if plan.n != d_out:
        raise ValueError(f"plan length {plan.n} != d_out {d_out}")
    if w_t.dtype != torch.float32 or not w_t.is_contiguous():
        raise ValueError("w_t must be contiguous fp32")
    if stream is not None:
        with torch.cuda.stream(stream):
            return optq_quantize(plan, w_t, h, chunk, damp, lloyd_iters, record, None, exact, factor)
    u, v = factor if factor is not None else compensation_factor(h, damp, want_v=not exact)
    nb = (d_out + 3) // 4
    dev = w_t.device
    cu = torch.empty((d_in, nb), dtype=torch.uint8, device=dev)
    cv = torch.empty_like(cu)
    ce = torch.empty((d_in, 2, 4), dtype=torch.float32, device=dev)
    q_t = torch.empty_like(w_t)
    work = torch.empty(K.kashin_optq_workspace_bytes(d_in, d_out, chunk), dtype=torch.uint8, device=dev)
    if record is None:
        K.kashin_optq_quantize(plan, w_t, u, v, chunk, exact, lloyd_iters, cu, cv, ce, q_t, work)
        return cu, cv, ce, q_t
    step = 1 if exact else chunk
    for c0 in range(0, d_in, step):
        c1 = min(c0 + step, d_in)
        snap = {"c0": c0, "c1": c1, "w_chunk": w_t[c0:c1].clone()}
        K.kashin_optq_quantize(plan, w_t[c0:], u[c0:, c0:], None if v is None else v[c0:, c0:], chunk, exact,
                               lloyd_iters, cu[c0:c1], cv[c0:c1], ce[c0:c1], q_t[c0:c1], work,
                               quantize_rows=c1 - c0)
        snap["w_rest_after"] = w_t[c1:].clone()
        record.append(snap)
    return cu, cv, ce, q_t
