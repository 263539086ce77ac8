"""Error-compensated quantisation of a weight matrix (Sec. 5, Fig. 1; eq. optq_update).

The columns of W (d_out x d_in) are the vectors quantised here; the matrix is held transposed,
w_t = W^T (d_in x d_out), so that each column is a row of length d_out for the library kernels.
Chunks of `chunk` columns are quantised at once (kashin_quantize: Alg. 2 + 2-bit clustering),
dequantised (kashin_reconstruct), and their error Delta = W_c - Q_c is carried into the columns
not yet quantised through the upper Cholesky factor U of (H + damp mean(diag H) I)^-1
(U_cc^-1 is the diagonal block of V = U^-1, see compensation_factor):

    W_r <- W_r - Delta U_cc^-1 U_cr        (held transposed: w_t[r] -= (U_cc^-1 U_cr)^T Delta^T)

With chunk = 1 this is eq. optq_update column by column.  With exact=True the columns of a chunk
are quantised one at a time and each one's error reaches the chunk's later columns before they are
quantised (err_i = Delta_i / U_ii, w_j -= err_i U_ij inside the chunk); the chunk's errors reach
the remaining columns in one product at the chunk's end (W_r -= E U_cr): OPTQ's lazy block
update, which equals eq. optq_update applied column by column for any chunk size.  The chunk
form (exact=False) quantises a chunk's columns together, which is exact only at chunk = 1.
The factorisation of the d_in x d_in Hessian (float64) and the trailing update (an fp32 GEMM)
use the ROCm libraries through torch; every decomposition, clustering and reconstruction runs in
libkashin.
"""
from __future__ import annotations

from . import kashin as K


def compensation_factor(h, damp: float = 0.01):
    """(U, V): U the upper Cholesky factor of Hd^-1, Hd = H + damp mean(diag H) I, and V = U^-1
    (float64, on H's device).  With J the exchange matrix, the lower Cholesky factor L of J Hd J
    gives Hd = V V^T for the upper triangular V = J L J, so Hd^-1 = (V^-1)^T V^-1 and U = V^-1 (its
    diagonal is positive): one factorisation and one triangular solve, without forming Hd^-1.
    The diagonal blocks of V are the inverses of those of U."""
    import torch

    hd = h.to(torch.float64)
    d = hd.shape[0]
    eye = torch.eye(d, dtype=torch.float64, device=hd.device)
    hd = hd + damp * hd.diagonal().mean() * eye
    v = torch.linalg.cholesky(hd.flip(0, 1)).flip(0, 1)
    u = torch.linalg.solve_triangular(v, eye, upper=True)
    return u, v


def optq_quantize(plan, w_t, h, chunk: int = 128, damp: float = 0.01, lloyd_iters: int = 0, record=None,
                  stream=None, exact: bool = False):
    """Quantise the rows of w_t (d_in x d_out fp32, CUDA; the columns of W) with error
    compensation; w_t is updated in place to the compensated weights.  Returns
    (codes_u, codes_v, centers, q_t) for all d_in rows (q_t = the dequantised rows).
    `record`, if a list, receives per chunk a dict of snapshots (for tests).  Everything is
    queued on `stream` (a torch stream; default: the current one), so matrices given different
    streams are quantised concurrently."""
    import torch

    d_in, d_out = w_t.shape
    if plan.n != d_out:
        raise ValueError(f"plan length {plan.n} != d_out {d_out}")
    if w_t.dtype != torch.float32 or not w_t.is_contiguous():
        raise ValueError("w_t must be contiguous fp32")
    if stream is not None:
        with torch.cuda.stream(stream):
            return optq_quantize(plan, w_t, h, chunk, damp, lloyd_iters, record, None, exact)
    stream = torch.cuda.current_stream()
    u, v = compensation_factor(h, damp)
    nb = (d_out + 3) // 4
    cu = torch.empty((d_in, nb), dtype=torch.uint8, device=w_t.device)
    cv = torch.empty_like(cu)
    ce = torch.empty((d_in, 2, 4), dtype=torch.float32, device=w_t.device)
    q_t = torch.empty_like(w_t)
    u32 = u.to(torch.float32) if exact else None
    for c0 in range(0, d_in, chunk):
        c1 = min(c0 + chunk, d_in)
        wc = w_t[c0:c1]
        if exact:
            # one column at a time; its error reaches the chunk's later columns at once
            for i in range(c0, c1):
                if record is not None:
                    record.append({"c0": i, "c1": i + 1, "w_chunk": w_t[i:i + 1].clone()})
                K.kashin_quantize(plan, w_t[i:i + 1], lloyd_iters, cu[i:i + 1], cv[i:i + 1], ce[i:i + 1], stream)
                K.kashin_reconstruct(plan, cu[i:i + 1], cv[i:i + 1], ce[i:i + 1], q_t[i:i + 1], stream)
                if i + 1 < c1:
                    err = (w_t[i] - q_t[i]) / u32[i, i]
                    w_t[i + 1:c1] -= torch.outer(u32[i, i + 1:c1], err)
            if c1 < d_in:
                err = (wc - q_t[c0:c1]) / u32[c0:c1, c0:c1].diagonal()[:, None]  # E, chunk x d_out
                w_t[c1:] -= torch.matmul(u32[c0:c1, c1:].t().contiguous(), err)
            if record is not None:
                record[-1]["w_rest_after"] = w_t[c1:].clone()
            continue
        snap = {"c0": c0, "c1": c1, "w_chunk": wc.clone()} if record is not None else None
        K.kashin_quantize(plan, wc, lloyd_iters, cu[c0:c1], cv[c0:c1], ce[c0:c1], stream)
        K.kashin_reconstruct(plan, cu[c0:c1], cv[c0:c1], ce[c0:c1], q_t[c0:c1], stream)
        if c1 < d_in:
            delta = wc - q_t[c0:c1]
            m = torch.matmul(v[c0:c1, c0:c1], u[c0:c1, c1:])  # U_cc^-1 U_cr
            w_t[c1:] -= torch.matmul(m.t().contiguous().to(torch.float32), delta)
        if snap is not None:
            snap["w_rest_after"] = w_t[c1:].clone()
            record.append(snap)
    return cu, cv, ce, q_t
