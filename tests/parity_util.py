"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI and compare
it with the float64 oracle.

Tolerances (the stated target of the method's GPU port): per row
  max |u - u_ref|, |vhat - vhat_ref| <= 1e-4 ||w||_inf,
  max |w - r - u - P vhat|          <= 1e-5 ||w||_inf   (P applied by the oracle in float64;
                                                       r = the oracle's residual, negligible
                                                       once k is large),
  2-bit codes equal in >= 99.99 % of entries, each mismatch within 1e-5 ||w||_inf of a
  decision boundary (a midpoint of the centres).

Near-ties.  A sign decision of Alg. 2 on an entry whose float64 value lies within fp32
rounding of zero is not determined by the input at fp32 precision, and the greedy
trajectory amplifies such a flip (it moves one entry of u by 2c).  The comparison
therefore replays the oracle with the GPU's own choices for entries inside a tie band
|x_i| <= tau = 1e-6 ||w||_inf (while the step size c >= tau), and requires every
decision outside that band to agree with float64.  That is a validity check of the
GPU's choices where several results are correct; everything else is the oracle's own
float64 arithmetic.  The direct (no replay) agreement is reported too.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle.kashin_ref as ref
from paper_2609_11687_amd import kashin as K

TOL_FACTOR = 1e-4
TOL_RECON = 1e-5
TOL_CODE_BOUNDARY = 1e-5
TAU_REL = 1e-6


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def gpu_trace(plan, w_dev, rows, k):
    n = plan.n
    rows_t = torch.as_tensor(np.asarray(rows, dtype=np.int64)).cuda()
    nr = rows_t.numel()
    signs = torch.empty((nr, 4 * k, n), dtype=torch.int8, device="cuda")
    cs = torch.empty((nr, 4 * k), dtype=torch.float32, device="cuda")
    u = torch.empty((nr, n), dtype=torch.float32, device="cuda")
    v = torch.empty((nr, n), dtype=torch.float32, device="cuda")
    K.kashin_trace(plan, w_dev, rows_t, signs, cs, u, v)
    torch.cuda.synchronize()
    return signs.cpu().numpy(), cs.cpu().numpy(), u.cpu().numpy().astype(np.float64), v.cpu().numpy().astype(np.float64)


def replay_parity(w64, eps, k, signs, u_gpu, v_gpu, direct=True):
    """Replay the oracle with the GPU's near-tie choices; return per-row error figures.  With
    `direct`, the plain float64 run (no replay) is done in the same batch and the fraction of rows
    it already matches within tolerance is reported (None without it)."""
    winf = np.abs(w64).max(axis=1)
    tau = TAU_REL * winf
    b = w64.shape[0]
    if direct:
        # replayed rows and plain float64 rows in one batch (tau < 0 switches replay off)
        both = ref.decompose(np.concatenate([w64, w64]), eps, k, replay_signs=np.concatenate([signs, signs]),
                             tau=np.concatenate([tau, -np.ones(b)]))
        rep = {key: (v[:b] if isinstance(v, np.ndarray) else v) for key, v in both.items()}
        plain = {key: v[b:] for key, v in both.items() if isinstance(v, np.ndarray)}
    else:
        rep = ref.decompose(w64, eps, k, replay_signs=signs, tau=tau)
        plain = None
    du = np.abs(u_gpu - rep["u"]).max(axis=1) / winf
    dv = np.abs(v_gpu - rep["vhat"]).max(axis=1) / winf
    # reconstruction identity of Alg. 2: u + P vhat = w - r (r from the replayed oracle; after
    # enough blocks r is far below fp32 resolution and this is |w - u - P vhat|)
    rec = np.abs(w64 - rep["r"] - u_gpu - ref.apply_p(v_gpu, eps)).max(axis=1) / winf
    frac = None
    if plain is not None:
        dd = np.maximum(np.abs(u_gpu - plain["u"]).max(axis=1), np.abs(v_gpu - plain["vhat"]).max(axis=1)) / winf
        frac = float(np.mean(dd <= TOL_FACTOR))
    return {
        "outside": rep["replay_outside"],
        "in_band_flips": rep["replay_in_band_flips"],
        "du": du,
        "dv": dv,
        "rec": rec,
        "direct_frac_ok": frac,
        "rep": rep,
        "winf": winf,
    }


def assert_replay_ok(res, label=""):
    bad = np.nonzero(res["outside"])[0]
    assert bad.size == 0, f"{label}: GPU sign decisions outside the tie band disagree with float64 in rows {bad[:10]}"
    assert res["du"].max() <= TOL_FACTOR, f"{label}: max |u - u_ref| / ||w||_inf = {res['du'].max():.3e}"
    assert res["dv"].max() <= TOL_FACTOR, f"{label}: max |vhat - vhat_ref| / ||w||_inf = {res['dv'].max():.3e}"
    assert res["rec"].max() <= TOL_RECON, f"{label}: reconstruction error {res['rec'].max():.3e}"


def boundary_distance(x, q):
    """Distance of each x (B, n) to the nearest midpoint of its row's sorted centres q (B, 4)."""
    mids = (q[:, :-1] + q[:, 1:]) * 0.5
    return np.min(np.abs(x[:, :, None] - mids[:, None, :]), axis=2)


def code_mismatches(codes_gpu, x_ref, q_ref, winf, label="", slack=None):
    """Compare GPU codes with the oracle's (decision taken in fp32 on the oracle's factor and
    centres); returns (mismatch count, total) and checks every mismatch is near a boundary (within
    1e-5 ||w||_inf, plus a per-row `slack` in the units of x by which the GPU's own midpoints may
    differ from the oracle's, e.g. after Lloyd passes)."""
    codes_ref = ref.assign_codes(x_ref, q_ref, np.float32)
    mism = codes_gpu != codes_ref
    if mism.any():
        extra = 0.0 if slack is None else (np.asarray(slack) / winf)[:, None]
        dist = boundary_distance(x_ref, q_ref) / winf[:, None] - extra
        worst = dist[mism].max()
        assert worst <= TOL_CODE_BOUNDARY, f"{label}: a code mismatch lies {worst:.3e} ||w||_inf from any boundary"
    return int(mism.sum()), int(mism.size)


def unpack(packed, n):
    return ref.unpack2bit(packed, n)


def assert_centres_close(ce, q, rel=1e-5):
    """Centres of one factor per row ([-(a+b), -|a-b|, |a-b|, a+b]) against the oracle's.  The
    inner centre |a-b| cancels when a ~ b, so its error is bounded by the errors of a and b:
    every centre is compared relative to the row's outer centre a+b."""
    ce = np.asarray(ce, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    scale = np.abs(q).max(axis=1)
    err = np.abs(ce - q).max(axis=1)
    bad = err > rel * scale + 1e-30
    assert not bad.any(), f"centres differ: rows {np.nonzero(bad)[0][:8]}, rel err {(err / np.maximum(scale, 1e-30)).max():.2e}"


def lloyd_tolerance(x, q0, passes, winf, band=TOL_CODE_BOUNDARY):
    """Per-row bound on how far the centres after `passes` Lloyd passes (from q0) may move when the
    entries of x lying within band ||w||_inf of a midpoint (a near-tie: the GPU's fp32 factor may
    sit on the other side) are assigned to the other cluster.  Moving one entry between adjacent
    clusters shifts each mean by at most (q_3 - q_0) / (its count); a shifted centre moves the next
    pass's midpoints, so the band of the next pass widens by the bound so far."""
    q = np.array(q0, dtype=np.float64, copy=True)
    tol = np.zeros(x.shape[0])
    for _ in range(passes):
        mids = (q[:, :-1] + q[:, 1:]) * 0.5
        dist = np.abs(x[:, :, None] - mids[:, None, :]).min(axis=2)
        near = (dist <= band * winf[:, None] + tol[:, None]).sum(axis=1)
        codes = ref.assign_codes(x, q)
        counts = np.stack([(codes == c).sum(axis=1) for c in range(4)], axis=1)
        smallest = np.where(counts > 0, counts, np.iinfo(np.int64).max).min(axis=1)
        tol = tol + near * (q[:, 3] - q[:, 0]) / np.maximum(smallest - near, 1)
        q = ref.lloyd(x, q, 1)
    return tol


def assert_lloyd_centres_close(ce, q, tol, rel=1e-5):
    """Lloyd centres against the oracle's, within rel of the row's outer centre plus the near-tie
    bound of lloyd_tolerance."""
    ce = np.asarray(ce, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    scale = np.abs(q).max(axis=1)
    err = np.abs(ce - q).max(axis=1)
    bad = err > rel * scale + tol + 1e-30
    assert not bad.any(), (f"Lloyd centres differ: rows {np.nonzero(bad)[0][:8]}, err {err[bad][:4]}, "
                           f"allowed {(rel * scale + tol)[bad][:4]}")


def near_boundary_count(x, q, winf, slack):
    """Entries of x within 1e-5 ||w||_inf + slack (per row, units of x) of a midpoint of q: the codes
    that may legitimately differ when the other side's midpoints are off by up to `slack`."""
    dist = boundary_distance(x, q)
    return int((dist <= TOL_CODE_BOUNDARY * winf[:, None] + np.asarray(slack)[:, None]).sum())
