"""Float64 CPU oracle for the Kashin-DCT hot path.

TEST INFRASTRUCTURE ONLY.  This module is imported by ``tests/``, by
``__graft_entry__.smoke()`` and by the ``cpu_baseline`` leg of ``bench.py``,
nothing else.  The product path (the HIP library under
``paper_2609_11687_amd/`` and its Python binding) never imports, links or
calls anything in ``oracle/``, and this module imports nothing from it.

It is a plain, slow restatement of what the method computes, in float64,
written from the paper ("Structured Transforms for Low-Overhead Quantization
of Language Models"):

* ``dct2_matrix`` -- the orthonormal DCT-II basis written out from its cosine
  definition (Sec. 4.1 and its footnote on the ``norm='ortho'`` convention;
  App. C footnote: IDCT is the transpose of DCT).
* ``apply_p`` / ``p_matrix`` -- the sign-randomised operator
  P z = IDCT(eps * DCT(z)) (Sec. 4.1, operator U_{E,Phi}; Alg. 2 input block),
  a symmetric involution (App. C, App. E).
* ``sign_mask`` -- the Rademacher mask eps drawn from a seed.  The paper only
  says it is generated once from a fixed seed (Sec. 5, App. C); the generator
  used here is splitmix64 (Steele, Lea, Flood 2014), re-implemented from its
  published definition, with eps_i = -1 when the top output bit is set.
* ``decompose`` -- the Greedy Algorithm with Alternating Updates (Alg. 2) run
  step by step in the paper's order: per block two steps on the cube Q_N
  accumulating into u, then two steps on P Q_N accumulating into v-hat, each
  v-hat step recomputing P rho and subtracting P(delta).  sign(0) = 0 and the
  step size is ||.||_1 / N, exactly as Alg. 2 prints them.
* ``closed_form_centers`` / ``lloyd`` / ``assign_codes`` -- the closed-form
  four-peak centres +-c1 +- c2 and the optional k-means refinement (Sec. 3.1).
* ``pack2bit`` / ``unpack2bit`` / ``reconstruct`` -- 2-bit codes, four per
  byte, and the load-time reconstitution w = u_q + P v_q (App. C).
* ``optimal4_sse`` -- exact optimum of 1-D 4-level clustering (brute force over
  contiguous partitions of the sorted values, or an O(4 n^2) dynamic program),
  used to pin the clustering.
* ``decompose_schedule`` -- the same greedy over the dictionary Q_N u P Q_N with
  other step schedules: Alg. 2's blocks in reverse order (Sec. 4.2), the
  adaptive choice of the half with the larger l1 correlation at every step
  (the single-step global greedy selection the paper contrasts with Alg. 2),
  and the original vector greedy of App. B (Alg. 1: that choice, with the
  step the orthogonal projection onto the sign vector).
* ``synthetic_hessian`` / ``optq_kashin`` -- the error-compensated pipeline of
  Sec. 5 (Fig. 1): the columns of W are quantised chunk by chunk (Alg. 2 +
  2-bit clustering on each column vector) and each chunk's error is carried
  into the columns not yet quantised through the Cholesky factor of H^-1
  (eq. optq_update, applied to a chunk at once); ``optq_reference`` is the
  same compensation written with the explicit inverse-Hessian downdate.
* ``hadamard_matrix`` / ``rotation_matrix`` / ``rotate`` -- the incoherence
  pre-rotation applied to weight rows before the decomposition (the "+H"
  preprocessing of Sec. 5; the paper only names a QuIP-style randomised
  Hadamard transform, with a Kronecker variant).  Reading: for n = 2^a b with
  b odd, R = (H_{2^a} / sqrt(2^a) kron C_b) diag(s), H the Sylvester Hadamard
  matrix, C_b the orthonormal DCT-II of length b (C_1 = [1]), s = sign_mask(n,
  seed).

Every function is pinned by ``tests/test_oracle_*.py`` against facts the paper
and the mathematics fix (library DCT, orthonormality, involution, the exact
one-step energy identity of App. E, hand-solvable inputs, brute-force optimal
clustering).  The convergence *rate* constants of Thm. 2 are not computable
(they depend on the unknown absolute constant c_3): parity unpinned for the
rate itself; only its computable intermediate bounds are tested.
"""
from __future__ import annotations

import functools
import itertools

import numpy as np

__all__ = [
    "splitmix64",
    "sign_mask",
    "dct2_matrix",
    "p_matrix",
    "apply_p",
    "decompose",
    "closed_form_centers",
    "assign_codes",
    "lloyd",
    "cluster2bit",
    "pack2bit",
    "unpack2bit",
    "dequantize",
    "reconstruct",
    "quantize",
    "optimal4_sse",
    "sse4",
    "hadamard_matrix",
    "rotation_matrix",
    "rotate",
    "SCHEDULES",
    "decompose_schedule",
    "synthetic_hessian",
    "damped_hessian",
    "compensation_factor",
    "optq_kashin",
    "optq_reference",
]

_MASK64 = (1 << 64) - 1


# ---------------------------------------------------------------------------
# Sign mask eps (Sec. 4.1: T_E multiplies DCT coefficient j by eps_j; Sec. 5 and
# App. C: one mask per layer, generated once from a fixed seed).
# ---------------------------------------------------------------------------
def splitmix64(seed: int, count: int) -> list[int]:
    """First ``count`` outputs of splitmix64 started from state ``seed``.

    Published definition (Steele, Lea, Flood, "Fast splittable pseudorandom
    number generators", OOPSLA 2014; the 64-bit finaliser constants of the
    public reference implementation): add the golden-gamma increment to the
    state, then xor-shift-multiply twice and xor-shift once.
    """
    s = seed & _MASK64
    out = []
    for _ in range(count):
        s = (s + 0x9E3779B97F4A7C15) & _MASK64
        z = s
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
        z ^= z >> 31
        out.append(z)
    return out


def sign_mask(n: int, seed: int) -> np.ndarray:
    """eps in {-1,+1}^n: eps_j = -1 iff the top bit of the j-th splitmix64 output is set."""
    vals = splitmix64(seed, n)
    return np.array([-1 if (v >> 63) else 1 for v in vals], dtype=np.int8)


# ---------------------------------------------------------------------------
# Orthonormal DCT-II and the operator P (Sec. 4.1; App. C).
# ---------------------------------------------------------------------------
@functools.lru_cache(maxsize=2)
def dct2_matrix(n: int) -> np.ndarray:
    """C[k, j] = sqrt(2/n) * s_k * cos(pi (2j+1) k / (2n)), s_0 = 1/sqrt(2), s_k = 1.

    Sec. 4.1 writes the basis with sqrt(2/N) for every index; under the stated
    norm='ortho' convention (Sec. 4.1 footnote, App. C footnote) the k = 0 row
    carries the extra 1/sqrt(2) that makes C orthonormal.  The angle index
    (2j+1)k is reduced modulo 4n in exact integer arithmetic before the cosine
    is taken, so every entry is a correctly-rounded cosine of a small angle.
    """
    if n < 1:
        raise ValueError("n must be >= 1")
    table = np.cos(np.pi * np.arange(4 * n, dtype=np.float64) / (2.0 * n))
    out = np.empty((n, n), dtype=np.float64)
    j = np.arange(n, dtype=np.int64)
    scale = np.sqrt(2.0 / n)
    for k in range(n):
        idx = ((2 * j + 1) * k) % (4 * n)
        out[k] = table[idx] * scale
    out[0] *= 1.0 / np.sqrt(2.0)
    out.setflags(write=False)
    return out


def p_matrix(eps: np.ndarray) -> np.ndarray:
    """Dense P = C^T diag(eps) C (Sec. 4.1, U_{E,Phi} = F^{-1} T_E F with F^{-1} = F^T)."""
    eps = np.asarray(eps, dtype=np.float64)
    c = dct2_matrix(eps.shape[0])
    return c.T @ (eps[:, None] * c)


def apply_p(x: np.ndarray, eps: np.ndarray) -> np.ndarray:
    """Row-wise P x = IDCT(eps * DCT(x)) for a batch of rows x (B, n) (Alg. 2 definition of P)."""
    x = np.asarray(x, dtype=np.float64)
    eps = np.asarray(eps, dtype=np.float64)
    c = dct2_matrix(eps.shape[0])
    return ((x @ c.T) * eps[None, :]) @ c


# ---------------------------------------------------------------------------
# Greedy Algorithm with Alternating Updates (Alg. 2).
# ---------------------------------------------------------------------------
def decompose(w, eps, k, *, replay_signs=None, tau=None, trace=False):
    """Run Alg. 2 on every row of ``w`` (B, n) for ``k`` blocks of four atomic steps.

    Returns a dict with
      ``u``, ``vhat``, ``r``  -- factors and residual, x = u + P vhat + r (Alg. 2 output),
      ``cstep``               -- (B, 4) magnitudes c of the four steps of block 0
                                 (c1, c2 from the u-steps, c3, c4 from the v-hat steps; Sec. 3.1),
      ``csum``                -- (B, 2) sums of all u-step and all v-hat-step magnitudes, the
                                 coefficient-sum bounds on ||u||_inf and ||vhat||_inf (App. F),
    and, with ``trace=True``, per-step records (see below).

    Replay (a validity check of another implementation's choices at near-ties,
    used by the GPU parity tests): with ``replay_signs`` (B, 4k, n) int8 and
    ``tau`` (B,), at atomic step s of row b, while that step's c >= tau[b] >= 0 (a
    negative tau switches replay off for that row), every
    entry whose float64 value satisfies |x_i| <= tau[b] takes the sign given in
    ``replay_signs[b, s, i]`` instead of sign(x_i).  All other decisions and all
    arithmetic stay float64 and the oracle's own.  ``out['replay_outside']``
    counts, per row, entries outside that band whose given sign disagrees with
    sign(x_i) (a wrong decision, not a tie).
    """
    w = np.array(w, dtype=np.float64, copy=True)
    if w.ndim == 1:
        w = w[None, :]
    eps = np.asarray(eps)
    bsz, n = w.shape
    if eps.shape != (n,):
        raise ValueError("eps must have shape (n,)")
    if k < 1:
        raise ValueError("k must be >= 1")
    rho = w.copy()
    u = np.zeros_like(w)
    vhat = np.zeros_like(w)
    cstep = np.zeros((bsz, 4))
    csum = np.zeros((bsz, 2))
    nsteps = 4 * k
    rec = None
    if trace:
        rec = {
            "c": np.zeros((bsz, nsteps)),
            "l1": np.zeros((bsz, nsteps)),
            "nnz": np.zeros((bsz, nsteps), dtype=np.int64),
            "r2_before": np.zeros((bsz, nsteps)),
            "r2_after": np.zeros((bsz, nsteps)),
            "min_margin": np.zeros((bsz, nsteps)),
            "signs": np.zeros((bsz, nsteps, n), dtype=np.int8),
        }
    outside = np.zeros(bsz, dtype=np.int64)
    in_band = np.zeros(bsz, dtype=np.int64)
    if replay_signs is not None:
        replay_signs = np.asarray(replay_signs)
        if replay_signs.shape != (bsz, nsteps, n):
            raise ValueError("replay_signs must have shape (B, 4k, n)")
        tau = np.broadcast_to(np.asarray(tau, dtype=np.float64), (bsz,))

    def take_signs(x, c, step):
        s = np.sign(x)
        if replay_signs is not None:
            gs = replay_signs[:, step, :].astype(np.float64)
            live = ((c >= tau) & (tau >= 0))[:, None]
            band = live & (np.abs(x) <= tau[:, None])
            wrong = live & ~band & (gs != s)
            outside[:] += wrong.sum(axis=1)
            in_band[:] += (band & (gs != s)).sum(axis=1)
            s = np.where(band, gs, s)
        return s

    # Alg. 2 visits the two halves of the dictionary in a fixed cycle of four atomic steps: the
    # cube Q_N twice, then its image P Q_N twice.  An atom of the cube half is a sign vector
    # itself; an atom of the other half is P applied to one, so its correlation with the residual
    # is read off P rho, and removing it subtracts P Delta from rho.
    cycle = ("cube", "cube", "rotated", "rotated")
    for step in range(nsteps):
        half = cycle[step % 4]
        x = rho if half == "cube" else apply_p(rho, eps)
        l1 = np.abs(x).sum(axis=1)
        c = l1 / n  # step size ||x||_1 / N; sign(0) = 0 below
        s = take_signs(x, c, step)
        d = s * c[:, None]
        if trace:
            rec["r2_before"][:, step] = (rho * rho).sum(axis=1)
        if half == "cube":
            u += d
            rho = rho - d
        else:
            vhat += d
            rho = rho - apply_p(d, eps)
        if trace:
            _record(rec, step, c, l1, x, s, rho)
        if step < 4:
            cstep[:, step] = c  # Sec. 3.1: the first block's four magnitudes fix the centres
        csum[:, 0 if half == "cube" else 1] += c
    out = {"u": u, "vhat": vhat, "r": rho, "cstep": cstep, "csum": csum}
    if trace:
        out["trace"] = rec
    if replay_signs is not None:
        out["replay_outside"] = outside
        out["replay_in_band_flips"] = in_band
    return out


def _record(rec, step, c, l1, x, s, rho):
    rec["c"][:, step] = c
    rec["l1"][:, step] = l1
    rec["nnz"][:, step] = (x != 0).sum(axis=1)
    rec["r2_after"][:, step] = (rho * rho).sum(axis=1)
    rec["min_margin"][:, step] = np.abs(x).min(axis=1)
    rec["signs"][:, step, :] = s.astype(np.int8)


# ---------------------------------------------------------------------------
# Four-peak 2-bit clustering (Sec. 3.1).
# ---------------------------------------------------------------------------
def closed_form_centers(a, b, dtype=np.float64):
    """Sorted centres of the four peaks +-a +- b left by two greedy updates of sizes a, b (Sec. 3.1)."""
    a = np.asarray(a, dtype=dtype)
    b = np.asarray(b, dtype=dtype)
    s = a + b
    d = np.abs(a - b)
    q = np.stack([-s, -d, d, s], axis=-1)
    return np.sort(q, axis=-1)


def assign_codes(x, q, dtype=np.float64):
    """code_i = number of midpoints of the sorted centres q strictly below x_i (ties go to the lower code).

    ``x`` is (B, n), ``q`` is (B, 4).  ``dtype`` is the precision the decision is
    taken in (midpoints and comparison).
    """
    x = np.asarray(x).astype(dtype)
    q = np.asarray(q).astype(dtype)
    half = dtype(0.5)
    mids = (q[:, :-1] + q[:, 1:]) * half
    return (x[:, :, None] > mids[:, None, :]).sum(axis=2).astype(np.uint8)


def lloyd(x, q, iters):
    """``iters`` plain 1-D k-means passes from centres q (B, 4): assign, recompute means,
    keep the previous centre for an empty cluster, re-sort (Sec. 3.1: a small number of
    refinement iterations, no restarts)."""
    x = np.asarray(x, dtype=np.float64)
    q = np.array(q, dtype=np.float64, copy=True)
    for _ in range(iters):
        codes = assign_codes(x, q)
        for b in range(x.shape[0]):
            for c in range(4):
                sel = codes[b] == c
                if sel.any():
                    q[b, c] = x[b, sel].mean()
        q = np.sort(q, axis=1)
    return q


def cluster2bit(u, vhat, cstep, lloyd_iters=0, decide_dtype=np.float64):
    """2-bit codes and centres for both factors.

    Centres start at the closed form: +-c1 +- c2 for u and +-c3 +- c4 for v-hat,
    where c1..c4 are the magnitudes of the four atomic steps of block 0 (Sec. 3.1).
    Returns (codes_u, codes_v, centers) with centers (B, 2, 4) ascending.
    """
    u = np.asarray(u, dtype=np.float64)
    vhat = np.asarray(vhat, dtype=np.float64)
    cstep = np.asarray(cstep, dtype=np.float64)
    qu = closed_form_centers(cstep[:, 0], cstep[:, 1])
    qv = closed_form_centers(cstep[:, 2], cstep[:, 3])
    if lloyd_iters:
        qu = lloyd(u, qu, lloyd_iters)
        qv = lloyd(vhat, qv, lloyd_iters)
    cu = assign_codes(u, qu, decide_dtype)
    cv = assign_codes(vhat, qv, decide_dtype)
    return cu, cv, np.stack([qu, qv], axis=1)


def pack2bit(codes):
    """Four 2-bit codes per byte: byte[i >> 2] |= code_i << 2 (i & 3) (two bits per entry, App. C)."""
    codes = np.asarray(codes, dtype=np.uint8)
    bsz, n = codes.shape
    nb = (n + 3) // 4
    out = np.zeros((bsz, nb), dtype=np.uint8)
    for i in range(n):
        out[:, i >> 2] |= (codes[:, i] & 3) << (2 * (i & 3))
    return out


def unpack2bit(packed, n):
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.zeros((packed.shape[0], n), dtype=np.uint8)
    for i in range(n):
        out[:, i] = (packed[:, i >> 2] >> (2 * (i & 3))) & 3
    return out


def dequantize(codes_u, codes_v, centers):
    """Quantised factors u_q = q_u[code], v_q = q_v[code] per row."""
    centers = np.asarray(centers, dtype=np.float64)
    rows = np.arange(centers.shape[0])[:, None]
    uq = centers[rows, 0, np.asarray(codes_u, dtype=np.int64)]
    vq = centers[rows, 1, np.asarray(codes_v, dtype=np.int64)]
    return uq, vq


def reconstruct(codes_u, codes_v, centers, eps):
    """Load-time reconstitution w_hat = u_q + P v_q (App. C)."""
    uq, vq = dequantize(codes_u, codes_v, centers)
    return uq + apply_p(vq, eps)


def quantize(w, eps, k, lloyd_iters=0):
    """Decompose (Alg. 2) then cluster and pack both factors (Sec. 3.1, App. C)."""
    d = decompose(w, eps, k)
    cu, cv, centers = cluster2bit(d["u"], d["vhat"], d["cstep"], lloyd_iters)
    return pack2bit(cu), pack2bit(cv), centers, d


# ---------------------------------------------------------------------------
# Exact 1-D 4-level clustering (pins the clustering; textbook result that an
# optimal 1-D k-means partition is contiguous in sorted order).
# ---------------------------------------------------------------------------
def sse4(x, q):
    """Sum of squared distances of x to its nearest centre among q."""
    x = np.asarray(x, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    return float(np.min((x[:, None] - q[None, :]) ** 2, axis=1).sum())


def optimal4_sse(x):
    """Minimum SSE over all partitions of x into at most four clusters.

    Brute force over every placement of three cuts in the sorted sequence for
    n <= 24; an O(4 n^2) dynamic program over prefix sums otherwise.
    """
    x = np.sort(np.asarray(x, dtype=np.float64))
    n = x.shape[0]
    if n == 0:
        return 0.0

    def seg(i, j):  # SSE of x[i:j]
        if j <= i:
            return 0.0
        s = x[i:j]
        return float(((s - s.mean()) ** 2).sum())

    if n <= 24:
        best = np.inf
        for c1, c2, c3 in itertools.combinations_with_replacement(range(n + 1), 3):
            v = seg(0, c1) + seg(c1, c2) + seg(c2, c3) + seg(c3, n)
            best = min(best, v)
        return best
    p1 = np.concatenate([[0.0], np.cumsum(x)])
    p2 = np.concatenate([[0.0], np.cumsum(x * x)])

    def cost(i, j):
        m = j - i
        if m <= 0:
            return 0.0
        s = p1[j] - p1[i]
        return max(p2[j] - p2[i] - s * s / m, 0.0)

    dp = np.array([cost(0, j) for j in range(n + 1)])
    for _ in range(3):
        nd = np.empty_like(dp)
        for j in range(n + 1):
            nd[j] = min(dp[i] + cost(i, j) for i in range(j + 1))
        dp = nd
    return float(dp[n])


# ---------------------------------------------------------------------------
# Incoherence pre-rotation (Sec. 5: the "+H" variant rotates the weights with a
# randomised Hadamard transform before the decomposition; the Kronecker form covers
# widths that are not powers of two).
# ---------------------------------------------------------------------------
def hadamard_matrix(m: int) -> np.ndarray:
    """Sylvester's Hadamard matrix of order m = 2^a (entries +-1): H_1 = [1],
    H_2k = [[H_k, H_k], [H_k, -H_k]]."""
    if m < 1 or m & (m - 1):
        raise ValueError("order must be a power of two")
    h = np.ones((1, 1))
    while h.shape[0] < m:
        h = np.block([[h, h], [h, -h]])
    return h


def _split_pow2(n: int) -> tuple[int, int]:
    """n = 2^a * b with b odd -> (2^a, b)."""
    p2 = n & -n
    return p2, n // p2


@functools.lru_cache(maxsize=2)
def rotation_matrix(n: int, seed: int) -> np.ndarray:
    """R = (H_{2^a} / sqrt(2^a) kron C_b) diag(s) for n = 2^a b, b odd (orthogonal)."""
    p2, b = _split_pow2(n)
    hb = hadamard_matrix(p2) / np.sqrt(p2)
    cb = dct2_matrix(b) if b > 1 else np.ones((1, 1))
    r = np.kron(hb, cb) * sign_mask(n, seed).astype(np.float64)[None, :]
    r.setflags(write=False)
    return r


def rotate(x: np.ndarray, seed: int, inverse: bool = False) -> np.ndarray:
    """Row-wise R x (or R^T x with inverse) for a batch of rows x (B, n)."""
    x = np.asarray(x, dtype=np.float64)
    r = rotation_matrix(x.shape[1], seed)
    return x @ r if inverse else x @ r.T


# ---------------------------------------------------------------------------
# Step schedules of the greedy over Q_N u P Q_N (Sec. 4.2; App. B, Alg. 1).
# ---------------------------------------------------------------------------
SCHEDULES = ("alternating", "reverse", "adaptive", "original")


def decompose_schedule(w, eps, nsteps, schedule, *, tol=0.0, replay_signs=None, replay_choices=None,
                       tau=None, choice_band=0.0):
    """Greedy decomposition x = u + P vhat + r with ``nsteps`` atomic steps in the given schedule.

    alternating  blocks (u, u, vhat, vhat): Alg. 2 (equals ``decompose`` for nsteps = 4k)
    reverse      blocks (vhat, vhat, u, u): the reverse order named in Sec. 4.2
    adaptive     every step takes the u-half when ||rho||_1 > ||P rho||_1, else the vhat-half,
                 step size ||.||_1 / N (greedy selection over the whole dictionary)
    original     Alg. 1 (App. B): the same choice, the step the orthogonal projection of the
                 current vector onto its sign vector s (coefficient <x, s> / <s, s>); a row stops
                 (takes no further steps) once ||rho||_2 < tol.
    A u-step on rho: Delta = c sign(rho), u += Delta, rho -= Delta.  A vhat-step on x = P rho:
    Delta = c sign(x), vhat += Delta, rho -= P Delta.

    Replay, as in ``decompose``: ``replay_signs`` (B, nsteps, n) and ``tau`` (B,) settle sign
    decisions on entries with |x_i| <= tau while c >= tau; ``replay_choices`` (B, nsteps) int8
    (0 u, 1 vhat, -1 stopped) settles the adaptive choice when | ||rho||_1 - ||P rho||_1 | <=
    choice_band (||rho||_1 + ||P rho||_1), and the stopping test of ``original`` when
    | ||rho||_2 - tol | <= choice_band tol; a given decision outside its band that differs from the
    oracle's is counted in ``choice_outside``.
    Trace: ``choice`` (B, nsteps) int8 (0 u, 1 vhat, -1 stopped), ``c``, ``l1u`` = ||rho||_1,
    ``l1v`` = ||P rho||_1 before the step, ``r2`` = ||rho||_2^2 after it, ``signs``.
    """
    if schedule not in SCHEDULES:
        raise ValueError(f"schedule must be one of {SCHEDULES}")
    w = np.array(w, dtype=np.float64, copy=True)
    if w.ndim == 1:
        w = w[None, :]
    bsz, n = w.shape
    rho = w.copy()
    u = np.zeros_like(w)
    vhat = np.zeros_like(w)
    tr = {"choice": np.zeros((bsz, nsteps), dtype=np.int8), "c": np.zeros((bsz, nsteps)),
          "l1u": np.zeros((bsz, nsteps)), "l1v": np.zeros((bsz, nsteps)), "r2": np.zeros((bsz, nsteps)),
          "signs": np.zeros((bsz, nsteps, n), dtype=np.int8)}
    outside = np.zeros(bsz, dtype=np.int64)
    choice_outside = np.zeros(bsz, dtype=np.int64)
    if replay_signs is not None:
        tau = np.broadcast_to(np.asarray(tau, dtype=np.float64), (bsz,))
    for step in range(nsteps):
        xu = rho
        xv = apply_p(rho, eps)
        l1u = np.abs(xu).sum(axis=1)
        l1v = np.abs(xv).sum(axis=1)
        pos = step % 4
        if schedule == "alternating":
            take_v = np.full(bsz, pos >= 2)
        elif schedule == "reverse":
            take_v = np.full(bsz, pos < 2)
        else:
            take_v = ~(l1u > l1v)
        active = np.ones(bsz, dtype=bool)
        if schedule == "original" and tol > 0:
            norm = np.sqrt((rho * rho).sum(axis=1))
            active = norm >= tol
            if replay_choices is not None:
                stopped = np.asarray(replay_choices)[:, step] == -1
                band = np.abs(norm - tol) <= choice_band * tol
                choice_outside += (~band & (stopped == active)).astype(np.int64)
                active = np.where(band, ~stopped, active)
        if schedule in ("adaptive", "original") and replay_choices is not None:
            given = np.asarray(replay_choices)[:, step]
            band = active & (given >= 0) & (np.abs(l1u - l1v) <= choice_band * (l1u + l1v))
            choice_outside += (active & (given >= 0) & ~band & ((given == 1) != take_v)).astype(np.int64)
            take_v = np.where(band, given == 1, take_v)
        x = np.where(take_v[:, None], xv, xu)
        l1 = np.where(take_v, l1v, l1u)
        s = np.sign(x)
        c0 = l1 / n
        if replay_signs is not None:
            gs = replay_signs[:, step, :].astype(np.float64)
            live = ((c0 >= tau) & (tau >= 0))[:, None]
            band = live & (np.abs(x) <= tau[:, None])
            outside += (live & ~band & (gs != s)).sum(axis=1)
            s = np.where(band, gs, s)
        if schedule == "original":
            ss = (s * s).sum(axis=1)
            c = np.where(ss > 0, (x * s).sum(axis=1) / np.maximum(ss, 1), 0.0)
        else:
            c = c0
        c = np.where(active, c, 0.0)
        d = s * c[:, None]
        du = np.where(take_v[:, None], 0.0, d)
        dv = np.where(take_v[:, None], d, 0.0)
        u += du
        vhat += dv
        rho = rho - du - apply_p(dv, eps)
        tr["choice"][:, step] = np.where(active, take_v.astype(np.int8), -1)
        tr["c"][:, step] = c
        tr["l1u"][:, step] = l1u
        tr["l1v"][:, step] = l1v
        tr["r2"][:, step] = (rho * rho).sum(axis=1)
        tr["signs"][:, step] = s.astype(np.int8)
    return {"u": u, "vhat": vhat, "r": rho, "trace": tr, "replay_outside": outside,
            "choice_outside": choice_outside}


# ---------------------------------------------------------------------------
# Error-compensated quantisation (Sec. 5, Fig. 1; eq. optq_update of App. on the stress tests).
# ---------------------------------------------------------------------------
def synthetic_hessian(d: int, nsamples: int, seed: int, outlier_cols: int = 0, outlier_scale: float = 1.0):
    """H = X^T X / nsamples for seeded Gaussian activations X (nsamples, d); `outlier_cols`
    channels scaled by `outlier_scale` (the activation outliers that make H ill-conditioned)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((nsamples, d))
    if outlier_cols:
        x[:, rng.choice(d, outlier_cols, replace=False)] *= outlier_scale
    return x.T @ x / nsamples


def damped_hessian(h, damp=0.01):
    """H + lambda I with lambda = damp * mean(diag H): the 1 % damping of the compensation (a
    remark in Sec. 5 sets damp = 0.01)."""
    h = np.asarray(h, dtype=np.float64)
    return h + damp * np.mean(np.diag(h)) * np.eye(h.shape[0])


def compensation_factor(h, damp=0.01):
    """Upper-triangular U with U^T U = (H + lambda I)^-1: the Cholesky factor of the damped
    inverse Hessian whose rows carry a quantised chunk's error forward (eq. optq_update)."""
    hinv = np.linalg.inv(damped_hessian(h, damp))
    return np.linalg.cholesky(hinv).T


def _quantise_columns(cols, eps, k, lloyd_iters):
    """Quantise each row of `cols` (one column vector of W per row) and dequantise it."""
    cu, cv, centers, _ = quantize(cols, eps, k, lloyd_iters)
    n = cols.shape[1]
    return reconstruct(unpack2bit(cu, n), unpack2bit(cv, n), centers, eps), (cu, cv, centers)


def optq_kashin(w, h, eps, k, chunk, damp=0.01, lloyd_iters=0, quantiser=None):
    """W (d_out, d_in), H (d_in, d_in): quantise the columns of W (vectors of length d_out) in
    chunks of `chunk` columns; after each chunk c, with Delta = W_c - Q_c and U the upper Cholesky
    factor of (H + damp mean(diag H) I)^-1, the remaining columns become W_r - Delta U_cc^-1 U_cr.
    Returns (Q, W_final, codes) with codes = per chunk (codes_u, codes_v, centers).

    ``quantiser(cols, c0)`` (optional) replaces the column quantiser: it maps the chunk starting
    at column c0 (one column vector per row of ``cols``) to (dequantised rows, codes); a test uses
    it to replay another implementation's near-tie decisions chunk by chunk."""
    w = np.array(w, dtype=np.float64, copy=True)
    d_in = w.shape[1]
    u = compensation_factor(h, damp)  # hinv = u^T u, u upper triangular
    q = np.zeros_like(w)
    codes = []
    for c0 in range(0, d_in, chunk):
        c1 = min(c0 + chunk, d_in)
        if quantiser is None:
            qc, cd = _quantise_columns(w[:, c0:c1].T, eps, k, lloyd_iters)
        else:
            qc, cd = quantiser(w[:, c0:c1].T, c0)
        q[:, c0:c1] = qc.T
        codes.append(cd)
        delta = w[:, c0:c1] - q[:, c0:c1]
        if c1 < d_in:
            w[:, c1:] -= delta @ np.linalg.solve(u[c0:c1, c0:c1], u[c0:c1, c1:])
    return q, w, codes


def optq_reference(w, h, chunk, quantiser, damp=0.01):
    """The same compensation written with the inverse Hessian of the remaining columns, downdated
    after each chunk (Schur complement): W_r -= Delta [G_cc]^-1 G_cr, G <- G_rr - G_rc [G_cc]^-1 G_cr,
    G = H^-1 at the start.  `quantiser(cols)` maps the chunk's column vectors (rows) to their
    dequantised values.  With chunk = 1 the update is eq. optq_update with [H^-1]_ii."""
    w = np.array(w, dtype=np.float64, copy=True)
    d_in = w.shape[1]
    g = np.linalg.inv(damped_hessian(h, damp))
    q = np.zeros_like(w)
    for c0 in range(0, d_in, chunk):
        c1 = min(c0 + chunk, d_in)
        b = c1 - c0
        q[:, c0:c1] = quantiser(w[:, c0:c1].T).T
        delta = w[:, c0:c1] - q[:, c0:c1]
        gcc, gcr, grr = g[:b, :b], g[:b, b:], g[b:, b:]
        if c1 < d_in:
            w[:, c1:] -= delta @ np.linalg.solve(gcc, gcr)
            g = grr - gcr.T @ np.linalg.solve(gcc, gcr)
    return q, w

