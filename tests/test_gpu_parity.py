"""GPU parity of the HIP path (called through the C ABI) against the float64 oracle.

See parity_util for the tolerances and the tie-band replay.  Inputs are seeded and
synthetic (paper_2609_11687_amd.synth); every size spans several FFT tiles, and the
odd row counts exercise the unpaired last row.
"""
import sys

import numpy as np
import pytest
import torch

import oracle.kashin_ref as ref
from paper_2609_11687_amd import kashin as K
from paper_2609_11687_amd import synth
import parity_util as pu

pytestmark = pytest.mark.gpu

ALL_N = [64, 96, 172, 256, 512, 768, 1024, 2048, 3072, 4096, 5120, 6144, 8192, 10000, 11008, 13824, 14336, 16384]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    K.lib()


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _rows(rng, m, n, dist="gauss", std=0.02):
    if dist == "gauss":
        w = rng.standard_normal((m, n)) * std
    elif dist == "t4":
        w = rng.standard_t(4, (m, n)) * (std / np.sqrt(2.0))
    elif dist == "outlier":
        w = rng.standard_normal((m, n)) * std
        w[:, rng.choice(n, max(1, n // 1000), replace=False)] *= 20.0
    else:
        raise ValueError(dist)
    return w.astype(np.float32)


# ----------------------------------------------------------------------------- operator P
@pytest.mark.parametrize("n", ALL_N)
def test_apply_p_matches_oracle(n):
    rng = np.random.default_rng(n)
    seed = 1000 + n
    eps = ref.sign_mask(n, seed)
    plan = K.kashin_plan(n, seed, 1)
    np.testing.assert_array_equal(K.kashin_plan_signs(plan), eps)
    x = rng.standard_normal((5, n)).astype(np.float32)
    xd = pu.to_dev(x)
    y = torch.empty_like(xd)
    K.kashin_apply_p(plan, xd, y)
    y2 = torch.empty_like(xd)
    K.kashin_apply_p(plan, y, y2)
    torch.cuda.synchronize()
    yref = ref.apply_p(x.astype(np.float64), eps)
    scale = max(np.abs(x).max(), np.abs(yref).max())
    err = np.abs(y.cpu().numpy() - yref).max() / scale
    _say(f"apply_p N={n}: max err / scale = {err:.2e}")
    assert err <= 5e-6
    # involution: P(P x) = x
    assert np.abs(y2.cpu().numpy() - x).max() / scale <= 1e-5


@pytest.mark.parametrize("n", [4096, 11008])
def test_apply_p_bench_batch(n):
    """y = P x on the benchmark's activation batch (16384 fp32 rows per width, one launch as
    bench.py --op apply_p times it): sampled rows against the oracle."""
    g = torch.Generator(device="cuda").manual_seed(n)
    x = torch.randn((16384, n), dtype=torch.float32, device="cuda", generator=g)
    y = torch.empty_like(x)
    plan = K.kashin_plan(n, 0, 1)
    K.kashin_apply_p(plan, x, y)
    torch.cuda.synchronize()
    rows = [0, 1, 2, 4097, 8191, 12345, 16382, 16383]
    xs = x[rows].cpu().numpy().astype(np.float64)
    yref = ref.apply_p(xs, ref.sign_mask(n, 0))
    err = np.abs(y[rows].cpu().numpy() - yref).max() / max(np.abs(xs).max(), np.abs(yref).max())
    _say(f"apply_p batch N={n}: max err / scale = {err:.2e}")
    assert err <= 5e-6


def test_reconstruct_layer_sampled_rows():
    """w_hat = u_q + P v_q for the llama7b layer's down_proj and q_proj (full matrices, one
    launch each as bench.py --op reconstruct times them), sampled rows against the oracle's
    reconstruction from the same codes and centres."""
    wl = synth.WORKLOADS["llama7b"]
    names = [s.name for s in wl.matrices]
    for name in ("q_proj", "down_proj"):
        idx = names.index(name)
        spec = wl.matrices[idx]
        seed = synth.sign_seed(wl, 0, idx)
        plan = K.kashin_plan(spec.n, seed, wl.iters)
        wd = pu.to_dev(synth.make_matrix(wl, 0, idx)).to(torch.float16)
        cu, cv, ce = K.quantize_alloc(plan, wd, 0)
        wh = torch.empty((spec.rows, spec.n), dtype=torch.float32, device="cuda")
        K.kashin_reconstruct(plan, cu, cv, ce, wh)
        torch.cuda.synchronize()
        rows = [0, 1, spec.rows // 2, spec.rows - 1]
        cu_s = pu.unpack(cu.cpu().numpy()[rows], spec.n)
        cv_s = pu.unpack(cv.cpu().numpy()[rows], spec.n)
        ce_s = ce.cpu().numpy()[rows].astype(np.float64)
        wref = ref.reconstruct(cu_s, cv_s, ce_s, ref.sign_mask(spec.n, seed))
        err = np.abs(wh.cpu().numpy()[rows] - wref).max() / np.abs(wref).max()
        _say(f"reconstruct {name} N={spec.n}: max err / max|w_hat| = {err:.2e}")
        assert err <= 1e-5


# ----------------------------------------------------------------------------- Alg. 2 on small batches
CASES = [(64, 3, "gauss"), (96, 20, "gauss"), (172, 20, "t4"), (256, 1, "gauss"), (512, 20, "gauss"),
         (768, 30, "outlier"), (1024, 8, "t4"), (2048, 20, "gauss"), (3072, 30, "outlier"), (4096, 30, "t4"),
         (5120, 20, "gauss"), (6144, 12, "t4"), (8192, 30, "t4"), (10000, 20, "gauss"), (11008, 4, "outlier"),
         (11008, 30, "t4"), (13824, 8, "outlier"), (14336, 8, "t4"), (16384, 30, "gauss")]


@pytest.mark.parametrize("n,k,dist", CASES)
def test_decompose_replay_parity(n, k, dist):
    """kashin_decompose (u, vhat, r, block-0 step sizes, factor bounds) against the oracle replayed
    on the GPU's near-tie signs, on every transform shape (odd row count: an unpaired last row)."""
    rng = np.random.default_rng(7 * n + k)
    m = 7 if n * k <= 100000 else 3
    w = _rows(rng, m, n, dist)
    seed = 17 + n
    eps = ref.sign_mask(n, seed)
    plan = K.kashin_plan(n, seed, k)
    wd = pu.to_dev(w)
    u, vh, r, cs, bd = K.decompose_alloc(plan, wd, want_r=True)
    signs, c_tr, u_tr, v_tr = pu.gpu_trace(plan, wd, list(range(m)), k)
    u, vh, r, cs, bd = (t.cpu().numpy() for t in (u, vh, r, cs, bd))
    # the trace run is the same computation as decompose: identical bits
    np.testing.assert_array_equal(u_tr, u.astype(np.float64))
    np.testing.assert_array_equal(v_tr, vh.astype(np.float64))
    w64 = w.astype(np.float64)
    res = pu.replay_parity(w64, eps, k, signs, u.astype(np.float64), vh.astype(np.float64))
    _say(f"decompose N={n} k={k} {dist}: du={res['du'].max():.2e} dv={res['dv'].max():.2e} "
         f"rec={res['rec'].max():.2e} in-band flips={res['in_band_flips'].sum()} direct ok={res['direct_frac_ok']}")
    pu.assert_replay_ok(res, f"N={n}")
    rep = res["rep"]
    winf = res["winf"]
    # step magnitudes: block-0 c's and the whole c trace agree with the replayed oracle
    np.testing.assert_allclose(cs, rep["cstep"], rtol=1e-5, atol=1e-7 * winf.max())
    # factor bounds: max norms of the returned factors, coefficient sums of App. F
    np.testing.assert_allclose(bd[:, 0], np.abs(u).max(axis=1), rtol=1e-6)
    np.testing.assert_allclose(bd[:, 1], np.abs(vh).max(axis=1), rtol=1e-6)
    np.testing.assert_allclose(bd[:, 2], rep["csum"][:, 0], rtol=1e-5)
    np.testing.assert_allclose(bd[:, 3], rep["csum"][:, 1], rtol=1e-5)
    assert np.all(bd[:, 0] <= bd[:, 2] * (1 + 1e-5)) and np.all(bd[:, 1] <= bd[:, 3] * (1 + 1e-5))
    # residual output: w = u + P vhat + r, and r itself against the oracle's residual
    rec = np.abs(w64 - u - ref.apply_p(vh.astype(np.float64), eps) - r).max(axis=1) / winf
    assert rec.max() <= 1e-5
    assert (np.abs(r - rep["r"]).max(axis=1) / winf).max() <= 1e-5


# ----------------------------------------------------------------------------- clustering and packing
@pytest.mark.parametrize("n,k,lloyd", [(512, 20, 0), (768, 30, 0), (512, 20, 2), (4096, 30, 0), (96, 5, 3),
                                         (3072, 20, 1), (11008, 8, 2)])
def test_quantize_codes_and_reconstruct(n, k, lloyd):
    rng = np.random.default_rng(n + 100 * lloyd)
    m = 9
    w = _rows(rng, m, n, "t4")
    seed = 5 + n
    eps = ref.sign_mask(n, seed)
    plan = K.kashin_plan(n, seed, k)
    wd = pu.to_dev(w)
    cu, cv, ce = K.quantize_alloc(plan, wd, lloyd)
    u, vh, _, cs, _ = K.decompose_alloc(plan, wd)
    nb = (n + 3) // 4
    cu2 = torch.empty((m, nb), dtype=torch.uint8, device="cuda")
    cv2 = torch.empty_like(cu2)
    ce2 = torch.empty((m, 2, 4), dtype=torch.float32, device="cuda")
    K.kashin_cluster2bit(plan, u, vh, cs, lloyd, cu2, cv2, ce2)
    what = torch.empty((m, n), dtype=torch.float32, device="cuda")
    K.kashin_reconstruct(plan, cu, cv, ce, what)
    torch.cuda.synchronize()
    cu, cv, ce = cu.cpu().numpy(), cv.cpu().numpy(), ce.cpu().numpy().astype(np.float64)
    u64, v64, cs64 = (t.cpu().numpy().astype(np.float64) for t in (u, vh, cs))
    winf = np.abs(w).max(axis=1).astype(np.float64)
    codes_u, codes_v = pu.unpack(cu, n), pu.unpack(cv, n)
    # (1) fused clustering == standalone clustering of the same factors
    if lloyd == 0:
        np.testing.assert_array_equal(cu, cu2.cpu().numpy())
        np.testing.assert_array_equal(cv, cv2.cpu().numpy())
        np.testing.assert_array_equal(ce, ce2.cpu().numpy())
    # (2) centres: closed form from the oracle's c's then Lloyd, and codes, vs the oracle
    qu = ref.closed_form_centers(cs64[:, 0], cs64[:, 1])
    qv = ref.closed_form_centers(cs64[:, 2], cs64[:, 3])
    if lloyd:
        qu = ref.lloyd(u64, qu, lloyd)
        qv = ref.lloyd(v64, qv, lloyd)
    np.testing.assert_allclose(ce[:, 0], qu, rtol=0, atol=1e-5 * winf.max())
    np.testing.assert_allclose(ce[:, 1], qv, rtol=0, atol=1e-5 * winf.max())
    mu, tot = pu.code_mismatches(codes_u, u64, qu, winf, "u")
    mv, _ = pu.code_mismatches(codes_v, v64, qv, winf, "vhat")
    _say(f"quantize N={n} lloyd={lloyd}: code mismatches u={mu} v={mv} of {tot}")
    assert mu + mv <= max(1, int(1e-4 * 2 * tot))
    # (3) reconstruction from codes == the oracle's dequantisation of the same codes
    wref = ref.reconstruct(codes_u, codes_v, ce, eps)
    err = np.abs(what.cpu().numpy() - wref).max(axis=1) / winf
    assert err.max() <= 1e-5
    # packing layout: bytes decode to in-range codes and the padded tail is zero
    if n % 4:
        assert not (cu[:, -1] >> (2 * (n % 4))).any()


def test_codes_against_oracle_decomposition():
    """Codes of the fused path versus codes the oracle derives from its own (replayed)
    decomposition, closed-form centres, decisions in fp32."""
    n, k, m = 1024, 20, 11
    rng = np.random.default_rng(99)
    w = _rows(rng, m, n, "t4")
    eps = ref.sign_mask(n, 21)
    plan = K.kashin_plan(n, 21, k)
    wd = pu.to_dev(w)
    cu, cv, ce = K.quantize_alloc(plan, wd, 0)
    signs, _, u_tr, v_tr = pu.gpu_trace(plan, wd, list(range(m)), k)
    w64 = w.astype(np.float64)
    res = pu.replay_parity(w64, eps, k, signs, u_tr, v_tr)
    pu.assert_replay_ok(res)
    rep = res["rep"]
    qu = ref.closed_form_centers(rep["cstep"][:, 0], rep["cstep"][:, 1])
    qv = ref.closed_form_centers(rep["cstep"][:, 2], rep["cstep"][:, 3])
    pu.assert_centres_close(ce.cpu().numpy()[:, 0], qu)
    pu.assert_centres_close(ce.cpu().numpy()[:, 1], qv)
    mu, tot = pu.code_mismatches(pu.unpack(cu.cpu().numpy(), n), rep["u"], qu, res["winf"], "u")
    mv, _ = pu.code_mismatches(pu.unpack(cv.cpu().numpy(), n), rep["vhat"], qv, res["winf"], "vhat")
    assert mu + mv <= max(1, int(2e-4 * tot))


GROUPED = [  # (n, k, dtype, lloyd, rows per matrix, rotation seed): sizes on every transform shape,
    # empty and single-row matrices, more matrices than one launch takes, the fused rotation
    (96, 5, torch.float32, 0, [5, 0, 1, 12], None),
    (256, 10, torch.float32, 0, [3, 1, 2, 5, 4, 1, 7, 2, 3, 6, 1, 2, 9, 4, 1, 3, 2, 5, 8], None),
    (512, 20, torch.float32, 2, [7, 4, 0], None),
    (768, 30, torch.float32, 0, [9, 1, 6], None),
    (3072, 30, torch.float32, 0, [4, 7], None),
    (4096, 30, torch.float16, 0, [6, 0, 3, 10], None),
    (11008, 30, torch.float16, 0, [3, 2, 0, 5], None),
    (16384, 8, torch.float32, 0, [2, 3], None),
    (5120, 10, torch.float16, 0, [3, 4], None),
    (10000, 6, torch.float32, 1, [3, 0, 2], None),
    (13824, 4, torch.float16, 0, [2, 3], None),
    (14336, 4, torch.float32, 2, [3, 2], None),
    (768, 30, torch.float32, 0, [5, 4], 99),
    (6144, 10, torch.float16, 0, [3, 2], 99),
    (4096, 30, torch.float16, 0, [6, 3, 1], 99),
    (11008, 30, torch.float16, 0, [3, 4], 99),
]


@pytest.mark.parametrize("n,k,dtype,lloyd,rows,rot", GROUPED)
def test_grouped_quantize_equals_per_matrix(n, k, dtype, lloyd, rows, rot):
    """kashin_quantize_grouped: every matrix (its own plan and sign mask, one of them strided) gives
    the codes and centres of kashin_quantize (kashin_quantize_rotated with a rotation seed) on it
    alone, bit for bit; without rotation one matrix is checked against the oracle's decomposition
    (tie-band replay) as well."""
    _say(f"grouped quantize N={n} k={k} rows={rows} rotation={rot}")
    rng = np.random.default_rng(n + 7)
    items, ref_out, host = [], [], []
    for i, m in enumerate(rows):
        w = _rows(rng, m, n, "t4" if i % 2 else "gauss")
        plan = K.kashin_plan(n, 1000 + 13 * i, k)
        if i == 1 and m > 0:  # strided rows: ld = n + 8
            big = torch.zeros((m, n + 8), dtype=dtype, device="cuda")
            big[:, :n] = pu.to_dev(w, dtype)
            wd = big[:, :n]
        else:
            wd = pu.to_dev(w, dtype)
        nb = (n + 3) // 4
        cu = torch.full((m, nb), 0xAB, dtype=torch.uint8, device="cuda")
        cv = torch.full_like(cu, 0xCD)
        ce = torch.full((m, 2, 4), float("nan"), dtype=torch.float32, device="cuda")
        items.append((plan, wd, cu, cv, ce))
        if rot is None:
            ref_out.append(K.quantize_alloc(plan, wd, lloyd))
        else:
            r1 = (torch.empty_like(cu), torch.empty_like(cv), torch.empty_like(ce))
            K.kashin_quantize_rotated(plan, rot, wd, lloyd, *r1)
            ref_out.append(r1)
        host.append(w)
    K.kashin_quantize_grouped(items, lloyd, rot_seed=rot)
    torch.cuda.synchronize()
    for i, ((plan, wd, cu, cv, ce), (cu1, cv1, ce1)) in enumerate(zip(items, ref_out)):
        assert torch.equal(cu, cu1), f"matrix {i}: codes_u"
        assert torch.equal(cv, cv1), f"matrix {i}: codes_v"
        assert torch.equal(ce.view(torch.int32), ce1.view(torch.int32)), f"matrix {i}: centres"
    if rot is not None:
        return  # the rotated path alone is checked against the oracle by the rotation tests
    # the largest matrix against the oracle
    i = int(np.argmax(rows))
    plan, wd, cu, cv, ce = items[i]
    m = rows[i]
    eps = ref.sign_mask(n, 1000 + 13 * i)
    signs, _, u_tr, v_tr = pu.gpu_trace(plan, wd, list(range(m)), k)
    w64 = wd.float().cpu().numpy().astype(np.float64)
    res = pu.replay_parity(w64, eps, k, signs, u_tr, v_tr)
    pu.assert_replay_ok(res)
    if lloyd == 0:
        rep = res["rep"]
        qu = ref.closed_form_centers(rep["cstep"][:, 0], rep["cstep"][:, 1])
        qv = ref.closed_form_centers(rep["cstep"][:, 2], rep["cstep"][:, 3])
        pu.assert_centres_close(ce.cpu().numpy()[:, 0], qu)
        pu.assert_centres_close(ce.cpu().numpy()[:, 1], qv)
        mu, tot = pu.code_mismatches(pu.unpack(cu.cpu().numpy(), n), rep["u"], qu, res["winf"], "u")
        mv, _ = pu.code_mismatches(pu.unpack(cv.cpu().numpy(), n), rep["vhat"], qv, res["winf"], "vhat")
        assert mu + mv <= max(1, int(2e-4 * tot))


RECON_GROUPED = [(n, rows) for n, _, _, _, rows, rot in GROUPED if rot is None] + [
    (256, [3000, 5, 2000]),  # more row pairs than the persistent grid: several pairs per workgroup
    (4096, [700, 1, 1300]),
]


@pytest.mark.parametrize("n,rows", RECON_GROUPED)
def test_grouped_reconstruct_equals_per_matrix(n, rows):
    """kashin_reconstruct_grouped: every matrix (its own plan, codes and centres; one output
    strided) gives kashin_reconstruct's w_hat on it alone, bit for bit, including matrices with
    fewer row pairs than workgroups and ones whose workgroups take several pairs each."""
    _say(f"grouped reconstruct N={n} rows={rows}")
    rng = np.random.default_rng(n + 11)
    items, ref_out = [], []
    for i, m in enumerate(rows):
        plan = K.kashin_plan(n, 2000 + 7 * i, 30)
        w = pu.to_dev(_rows(rng, m, n, "t4" if i % 2 else "gauss"), torch.float32)
        cu, cv, ce = K.quantize_alloc(plan, w, 0)
        if i == 1 and m > 0:  # strided output rows: ld = n + 8
            big = torch.full((m, n + 8), float("nan"), dtype=torch.float32, device="cuda")
            wh = big[:, :n]
        else:
            wh = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
        r1 = torch.empty((m, n), dtype=torch.float32, device="cuda")
        K.kashin_reconstruct(plan, cu, cv, ce, r1)
        items.append((plan, cu, cv, ce, wh))
        ref_out.append(r1)
    K.kashin_reconstruct_grouped(items)
    torch.cuda.synchronize()
    for i, ((plan, cu, cv, ce, wh), r1) in enumerate(zip(items, ref_out)):
        assert torch.equal(wh.contiguous().view(torch.int32), r1.view(torch.int32)), f"matrix {i}: w_hat"
    if len(rows) > 1 and rows[1] > 0:  # the padding of the strided output is left alone
        assert torch.isnan(items[1][4].as_strided((rows[1], 8), (n + 8, 1), n)).all()


# ----------------------------------------------------------------------------- properties and edges
def test_deterministic_and_pow2_homogeneous():
    n, k, m = 512, 20, 6
    rng = np.random.default_rng(3)
    w = _rows(rng, m, n)
    plan = K.kashin_plan(n, 9, k)
    out1 = K.decompose_alloc(plan, pu.to_dev(w))
    out2 = K.decompose_alloc(plan, pu.to_dev(w))
    out4 = K.decompose_alloc(plan, pu.to_dev(w * 4.0))
    outn = K.decompose_alloc(plan, pu.to_dev(-w))
    torch.cuda.synchronize()
    for i in (0, 1):
        a = out1[i].cpu().numpy()
        np.testing.assert_array_equal(a, out2[i].cpu().numpy())
        np.testing.assert_array_equal(4.0 * a, out4[i].cpu().numpy())
        np.testing.assert_array_equal(-a, outn[i].cpu().numpy())


def test_fp16_input_equals_fp32_of_same_values():
    n, k, m = 4096, 10, 4
    rng = np.random.default_rng(4)
    w16 = _rows(rng, m, n).astype(np.float16)
    plan = K.kashin_plan(n, 2, k)
    a = K.decompose_alloc(plan, pu.to_dev(w16))
    b = K.decompose_alloc(plan, pu.to_dev(w16.astype(np.float32)))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(a[0].cpu().numpy(), b[0].cpu().numpy())
    np.testing.assert_array_equal(a[1].cpu().numpy(), b[1].cpu().numpy())


@pytest.mark.parametrize("n", [512, 4096, 11008])
def test_bf16_input_equals_fp32_of_same_values(n):
    """bfloat16 rows (widened exactly) give what fp32 rows of the same values give, bit for bit, in
    every entry point that reads weight rows: decompose (u, vhat, r), quantize (plain, grouped,
    rotated), trace, the schedules and the rotation (odd row count: an unpaired last row)."""
    k, m = 6, 5
    rng = np.random.default_rng(n + 8)
    wb = torch.from_numpy(_rows(rng, m, n, "t4")).to(torch.bfloat16).cuda()
    wf = wb.float()
    plan = K.kashin_plan(n, 21, k)
    outs = []
    for w in (wb, wf):
        r = {}
        u, vh = torch.empty((m, n), device="cuda"), torch.empty((m, n), device="cuda")
        rr = torch.empty_like(u)
        K.kashin_decompose(plan, w, u, vh, rr)
        r["decompose"] = (u, vh, rr)
        r["quantize"] = K.quantize_alloc(plan, w, 1)
        nb = (n + 3) // 4
        g = (torch.empty((m, nb), dtype=torch.uint8, device="cuda"), torch.empty((m, nb), dtype=torch.uint8,
             device="cuda"), torch.empty((m, 2, 4), device="cuda"))
        K.kashin_quantize_grouped([(plan, w) + g], 0)
        r["grouped"] = g
        rows = torch.arange(m, dtype=torch.int64, device="cuda")
        sg = torch.empty((m, 4 * k, n), dtype=torch.int8, device="cuda")
        ct = torch.empty((m, 4 * k), device="cuda")
        ut, vt = torch.empty_like(u), torch.empty_like(u)
        K.kashin_trace(plan, w, rows, sg, ct, ut, vt)
        r["trace"] = (sg, ct, ut, vt)
        us, vs = torch.empty_like(u), torch.empty_like(u)
        K.kashin_decompose_schedule(plan, "adaptive", w, us, vs)
        r["schedule"] = (us, vs)
        y = torch.empty_like(u)
        K.kashin_rotate(n, 5, w, y)
        r["rotate"] = (y,)
        cr = (torch.empty((m, nb), dtype=torch.uint8, device="cuda"), torch.empty((m, nb), dtype=torch.uint8,
              device="cuda"), torch.empty((m, 2, 4), device="cuda"))
        K.kashin_quantize_rotated(plan, 5, w, 0, *cr)
        r["rotated"] = cr
        torch.cuda.synchronize()
        outs.append({key: [t.cpu().numpy() for t in v] for key, v in r.items()})
    assert outs[0].keys() == outs[1].keys()
    for key in outs[0]:
        for a_, b_ in zip(outs[0][key], outs[1][key]):
            np.testing.assert_array_equal(a_, b_, err_msg=key)


# one length per transform shape: generic (256), lane-paired resident (512, 4096), odd inner pass
# (768), palindromic resident (1024, 16384), split radix-43 (11008)
@pytest.mark.parametrize("n", [256, 512, 768, 1024, 3072, 4096, 11008, 16384])
def test_empty_single_and_strided_rows(n):
    """m = 0 is a no-op; a strided 3-row call (ldw = n + 40) satisfies w = u + P vhat + r with
    its own residual and matches float64 under the tie-band replay (k = 5 leaves a residual
    above fp32 resolution, where a sign decision near a tie may go either way, Alg. 2); its
    unpaired last row equals a 1-row call bit for bit."""
    k = 5
    plan = K.kashin_plan(n, 1, k)
    rng = np.random.default_rng(5)
    # m = 0: no-op
    w0 = torch.empty((0, n), dtype=torch.float32, device="cuda")
    K.kashin_decompose(plan, w0, w0, w0)
    # m = 1 (unpaired row) and a strided view (ldw = n + 40)
    wide = _rows(rng, 3, n + 40)
    wv = pu.to_dev(wide)[:, 5:5 + n]
    assert wv.stride(0) == n + 40
    u, vh, r, _, _ = K.decompose_alloc(plan, wv, want_r=True)
    u1, vh1, _, _, _ = K.decompose_alloc(plan, pu.to_dev(wide[2:3, 5:5 + n]))
    signs, _, u_tr, v_tr = pu.gpu_trace(plan, wv, [0, 1, 2], k)
    torch.cuda.synchronize()
    eps = ref.sign_mask(n, 1)
    w64 = wide[:, 5:5 + n].astype(np.float64)
    u, vh, r = (t.cpu().numpy().astype(np.float64) for t in (u, vh, r))
    own = np.abs(w64 - u - ref.apply_p(vh, eps) - r).max() / np.abs(w64).max()
    res = pu.replay_parity(w64, eps, k, signs, u_tr, v_tr)
    _say(f"empty/single/strided N={n}: own identity {own:.2e}, replay du={res['du'].max():.2e} "
         f"in-band flips={res['in_band_flips'].sum()}")
    assert own <= 1e-5
    pu.assert_replay_ok(res, f"N={n}")
    np.testing.assert_array_equal(u_tr, u)  # the trace run is the same computation
    # the unpaired last row of the 3-row call equals the 1-row call bit for bit
    np.testing.assert_array_equal(u[2], u1.cpu().numpy()[0].astype(np.float64))


def test_unaligned_and_strided_p_map_io():
    """apply_p from/to buffers that are not 16-byte aligned and reconstruct into strided rows
    take the scalar staging path; results equal the aligned, contiguous calls bit for bit."""
    n, m = 512, 5
    plan = K.kashin_plan(n, 3, 6)
    rng = np.random.default_rng(8)
    x = pu.to_dev(_rows(rng, m, n))
    y = torch.empty_like(x)
    K.kashin_apply_p(plan, x, y)
    xbuf = torch.zeros(m * n + 1, dtype=torch.float32, device="cuda")
    ybuf = torch.zeros(m * n + 1, dtype=torch.float32, device="cuda")
    xbuf[1:].copy_(x.reshape(-1))
    xo, yo = xbuf[1:].view(m, n), ybuf[1:].view(m, n)
    K.kashin_apply_p(plan, xo, yo)
    cu, cv, ce = K.quantize_alloc(plan, x, 0)
    wh = torch.empty((m, n), dtype=torch.float32, device="cuda")
    K.kashin_reconstruct(plan, cu, cv, ce, wh)
    wide = torch.zeros((m, n + 3), dtype=torch.float32, device="cuda")
    K.kashin_reconstruct(plan, cu, cv, ce, wide[:, :n])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(yo.cpu().numpy(), y.cpu().numpy())
    np.testing.assert_array_equal(wide[:, :n].cpu().numpy(), wh.cpu().numpy())
    assert (wide[:, n:] == 0).all()


def test_nonfinite_row_is_isolated():
    n, k, m = 512, 10, 4
    rng = np.random.default_rng(6)
    w = _rows(rng, m, n)
    w_bad = w.copy()
    w_bad[2, 17] = np.nan
    w_bad[1, 3] = np.inf
    plan = K.kashin_plan(n, 4, k)
    u, vh, _, cs, _ = K.decompose_alloc(plan, pu.to_dev(w_bad))
    cu, cv, ce = K.quantize_alloc(plan, pu.to_dev(w_bad))
    torch.cuda.synchronize()
    u, vh, ce = u.cpu().numpy(), vh.cpu().numpy(), ce.cpu().numpy()
    assert np.isnan(u[2]).all() and np.isnan(vh[2]).all() and np.isnan(u[1]).all()
    assert np.isnan(ce[1]).all() and np.isnan(ce[2]).all()
    assert not cu.cpu().numpy()[1:3].any()
    # partners (rows 0 and 3) are finite and still decompose their own rows
    eps = ref.sign_mask(n, 4)
    for row in (0, 3):
        assert np.isfinite(u[row]).all()
        rec = np.abs(w[row] - u[row] - ref.apply_p(vh[row:row + 1].astype(np.float64), eps)[0]).max()
        assert rec <= 1e-5 * np.abs(w[row]).max()


def test_lloyd_keeps_emptied_centres_fused():
    """Rows a s with s in {-1,1}^N and a = 2^-6 (every sum exact in fp32): one u-step takes the
    whole row (u = w, c1 = a, every later step 0), so the closed-form centres are [-a, -a, a, a],
    the codes are 0 and 2, and Lloyd passes leave clusters 1 and 3 (and three clusters of vhat = 0)
    empty.  The fused quantizer's codes and centres equal the oracle's exactly, for 1 and 2 passes
    (an emptied cluster keeps its centre: Sec. 3.1)."""
    n, k = 512, 3
    rng = np.random.default_rng(3)
    s = np.where(rng.random((5, n)) < 0.5, -1.0, 1.0)
    w = (2.0 ** -6 * s).astype(np.float32)
    w[4] = 2.0 ** -6  # a constant row: a single occupied cluster
    seed = 77
    eps = ref.sign_mask(n, seed)
    plan = K.kashin_plan(n, seed, k)
    wd = pu.to_dev(w)
    d = ref.decompose(w.astype(np.float64), eps, k)
    for lloyd in (1, 2):
        cu, cv, ce = K.quantize_alloc(plan, wd, lloyd)
        torch.cuda.synchronize()
        ru, rv, rc = ref.cluster2bit(d["u"], d["vhat"], d["cstep"], lloyd)
        np.testing.assert_array_equal(ce.cpu().numpy(), rc.astype(np.float32))
        np.testing.assert_array_equal(pu.unpack(cu.cpu().numpy(), n), ru)
        np.testing.assert_array_equal(pu.unpack(cv.cpu().numpy(), n), rv)
        np.testing.assert_array_equal(rc[0, 0], [-2.0 ** -6, -2.0 ** -6, 2.0 ** -6, 2.0 ** -6])


def test_lloyd_keeps_emptied_centres_standalone():
    """kashin_cluster2bit on hand-built factors (values exact in fp32): u rows with values -2.5, 0.5
    and 4 around the closed-form centres [-3, -1, 1, 3] (c1 = 2, c2 = 1) leave cluster 1 empty,
    vhat rows with -3.5, -0.75 and 2.5 leave cluster 2 empty; one and two Lloyd passes give the
    oracle's centres and codes exactly (the emptied centre is kept)."""
    n, m = 64, 3
    rng = np.random.default_rng(4)
    u = np.concatenate([np.full(16, -2.5), np.full(16, 0.5), np.full(32, 4.0)])
    v = np.concatenate([np.full(20, -3.5), np.full(20, -0.75), np.full(24, 2.5)])
    uu = np.stack([rng.permutation(u) for _ in range(m)]).astype(np.float32)
    vv = np.stack([rng.permutation(v) for _ in range(m)]).astype(np.float32)
    cs = np.tile(np.array([2.0, 1.0, 2.0, 1.0], np.float32), (m, 1))
    plan = K.kashin_plan(n, 1, 1)
    for lloyd in (1, 2):
        cu = torch.empty((m, n // 4), dtype=torch.uint8, device="cuda")
        cv = torch.empty_like(cu)
        ce = torch.empty((m, 2, 4), dtype=torch.float32, device="cuda")
        K.kashin_cluster2bit(plan, pu.to_dev(uu), pu.to_dev(vv), pu.to_dev(cs), lloyd, cu, cv, ce)
        torch.cuda.synchronize()
        ru, rv, rc = ref.cluster2bit(uu, vv, cs, lloyd)
        np.testing.assert_array_equal(rc[0, 0], [-2.5, -1.0, 0.5, 4.0])
        np.testing.assert_array_equal(rc[0, 1], [-3.5, -0.75, 1.0, 2.5])
        np.testing.assert_array_equal(ce.cpu().numpy(), rc.astype(np.float32))
        np.testing.assert_array_equal(pu.unpack(cu.cpu().numpy(), n), ru)
        np.testing.assert_array_equal(pu.unpack(cv.cpu().numpy(), n), rv)


def test_subnormal_row():
    """A fp32 row whose entries are all subnormal (|w| < 2^-126): the row scale is clamped so it
    stays finite; factors and centres are finite and equal those of the same row scaled by 2^126
    (a normal row: the decomposition is homogeneous), divided back, to fp32 resolution of the
    normal row.  Each row is decomposed alone (no partner)."""
    n, k = 512, 10
    rng = np.random.default_rng(8)
    tiny = (rng.standard_normal(n) * 1e-40).astype(np.float32)
    assert np.abs(tiny).max() < 2.0 ** -126 and np.count_nonzero(tiny) > n // 2
    big = (tiny.astype(np.float64) * 2.0 ** 126).astype(np.float32)
    np.testing.assert_array_equal(big.astype(np.float64) * 2.0 ** -126, tiny.astype(np.float64))
    plan = K.kashin_plan(n, 3, k)
    outs = []
    for row in (tiny, big):
        wd = pu.to_dev(np.stack([row]))
        u, vh, _, cs, _ = K.decompose_alloc(plan, wd)
        cu, cv, ce = K.quantize_alloc(plan, wd, 0)
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy().astype(np.float64) for t in (u, vh, cs, ce)])
    for t in outs[0]:
        assert np.isfinite(t).all()
    scale = np.abs(big).max()
    for a, b in zip(outs[0], outs[1]):
        err = np.abs(a * 2.0 ** 126 - b).max() / scale
        assert err <= 1e-5, err
    # and the normal row against the oracle
    eps = ref.sign_mask(n, 3)
    signs, _, u_tr, v_tr = pu.gpu_trace(plan, pu.to_dev(np.stack([big])), [0], k)
    pu.assert_replay_ok(pu.replay_parity(np.stack([big]).astype(np.float64), eps, k, signs, u_tr, v_tr), "normal")


def test_row_pairing_permutation():
    """A row's last bits depend on the row it shares a complex FFT with.  Quantising the rows in a
    permuted order (every row gets another partner) changes nothing beyond that: both orders pass
    the replay parity against the oracle row by row, and their codes differ only where the
    parity rule allows (near a decision boundary, at most 1e-4 of the codes)."""
    n, k, m = 1024, 20, 12
    rng = np.random.default_rng(31)
    w = _rows(rng, m, n, "t4")
    perm = rng.permutation(m)
    seed = 55
    eps = ref.sign_mask(n, seed)
    plan = K.kashin_plan(n, seed, k)
    w64 = w.astype(np.float64)
    codes = []
    for order in (np.arange(m), perm):
        wd = pu.to_dev(w[order])
        cu, cv, ce = K.quantize_alloc(plan, wd, 0)
        signs, _, u_tr, v_tr = pu.gpu_trace(plan, wd, list(range(m)), k)
        res = pu.replay_parity(w64[order], eps, k, signs, u_tr, v_tr)
        pu.assert_replay_ok(res, "pairing")
        inv = np.argsort(order)
        codes.append((pu.unpack(cu.cpu().numpy(), n)[inv], pu.unpack(cv.cpu().numpy(), n)[inv],
                      ce.cpu().numpy()[inv]))
    diff = int((codes[0][0] != codes[1][0]).sum() + (codes[0][1] != codes[1][1]).sum())
    _say(f"pairing permutation: {diff} of {2 * m * n} codes differ")
    assert diff <= max(1, int(1e-4 * 2 * m * n))
    np.testing.assert_allclose(codes[0][2], codes[1][2], rtol=1e-5, atol=1e-7)


def test_rotation_rejected_for_other_odd_parts():
    """Plans whose length has an odd part other than 1, 3 or 43 take every entry point except the
    rotated ones, which return KASHIN_E_UNSUPPORTED_N before launching anything."""
    for n in (5120, 10000, 13824, 14336):
        plan = K.kashin_plan(n, 1, 2)
        wd = torch.zeros((2, n), dtype=torch.float32, device="cuda")
        cu, cv, ce = K.quantize_alloc(plan, wd, 0)
        for call in (lambda: K.kashin_quantize_rotated(plan, 5, wd, 0, cu, cv, ce),
                     lambda: K.kashin_reconstruct_rotated(plan, 5, cu, cv, ce, wd),
                     lambda: K.kashin_quantize_grouped([(plan, wd, cu, cv, ce)], 0, rot_seed=5)):
            with pytest.raises(K.KashinError) as e:
                call()
            assert e.value.status == K.KASHIN_E_UNSUPPORTED_N
        torch.cuda.synchronize()


def test_zero_and_cube_vertex_rows():
    """A zero row stays zero; a row a*s (s in {-1,1}^N) is all u after one step (T11)."""
    n, k = 512, 4
    s = np.where(np.arange(n) % 3 == 0, -1.0, 1.0).astype(np.float32)
    w = np.stack([np.zeros(n, np.float32), 0.75 * s, 0.25 * s, np.zeros(n, np.float32)])
    plan = K.kashin_plan(n, 8, k)
    u, vh, _, cs, _ = K.decompose_alloc(plan, pu.to_dev(w))
    torch.cuda.synchronize()
    u, vh, cs = u.cpu().numpy(), vh.cpu().numpy(), cs.cpu().numpy()
    assert not u[0].any() and not vh[0].any() and not u[3].any()
    np.testing.assert_allclose(u[1], w[1], atol=1e-6)
    assert np.abs(vh[1]).max() <= 1e-6
    np.testing.assert_allclose(cs[1], [0.75, 0, 0, 0], atol=1e-7)


# ----------------------------------------------------------------------------- full-size workloads, sampled rows
def _sample_rows(w, count, rng):
    """Row 0, the last row, the three rows of largest ||w||_inf, then random rows up to `count`."""
    m = w.shape[0]
    mx = np.abs(w.astype(np.float32)).max(axis=1)
    pick = {0, m - 1} | {int(i) for i in np.argsort(mx)[-3:]}
    while len(pick) < min(count, m):
        pick.add(int(rng.integers(0, m)))
    return sorted(pick)


WL_ROWS = {"gauss512": None, "opt125m": 8, "llama7b": 8, "pythia7b": 8}  # sampled rows per matrix (None: all)


def _load_matrix(wl, layer, idx):
    """(host rows, device rows, plan, (codes_u, codes_v, centres) buffers) of one matrix."""
    spec = wl.matrices[idx]
    w = synth.make_matrix(wl, layer, idx)
    plan = K.kashin_plan(spec.n, synth.sign_seed(wl, layer, idx), wl.iters)
    dt = torch.float16 if spec.dtype == "f16" else torch.float32
    wd = pu.to_dev(w).to(dt)
    nb = (spec.n + 3) // 4
    out = (torch.empty((spec.rows, nb), dtype=torch.uint8, device="cuda"),
           torch.empty((spec.rows, nb), dtype=torch.uint8, device="cuda"),
           torch.empty((spec.rows, 2, 4), dtype=torch.float32, device="cuda"))
    return w, wd, plan, out


def _check_matrix(key, wl, layer, idx, per_matrix, rng, loaded, lloyd=0):
    """Replay sampled rows (all rows if per_matrix is None) of matrix idx, already quantised in
    full in the benchmark's launch configuration, against the oracle: factors, reconstruction,
    centres (closed form from the replayed step sizes, then `lloyd` passes of the oracle's Lloyd on
    the replayed factors) and codes.  Returns (code mismatches, codes compared)."""
    spec = wl.matrices[idx]
    w, wd, plan, (cu, cv, ce) = loaded
    seed = synth.sign_seed(wl, layer, idx)
    rows = list(range(w.shape[0])) if per_matrix is None else _sample_rows(w, per_matrix, rng)
    signs, _, u_tr, v_tr = pu.gpu_trace(plan, wd, rows, wl.iters)
    eps = ref.sign_mask(spec.n, seed)
    w64 = w[rows].astype(np.float64)
    res = pu.replay_parity(w64, eps, wl.iters, signs, u_tr, v_tr, direct=spec.n < 11008)
    _say(f"{key}/L{layer}/{spec.name} N={spec.n} rows={len(rows)} lloyd={lloyd}: du={res['du'].max():.2e} "
         f"dv={res['dv'].max():.2e} rec={res['rec'].max():.2e} direct ok={res['direct_frac_ok']}")
    pu.assert_replay_ok(res, f"{key}/L{layer}/{spec.name}")
    rep = res["rep"]
    qu = ref.closed_form_centers(rep["cstep"][:, 0], rep["cstep"][:, 1])
    qv = ref.closed_form_centers(rep["cstep"][:, 2], rep["cstep"][:, 3])
    ce_s = ce.cpu().numpy()[rows].astype(np.float64)
    slack = [None, None]
    if lloyd:
        # Lloyd's means jump when a near-tie entry lands in the other cluster: the centres are
        # checked within the bound that near-ties allow, and codes near the shifted midpoints
        for f, (x, q0) in enumerate(((rep["u"], qu), (rep["vhat"], qv))):
            tol = pu.lloyd_tolerance(x, q0, lloyd, res["winf"])
            q = ref.lloyd(x, q0, lloyd)
            pu.assert_lloyd_centres_close(ce_s[:, f], q, tol)
            slack[f] = np.abs(ce_s[:, f] - q).max(axis=1)
            if f == 0:
                qu = q
            else:
                qv = q
        _say(f"  lloyd: near-tie centre bound {slack[0].max():.2e} / {slack[1].max():.2e}")
    else:
        pu.assert_centres_close(ce_s[:, 0], qu)
        pu.assert_centres_close(ce_s[:, 1], qv)
    codes_u = pu.unpack(cu.cpu().numpy()[rows], spec.n)
    codes_v = pu.unpack(cv.cpu().numpy()[rows], spec.n)
    mu, tot = pu.code_mismatches(codes_u, rep["u"], qu, res["winf"], "u", slack[0])
    mv, _ = pu.code_mismatches(codes_v, rep["vhat"], qv, res["winf"], "vhat", slack[1])
    # every row of the matrix got finite centres
    assert np.isfinite(ce.cpu().numpy()).all()
    if lloyd:
        # codes between the GPU's and the oracle's (shifted) Lloyd midpoints may flip: they are not
        # counted against the 1e-4 budget (each was checked to lie in that band above)
        band = pu.near_boundary_count(rep["u"], qu, res["winf"], slack[0]) + \
            pu.near_boundary_count(rep["vhat"], qv, res["winf"], slack[1])
        _say(f"  lloyd: {mu + mv} code mismatches, {band} entries in the shifted-midpoint band")
        return max(0, mu + mv - band), 2 * tot
    return mu + mv, 2 * tot


def _quantize_grouped(loaded, lloyd=0):
    """One kashin_quantize_grouped call per vector length (at most 16 matrices each), as the
    benchmark launches them."""
    by_n = {}
    for w, wd, plan, out in loaded:
        by_n.setdefault(plan.n, []).append((plan, wd) + out)
    for items in by_n.values():
        for c0 in range(0, len(items), 16):
            K.kashin_quantize_grouped(items[c0:c0 + 16], lloyd)
    torch.cuda.synchronize()


_WL_CACHE = {}


def _workload_quantised(key, lloyd=0):
    """Every matrix of the workload's first layer, quantised in full by the grouped launches the
    benchmark times; kept for the tests of one workload (one workload's buffers at a time)."""
    ck = (key, lloyd)
    if ck not in _WL_CACHE:
        _WL_CACHE.clear()
        torch.cuda.empty_cache()
        wl = synth.WORKLOADS[key]
        loaded = [_load_matrix(wl, 0, idx) for idx in range(len(wl.matrices))]
        _quantize_grouped(loaded, lloyd)
        _WL_CACHE[ck] = loaded
    return _WL_CACHE[ck]


WL_MATRICES = [(key, i) for key in WL_ROWS for i in range(len(synth.WORKLOADS[key].matrices))]


@pytest.mark.parametrize("key,idx", WL_MATRICES)
def test_workload_matrix_sampled_rows(key, idx):
    """Every matrix of every single-layer workload (each with its own sign mask), quantised in full
    by the grouped launches of the benchmark; row 0, the last row, the three largest-||w||_inf rows
    and random rows (8 per matrix; all rows of the 256-row matrix) replayed against the oracle."""
    wl = synth.WORKLOADS[key]
    loaded = _workload_quantised(key)
    mm, tot = _check_matrix(key, wl, 0, idx, WL_ROWS[key], np.random.default_rng(11 + idx), loaded[idx])
    _say(f"{key}/{wl.matrices[idx].name}: code mismatches {mm} of {tot}")
    assert mm <= max(1, int(1e-4 * tot))


@pytest.mark.parametrize("idx", [0, 4, 6])
def test_llama7b_layer_lloyd2(idx):
    """The llama7b layer quantised with two Lloyd passes (all seven matrices, grouped launches):
    sampled rows against the oracle's replayed decomposition followed by the oracle's Lloyd passes
    on the replayed factors (centres and codes)."""
    wl = synth.WORKLOADS["llama7b"]
    loaded = _workload_quantised("llama7b", lloyd=2)
    mm, tot = _check_matrix("llama7b", wl, 0, idx, 5, np.random.default_rng(40 + idx), loaded[idx], lloyd=2)
    _say(f"llama7b lloyd=2 {wl.matrices[idx].name}: code mismatches {mm} of {tot}")
    assert mm <= max(1, int(1e-4 * tot))


def test_stack_first_and_last_layer():
    """The 32-layer stack (Student-t(3), outlier columns x50, k = 40): q_proj and down_proj of
    the first and the last layer quantised in full, four sampled rows each replayed."""
    _WL_CACHE.clear()
    wl = synth.WORKLOADS["llama7b_stack"]
    rng = np.random.default_rng(12)
    names = [s.name for s in wl.matrices]
    total_m = total_codes = 0
    for layer in (0, wl.layers - 1):
        for name in ("q_proj", "down_proj"):
            loaded = _load_matrix(wl, layer, names.index(name))
            _quantize_grouped([loaded])
            mm, tot = _check_matrix("llama7b_stack", wl, layer, names.index(name), 4, rng, loaded)
            total_m += mm
            total_codes += tot
    _say(f"llama7b_stack: code mismatches {total_m} of {total_codes}")
    assert total_m <= max(1, int(1e-4 * total_codes))


# ----------------------------------------------------------------------------- incoherence rotation
ROT_N = [n for n in ALL_N if n // (n & -n) in (1, 3, 43)]  # the lengths the rotation takes


@pytest.mark.parametrize("n", ROT_N)
def test_rotate_matches_oracle(n):
    """y = R x and x = R^T y against the oracle's dense R, fp32 rows; fp16 input equals fp32
    input of the same values bit for bit; in place equals out of place bit for bit."""
    rng = np.random.default_rng(3 * n)
    seed = 77 + n
    m = 5
    x = _rows(rng, m, n, "outlier")
    xd = pu.to_dev(x)
    y = torch.empty_like(xd)
    K.kashin_rotate(n, seed, xd, y)
    back = torch.empty_like(xd)
    K.kashin_rotate(n, seed, y, back, inverse=True)
    yh = torch.empty_like(xd)
    xh = xd.half()
    K.kashin_rotate(n, seed, xh, yh)
    yf = torch.empty_like(xd)
    K.kashin_rotate(n, seed, xh.float(), yf)
    inplace = xd.clone()
    K.kashin_rotate(n, seed, inplace, inplace)
    torch.cuda.synchronize()
    yref = ref.rotate(x.astype(np.float64), seed)
    scale = max(np.abs(x).max(), np.abs(yref).max())
    err = np.abs(y.cpu().numpy() - yref).max() / scale
    inv_err = np.abs(back.cpu().numpy() - x).max() / scale
    _say(f"rotate N={n}: max err / scale = {err:.2e}, round trip {inv_err:.2e}")
    assert err <= 2e-6
    assert inv_err <= 4e-6
    yinv_ref = ref.rotate(x.astype(np.float64), seed, inverse=True)
    yinv = torch.empty_like(xd)
    K.kashin_rotate(n, seed, xd, yinv, inverse=True)
    torch.cuda.synchronize()
    assert np.abs(yinv.cpu().numpy() - yinv_ref).max() / scale <= 2e-6
    np.testing.assert_array_equal(yh.cpu().numpy(), yf.cpu().numpy())
    np.testing.assert_array_equal(inplace.cpu().numpy(), y.cpu().numpy())


def test_rotated_quantization_pipeline():
    """The +H composition on full llama7b matrices (q_proj, down_proj; fp16 rows): R w on the
    GPU, quantised, reconstructed and rotated back.  Sampled rows: R w against the oracle, and
    w_hat against the oracle's R^T (u_q + P v_q) from the same codes and centres."""
    wl = synth.WORKLOADS["llama7b"]
    names = [s.name for s in wl.matrices]
    rot_seed = 1234
    for name in ("q_proj", "down_proj"):
        idx = names.index(name)
        spec = wl.matrices[idx]
        seed = synth.sign_seed(wl, 0, idx)
        w = synth.make_matrix(wl, 0, idx)
        wd = pu.to_dev(w).to(torch.float16)
        wr = torch.empty((spec.rows, spec.n), dtype=torch.float32, device="cuda")
        K.kashin_rotate(spec.n, rot_seed, wd, wr)
        plan = K.kashin_plan(spec.n, seed, wl.iters)
        cu, cv, ce = K.quantize_alloc(plan, wr, 0)
        wh = torch.empty_like(wr)
        K.kashin_reconstruct(plan, cu, cv, ce, wh)
        K.kashin_rotate(spec.n, rot_seed, wh, wh, inverse=True)
        torch.cuda.synchronize()
        rows = [0, 3, spec.rows // 2, spec.rows - 1]
        w64 = w[rows].astype(np.float64)
        rref = ref.rotate(w64, rot_seed)
        rerr = np.abs(wr.cpu().numpy()[rows] - rref).max() / np.abs(rref).max()
        cu_s = pu.unpack(cu.cpu().numpy()[rows], spec.n)
        cv_s = pu.unpack(cv.cpu().numpy()[rows], spec.n)
        ce_s = ce.cpu().numpy()[rows].astype(np.float64)
        whref = ref.rotate(ref.reconstruct(cu_s, cv_s, ce_s, ref.sign_mask(spec.n, seed)), rot_seed, inverse=True)
        herr = np.abs(wh.cpu().numpy()[rows] - whref).max() / np.abs(whref).max()
        rel = np.linalg.norm(wh.cpu().numpy()[rows] - w64) / np.linalg.norm(w64)
        _say(f"+H {name} N={spec.n}: rotate err {rerr:.2e}, w_hat err {herr:.2e}, "
             f"relative reconstruction error {rel:.3f}")
        assert rerr <= 2e-6
        assert herr <= 1e-5
        del plan


# ----------------------------------------------------------------------------- step schedules
SCHED_CASES = [(n, s) for n in (512, 4096, 11008) for s in ("alternating", "reverse", "adaptive", "original")] + \
    [(768, "original"), (3072, "adaptive")] + [(10000, s) for s in ("alternating", "adaptive", "original")]


@pytest.mark.parametrize("n,schedule", SCHED_CASES)
def test_schedule_replay_parity(n, schedule):
    """kashin_decompose_schedule against the oracle's schedules: every row traced (signs, step
    sizes, choices, ||rho||^2), the oracle replayed on the GPU's near-tie signs and near-tie
    choices; decisions outside the bands must agree, factors within 1e-4 ||w||_inf, and
    w = u + P vhat + r.  The traced factors equal the untraced call bit for bit."""
    k = 5
    steps = 4 * k
    m = 5
    rng = np.random.default_rng(17 * n + len(schedule))
    w = _rows(rng, m, n, "t4")
    seed = 300 + n
    eps = ref.sign_mask(n, seed)
    plan = K.kashin_plan(n, seed, k)
    wd = pu.to_dev(w)
    tol = 0.05 * float(np.sqrt((w.astype(np.float64) ** 2).sum(axis=1)).min()) if schedule == "original" else 0.0
    u = torch.empty_like(wd)
    vh = torch.empty_like(wd)
    r = torch.empty_like(wd)
    K.kashin_decompose_schedule(plan, schedule, wd, u, vh, r, tol=tol)
    rows_t = torch.arange(m, dtype=torch.int64, device="cuda")
    sg = torch.empty((m, steps, n), dtype=torch.int8, device="cuda")
    cs = torch.empty((m, steps), dtype=torch.float32, device="cuda")
    ch = torch.empty((m, steps), dtype=torch.int8, device="cuda")
    r2 = torch.empty((m, steps), dtype=torch.float32, device="cuda")
    ut = torch.empty_like(wd)
    vt = torch.empty_like(wd)
    K.kashin_trace_schedule(plan, schedule, wd, rows_t, sg, cs, ch, r2, ut, vt, tol=tol)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ut.cpu().numpy(), u.cpu().numpy())
    np.testing.assert_array_equal(vt.cpu().numpy(), vh.cpu().numpy())
    w64 = w.astype(np.float64)
    winf = np.abs(w64).max(axis=1)
    rep = ref.decompose_schedule(w64, eps, steps, schedule, tol=tol, replay_signs=sg.cpu().numpy(),
                                 replay_choices=ch.cpu().numpy(), tau=pu.TAU_REL * winf, choice_band=1e-5)
    ug, vg, rg = (t.cpu().numpy().astype(np.float64) for t in (u, vh, r))
    du = (np.abs(ug - rep["u"]).max(axis=1) / winf).max()
    dv = (np.abs(vg - rep["vhat"]).max(axis=1) / winf).max()
    rec = (np.abs(w64 - ug - ref.apply_p(vg, eps) - rg).max(axis=1) / winf).max()
    gch = ch.cpu().numpy()
    _say(f"schedule {schedule} N={n}: du={du:.2e} dv={dv:.2e} rec={rec:.2e} vhat-steps "
         f"{(gch == 1).mean():.2f} stopped {(gch == -1).mean():.2f}")
    assert not rep["replay_outside"].any(), "sign decisions outside the tie band disagree"
    assert not rep["choice_outside"].any(), "step choices outside the tie band disagree"
    np.testing.assert_array_equal(gch, rep["trace"]["choice"])
    assert du <= pu.TOL_FACTOR and dv <= pu.TOL_FACTOR
    assert rec <= pu.TOL_RECON
    np.testing.assert_allclose(cs.cpu().numpy(), rep["trace"]["c"], rtol=1e-4, atol=1e-7 * winf.max())
    np.testing.assert_allclose(r2.cpu().numpy(), rep["trace"]["r2"], rtol=1e-3, atol=1e-10 * (winf.max() ** 2) * n)
    if schedule == "original":
        assert (gch == -1).any()  # the tolerance stopped some rows


@pytest.mark.parametrize("n", [172, 4096, 11008])
def test_schedule_outputs_unaligned(n):
    """The schedule kernel writes its outputs in row order through LDS as 16-byte stores where a
    row is 16-byte aligned and 4-byte stores where it is not: outputs placed one float off
    alignment equal the aligned ones bit for bit (odd row count: an unpaired last row)."""
    k, m = 3, 5
    rng = np.random.default_rng(n + 5)
    wd = pu.to_dev(_rows(rng, m, n, "t4"))
    plan = K.kashin_plan(n, 9, k)
    outs = []
    for off in (0, 1):
        flat = torch.full((3, m * n + 4), float("nan"), dtype=torch.float32, device="cuda")
        u, vh, r = (flat[j, off:off + m * n].view(m, n) for j in range(3))
        K.kashin_decompose_schedule(plan, "adaptive", wd, u, vh, r)
        torch.cuda.synchronize()
        assert not torch.isnan(flat[:, off:off + m * n]).any()
        assert torch.isnan(flat[:, :off]).all() and torch.isnan(flat[:, off + m * n:]).all()  # nothing outside
        outs.append([t.cpu().numpy().copy() for t in (u, vh, r)])
    for a_, b_ in zip(*outs):
        np.testing.assert_array_equal(a_, b_)


# ----------------------------------------------------------------------------- error compensation
def test_optq_pipeline_stepwise():
    """The chunked error-compensated pipeline, checked chunk by chunk on the GPU's own state:
    each chunk's codes against the oracle's decomposition of the same columns (replayed at
    near-ties), its dequantised columns against the oracle's reconstruction of the GPU codes, and
    the carried error against the oracle's U_cc^-1 U_cr applied to the GPU's Delta."""
    from paper_2609_11687_amd import optq

    d_out, d_in, chunk, k = 512, 192, 64, 20
    rng = np.random.default_rng(21)
    w = _rows(rng, d_in, d_out, "t4")  # W^T: one row per column of W
    h = ref.synthetic_hessian(d_in, 400, 9, outlier_cols=4, outlier_scale=10.0)
    seed = 41
    eps = ref.sign_mask(d_out, seed)
    plan = K.kashin_plan(d_out, seed, k)
    w_t = pu.to_dev(w)
    record = []
    cu, cv, ce, q_t = optq.optq_quantize(plan, w_t, pu.to_dev(h), chunk, record=record)
    torch.cuda.synchronize()
    u = ref.compensation_factor(h)  # the oracle's damping (0.01 mean diag H) and factor
    scale = np.abs(w).max()
    for snap in record:
        c0, c1 = snap["c0"], snap["c1"]
        wc = snap["w_chunk"].cpu().numpy().astype(np.float64)
        qc = q_t[c0:c1].cpu().numpy().astype(np.float64)
        # dequantised columns: the oracle's reconstruction of the GPU codes
        qref = ref.reconstruct(pu.unpack(cu[c0:c1].cpu().numpy(), d_out), pu.unpack(cv[c0:c1].cpu().numpy(), d_out),
                               ce[c0:c1].cpu().numpy().astype(np.float64), eps)
        assert np.abs(qc - qref).max() <= 1e-5 * np.abs(qref).max()
        # the decomposition of the chunk's columns, sampled rows replayed against the oracle
        rows = [0, (c1 - c0) // 2, c1 - c0 - 1]
        signs, _, u_tr, v_tr = pu.gpu_trace(plan, snap["w_chunk"], rows, k)
        res = pu.replay_parity(wc[rows], eps, k, signs, u_tr, v_tr)
        pu.assert_replay_ok(res, f"optq chunk {c0}")
        if c0 > 0:
            np.testing.assert_array_equal(wc, wc_rest[:c1 - c0])  # the chunk starts from the carried state
        # the carried error
        if c1 < d_in:
            before = wc_rest if c0 > 0 else w.astype(np.float64)
            before = before[c1 - c0:] if c0 > 0 else before[c1:]
            m = np.linalg.solve(u[c0:c1, c0:c1], u[c0:c1, c1:])
            expect = before - m.T @ (wc - qc)
            got = snap["w_rest_after"].cpu().numpy().astype(np.float64)
            err = np.abs(got - expect).max() / scale
            _say(f"optq chunk {c0}:{c1}: carried-error mismatch {err:.2e}, du={res['du'].max():.2e}")
            assert err <= 1e-5
            wc_rest = got
    del plan


@pytest.mark.parametrize("d,outliers", [(1, 0), (96, 3), (512, 4), (4096, 8)])
def test_optq_factor_matches_oracle(d, outliers):
    """kashin_optq_factor (rocSOLVER Cholesky of the exchange-flipped damped Hessian and its triangular
    inverse, float64) against the oracle's factor of the inverse: U upper with U^T U = (H + lambda
    I)^-1, lambda = 0.01 mean(diag H), and V = U^-1."""
    from paper_2609_11687_amd import optq

    h = ref.synthetic_hessian(d, 2 * d + 8, d, outlier_cols=outliers, outlier_scale=20.0).astype(np.float32)
    u, v = optq.compensation_factor(pu.to_dev(h))
    torch.cuda.synchronize()
    u_ref = ref.compensation_factor(h.astype(np.float64))
    ug, vg = u.cpu().numpy(), v.cpu().numpy()
    err_u = np.abs(ug - u_ref).max() / np.abs(u_ref).max()
    err_v = np.abs(vg @ ug - np.eye(d)).max()
    _say(f"optq factor d={d}: max |U - U_ref| / max |U_ref| = {err_u:.2e}, max |V U - I| = {err_v:.2e}")
    assert err_u <= 1e-9
    assert err_v <= 1e-9
    assert np.all(np.tril(ug, -1) == 0) and np.all(np.diag(ug) > 0)


def _replaying_quantiser(plan, eps, k, record, codes_u, codes_v, n):
    """Column quantiser for ref.optq_kashin that follows the GPU run chunk by chunk: the oracle
    decomposes its own columns in float64, taking the GPU's sign only on entries within the tie
    band (the GPU's record of the same chunk, traced again), and takes the GPU's code only where its
    own decision lies within the boundary band; everything else is the oracle's."""
    by_c0 = {snap["c0"]: snap for snap in record}

    def quantiser(cols, c0):
        snap = by_c0[c0]
        nr = cols.shape[0]
        signs, _, _, _ = pu.gpu_trace(plan, snap["w_chunk"], list(range(nr)), k)
        winf = np.abs(cols).max(axis=1)
        d = ref.decompose(cols, eps, k, replay_signs=signs, tau=pu.TAU_REL * winf)
        assert not d["replay_outside"].any(), f"chunk {c0}: a sign decision outside the tie band differs"
        cu, cv, ce = ref.cluster2bit(d["u"], d["vhat"], d["cstep"], 0, decide_dtype=np.float32)
        gu = pu.unpack(codes_u[c0:c0 + nr].cpu().numpy(), n)
        gv = pu.unpack(codes_v[c0:c0 + nr].cpu().numpy(), n)
        for mine, gpu, x, q in ((cu, gu, d["u"], ce[:, 0]), (cv, gv, d["vhat"], ce[:, 1])):
            mism = mine != gpu
            if mism.any():
                dist = pu.boundary_distance(x, q) / winf[:, None]
                assert dist[mism].max() <= pu.TOL_CODE_BOUNDARY, f"chunk {c0}: a code differs away from a boundary"
                mine[mism] = gpu[mism]
        return ref.reconstruct(cu, cv, ce, eps), (ref.pack2bit(cu), ref.pack2bit(cv), ce)

    return quantiser


@pytest.mark.parametrize("lloyd,exact", [(0, False), (2, False), (2, True)])
def test_optq_single_chunk_is_plain_quantisation(lloyd, exact):
    """With one chunk covering every column nothing is carried: kashin_optq_quantize must give
    kashin_quantize's codes and centres (Lloyd passes included) and kashin_reconstruct's rows bit
    for bit, and leave w_t as it was (the exact form carries inside the chunk, so only its first
    column is plain quantisation and the rest differ)."""
    from paper_2609_11687_amd import optq

    d_in, n = 64, 512
    rng = np.random.default_rng(5 + lloyd)
    w = _rows(rng, d_in, n, "t4")
    h = ref.synthetic_hessian(d_in, 200, 3, outlier_cols=2, outlier_scale=5.0).astype(np.float32)
    plan = K.kashin_plan(n, 77, 12)
    w_t = pu.to_dev(w)
    cu, cv, ce, q_t = optq.optq_quantize(plan, w_t, pu.to_dev(h), 128, lloyd_iters=lloyd, exact=exact)
    # the exact form quantises its first column alone (no partner row in its complex FFT)
    ref_rows = 1 if exact else d_in
    rcu, rcv, rce = K.quantize_alloc(plan, pu.to_dev(w[:ref_rows]), lloyd)
    rq = torch.empty((ref_rows, n), dtype=torch.float32, device="cuda")
    K.kashin_reconstruct(plan, rcu, rcv, rce, rq)
    torch.cuda.synchronize()
    for got, want in ((cu, rcu), (cv, rcv), (ce, rce), (q_t, rq)):
        np.testing.assert_array_equal(got[:ref_rows].cpu().numpy(), want.cpu().numpy())
    if exact:
        assert not np.array_equal(w_t.cpu().numpy()[1:], w[1:])  # later columns were compensated
    else:
        np.testing.assert_array_equal(w_t.cpu().numpy(), w)


@pytest.mark.parametrize("chunk,exact", [(32, False), (32, True), (1, False)])
def test_optq_pipeline_end_to_end(chunk, exact):
    """The whole compensated pipeline against ref.optq_kashin: the final dequantised Q and the
    compensated W.  The chunk form at chunk 32 against the oracle's chunk form at 32; the exact form
    (columns one at a time inside chunks of 32, lazy trailing update) and chunk 1 against the
    oracle's per-column form (eq. optq_update column by column).  The oracle follows the GPU only at
    near-ties (see _replaying_quantiser)."""
    from paper_2609_11687_amd import optq

    d_out, d_in, k = 512, 96, 20
    rng = np.random.default_rng(23)
    w = _rows(rng, d_in, d_out, "t4")  # W^T
    h = ref.synthetic_hessian(d_in, 300, 10, outlier_cols=3, outlier_scale=8.0)
    seed = 43
    eps = ref.sign_mask(d_out, seed)
    plan = K.kashin_plan(d_out, seed, k)
    w_t = pu.to_dev(w)
    record = []
    cu, cv, ce, q_t = optq.optq_quantize(plan, w_t, pu.to_dev(h), chunk, record=record, exact=exact)
    torch.cuda.synchronize()
    oracle_chunk = 1 if (exact or chunk == 1) else chunk
    q_ref, w_ref, _ = ref.optq_kashin(w.T.astype(np.float64), h, eps, k, oracle_chunk,
                                      quantiser=_replaying_quantiser(plan, eps, k, record, cu, cv, d_out))
    scale = np.abs(w).max()
    dq = np.abs(q_t.cpu().numpy().astype(np.float64) - q_ref.T).max() / scale
    dw = np.abs(w_t.cpu().numpy().astype(np.float64) - w_ref.T).max() / scale
    _say(f"optq end to end chunk={chunk} exact={exact}: max |Q - Q_ref| = {dq:.2e}, max |W - W_ref| = {dw:.2e} "
         f"(of max |W|)")
    assert dq <= 1e-4 and dw <= 1e-4


@pytest.mark.parametrize("n", [172, 512, 768, 4096, 11008])
def test_fused_rotation_equals_separate_passes(n):
    """kashin_quantize_rotated (rotation fused into the load) gives the codes and centres of
    kashin_rotate followed by kashin_quantize, bit for bit, for fp16 and fp32 rows (odd row count:
    an unpaired last row); kashin_reconstruct_rotated equals kashin_reconstruct followed by the
    inverse rotation bit for bit."""
    rng = np.random.default_rng(5 * n)
    m, k, rot_seed = 5, 8, 99 + n
    plan = K.kashin_plan(n, 7 + n, k)
    for dt in (torch.float32, torch.float16):
        wd = pu.to_dev(_rows(rng, m, n, "outlier")).to(dt)
        wr = torch.empty((m, n), dtype=torch.float32, device="cuda")
        K.kashin_rotate(n, rot_seed, wd, wr)
        cu, cv, ce = K.quantize_alloc(plan, wr, 0)
        fu, fv, fc = torch.empty_like(cu), torch.empty_like(cv), torch.empty_like(ce)
        K.kashin_quantize_rotated(plan, rot_seed, wd, 0, fu, fv, fc)
        wh = torch.empty((m, n), dtype=torch.float32, device="cuda")
        K.kashin_reconstruct(plan, cu, cv, ce, wh)
        K.kashin_rotate(n, rot_seed, wh, wh, inverse=True)
        fh = torch.empty_like(wh)
        K.kashin_reconstruct_rotated(plan, rot_seed, cu, cv, ce, fh)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(fu.cpu().numpy(), cu.cpu().numpy())
        np.testing.assert_array_equal(fv.cpu().numpy(), cv.cpu().numpy())
        np.testing.assert_array_equal(fc.cpu().numpy(), ce.cpu().numpy())
        np.testing.assert_array_equal(fh.cpu().numpy(), wh.cpu().numpy())
    _say(f"fused rotation N={n}: equal to the separate passes")
