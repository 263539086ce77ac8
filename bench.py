#!/usr/bin/env python3
"""Throughput of the Kashin-DCT hot path on one MI355X.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload llama7b] [--lloyd 0] [--op quantize]

--op quantize (default): one step = kashin_quantize_grouped (decompose with Alg. 2 + four-peak
  2-bit clustering + packing) over every matrix of the workload (default: one Llama-2-7B-shaped
  decoder layer, fp16-stored, 30 blocks, closed-form centres), one launch per vector length and 16
  matrices (--per-matrix: one kashin_quantize launch per matrix), inputs already resident in HBM.
--op apply_p: one step = y = P x (kashin_apply_p) over --act-rows fp32 activation rows for each
  input width N of the workload (the inference-side product of App. C).
--op reconstruct: one step = w_hat = u_q + P v_q from the codes and centres of every matrix of
  the workload (quantized once, untimed), one kashin_reconstruct_grouped launch per vector length
  and 16 matrices (--per-matrix: one kashin_reconstruct launch per matrix).
--op rotate: one step = the incoherence pre-rotation R w (kashin_rotate) of every matrix of the
  workload, fp16 rows in, fp32 rows out.
--op quantize_h: one step = the "+H" pipeline, R w formed in the load, then quantised
  (kashin_quantize_grouped with a rotation seed; --per-matrix: kashin_quantize_rotated per matrix).
--op schedule: one step = kashin_decompose_schedule (--schedule alternating | reverse | adaptive |
  original) over every matrix of the workload, 4k atomic steps, factors and residual written.
--op optq: one step = the chunked error-compensated pipeline (paper_2609_11687_amd.optq) on one
  matrix of the workload (--matrix, default q_proj): its columns quantised in chunks of --chunk
  with the error carried through a synthetic Hessian (seeded activations with outlier channels).
--op fig2: the convergence comparison of Fig. 2: --fig2-rows vectors x of length N = 10^4 drawn
  from N(0, I), --fig2-steps greedy updates with Alg. 2's alternating schedule and with Alg. 1
  (kashin_decompose_schedule, "original"); one step = both decompositions.  Reports the residual
  ||x - u - P vhat||_2 / ||x||_2 after selected updates (mean over the vectors and for vector 0),
  and how much of each factor sits at four peaks.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time
from dataclasses import dataclass
from typing import Callable

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "weight vectors decomposed/s (N=4096, fixed iters); % of HBM / FP32 VALU roofline"
METRIC_APPLY_P = "activation rows transformed/s (y = P x, fp32); % of HBM roofline"
METRIC_RECON = "weight rows reconstructed/s (w_hat = u_q + P v_q from 2+2-bit codes, fp32 out); % of HBM roofline"
METRIC_ROTATE = "weight rows rotated/s (R w, fp16 in, fp32 out); % of HBM roofline"
METRIC_QUANT_H = "weight vectors rotated + decomposed + quantised/s (+H pipeline, N=4096, fixed iters)"
METRIC_SCHED = "weight vectors decomposed/s with the {} step schedule (4k steps, both residual domains kept)"
METRIC_OPTQ = "weight columns quantised/s with error compensation (chunks of {}, synthetic Hessian)"
ROT_SEED = 1234  # seed of the rotation's sign vector
PEAK_FP32_TFLOPS = 157.3   # MI355X published FP32 vector peak (256 CU x 2.4 GHz x 256 flop/clk)
PEAK_HBM_GBPS = 8000.0     # MI355X published HBM3E bandwidth
PMAP_GRID = 2048           # workgroups of a P-only launch (the library's cap; each walks several pairs)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def transform_flops(n: int) -> float:
    """Counted flops of one length-n DCT-II or DCT-III: 2.5 n log2 n."""
    return 2.5 * n * math.log2(n)


def counted_flops_per_vector(n: int, k: int) -> float:
    """Algorithmic count: 4k - 2 transforms (two P per block, the last one not needed for the
    factors), each 2.5 N log2 N flops."""
    return (4 * k - 2) * transform_flops(n)


def hbm_bytes_per_vector(n: int, in_bytes: int) -> int:
    """Algorithmic traffic: read the row once, write 2 x N/4 bytes of codes and 32 B of centres."""
    return n * in_bytes + 2 * ((n + 3) // 4) + 32


@dataclass
class Launch:
    n: int
    rows: int
    flops: float          # counted flops of the launch
    nbytes: float         # algorithmic HBM bytes of the launch
    run: Callable         # run(stream)
    kind: str = "quantize"  # which kernel the launch runs: quantize, pmap or rotate
    wgs: int = 0          # workgroups of the launch's one kernel dispatch (0: one per row pair)

    def workgroups(self) -> int:
        return self.wgs or (self.rows + 1) // 2


def measured_traffic(op: str, workload: str, kernel: str, launches) -> float | None:
    """HBM bytes per launch of the dominant kernel from the committed counter summary of this
    op and workload (profiles/<kernel>__<op>_<workload>.txt, line TRAFFIC_JSON), averaged over
    `launches` = [(n, workgroups)], or None when that summary was not taken on the current
    kernel sources."""
    from paper_2609_11687_amd.build import source_digest

    path = os.path.join(ROOT, "profiles", f"{kernel.split('[')[0]}__{op}_{workload}.txt")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        for line in fh:
            if line.startswith("TRAFFIC_JSON "):
                rec = json.loads(line[len("TRAFFIC_JSON "):])
                keys = [f"{kernel}|{n}/{wg}" for n, wg in launches]
                if rec.get("digest") == source_digest() and all(k in rec["bytes"] for k in keys):
                    return sum(rec["bytes"][k] for k in keys) / len(keys)
    return None


def _blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info

        return max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return os.cpu_count() or 1


def cpu_baseline(wl, rows: int, loaded=None):
    """The float64 oracle on a bounded sample of the workload: the first `rows` rows of the first
    matrix, and for every other vector length the first rows of its first matrix in proportion to
    the oracle's cost (8 N^2 k flops per vector), timed separately (the dense explicit-cosine
    matrix is built before timing).  `value` is the rate at the first matrix's length; `per_n` has
    every length's rate and `extrapolated_step_s` the time the oracle would take for one whole step
    at those rates (labelled as extrapolated: it is not measured).  With `loaded` (the
    benchmarked matrices: (plan, rows, codes_u, codes_v, centres) per matrix, first layer) the GPU's
    codes of the sampled rows are compared with the oracle's (plain float64 decisions, no replay),
    and a few rows per length are replayed (see _parity_sample)."""
    import numpy as np

    import oracle.kashin_ref as ref
    from paper_2609_11687_amd import synth

    first = {}
    for idx, spec in enumerate(wl.matrices):
        first.setdefault(spec.n, idx)
    n0 = wl.matrices[0].n
    per_n, agree = {}, {}
    total = 0.0
    for n, idx in first.items():
        spec = wl.matrices[idx]
        nr = max(8, int(rows * (n0 / n) ** 2)) if n != n0 else rows
        nr = min(nr, spec.rows)
        w = synth.make_matrix(wl, 0, idx, rows=slice(0, nr)).astype(np.float64)
        eps = ref.sign_mask(n, synth.sign_seed(wl, 0, idx))
        ref.dct2_matrix(n)
        t0 = time.perf_counter()
        cu, cv, ce, _ = ref.quantize(w, eps, wl.iters, 0)
        dt = time.perf_counter() - t0
        per_n[str(n)] = {"vectors_per_s": nr / dt, "rows": nr, "seconds": dt, "matrix": spec.name}
        total += dt
        if loaded is not None:
            _, _, gu, gv, _ = loaded[idx]
            same = (ref.unpack2bit(gu[:nr].cpu().numpy(), n) == ref.unpack2bit(cu, n)).sum() + \
                (ref.unpack2bit(gv[:nr].cpu().numpy(), n) == ref.unpack2bit(cv, n)).sum()
            agree[str(n)] = float(same) / (2 * nr * n)
    counts = {}
    for spec in wl.matrices:
        counts[spec.n] = counts.get(spec.n, 0) + spec.rows * wl.layers
    extrap = sum(counts[n] / per_n[str(n)]["vectors_per_s"] for n in counts)
    s0 = per_n[str(n0)]
    out = {
        "value": s0["vectors_per_s"],
        "unit": "vectors/s",
        "cores": int(_blas_threads()),
        "kind": "oracle",
        "sample": "float64 literal Alg. 2 with a dense P (4 GEMMs per block) + closed-form clustering + "
                  "packing, k=%d; " % wl.iters + "; ".join(
                      f"{d['rows']} rows of {d['matrix']} (N={n}) in {d['seconds']:.1f} s" for n, d in per_n.items())
                  + "; cosine-matrix construction excluded",
        "per_n": per_n,
        "extrapolated_step_s": extrap,
        "extrapolated_note": "time the oracle would take for one whole step at the sampled per-length rates "
                             "(extrapolated, not measured)",
    }
    if agree:
        out["code_agreement_direct"] = agree
    if loaded is not None:
        out["parity"] = _parity_sample(wl, loaded)
    return out


def _parity_sample(wl, loaded, rows_per_matrix: int = 4):
    """Replay parity of the benchmarked launches on sampled rows: for the first matrix of each
    vector length, `rows_per_matrix` rows (row 0, the largest ||w||_inf row, the last row, ...) are
    traced on the GPU and the oracle is replayed on the GPU's near-tie signs; reports the largest
    factor and reconstruction errors (fractions of ||w||_inf), the sign decisions outside the tie
    band that differ from float64 (must be 0) and the code agreement with the oracle's codes."""
    import numpy as np
    import torch

    import oracle.kashin_ref as ref
    from paper_2609_11687_amd import kashin as K
    from paper_2609_11687_amd import synth

    first = {}
    for idx, spec in enumerate(wl.matrices):
        first.setdefault(spec.n, idx)
    out = {}
    for n, idx in first.items():
        plan, wd, cu, cv, ce = loaded[idx]
        w = wd.float()
        m = w.shape[0]
        mx = w.abs().amax(dim=1)
        rows = sorted({0, m - 1, int(torch.argmax(mx))} | {int(i) for i in torch.topk(mx, 2).indices})[:rows_per_matrix]
        k = wl.iters
        rt = torch.tensor(rows, dtype=torch.int64, device=wd.device)
        sg = torch.empty((len(rows), 4 * k, n), dtype=torch.int8, device=wd.device)
        ct = torch.empty((len(rows), 4 * k), dtype=torch.float32, device=wd.device)
        ut = torch.empty((len(rows), n), dtype=torch.float32, device=wd.device)
        vt = torch.empty_like(ut)
        K.kashin_trace(plan, wd, rt, sg, ct, ut, vt)
        torch.cuda.synchronize()
        w64 = w[rows].cpu().numpy().astype(np.float64)
        winf = np.abs(w64).max(axis=1)
        eps = ref.sign_mask(n, synth.sign_seed(wl, 0, idx))
        d = ref.decompose(w64, eps, k, replay_signs=sg.cpu().numpy(), tau=1e-6 * winf)
        u, v = ut.cpu().numpy().astype(np.float64), vt.cpu().numpy().astype(np.float64)
        du = float((np.abs(u - d["u"]).max(axis=1) / winf).max())
        dv = float((np.abs(v - d["vhat"]).max(axis=1) / winf).max())
        rec = float((np.abs(w64 - d["r"] - u - ref.apply_p(v, eps)).max(axis=1) / winf).max())
        same = tot = 0
        for packed, x, c1, c2 in ((cu, d["u"], 0, 1), (cv, d["vhat"], 2, 3)):
            q = ref.closed_form_centers(d["cstep"][:, c1], d["cstep"][:, c2])
            codes = ref.unpack2bit(packed[rows].cpu().numpy(), n)
            same += int((codes == ref.assign_codes(x, q, np.float32)).sum())
            tot += codes.size
        out[str(n)] = {"matrix": wl.matrices[idx].name, "rows": rows, "max_du": du, "max_dv": dv, "max_rec": rec,
                       "outside_tie_band": int(d["replay_outside"].sum()), "code_agreement": same / tot,
                       "tolerances": {"factors": 1e-4, "reconstruction": 1e-5, "codes": 0.9999}}
    return out


def held_clock_mhz(run_for_ms):
    """SCLK of the GPU while the benchmark's step keeps it busy: `run_for_ms()` queues about two
    seconds of steps without waiting, rocm-smi reads the current clock meanwhile."""
    import subprocess

    import torch

    if any(k.startswith("ROCPROF") for k in os.environ):
        # under rocprofv3 every child process loads the profiler, which starts the GPU runtime
        # before rocm-smi's interpreter is exec'd: no clock probe in profiled runs
        return None
    run_for_ms()
    try:
        res = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True, text=True, timeout=30)
        torch.cuda.synchronize()
        data = json.loads(res.stdout)
        for card in data.values():
            for key, val in card.items():
                if "sclk" in key.lower():
                    digits = "".join(ch for ch in str(val).split("Mhz")[0] if ch.isdigit())
                    if digits:
                        return int(digits)
    except Exception:  # pragma: no cover - no rocm-smi, unparsable output
        torch.cuda.synchronize()
    return None


def copy_bandwidth_gbps():
    """Achievable HBM bandwidth: a plain 1 GiB device-to-device copy (read + write bytes / time)."""
    import torch

    x = torch.ones(256 << 20, dtype=torch.float32, device="cuda:0")
    y = torch.empty_like(x)
    for _ in range(2):
        y.copy_(x)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(5):
        y.copy_(x)
    t1.record()
    torch.cuda.synchronize()
    gbps = 5 * 2 * x.numel() * 4 / (t0.elapsed_time(t1) / 1e3) / 1e9
    del x, y
    torch.cuda.empty_cache()
    return gbps


def cpu_baseline_apply_p(n: int, rows: int):
    """The oracle's P (two dense float64 GEMMs with the explicit cosine matrix) on `rows` rows."""
    import numpy as np

    import oracle.kashin_ref as ref

    x = np.random.default_rng(0).standard_normal((rows, n))
    eps = ref.sign_mask(n, 0)
    ref.dct2_matrix(n)
    t0 = time.perf_counter()
    ref.apply_p(x, eps)
    dt = time.perf_counter() - t0
    return {"value": rows / dt, "unit": "rows/s", "cores": int(_blas_threads()), "kind": "oracle",
            "sample": f"{rows} Gaussian rows of width {n}, float64 dense P; {dt:.1f} s; "
                      f"cosine-matrix construction excluded"}


def time_launches(launches, steps: int, warmup: int, stream):
    """Whole-step time (no events inside the step) and the average duration of every launch
    (HIP events recorded on the launch stream around each one)."""
    import torch

    def step(events=None):
        for i, l in enumerate(launches):
            if events is not None:
                events[i][0].record(stream)
            l.run(stream)
            if events is not None:
                events[i][1].record(stream)

    log(f"warmup {warmup} steps")
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    log(f"timing {steps} steps")
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = t0.elapsed_time(t1) / steps
    launch_ms = [0.0] * len(launches)
    for _ in range(steps):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in launches]
        step(ev)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(ev):
            launch_ms[i] += a.elapsed_time(b) / steps
    return ms_per_step, launch_ms


def per_n_figures(launches, launch_ms):
    by_n = {}
    for l, ms in zip(launches, launch_ms):
        d = by_n.setdefault(l.n, {"vectors": 0, "ms": 0.0, "flops": 0.0, "bytes": 0.0})
        d["vectors"] += l.rows
        d["ms"] += ms
        d["flops"] += l.flops
        d["bytes"] += l.nbytes
    out = {}
    for n, d in sorted(by_n.items()):
        s = d["ms"] / 1e3
        out[str(n) if n else "mixed lengths"] = {
            "vectors_per_s": d["vectors"] / s,
            "counted_tflops": d["flops"] / s / 1e12,
            "valu_frac": d["flops"] / s / 1e12 / PEAK_FP32_TFLOPS,
            "hbm_gbps": d["bytes"] / s / 1e9,
            "hbm_frac": d["bytes"] / s / 1e9 / PEAK_HBM_GBPS,
            "ms_per_step": d["ms"],
        }
    return by_n, out


def peak_mass(x, a, b):
    """Fraction of the entries of each row of x within a tenth of the smallest centre gap of the
    nearest of the four centres +-a +- b (the peaks of Sec. 3.1), averaged over rows."""
    import numpy as np

    q = np.sort(np.stack([-(a + b), -np.abs(a - b), np.abs(a - b), a + b], axis=1), axis=1)
    gap = np.maximum(np.diff(q, axis=1).min(axis=1), 1e-30)
    dist = np.abs(x[:, :, None] - q[:, None, :]).min(axis=2)
    return float((dist <= 0.1 * gap[:, None]).mean())


def histogram_modes(x, bins=48, prominence=0.1):
    """Per row of x: the number of modes of its density, counted as the peaks of a `bins`-bin
    histogram over [-max|x|, max|x|] (smoothed with weights 1, 2, 1) that rise at least
    `prominence` times the tallest bin above the deeper of the valleys around them."""
    import numpy as np
    from scipy.signal import find_peaks

    out = []
    for row in x:
        lim = float(np.abs(row).max()) or 1.0
        h, _ = np.histogram(row, bins=bins, range=(-lim, lim))
        hs = np.convolve(np.concatenate([[0], h, [0]]), [0.25, 0.5, 0.25], mode="same")
        peaks, _ = find_peaks(np.concatenate([[0], hs, [0]]), prominence=prominence * hs.max())
        out.append(len(peaks))
    return np.array(out)


def fig2(args) -> int:
    """Fig. 2's comparison on the GPU: Alg. 2 (alternating blocks) against Alg. 1 (the original
    greedy: the half with the larger correlation, projection steps) on N(0, I) vectors, N = 10^4."""
    import numpy as np
    import torch

    from paper_2609_11687_amd import kashin as K

    n, rows, steps = 10000, args.fig2_rows, args.fig2_steps
    k = (steps + 3) // 4
    dev = torch.device("cuda:0")
    x = torch.randn((rows, n), dtype=torch.float32, device=dev, generator=torch.Generator(device=dev).manual_seed(0))
    plan = K.kashin_plan(n, 0, k)
    x2 = (x.double() ** 2).sum(dim=1)
    out = {}
    launches = []
    for sched in ("alternating", "original"):
        u, vh, r = torch.empty_like(x), torch.empty_like(x), torch.empty_like(x)
        rows_t = torch.arange(rows, dtype=torch.int64, device=dev)
        sg = torch.empty((rows, 4 * k, n), dtype=torch.int8, device=dev)
        cs = torch.empty((rows, 4 * k), dtype=torch.float32, device=dev)
        ch = torch.empty((rows, 4 * k), dtype=torch.int8, device=dev)
        r2 = torch.empty((rows, 4 * k), dtype=torch.float32, device=dev)
        ut, vt = torch.empty_like(x), torch.empty_like(x)
        K.kashin_trace_schedule(plan, sched, x, rows_t, sg, cs, ch, r2, ut, vt)
        torch.cuda.synchronize()
        rel = (r2.double() / x2[:, None]).sqrt().cpu().numpy()
        chc = ch.cpu().numpy()
        csc = cs.cpu().numpy().astype(np.float64)
        # centres of each factor from its first two steps (Sec. 3.1; for Alg. 1 the first two
        # steps it happened to take in that half)
        ab = {}
        for half, code in (("u", 0), ("vhat", 1)):
            a = np.zeros(rows)
            b = np.zeros(rows)
            for i in range(rows):
                idx = np.nonzero(chc[i] == code)[0]
                if idx.size >= 2:
                    a[i], b[i] = csc[i, idx[0]], csc[i, idx[1]]
            ab[half] = (a, b)
        # u and v-hat: Fig. 2's densities are those of u_k and of U v_k = v-hat (x = u_k + v_k)
        uu, vv = ut.cpu().numpy().astype(np.float64), vt.cpu().numpy().astype(np.float64)
        marks = [s_ for s_ in (4, 8, 16, 32, 64, 128, 200, 400) if s_ <= 4 * k]
        out[sched] = {
            "residual_rel_mean": {str(s_): float(rel[:, s_ - 1].mean()) for s_ in marks},
            "residual_rel_vector0": {str(s_): float(rel[0, s_ - 1]) for s_ in marks},
            "vhat_steps_frac": float((chc == 1).mean()),
            "peak_mass_u": peak_mass(uu, *ab["u"]),
            "peak_mass_vhat": peak_mass(vv, *ab["vhat"]),
            "modes_u": np.bincount(histogram_modes(uu), minlength=6).tolist(),
            "modes_vhat": np.bincount(histogram_modes(vv), minlength=6).tolist(),
        }
        launches.append(lambda s, a=(sched, u, vh, r): K.kashin_decompose_schedule(plan, a[0], x, a[1], a[2], a[3],
                                                                                   stream=s))
    stream = torch.cuda.current_stream()

    class _L:
        def __init__(self, f):
            self.run = f

    ms_per_step, launch_ms = time_launches([_L(f) for f in launches], args.steps, args.warmup, stream)
    baseline = None if args.no_cpu_baseline else fig2_cpu_baseline(x[:1], n)
    result = {
        "metric": "Fig. 2 set-up: residual after greedy updates, Alg. 2 vs Alg. 1, N = 10^4",
        "value": 2 * rows / (ms_per_step / 1e3),
        "unit": "vectors/s (both schedules)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"fig2: {rows} vectors of N(0, I_N), N = {n}, {4 * k} greedy updates, "
                               f"schedules alternating (Alg. 2) and original (Alg. 1, no tolerance)",
                   "ms_alternating": launch_ms[0], "ms_original": launch_ms[1]},
        "fig2": out,
    }
    if baseline is not None:
        result["cpu_baseline"] = baseline
    print(json.dumps(result), flush=True)
    return 0


def fig2_cpu_baseline(x0, n, steps: int = 24):
    """The oracle on vector 0 of the Fig. 2 set-up, both schedules, the first `steps` updates: its
    rate, and the GPU's factors after those updates (traced with a plan of steps / 4 blocks)
    against the oracle replayed on the GPU's near-tie decisions (signs within 1e-6 ||x||_inf of
    zero, choices within 1e-5 of a tie).  24 updates leave a residual near 1e-5 of ||x||_2: once it
    nears fp32's resolution of x (after about 32), the two residuals share no more digits and
    Alg. 1's half choices, decided by comparing two l1 norms of that residual, no longer need to
    agree (the factors, then changed by steps of that size, still do)."""
    import numpy as np
    import torch

    import oracle.kashin_ref as ref
    from paper_2609_11687_amd import kashin as K

    dev = x0.device
    k = steps // 4
    plan = K.kashin_plan(n, 0, k)
    x64 = x0.double().cpu().numpy()
    winf = float(np.abs(x64).max())
    eps = ref.sign_mask(n, 0)
    ref.dct2_matrix(n)  # the dense cosine matrix, built outside the timing
    rows_t = torch.zeros(1, dtype=torch.int64, device=dev)
    parity, seconds = {}, 0.0
    for sched in ("alternating", "original"):
        sg = torch.empty((1, 4 * k, n), dtype=torch.int8, device=dev)
        cs = torch.empty((1, 4 * k), dtype=torch.float32, device=dev)
        ch = torch.empty((1, 4 * k), dtype=torch.int8, device=dev)
        r2 = torch.empty((1, 4 * k), dtype=torch.float32, device=dev)
        ut, vt = torch.empty_like(x0), torch.empty_like(x0)
        K.kashin_trace_schedule(plan, sched, x0, rows_t, sg, cs, ch, r2, ut, vt)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rep = ref.decompose_schedule(x64, eps, 4 * k, sched, replay_signs=sg.cpu().numpy(),
                                     replay_choices=ch.cpu().numpy(), tau=1e-6 * winf, choice_band=1e-5)
        seconds += time.perf_counter() - t0
        parity[sched] = {
            "updates": 4 * k,
            "max_du": float(np.abs(ut.double().cpu().numpy() - rep["u"]).max() / winf),
            "max_dv": float(np.abs(vt.double().cpu().numpy() - rep["vhat"]).max() / winf),
            "outside_tie_band": int(np.asarray(rep["replay_outside"]).sum()),
            "choices_outside_band": int(np.asarray(rep["choice_outside"]).sum()),
            "tolerance_factors": 1e-4,
        }
    return {"value": 2 / seconds, "unit": "vectors/s", "cores": int(_blas_threads()), "kind": "oracle",
            "sample": f"vector 0, {4 * k} updates of each schedule, float64 dense P (N = {n}); {seconds:.1f} s; "
                      f"cosine-matrix construction excluded",
            "parity": parity}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama7b")
    ap.add_argument("--op", choices=("quantize", "apply_p", "reconstruct", "rotate", "quantize_h", "schedule",
                                     "optq", "fig2"), default="quantize")
    ap.add_argument("--fig2-rows", type=int, default=64)
    ap.add_argument("--fig2-steps", type=int, default=200)
    ap.add_argument("--exact", action="store_true", help="--op optq: columns one at a time inside each chunk")
    ap.add_argument("--matrix", default="q_proj", help="matrix of the workload (--op optq)")
    ap.add_argument("--chunk", type=int, default=128, help="columns per compensation chunk (--op optq)")
    ap.add_argument("--model-layers", type=int, default=0,
                    help="--op optq --matrix all: one step = this many layers, each factorising its four "
                         "Hessians (inputs of q/k/v, o, gate/up, down) inside the timed region, then the "
                         "compensated quantisation of its seven matrices")
    ap.add_argument("--schedule", choices=("alternating", "reverse", "adaptive", "original"), default="adaptive")
    ap.add_argument("--lloyd", type=int, default=0)
    ap.add_argument("--per-matrix", action="store_true",
                    help="--op quantize / quantize_h / reconstruct: one kashin_quantize(_rotated) or "
                         "kashin_reconstruct launch per matrix instead of one grouped launch per vector "
                         "length (up to 16 matrices each)")
    ap.add_argument("--act-rows", type=int, default=16384, help="activation rows per width (--op apply_p)")
    ap.add_argument("--cpu-rows", type=int, default=1536)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device-to-device copy (HBM counter calibration)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: rows are independent, so a multi-GPU run would shard them "
              "with no communication; only --gpus 1 is supported.", file=sys.stderr)
        return 2
    if args.op == "optq":
        # one hardware queue per matrix chain: the runtime's default is four per process, and
        # chains sharing a queue run one after the other (read when the runtime starts)
        if int(os.environ.get("GPU_MAX_HW_QUEUES", "4")) < 8:
            os.environ["GPU_MAX_HW_QUEUES"] = "8"

    import torch

    if args.copy_calibration:
        x = torch.ones(64 << 20, dtype=torch.float32, device="cuda:0")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": x.numel() * 4, "copy_bytes_written": y.numel() * 4}), flush=True)
        return 0

    from paper_2609_11687_amd import kashin as K
    from paper_2609_11687_amd import synth
    from paper_2609_11687_amd.build import source_digest

    K.lib()
    if args.op == "fig2":
        return fig2(args)
    wl = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    launches: list[Launch] = []
    keep = []  # device buffers and plans referenced by the launches

    if args.op in ("quantize", "reconstruct", "rotate", "quantize_h", "schedule"):
        for layer in range(wl.layers):
            for idx, spec in enumerate(wl.matrices):
                log(f"generating {args.workload} layer {layer} {spec.name} {spec.rows}x{spec.n}")
                w = synth.make_matrix(wl, layer, idx)
                dt = torch.float16 if spec.dtype == "f16" else torch.float32
                wd = torch.from_numpy(w).to(dev).to(dt)
                del w
                plan = K.kashin_plan(spec.n, synth.sign_seed(wl, layer, idx), wl.iters)
                nb = (spec.n + 3) // 4
                cu = torch.empty((spec.rows, nb), dtype=torch.uint8, device=dev)
                cv = torch.empty_like(cu)
                ce = torch.empty((spec.rows, 2, 4), dtype=torch.float32, device=dev)
                if args.op == "schedule":
                    uu = torch.empty((spec.rows, spec.n), dtype=torch.float32, device=dev)
                    vv, rr_ = torch.empty_like(uu), torch.empty_like(uu)
                    keep.append((plan, wd, uu, vv, rr_))
                    launches.append(Launch(
                        spec.n, spec.rows, spec.rows * 2 * (4 * wl.iters + 2) * transform_flops(spec.n),
                        spec.rows * (spec.n * (2 if spec.dtype == "f16" else 4) + 12 * spec.n),
                        lambda s, a=(plan, wd, uu, vv, rr_): K.kashin_decompose_schedule(
                            a[0], args.schedule, a[1], a[2], a[3], a[4], stream=s),
                        kind="schedule"))
                elif args.op == "rotate":
                    wr = torch.empty((spec.rows, spec.n), dtype=torch.float32, device=dev)
                    keep.append((plan, wd, wr, cu, cv, ce))
                    p2 = spec.n & -spec.n
                    launches.append(Launch(
                        spec.n, spec.rows, spec.rows * spec.n * (math.log2(p2) + 2 * (spec.n // p2)),
                        spec.rows * spec.n * (2 + 4),
                        lambda s, a=(spec.n, wd, wr): K.kashin_rotate(a[0], ROT_SEED, a[1], a[2], stream=s),
                        kind="rotate"))
                elif args.op == "quantize_h" and not args.per_matrix:
                    keep.append((plan, wd, cu, cv, ce))  # grouped by vector length below
                elif args.op == "quantize_h":
                    keep.append((plan, wd, cu, cv, ce))
                    launches.append(Launch(
                        spec.n, spec.rows, spec.rows * counted_flops_per_vector(spec.n, wl.iters),
                        spec.rows * hbm_bytes_per_vector(spec.n, 2 if spec.dtype == "f16" else 4),
                        lambda s, a=(plan, wd, cu, cv, ce): K.kashin_quantize_rotated(
                            a[0], ROT_SEED, a[1], args.lloyd, a[2], a[3], a[4], s)))
                elif args.op == "quantize" and not args.per_matrix:
                    keep.append((plan, wd, cu, cv, ce))  # grouped by vector length below
                elif args.op == "quantize":
                    keep.append((plan, wd, cu, cv, ce))
                    launches.append(Launch(
                        spec.n, spec.rows, spec.rows * counted_flops_per_vector(spec.n, wl.iters),
                        spec.rows * hbm_bytes_per_vector(spec.n, 2 if spec.dtype == "f16" else 4),
                        lambda s, a=(plan, wd, cu, cv, ce): K.kashin_quantize(a[0], a[1], args.lloyd, a[2], a[3],
                                                                              a[4], s)))
                else:
                    K.kashin_quantize(plan, wd, args.lloyd, cu, cv, ce, stream)
                    torch.cuda.synchronize()
                    del wd
                    wh = torch.empty((spec.rows, spec.n), dtype=torch.float32, device=dev)
                    keep.append((plan, cu, cv, ce, wh))
                    if not args.per_matrix:
                        continue  # grouped by vector length below
                    launches.append(Launch(
                        spec.n, spec.rows, spec.rows * 2 * transform_flops(spec.n),
                        spec.rows * (2 * nb + 32 + 4 * spec.n),
                        lambda s, a=(plan, cu, cv, ce, wh): K.kashin_reconstruct(a[0], a[1], a[2], a[3], a[4], s),
                        kind="pmap"))
        if args.op in ("quantize", "quantize_h") and not args.per_matrix:
            # one grouped launch per vector length and 16 matrices: the row pairs of all of them
            # share one grid, so no launch ends in a partial wave of workgroups
            for n in sorted({spec.n for spec in wl.matrices}):
                items = [it for it in keep if it[0].n == n]
                for c0 in range(0, len(items), 16):
                    chunk = items[c0:c0 + 16]
                    rows = sum(it[1].shape[0] for it in chunk)
                    in_bytes = chunk[0][1].element_size()
                    launches.append(Launch(
                        n, rows, rows * counted_flops_per_vector(n, wl.iters), rows * hbm_bytes_per_vector(n, in_bytes),
                        lambda s, c=chunk: K.kashin_quantize_grouped(
                            c, args.lloyd, s, rot_seed=ROT_SEED if args.op == "quantize_h" else None),
                        wgs=sum((it[1].shape[0] + 1) // 2 for it in chunk)))
        if args.op == "reconstruct" and not args.per_matrix:
            # one grouped reconstruction per vector length and 16 matrices; each matrix takes a
            # share of the persistent grid in proportion to its row pairs
            for n in sorted({spec.n for spec in wl.matrices}):
                items = [it for it in keep if it[0].n == n]
                for c0 in range(0, len(items), 16):
                    chunk = items[c0:c0 + 16]
                    rows = sum(it[4].shape[0] for it in chunk)
                    nb = (n + 3) // 4
                    pairs = [(it[4].shape[0] + 1) // 2 for it in chunk]
                    grid = min(sum(pairs), 2048)
                    launches.append(Launch(
                        n, rows, rows * 2 * transform_flops(n), rows * (2 * nb + 32 + 4 * n),
                        lambda s, c=chunk: K.kashin_reconstruct_grouped(c, s), kind="pmap",
                        wgs=sum(max(1, min(p, grid * p // sum(pairs))) for p in pairs)))
    elif args.op == "optq":
        from paper_2609_11687_amd import optq

        names = [s_.name for s_ in wl.matrices]
        chosen = list(range(len(names))) if args.matrix == "all" else [names.index(args.matrix)]
        jobs = []
        gemm = 0.0
        g = torch.Generator(device=dev).manual_seed(0)
        hess_by_din = {}
        for idx in chosen:
            spec = wl.matrices[idx]
            log(f"generating {args.workload} {spec.name} {spec.rows}x{spec.n}")
            w0_t = torch.from_numpy(synth.make_matrix(wl, 0, idx).T.copy()).to(dev).to(torch.float32).contiguous()
            d_in, d_out = w0_t.shape
            if d_in not in hess_by_din:  # one synthetic Hessian per input width
                x = torch.randn((2 * d_in, d_in), dtype=torch.float32, device=dev, generator=g)
                x[:, torch.randperm(d_in, generator=g, device=dev)[: max(1, d_in // 1000)]] *= 20.0
                hess_by_din[d_in] = (x.t() @ x) / x.shape[0]
                del x
            plan = K.kashin_plan(d_out, synth.sign_seed(wl, 0, idx), wl.iters)
            jobs.append((plan, w0_t, torch.empty_like(w0_t), hess_by_din[d_in], None))
            gemm += sum(2.0 * min(args.chunk, d_in - c0) * d_out * (d_in - min(c0 + args.chunk, d_in))
                        for c0 in range(0, d_in, args.chunk))
        keep.append(jobs)
        nchunks = sum((j[1].shape[0] + args.chunk - 1) // args.chunk for j in jobs)
        # the factor of each input width's damped inverse Hessian (kashin_optq_factor), once, before
        # timing, as the Hessian itself: it stays alive for every step, so no stream ever reads a
        # factor whose memory the allocator could hand out again
        factors, factor_ms = {}, {}
        for d_in, hess in hess_by_din.items():
            # an untimed first call per size: it loads the library kernels that size uses
            optq.compensation_factor(hess, want_v=not args.exact)
            torch.cuda.synchronize()
            t0e, t1e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0e.record()
            factors[d_in] = optq.compensation_factor(hess, want_v=not args.exact)
            t1e.record()
            torch.cuda.synchronize()
            factor_ms[str(d_in)] = t0e.elapsed_time(t1e)
        keep.append(factors)

        # Each matrix is one chain of dependent chunks, on a stream of its own as long as the
        # hardware queues last (streams beyond them share queues, and chains on one queue run one
        # after the other); otherwise longest first onto the least loaded stream (a chain's cost
        # taken as chunks x vector length).
        n_streams = min(int(os.environ.get("GPU_MAX_HW_QUEUES", "4")), len(jobs))
        streams = [torch.cuda.Stream(dev) for _ in range(n_streams)]
        load = [0.0] * n_streams
        placed = []
        for j in sorted(jobs, key=lambda j: -((j[1].shape[0] + args.chunk - 1) // args.chunk) * j[1].shape[1]):
            k_ = min(range(n_streams), key=lambda i: load[i])
            load[k_] += ((j[1].shape[0] + args.chunk - 1) // args.chunk) * j[1].shape[1]
            placed.append(j[:4] + (streams[k_],))
        jobs = placed

        def run_optq(s):
            # every matrix on its own stream, joined back into the timing stream
            for plan, w0_t, w_t, hess, st in jobs:
                st.wait_stream(s)
                with torch.cuda.stream(st):
                    w_t.copy_(w0_t)
                optq.optq_quantize(plan, w_t, hess, args.chunk, lloyd_iters=args.lloyd, stream=st, exact=args.exact,
                                   factor=factors[w_t.shape[0]])
            for *_, st in jobs:
                s.wait_stream(st)

        if args.model_layers > 0:
            if args.matrix != "all":
                raise SystemExit("--model-layers needs --matrix all")
            one_layer = run_optq
            widths = sorted(hess_by_din)

            def run_optq(s):  # noqa: F811 - the model: every layer factorises its Hessians, then quantises
                for _ in range(args.model_layers):
                    for d_in in widths:
                        # three distinct inputs of width 4096 per layer (q/k/v, o, gate/up), one of 11008
                        for _rep in range(3 if d_in == widths[0] and len(widths) > 1 else 1):
                            factors[d_in] = optq.compensation_factor(hess_by_din[d_in], want_v=not args.exact)
                    one_layer(s)

        # one launch covers every matrix: its length is the matrices' common d_out, else 0 (mixed)
        d_outs = {j[1].shape[1] for j in jobs}
        d_out = d_outs.pop() if len(d_outs) == 1 else 0
        reps = max(1, args.model_layers)
        cols = reps * sum(j[1].shape[0] for j in jobs)
        flops = reps * (sum(j[1].shape[0] * counted_flops_per_vector(j[1].shape[1], wl.iters) for j in jobs) + gemm)
        launches.append(Launch(d_out, cols, flops, reps * sum(j[1].numel() * 12 for j in jobs), run_optq,
                               kind="optq"))
    else:
        g = torch.Generator(device=dev).manual_seed(0)
        for n in sorted({spec.n for spec in wl.matrices}):
            log(f"activation rows {args.act_rows}x{n}")
            x = torch.randn((args.act_rows, n), dtype=torch.float32, device=dev, generator=g)
            y = torch.empty_like(x)
            plan = K.kashin_plan(n, 0, 1)
            keep.append((plan, x, y))
            launches.append(Launch(n, args.act_rows, args.act_rows * 2 * transform_flops(n), args.act_rows * 8 * n,
                                   lambda s, a=(plan, x, y): K.kashin_apply_p(a[0], a[1], a[2], s), kind="pmap"))
    torch.cuda.synchronize()

    def step_all(s_):
        for l_ in launches:
            l_.run(s_)

    ms_per_step, launch_ms = time_launches(launches, args.steps, args.warmup, stream)
    total_vectors = sum(l.rows for l in launches)
    by_n, per_n = per_n_figures(launches, launch_ms)

    # dominant kernel: the N = 4096 launches (if present) of the op's main kernel, averaged over them
    main_kind = {"quantize": "quantize", "quantize_h": "quantize", "rotate": "rotate",
                 "schedule": "schedule", "optq": "optq"}.get(args.op, "pmap")
    dom_n = 4096 if 4096 in by_n else max(by_n, key=lambda n: by_n[n]["ms"])
    dom = [(l, ms) for l, ms in zip(launches, launch_ms) if l.n == dom_n and l.kind == main_kind]
    dom_s = sum(ms for _, ms in dom) / 1e3
    dom_flops = sum(l.flops for l, _ in dom)
    dom_bytes = sum(l.nbytes for l, _ in dom)
    layer = ", ".join(f"{s.name} {s.rows}x{s.n}" for s in wl.matrices) + f" x {wl.layers} layer(s)"
    if main_kind == "optq":
        achieved = dom_flops / dom_s / 1e12
        roofline = {
            "bound": "alu", "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP32_TFLOPS, "traffic": None,
            "kernel": f"optq pipeline ({len(jobs)} matrices, {nchunks} chunks: pair_greedy_kernel + pair_pmap_kernel "
                      f"+ update_gemm_kernel; factorisation once per input width, before timing)",
            "launches": len(dom), "counted_flops": dom_flops, "gemm_flops": gemm,
            "factor_ms_per_input_width": factor_ms,
        }
        metric, unit = METRIC_OPTQ.format(args.chunk) + (", exact per-column updates" if args.exact else ""), \
            "columns/s"
        workload = (f"optq: {args.workload} " + ", ".join(f"{wl.matrices[i].name} {wl.matrices[i].rows}x{wl.matrices[i].n}"
                                                           for i in chosen)
                    + f" (chains on {n_streams} streams, {os.environ.get('GPU_MAX_HW_QUEUES')} hardware queues), columns quantised in chunks of {args.chunk}, k={wl.iters}, "
                    f"Hessian of 2 d_in seeded Gaussian activations with 0.1% outlier channels x20")
        if args.model_layers > 0:
            workload += (f"; one step = {args.model_layers} such layers (the same synthetic matrices), each "
                         f"factorising four Hessians (3 at d_in 4096, 1 at 11008) inside the step")
    elif main_kind == "schedule":
        achieved = dom_flops / dom_s / 1e12
        roofline = {
            "bound": "alu", "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP32_TFLOPS, "traffic": None,
            "kernel": f"pair_schedule_kernel N={dom_n}", "launches": len(dom),
            "flops_per_vector": 2 * (4 * wl.iters + 2) * transform_flops(dom_n),
            "algorithmic_bytes_per_launch": dom_bytes / len(dom),
        }
        metric, unit = METRIC_SCHED.format(args.schedule), "vectors/s"
        workload = (f"{args.workload} {args.schedule} schedule: {layer}, {wl.matrices[0].dtype} storage, "
                    f"{4 * wl.iters} atomic steps")
    elif main_kind == "quantize":
        achieved = dom_flops / dom_s / 1e12
        kname = "pair_greedy_kernel[quantize" + (",lloyd" if args.lloyd > 0 else "") + \
            (",rotated]" if args.op == "quantize_h" else "]")
        roofline = {
            "bound": "alu", "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP32_TFLOPS,
            "traffic": measured_traffic(args.op, args.workload, kname, [(l.n, l.workgroups()) for l, _ in dom]),
            "kernel": f"{kname} N={dom_n}", "launches": len(dom),
            "flops_per_vector": counted_flops_per_vector(dom_n, wl.iters),
            "algorithmic_bytes_per_launch": dom_bytes / len(dom),
        }
        if args.op == "quantize":
            metric, unit = METRIC, "vectors/s"
            workload = (f"{args.workload}: {layer}, {wl.matrices[0].dtype} storage, k={wl.iters} blocks, "
                        f"lloyd={args.lloyd}, one row = one vector, "
                        + ("one launch per matrix" if args.per_matrix else
                           "one grouped launch per vector length (kashin_quantize_grouped)"))
        else:
            metric, unit = METRIC_QUANT_H, "vectors/s"
            workload = (f"{args.workload} +H: {layer}, {wl.matrices[0].dtype} rows rotated in the load (R w, seed "
                        f"{ROT_SEED}) and quantised, k={wl.iters} blocks, lloyd={args.lloyd}, "
                        + ("one launch per matrix" if args.per_matrix else
                           "one grouped launch per vector length (kashin_quantize_grouped)"))
    else:
        achieved = dom_bytes / dom_s / 1e9
        kname = f"rotate_kernel[b={dom_n // (dom_n & -dom_n)}]" if main_kind == "rotate" else "pair_pmap_kernel"
        grid = (lambda l: l.rows) if main_kind == "rotate" else (
            lambda l: l.wgs or min((l.rows + 1) // 2, PMAP_GRID))
        keyn = (lambda l: 0) if main_kind == "rotate" else (lambda l: l.n)  # the rotation kernel takes n at run time
        roofline = {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBPS,
            "traffic": measured_traffic(args.op, args.workload, kname, [(keyn(l), grid(l)) for l, _ in dom]),
            "kernel": f"{kname} N={dom_n}", "launches": len(dom),
            "valu_tflops": dom_flops / dom_s / 1e12,
            "algorithmic_bytes_per_launch": dom_bytes / len(dom),
        }
        if args.op == "apply_p":
            metric, unit = METRIC_APPLY_P, "rows/s"
            workload = (f"apply_p: {args.act_rows} Gaussian fp32 rows at each width "
                        + ", ".join(str(n) for n in sorted(by_n)) + f" ({args.workload} input widths)")
        elif args.op == "rotate":
            metric, unit = METRIC_ROTATE, "rows/s"
            workload = f"rotate: {args.workload} {layer}, fp16 rows in, fp32 rows out (seed {ROT_SEED})"
        else:
            metric, unit = METRIC_RECON, "rows/s"
            workload = (f"reconstruct: {args.workload} {layer} from their 2+2-bit codes (k={wl.iters}), "
                        f"fp32 output, " + ("one launch per matrix" if args.per_matrix else
                                            "one grouped launch per vector length (kashin_reconstruct_grouped)"))
    result = {
        "metric": metric,
        "value": total_vectors / (ms_per_step / 1e3),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workload, "vectors_per_step": total_vectors, "iters": wl.iters},
        "per_n": per_n,
        "roofline": roofline,
        "source_digest": source_digest(),
    }
    if args.op in ("quantize", "quantize_h", "schedule", "rotate"):
        # GB/s of weights quantised: the stored weight bytes the step reads, per second
        wbytes = wl.layers * sum(sp.rows * sp.n * (2 if sp.dtype == "f16" else 4) for sp in wl.matrices)
        result["weights_gbps"] = wbytes / (ms_per_step / 1e3) / 1e9
    if args.op == "schedule":
        # convergence (Fig. 2 style): ||rho||_2 / ||w||_2 after 4, 8, 16 and 32 atomic steps, the
        # mean over the first 8 rows of the first matrix (recorded by kashin_trace_schedule)
        plan, wd, *_ = keep[0]
        nr, n0, steps = 8, wd.shape[1], 4 * wl.iters
        rows_t = torch.arange(nr, dtype=torch.int64, device=dev)
        sg = torch.empty((nr, steps, n0), dtype=torch.int8, device=dev)
        cs = torch.empty((nr, steps), dtype=torch.float32, device=dev)
        ch = torch.empty((nr, steps), dtype=torch.int8, device=dev)
        r2 = torch.empty((nr, steps), dtype=torch.float32, device=dev)
        ut, vt = torch.empty((nr, n0), device=dev), torch.empty((nr, n0), device=dev)
        K.kashin_trace_schedule(plan, args.schedule, wd, rows_t, sg, cs, ch, r2, ut, vt)
        torch.cuda.synchronize()
        w2 = (wd[:nr].float() ** 2).sum(dim=1)
        result["convergence"] = {str(s_): (r2[:, s_ - 1] / w2).sqrt().mean().item() for s_ in (4, 8, 16, 32)
                                 if s_ <= steps}
    if main_kind in ("quantize", "pmap", "rotate"):
        # peaks as this machine delivers them: the clock it holds under this load and a plain copy
        mhz = held_clock_mhz(lambda: [step_all(stream) for _ in range(max(1, int(2000 / max(ms_per_step, 1e-3))))])
        copy = copy_bandwidth_gbps()
        roofline["measured_peaks"] = {
            "sclk_mhz": mhz,
            "fp32_tflops_at_held_clock": None if mhz is None else PEAK_FP32_TFLOPS * mhz / 2400.0,
            "hbm_copy_gbps": copy,
            "note": "published peaks assume 2400 MHz and 8 TB/s; these are the clock held during the step "
                    "(rocm-smi while steps run) and a 1 GiB device-to-device copy",
        }
        if roofline["unit"] == "TFLOP/s" and mhz:
            roofline["frac_of_held_clock_peak"] = roofline["achieved"] / (PEAK_FP32_TFLOPS * mhz / 2400.0)
        if roofline["unit"] == "GB/s":
            roofline["frac_of_copy_bandwidth"] = roofline["achieved"] / copy
    if not args.no_cpu_baseline:
        if args.op == "quantize":
            log(f"cpu baseline: oracle on {args.cpu_rows} rows at N = {wl.matrices[0].n} and proportionally "
                f"fewer at the other lengths, then a replay of sampled rows")
            result["cpu_baseline"] = cpu_baseline(wl, args.cpu_rows, keep[:len(wl.matrices)])
        elif args.op == "apply_p":
            result["cpu_baseline"] = cpu_baseline_apply_p(dom_n, 4 * args.cpu_rows)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
