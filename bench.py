#!/usr/bin/env python3
"""Throughput of the fused Kashin-DCT quantizer (decompose + four-peak 2-bit clustering +
packing) on one MI355X.

One step = kashin_quantize over every matrix of the workload (default: one
Llama-2-7B-shaped decoder layer, fp16-stored, 30 blocks of Alg. 2, closed-form
centres), inputs already resident in HBM.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload llama7b] [--lloyd 0]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "weight vectors decomposed/s (N=4096, fixed iters); % of HBM / FP32 VALU roofline"
PEAK_FP32_TFLOPS = 157.3   # MI355X published FP32 vector peak (256 CU x 2.4 GHz x 256 flop/clk)
PEAK_HBM_GBPS = 8000.0     # MI355X published HBM3E bandwidth


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def counted_flops_per_vector(n: int, k: int) -> float:
    """Algorithmic count: 4k - 2 transforms (two P per block, the last one not needed for the
    factors), each 2.5 N log2 N flops."""
    return (4 * k - 2) * 2.5 * n * math.log2(n)


def hbm_bytes_per_vector(n: int, in_bytes: int) -> int:
    """Algorithmic traffic: read the row once, write 2 x N/4 bytes of codes and 32 B of centres."""
    return n * in_bytes + 2 * ((n + 3) // 4) + 32


def measured_traffic(launches) -> float | None:
    """HBM bytes per launch of the dominant kernel from the committed counter summaries
    (profiles/*.txt, line TRAFFIC_JSON), averaged over `launches` = [(n, workgroups)], or None
    when no summary was taken on the current kernel sources."""
    import glob

    from paper_2609_11687_amd.build import source_digest

    digest = source_digest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.txt"))):
        with open(path) as fh:
            for line in fh:
                if not line.startswith("TRAFFIC_JSON "):
                    continue
                rec = json.loads(line[len("TRAFFIC_JSON "):])
                keys = [f"{n}/{wg}" for n, wg in launches]
                if rec.get("digest") == digest and all(k in rec["bytes"] for k in keys):
                    return sum(rec["bytes"][k] for k in keys) / len(keys)
    return None


def cpu_baseline(wl, rows: int):
    """The float64 oracle on a bounded sample of the workload: the first `rows` rows of the
    first matrix (the dense explicit-cosine matrix is built before timing)."""
    import numpy as np

    import oracle.kashin_ref as ref
    from paper_2609_11687_amd import synth

    spec = wl.matrices[0]
    w = synth.make_matrix(wl, 0, 0, rows=slice(0, rows)).astype(np.float64)
    eps = ref.sign_mask(spec.n, synth.sign_seed(wl, 0, 0))
    ref.dct2_matrix(spec.n)
    try:
        from threadpoolctl import threadpool_info

        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    t0 = time.perf_counter()
    ref.quantize(w, eps, wl.iters, 0)
    dt = time.perf_counter() - t0
    return {
        "value": rows / dt,
        "unit": "vectors/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": f"{rows} rows of {spec.name} ({spec.rows}x{spec.n}), k={wl.iters}, float64 literal Alg. 2 "
                  f"with a dense P (4 GEMMs per block) + closed-form clustering + packing; "
                  f"{dt:.1f} s; cosine-matrix construction excluded",
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="llama7b")
    ap.add_argument("--lloyd", type=int, default=0)
    ap.add_argument("--cpu-rows", type=int, default=2048)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device-to-device copy (HBM counter calibration)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: rows are independent, so a multi-GPU run would shard them "
              "with no communication; only --gpus 1 is supported in this build.", file=sys.stderr)
        return 2

    import numpy as np
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
    wl = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    mats = []
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
            mats.append((spec, wd, plan, cu, cv, ce))
    stream = torch.cuda.current_stream()

    def step(events=None):
        for i, (spec, wd, plan, cu, cv, ce) in enumerate(mats):
            if events is not None:
                events[i][0].record(stream)
            K.kashin_quantize(plan, wd, args.lloyd, cu, cv, ce, stream)
            if events is not None:
                events[i][1].record(stream)

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # whole-step timing (no per-launch events inside)
    log(f"timing {args.steps} steps")
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    ms_per_step = ms_total / args.steps

    # per-launch durations (HIP events on the launch stream), for the per-N figures and roofline
    per = [[0.0 for _ in mats]]
    for _ in range(args.steps):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in mats]
        step(ev)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(ev):
            per[0][i] += a.elapsed_time(b) / args.steps
    launch_ms = per[0]

    total_vectors = sum(spec.rows for spec, *_ in mats)
    value = total_vectors / (ms_per_step / 1e3)
    by_n = {}
    for (spec, *_), ms in zip(mats, launch_ms):
        d = by_n.setdefault(spec.n, {"vectors": 0, "ms": 0.0, "flops": 0.0, "bytes": 0})
        d["vectors"] += spec.rows
        d["ms"] += ms
        d["flops"] += spec.rows * counted_flops_per_vector(spec.n, wl.iters)
        d["bytes"] += spec.rows * hbm_bytes_per_vector(spec.n, 2 if spec.dtype == "f16" else 4)
    per_n = {}
    for n, d in sorted(by_n.items()):
        s = d["ms"] / 1e3
        per_n[str(n)] = {
            "vectors_per_s": d["vectors"] / s,
            "counted_tflops": d["flops"] / s / 1e12,
            "valu_frac": d["flops"] / s / 1e12 / PEAK_FP32_TFLOPS,
            "hbm_gbps": d["bytes"] / s / 1e9,
            "ms_per_step": d["ms"],
        }
    # dominant kernel: the N = 4096 pair kernel (if present), averaged over its launches
    dom_n = 4096 if 4096 in by_n else max(by_n, key=lambda n: by_n[n]["ms"])
    dom = [(spec, ms) for (spec, *_), ms in zip(mats, launch_ms) if spec.n == dom_n]
    dom_flops = sum(spec.rows * counted_flops_per_vector(spec.n, wl.iters) for spec, _ in dom)
    dom_s = sum(ms for _, ms in dom) / 1e3
    achieved = dom_flops / dom_s / 1e12
    dom_bytes = sum(spec.rows * hbm_bytes_per_vector(spec.n, 2 if spec.dtype == "f16" else 4)
                    for spec, _ in dom) / len(dom)
    traffic = measured_traffic([(spec.n, (spec.rows + 1) // 2) for spec, _ in dom])
    result = {
        "metric": METRIC,
        "value": value,
        "unit": "vectors/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: " + ", ".join(f"{s.name} {s.rows}x{s.n}" for s in wl.matrices)
                        + f" x {wl.layers} layer(s), {wl.matrices[0].dtype} storage, k={wl.iters} blocks, "
                        f"lloyd={args.lloyd}, one row = one vector",
            "vectors_per_step": total_vectors,
            "iters": wl.iters,
        },
        "per_n": per_n,
        "roofline": {
            "bound": "alu",
            "achieved": achieved,
            "peak": PEAK_FP32_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP32_TFLOPS,
            "traffic": traffic,
            "kernel": f"pair_greedy_kernel N={dom_n}",
            "launches": len(dom),
            "flops_per_vector": counted_flops_per_vector(dom_n, wl.iters),
            "algorithmic_bytes_per_launch": dom_bytes,
        },
        "source_digest": source_digest(),
    }
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle on {args.cpu_rows} rows")
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_rows)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
