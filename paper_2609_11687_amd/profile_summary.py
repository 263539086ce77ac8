"""Turns rocprofv3 result databases into the short text summaries kept with the measurements.

    python -m paper_2609_11687_amd.profile_summary --trace KT.db \
        [--fetch F.db --write W.db --copy-fetch CF.db --copy-write CW.db] \
        --command "..." [--command "..."] > summary.txt

--trace: a `rocprofv3 --kernel-trace --stats` run; per kernel and launch shape it lists the
number of dispatches and the average duration.  The four counter databases (one
`--pmc FETCH_SIZE` and one `--pmc WRITE_SIZE` run of the same program, and the same two of a
plain 256 MiB device copy) give HBM bytes per dispatch: the raw KiB figure times the factor
that makes the copy's counter read its known size.  The last line of the output,
`TRAFFIC_JSON {...}`, carries those bytes per (kernel, vector length, workgroups) together with
the digest of the kernel sources they were taken on.  --sq (repeatable) adds the shader
counters of `--pmc SQ_...` runs for the pair kernels, with the busy and wait ratios they give.
"""
from __future__ import annotations

import argparse
import collections
import json
import re
import sqlite3
import sys

from .build import source_digest

COPY_BYTES = 256 << 20  # the calibration copy reads and writes 256 MiB


def _short(name: str) -> tuple[str, int]:
    m = re.search(r"(pair_greedy_kernel|pair_pmap_kernel|pair_schedule_kernel|rotate_kernel|cluster_kernel|"
                  r"__amd_rocclr_copyBuffer\w*|elementwise_kernel|potf2\w*|\w*substitution\w*|Cijk_\w*)", name)
    c = re.search(r"Cfg<(\d+)", name)
    base = m.group(1) if m else name[:40]
    if base.startswith("Cijk_"):  # library GEMM: operand layout, type and macro tile
        base = base[:42]
    rot = re.search(r"rotate_kernel<(\d+), (true|false)", name)  # rotate_kernel<odd factor, inverse, input type>
    if rot:
        base += f"[b={rot.group(1)}" + (",inverse]" if rot.group(2) == "true" else "]")
    # pair_greedy_kernel<Cfg, LLOYD, QUANT, ROT>
    flags = re.search(r">, (true|false), (true|false), (true|false)>", name)
    if flags:
        base += ("[quantize" + (",lloyd" if flags.group(1) == "true" else "") +
                 (",rotated" if flags.group(3) == "true" else "") + "]"
                 if flags.group(2) == "true" else "[decompose]")
    return base, int(c.group(1)) if c else 0


def trace_stats(path: str):
    db = sqlite3.connect(path)
    rows = db.execute("select name, duration, grid_x, workgroup_x, scratch_size from kernels")
    agg = collections.defaultdict(list)
    meta = {}
    for name, dur, gx, wx, scratch in rows:
        k, n = _short(name)
        key = (k, n, gx // max(wx, 1), wx)
        agg[key].append(dur)
        meta[key] = scratch
    return agg, meta


def counter_per_dispatch(path: str, counter: str):
    db = sqlite3.connect(path)
    rows = db.execute("select kernel_name, grid_size, workgroup_size, value from counters_collection "
                      "where counter_name = ?", (counter,))
    agg = collections.defaultdict(list)
    for name, g, w, v in rows:
        k, n = _short(name)
        agg[(k, n, g // max(w, 1), w)].append(v)
    return {key: sum(v) / len(v) for key, v in agg.items()}


def counters_per_dispatch(path: str):
    """Every counter of a `--pmc` database, averaged per dispatch of each kernel shape."""
    db = sqlite3.connect(path)
    rows = db.execute("select kernel_name, grid_size, workgroup_size, counter_name, value from counters_collection")
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for name, g, w, c, v in rows:
        k, n = _short(name)
        agg[(k, n, g // max(w, 1), w)][c].append(v)
    return {key: {c: sum(v) / len(v) for c, v in cs.items()} for key, cs in agg.items()}


CU_NUM = 256
XCD_NUM = 8  # GRBM_GUI_ACTIVE comes summed over the XCDs: 8 x the dispatch's clock cycles


def sq_lines(paths):
    """Shader-sequencer counters of the pair kernels and the ratios read from them.  SQ_WAVE_CYCLES,
    SQ_ACTIVE_INST_ANY and the SQ_WAIT_* counters are quad-cycles summed over the waves (their
    ratios are shares of a wave's lifetime); SQ_INSTS_* count instructions; GRBM_GUI_ACTIVE / 8 is
    the dispatch's length in clock cycles."""
    merged = collections.defaultdict(dict)
    for p in paths:
        for key, cs in counters_per_dispatch(p).items():
            merged[key].update(cs)
    out = ["", "shader counters (--pmc SQ_*, GRBM_GUI_ACTIVE; per dispatch)"]
    for key in sorted(merged):
        k, n, wg, wx = key
        if not k.startswith(("pair_", "rotate_")):
            continue
        c = merged[key]
        out.append(f"  {k} N={n} WGs={wg} threads={wx}")
        for name in sorted(c):
            out.append(f"    {name:24s} {c[name]:16.6g}")
        ratios = []
        gui = c.get("GRBM_GUI_ACTIVE")
        if gui:
            cycles = gui / XCD_NUM
            simd_cycles = 4 * CU_NUM * cycles
            ratios.append(f"dispatch length {cycles:.4g} cycles")
            if "SQ_INSTS_VALU" in c:
                ratios.append(f"VALU instructions per SIMD per cycle {c['SQ_INSTS_VALU'] / simd_cycles:.3f} (a wave64 "
                              f"fp32 instruction takes 2 cycles: limit 0.5)")
            if "SQ_INSTS_LDS" in c:
                ratios.append(f"LDS instructions per CU per cycle {c['SQ_INSTS_LDS'] / (CU_NUM * cycles):.3f}")
            if "SQ_LDS_BANK_CONFLICT" in c:
                ratios.append(f"LDS bank-conflict stall cycles per CU cycle "
                              f"{c['SQ_LDS_BANK_CONFLICT'] / (CU_NUM * cycles):.3f}")
        wc = c.get("SQ_WAVE_CYCLES")
        if wc:
            for name, label in (("SQ_ACTIVE_INST_ANY", "issuing"), ("SQ_WAIT_INST_ANY", "waiting to issue"),
                                ("SQ_WAIT_INST_LDS", "waiting to issue LDS"),
                                ("SQ_WAIT_ANY", "waiting on a dependency or barrier")):
                if name in c:
                    ratios.append(f"share of wave time {label} {c[name] / wc:.3f}")
        out += [f"    -> {r}" for r in ratios]
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--command", action="append", default=[])
    ap.add_argument("--top", type=int, default=0, help="list only the kernels with the largest total time")
    ap.add_argument("--sq", action="append", default=[],
                    help="a `--pmc` database of shader-sequencer counters (repeatable: one per pass)")
    ap.add_argument("--bench-json", help="JSON line printed by the profiled bench run: its source_digest is "
                                         "recorded (default: the digest of the sources as they are now)")
    args = ap.parse_args()
    digest = source_digest()
    if args.bench_json:
        with open(args.bench_json) as fh:
            digest = json.loads(fh.read().strip().splitlines()[-1])["source_digest"]
    out = []
    out.append("commands (from the repository root, TMPDIR=/tmp):")
    out += [f"  {c}" for c in args.command]
    out.append("")
    agg, meta = trace_stats(args.trace)
    out.append("kernel trace (--kernel-trace --stats): average duration per dispatch")
    out.append(f"  {'kernel':28s} {'N':>6s} {'WGs':>6s} {'threads':>7s} {'calls':>5s} {'avg_us':>10s} "
               f"{'total_ms':>9s} {'scratch_B':>9s}")
    keys = sorted(agg, key=lambda k: (-sum(agg[k]), k))
    if args.top:
        rest = keys[args.top:]
        keys = keys[:args.top]
    for key in keys:
        k, n, wg, wx = key
        v = agg[key]
        out.append(f"  {k:28s} {n:6d} {wg:6d} {wx:7d} {len(v):5d} {sum(v) / len(v) / 1e3:10.2f} "
                   f"{sum(v) / 1e6:9.3f} {meta[key]:9d}")
    if args.top and rest:
        out.append(f"  ({len(rest)} more kernel shapes, {sum(sum(agg[k]) for k in rest) / 1e6:.3f} ms in total)")
    traffic = None
    if args.fetch and args.write and args.copy_fetch and args.copy_write:
        fetch = counter_per_dispatch(args.fetch, "FETCH_SIZE")
        write = counter_per_dispatch(args.write, "WRITE_SIZE")
        cf = [v for (k, *_), v in counter_per_dispatch(args.copy_fetch, "FETCH_SIZE").items() if "copyBuffer" in k]
        cw = [v for (k, *_), v in counter_per_dispatch(args.copy_write, "WRITE_SIZE").items() if "copyBuffer" in k]
        f_fac = COPY_BYTES / 1024 / cf[0]
        w_fac = COPY_BYTES / 1024 / cw[0]
        out.append("")
        out.append(f"HBM counters (--pmc FETCH_SIZE, --pmc WRITE_SIZE; KiB per dispatch)")
        out.append(f"  calibration: 256 MiB device copy reads FETCH_SIZE={cf[0]:.6g} KiB, WRITE_SIZE={cw[0]:.6g} KiB"
                   f" -> factors {f_fac:.4f} (fetch), {w_fac:.4f} (write)")
        out.append(f"  {'kernel':28s} {'N':>6s} {'WGs':>6s} {'FETCH_KiB':>11s} {'WRITE_KiB':>11s} {'bytes(cal)':>12s}")
        traffic = {"digest": digest, "fetch_factor": f_fac, "write_factor": w_fac, "bytes": {}}
        for key in sorted(set(fetch) & set(write)):
            k, n, wg, wx = key
            b = fetch[key] * 1024 * f_fac + write[key] * 1024 * w_fac
            out.append(f"  {k:28s} {n:6d} {wg:6d} {fetch[key]:11.1f} {write[key]:11.1f} {b:12.4g}")
            if k.startswith(("pair_", "rotate_")):
                traffic["bytes"][f"{k}|{n}/{wg}"] = b
    if args.sq:
        out += sq_lines(args.sq)
    print("\n".join(out))
    if traffic is not None:
        print("TRAFFIC_JSON " + json.dumps(traffic, sort_keys=True))
    return 0


if __name__ == "__main__":
    sys.exit(main())
