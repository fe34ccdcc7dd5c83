"""Per-kernel HBM traffic and matrix-core utilisation from rocprofv3 counter
passes over ``bench.py``.

Three passes of the same short bench command, each with one counter group
(rocprofv3 does not split counters over passes)::

    B="python3 bench.py --steps 2 --warmup 1 --no-extras --no-cpu-baseline \\
       --copy-calibration-mib 256"
    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/fetch -o run -- $B
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/write -o run -- $B
    rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE \\
        SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_BUSY_CYCLES --output-format csv \\
        -d OUT/mfma -o run -- $B
    python3 traffic.py --fetch OUT/fetch --write OUT/write \\
        --mfma OUT/mfma --key cfg2:carry:4

``--copy-calibration-mib 256`` makes the bench run one plain device copy of
256 MiB (256 MiB read, 256 MiB written) before the steps; the byte counters
are scaled by known / measured for that copy. The result is merged into
``profiles/traffic.json`` (bytes per launch per kernel, tagged with the hash
of the kernel sources so that bench.py ignores figures taken from older
kernels) and a summary table is printed.
"""
from __future__ import annotations

import argparse
import csv
import json
import os
import re
from collections import defaultdict

ROOT = os.path.dirname(os.path.abspath(__file__))
SIMDS = 256 * 4  # gfx950: 256 CUs x 4 SIMDs
XCDS = 8


def _rows(d):
    return list(csv.DictReader(open(os.path.join(d, "run_counter_collection.csv"))))


def bench_name(mangled: str) -> str:
    """rocprofv3's kernel name -> the name bench.py's per-kernel table uses."""
    n = re.sub(r"\(.*", "", mangled).replace("void ", "").replace("lrcnn::", "")
    n = n.replace("unsigned short", "bf16")
    m = re.match(r"conv_gemm_kernel<(\w+), (\d+), \d+, (true|false), (true|false), "
                 r"(true|false)(?:, (true|false))?", n)
    if m:
        kind = ("scalar" if m.group(4) != "true" else
                "1x1" if m.group(6) == "true" else "vec")
        return (f"conv_gemm_kernel<{m.group(1)}, {m.group(2)}, "
                f"{'dgrad' if m.group(3) == 'true' else 'fwd'}, {kind}>")
    if re.match(r"wgrad_rowg_kernel<\d+>", n):
        return "wgrad_kernel<bf16, vec>"
    m = re.match(r"wgrad_kernel<(\w+), (?:\d+, )?(true|false), (true|false)(?:, \d+)?>", n)
    if m:
        vec = m.group(2) == "true" and m.group(3) == "true"
        return f"wgrad_kernel<{m.group(1)}, {'vec' if vec else 'scalar'}>"
    for short in ("conv_split_epilogue", "wgrad_reduce_kernel"):
        if n.startswith(short):
            return short
    return n


def per_dispatch(rows, counter):
    out = {}
    for r in rows:
        if r["Counter_Name"] == counter:
            out[int(r["Dispatch_Id"])] = (r["Kernel_Name"], int(r["Grid_Size"]),
                                          float(r["Counter_Value"]))
    return out


def calibration(disp, known_kib):
    """Scale factor from the largest device-copy dispatch."""
    best = None
    for name, grid, val in disp.values():
        if "copyBuffer" in name and (best is None or val > best):
            best = val
    if not best:
        raise SystemExit("no calibration copy found (run bench.py with --copy-calibration-mib)")
    return known_kib / best, best


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--mfma")
    ap.add_argument("--copy-mib", type=int, default=256)
    ap.add_argument("--key", required=True, help="workload key, e.g. cfg2:carry:4")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "traffic.json"))
    args = ap.parse_args()

    fetch = per_dispatch(_rows(args.fetch), "FETCH_SIZE")
    write = per_dispatch(_rows(args.write), "WRITE_SIZE")
    known = args.copy_mib * 1024.0
    ff, fraw = calibration(fetch, known)
    fw, wraw = calibration(write, known)
    agg = defaultdict(lambda: [0, 0.0, 0.0])
    for d, (name, grid, fv) in fetch.items():
        if d not in write or write[d][0] != name or write[d][1] != grid:
            raise SystemExit(f"dispatch {d} differs between the two passes")
        if not name.startswith("void lrcnn::") and "lrcnn::" not in name:
            continue
        a = agg[bench_name(name)]
        a[0] += 1
        a[1] += fv * ff * 1024.0
        a[2] += write[d][2] * fw * 1024.0

    mf = {}
    if args.mfma:
        mrows = _rows(args.mfma)
        busy = per_dispatch(mrows, "SQ_VALU_MFMA_BUSY_CYCLES")
        gui = per_dispatch(mrows, "GRBM_GUI_ACTIVE")
        mops = per_dispatch(mrows, "SQ_INSTS_VALU_MFMA_MOPS_F32")
        mops.update(per_dispatch(mrows, "SQ_INSTS_VALU_MFMA_MOPS_BF16"))
        ma = defaultdict(lambda: [0.0, 0.0, 0.0])
        for d, (name, grid, b) in busy.items():
            if "lrcnn::" not in name:
                continue
            e = ma[bench_name(name)]
            e[0] += b
            e[1] += gui[d][2] / XCDS  # GRBM_GUI_ACTIVE is summed over the XCDs
            e[2] += mops[d][2] * 512.0 if d in mops else 0.0
        for k, (b, g, fl) in ma.items():
            mf[k] = {"mfma_busy_pct": round(100.0 * b / (g * SIMDS), 1) if g else None,
                     "mfma_flops_executed": fl}

    from bench import kernel_source_hash  # noqa: E402 (repo root on sys.path)
    h = kernel_source_hash()
    table = json.load(open(args.out)) if os.path.exists(args.out) else {}
    table["_calibration"] = {
        "copy_mib": args.copy_mib, "fetch_kib_measured": fraw, "write_kib_measured": wraw,
        "fetch_factor": round(ff, 4), "write_factor": round(fw, 4)}
    print(f"calibration: copy of {args.copy_mib} MiB -> FETCH_SIZE {fraw:.0f} KiB "
          f"(factor {ff:.3f}), WRITE_SIZE {wraw:.0f} KiB (factor {fw:.3f})")
    print(f"{'kernel':44s} {'launches':>8s} {'read MB/l':>10s} {'write MB/l':>10s} "
          f"{'MFMA busy %':>11s}")
    for k, (n, rb, wb) in sorted(agg.items(), key=lambda kv: -(kv[1][1] + kv[1][2])):
        ent = {"launches": n, "read_bytes_per_launch": rb / n,
               "write_bytes_per_launch": wb / n, "bytes_per_launch": (rb + wb) / n,
               "source_hash": h}
        ent.update(mf.get(k, {}))
        table[f"{args.key}:{k}"] = ent
        busy_s = f"{mf[k]['mfma_busy_pct']:>11}" if k in mf else f"{'':>11s}"
        print(f"{k:44s} {n:8d} {rb / n / 1e6:10.3f} {wb / n / 1e6:10.3f} {busy_s}")
    with open(args.out, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
    print("wrote", args.out)


if __name__ == "__main__":
    import sys
    sys.path.insert(0, ROOT)
    main()
