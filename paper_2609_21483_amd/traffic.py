"""HBM traffic of the megakernel from rocprofv3 counter collections.

Two `rocprofv3 --pmc` passes over the same `bench.py --copy-probe-mib M`
command, one with FETCH_SIZE and one with WRITE_SIZE (KiB per dispatch), give
the counters of every launch of the megakernel and of the plain device copies
of M MiB that the bench runs last.  Each counter is scaled by what it reads
for the copy against the bytes the copy is known to read and write, so the
record holds bytes, not counter units.  The record is keyed by workload and
kernel and by the megakernel's sources (comments and whitespace removed), and
bench.py reports it as `roofline.traffic` only while those sources are
unchanged.

    python -m paper_2609_21483_amd.traffic --fetch F.csv --write W.csv \
        --copy-mib 1024 --key large_stack:moe_megakernel_stack [--tcc T.csv]
"""
from __future__ import annotations

import argparse
import csv
import json
import os
import statistics
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OUT = os.path.join(ROOT, "profiles", "megakernel_traffic.json")
COPY_KERNEL = "copy"  # the device copy of torch (the runtime's copyBuffer kernel)


def per_dispatch(path: str, counter: str) -> dict:
    """Counter value per dispatch, grouped by kernel name."""
    out: dict = {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return out


def find(groups: dict, needle: str) -> list:
    vals = [v for k, vs in groups.items() if needle in k for v in vs]
    if not vals:
        raise SystemExit(f"no dispatch of a kernel named like {needle!r} in the counter file")
    return vals


def copy_reading(groups: dict, nbytes: int) -> float:
    """The counter of the copy dispatches (the largest dispatches of a copy
    kernel, one per copy): their median."""
    cands = [v for k, vs in groups.items() if COPY_KERNEL in k.lower() for v in vs]
    big = sorted(cands)[-3:]
    if not big:
        raise SystemExit("no copy dispatch in the counter file (run the bench with --copy-probe-mib)")
    return statistics.median(big)


def main(argv=None) -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--tcc", default="", help="optional counter file with TCC_HIT_sum and TCC_MISS_sum")
    ap.add_argument("--copy-mib", type=int, required=True)
    ap.add_argument("--key", required=True, help="workload:kernel, e.g. large_stack:moe_megakernel_stack")
    ap.add_argument("--out", default=OUT)
    args = ap.parse_args(argv)
    sys.path.insert(0, ROOT)
    import bench

    workload, kernel = args.key.split(":")
    nb = args.copy_mib << 20
    fetch, write = per_dispatch(args.fetch, "FETCH_SIZE"), per_dispatch(args.write, "WRITE_SIZE")
    needle = f"moe::{kernel}("
    f_k, w_k = find(fetch, needle), find(write, needle)
    # a copy of nb bytes reads nb and writes nb
    f_scale = nb / (copy_reading(fetch, nb) * 1024.0)
    w_scale = nb / (copy_reading(write, nb) * 1024.0)
    fb = statistics.mean(f_k) * 1024.0 * f_scale
    wb = statistics.mean(w_k) * 1024.0 * w_scale
    rec = {"sources": bench.kernel_sources_hash(), "bytes_per_launch": fb + wb, "fetch_bytes": fb,
           "write_bytes": wb, "fetch_scale": f_scale, "write_scale": w_scale, "launches": len(f_k),
           "how": "rocprofv3 --pmc FETCH_SIZE, then --pmc WRITE_SIZE (KiB per dispatch), each scaled by the "
                  f"same counter on a {args.copy_mib} MiB device copy"}
    if args.tcc:
        hit, miss = find(per_dispatch(args.tcc, "TCC_HIT_sum"), needle), find(per_dispatch(args.tcc, "TCC_MISS_sum"), needle)
        rec["l2_hit_rate"] = statistics.mean(hit) / (statistics.mean(hit) + statistics.mean(miss))
    try:
        with open(args.out) as f:
            d = json.load(f)
    except (OSError, ValueError):
        d = {}
    d[args.key] = rec
    with open(args.out, "w") as f:
        json.dump(d, f, indent=1)
        f.write("\n")
    print(json.dumps({args.key: rec}, indent=1))


if __name__ == "__main__":
    main()
