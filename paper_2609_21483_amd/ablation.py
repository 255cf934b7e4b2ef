"""Design ablation, cost-model accuracy and timeline metrics of the megakernel
on one GPU (the paper's design ablation of section 5, Fig 11; the prologue's
accuracy against an exhaustive (c, K) search, section 3.3; SM Active and
overlap, Fig 2).

    python -m paper_2609_21483_amd.ablation --workload mixtral_ep4 fine_zipf

For each workload share (layer 0, its own routing, the calibrated table):

  serial       w/o S+T: dispatch, GEMM0, GEMM1 and combine as four kernels on
               every CU, one after the other (no overlap);
  no_T         w/o T: the spatial split alone, c = the cost model's c*, K = 1,
               no bubble stealing, combine only on the movement workers;
  full         the prologue's plan (c*, K*, n_steal, final combine on every
               worker);
  static       a fixed split c = static_c (DeepEP's share of SMs), K = 1, no
               stealing;
  best_static  the fastest fixed split over the calibration grid, K = 1, no
               stealing (chosen in hindsight).

Accuracy: every (c, K) of the calibration grid runs as the cost model would
plan it there (the prologue evaluated on a one-point table picks that point's
n_steal and final combine); the exhaustive best is compared with the plan the
full table picks, gap = t(pick) / t(best) - 1.

Timeline: SM Active and overlap (timeline.metrics) from one traced launch of
full, no_T and static.  One JSON object per workload goes to stdout; --md
writes a markdown summary.
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np
import torch

from . import binding as B
from . import timeline as TL
from . import workloads as W
from .calibrate import _time, load_calib


def _traced(layer, x, idx, w, y, mode, forced=None) -> dict | None:
    buf = torch.zeros(64 + 32 * (1 << 18), dtype=torch.uint8, device="cuda")
    B.moe_set_trace(layer.h, buf)
    try:
        layer.forward(x, idx, w, y, mode, forced=forced)
        torch.cuda.synchronize()
    finally:
        B.moe_set_trace(layer.h, None)
    return TL.metrics(B.read_trace(buf))


def _interleaved(fns: dict, reps: int, rounds: int) -> dict:
    """Median over rounds of each configuration's median time; every round
    times every configuration once, so clock drift spreads over all of them."""
    res = {k: [] for k in fns}
    for _ in range(rounds):
        for k, fn in fns.items():
            res[k].append(_time(fn, reps))
    return {k: float(np.median(v)) for k, v in res.items()}


def run(workload: str, reps: int = 5, rounds: int = 3, log=print) -> dict:
    shape = W.WORKLOADS[workload]
    N = torch.cuda.get_device_properties(0).multi_processor_count
    d = load_calib(workload, N)
    if d is None:
        raise SystemExit(f"no calibration table for {workload} at N = {N}: run calibrate first")
    x = W.tokens(shape)
    wg = W.gate(shape, 0)
    bias = W.zipf_log_prior(shape, 0)
    w1, w3, w2 = W.experts(shape, 0)
    ws = W.shared_experts(shape, 0)
    layer = B.MoeLayer(shape, w1, w3, w2, *ws, calib=d)
    try:
        cal = B.moe_get_calib(layer.h)
        xd = x.cuda()
        idx = torch.empty((shape.T, shape.top_k), dtype=torch.int32, device="cuda")
        w = torch.empty((shape.T, shape.top_k), dtype=torch.float32, device="cuda")
        y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        layer.route(xd, wg.cuda(), None if bias is None else bias.cuda(), idx, w)
        st = layer.ws_view("stats", torch.int32, 16).cpu().numpy()
        X = int(st[0])
        flops = (X + shape.n_shared_experts * shape.tokens_per_rank) * 6.0 * shape.hidden * shape.ffn
        fwd = lambda mode, p=None: (lambda: layer.forward(xd, idx, w, y, mode, forced=p))

        layer.forward(xd, idx, w, y, "dynamic")
        pick = B.moe_get_plan(layer.h)
        no_t = B.moe_plan(pick.c, 1, 0, 0, 0.0)
        static = B.moe_plan(cal.static_c, 1, 0, 0, 0.0)
        cs = [cal.c[i] for i in range(cal.n_c)]
        Ks = [cal.k_chunks[j] for j in range(cal.n_k)]
        fns = {"serial": fwd("serial"), "full": fwd("dynamic"), "no_T": fwd("dynamic", no_t),
               "static": fwd("dynamic", static)}
        fns.update({("c", c): fwd("dynamic", B.moe_plan(c, 1, 0, 0, 0.0)) for c in cs})
        m = _interleaved(fns, reps, rounds)
        st_c = {c: m[("c", c)] for c in cs}
        best_static_c = min(st_c, key=st_c.get)
        t = {k: m[k] for k in ("serial", "full", "no_T", "static")}
        t["best_static"] = st_c[best_static_c]
        log(f"[ablation] {workload}: " + "  ".join(f"{k} {v * 1e6:.1f}" for k, v in t.items()) + " us")

        # every (c, K) as the cost model plans it there: the prologue on a
        # one-point table
        points = []
        for i, c in enumerate(cs):
            for j, K in enumerate(Ks):
                points.append((c, K, B.make_calib([c], [cal.bw_bytes_per_s[i]], [cal.comp_flop_per_s[i]], [K],
                                                  [cal.eff_chunk[j]], cal.alpha, cal.static_c, cal.literal_volumes,
                                                  cal.bw_all_bytes_per_s, cal.steal_window, cal.steal_ceil)))
        runs = {pt[:2]: [] for pt in points}
        plans = {}
        for _ in range(rounds):
            for c, K, one in points:
                B.moe_set_calib(layer.h, one)
                runs[(c, K)].append(_time(fwd("dynamic"), reps))
                plans[(c, K)] = B.moe_get_plan(layer.h)
        B.moe_set_calib(layer.h, cal)
        grid = [[c, K, plans[(c, K)].n_steal, plans[(c, K)].final_all, float(np.median(runs[(c, K)])) * 1e6,
                 plans[(c, K)].t_pred_s * 1e6] for c, K, _ in points]
        assert B.moe_sync_status(layer.h) == B.MOE_OK, B.moe_last_error()
        best = min(grid, key=lambda g: g[4])
        t_pick = next(g[4] for g in grid if g[0] == pick.c and g[1] == pick.K)
        log(f"[ablation] {workload}: pick c={pick.c} K={pick.K} {t_pick:.1f} us, exhaustive best c={best[0]} "
            f"K={best[1]} {best[4]:.1f} us, gap {t_pick / best[4] - 1:.3f}")

        tl = {"full": _traced(layer, xd, idx, w, y, "dynamic"),
              "no_T": _traced(layer, xd, idx, w, y, "dynamic", no_t),
              "static": _traced(layer, xd, idx, w, y, "dynamic", static)}
        assert B.moe_sync_status(layer.h) == B.MOE_OK, B.moe_last_error()
        us = {k: v * 1e6 for k, v in t.items()}
        return {
            "workload": workload, "N": N, "X": X, "gflop": flops / 1e9, "times_us": us,
            "plans": {"full": pick.as_tuple(), "no_T": no_t.as_tuple(), "static": static.as_tuple(),
                      "best_static": (best_static_c, 1, 0, 0)},
            "reduction": {"S": 1 - us["no_T"] / us["serial"], "T": 1 - us["full"] / us["no_T"],
                          "S+T": 1 - us["full"] / us["serial"]},
            "accuracy": {"pick": [pick.c, pick.K], "t_pick_us": t_pick, "best": best[:2], "t_best_us": best[4],
                         "gap": t_pick / best[4] - 1},
            "grid": grid, "timeline": tl, "device": torch.cuda.get_device_name(0),
        }
    finally:
        layer.close()


def markdown(results) -> str:
    out = ["| Workload | serial (w/o S+T) | w/o T | full | static | best static (c) | S | T | S+T |",
           "|---|---|---|---|---|---|---|---|---|"]
    for r in results:
        t, red = r["times_us"], r["reduction"]
        out.append(f"| {r['workload']} | {t['serial']:.1f} | {t['no_T']:.1f} (c {r['plans']['no_T'][0]}) | "
                   f"{t['full']:.1f} | {t['static']:.1f} | {t['best_static']:.1f} ({r['plans']['best_static'][0]}) | "
                   f"{red['S']:+.1%} | {red['T']:+.1%} | {red['S+T']:+.1%} |")
    out += ["", "| Workload | pick (c, K) | t pick µs | exhaustive best (c, K) | t best µs | gap |", "|---|---|---|---|---|---|"]
    for r in results:
        a = r["accuracy"]
        out.append(f"| {r['workload']} | {tuple(a['pick'])} | {a['t_pick_us']:.1f} | {tuple(a['best'])} | "
                   f"{a['t_best_us']:.1f} | {a['gap']:.1%} |")
    for r in results:
        # Fig 7b: the layer time over the (c, K) grid, each point run as the
        # cost model plans it there (its n_steal), next to the model's T_total
        g = {(c, K): (t, tp) for c, K, _, _, t, tp in r["grid"]}
        cs = sorted({c for c, _ in g})
        ks = sorted({K for _, K in g})
        best = min(g, key=lambda ck: g[ck][0])
        out += ["", f"(c, K) grid, {r['workload']}: measured µs (predicted T_total µs); fastest point in bold", "",
                "| c | " + " | ".join(f"K = {K}" for K in ks) + " |", "|---" * (len(ks) + 1) + "|"]
        for c in cs:
            cells = []
            for K in ks:
                t, tp = g[(c, K)]
                cell = f"{t:.1f} ({tp:.0f})"
                cells.append(f"**{cell}**" if (c, K) == best else cell)
            out.append(f"| {c} | " + " | ".join(cells) + " |")
    out += ["", "| Workload | plan | SM Active | overlap (of layer) | overlap (of movement) | prologue µs |",
            "|---|---|---|---|---|---|"]
    for r in results:
        for k, m in r["timeline"].items():
            if m:
                om = "–" if m["overlap_of_mov"] is None else f"{m['overlap_of_mov']:.1%}"
                out.append(f"| {r['workload']} | {k} | {m['sm_active']:.1%} | {m['overlap']:.1%} | {om} | "
                           f"{m['prologue_us']:.1f} |")
    return "\n".join(out) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", nargs="+", default=["mixtral_ep4"])
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--rounds", type=int, default=3)
    ap.add_argument("--md", default="", help="write a markdown summary to this file")
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("the ablation runs on the GPU")
    log = lambda s: print(s, file=sys.stderr, flush=True)
    results = []
    for wl in args.workload:
        r = run(wl, args.reps, args.rounds, log)
        print(json.dumps(r), flush=True)
        results.append(r)
    if args.md:
        with open(args.md, "w") as f:
            f.write(markdown(results))


if __name__ == "__main__":
    main()
