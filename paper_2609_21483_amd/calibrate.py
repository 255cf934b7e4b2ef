"""Measures the cost model's hardware input on this GPU (paper section 3:
calibrated communication bandwidth and GEMM throughput curves, Fig 4a/b; the
chunked-GEMM efficiency of Fig 7a; the overlap ratio alpha of Eq 6).

    python -m paper_2609_21483_amd.calibrate --workload mixtral_ep4

For a workload share (layer 0, its own routing):
  BW(c)         = (W_dispatch + W_combine) / time of dispatch + combine run as
                  separate kernels on c workgroups (the volumes the cost model
                  uses, Eq 2-3 as counted on one GPU);
  TFLOPS(N - c) = W_comp / time of GEMM0 + GEMM1 on N - c workgroups (Eq 1);
                  both measured in interleaved rounds over a shuffled c order
                  (medians), then made monotone (BW non-decreasing and
                  TFLOPS(N - c) non-increasing in c) by isotonic regression:
                  run-to-run noise of a few percent otherwise makes the curves
                  cross and decides c*;
  BW(N)         = the same movement on all N workgroups (the final combine
                  runs on every worker, section 4);
  eff_chunk(K), = identified together by linear least squares of Eq 15 on a
  alpha           grid of forced megakernel plans without bubble stealing
                  (n_steal = 0, the execution Eq 15 describes: GEMM on N - c
                  workers, the last combine after the last tile), over its
                  points that the model counts compute-bound: there
                  T = T_comp(c) / eff_chunk(K) + (1 - alpha) W_combine /
                  (BW_all K), linear in 1 / eff_chunk(K) and 1 - alpha.
                  Points the model counts communication-bound are left out:
                  on one GPU the compute workers copy rows themselves when
                  theirs are not dispatched yet (movement stealing), so few
                  movement workers are never the bound that Eq 8 predicts.
                  Also recorded: eff_total, the megakernel's best time over c
                  at K = 1 / its best time at K with free stealing (a whole-
                  layer ratio that already holds the 1/K tail of Eq 12, so
                  using it as eff_chunk counts that tail twice), and eff_gemm,
                  the ratio of GEMM-only runs.
The table is written to calib/<workload>.json and loaded by bench.py.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

from . import binding as B
from . import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
CALIB_DIR = os.path.join(HERE, "calib")


def calib_path(workload: str) -> str:
    return os.path.join(CALIB_DIR, f"{workload}.json")


def load_calib(workload: str, N: int):
    """The measured table for this workload and worker count, or None."""
    p = calib_path(workload)
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if int(d.get("N", -1)) != N:
        return None
    return B.make_calib(d["c"], d["bw"], d["flops"], d["K"], d["eff"], d["alpha"], d["static_c"], d.get("literal", 0),
                        d.get("bw_all", 0.0), d.get("steal_window", 1), d.get("steal_ceil", 1))


def _time(fn, reps: int) -> float:
    fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(reps):
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e-3)
    return float(np.median(ts))


def isotonic(y, increasing: bool):
    """Pool-adjacent-violators least-squares fit of a monotone sequence."""
    v = [float(t) for t in (y if increasing else [-t for t in y])]
    blocks = []  # [sum, count]
    for t in v:
        blocks.append([t, 1])
        while len(blocks) > 1 and blocks[-2][0] / blocks[-2][1] > blocks[-1][0] / blocks[-1][1]:
            s2, n2 = blocks.pop()
            blocks[-1][0] += s2
            blocks[-1][1] += n2
    out = []
    for s_, n_ in blocks:
        out += [s_ / n_] * n_
    return out if increasing else [-t for t in out]


def fit_eff_alpha(sweep0, Ks, w_comp, w_move, w_comb, fl, bw, bw_all):
    """eff_chunk(K) and alpha from Eq 15 on the compute-bound points of a
    no-stealing grid [(c index, K index, seconds)]: T = T_comp(c) u_K +
    W_combine / (BW_all K) v with u_1 = 1, u_K = 1 / eff_chunk(K), v = 1 -
    alpha; linear least squares, then eff clipped to (0, 1] and alpha to
    [0, 1).  Falls back to eff = 1, alpha = 0 where a K has no point.
    Returns (eff, alpha, points used, relative residuals, alpha before
    clipping)."""
    pts = []
    for ci, ki, t in sweep0:
        tc = w_comp / fl[ci]
        tl = w_comb / (bw_all * Ks[ki])
        if w_move / bw[ci] <= tc:  # compute-bound by the model (before the tail)
            pts.append((ki, tc, tl, t))
    nk = len(Ks)
    A, b = [], []
    for ki, tc, tl, t in pts:
        row = [0.0] * nk  # columns: u_2 .. u_K (nk - 1), then v
        if ki > 0:
            row[ki - 1] = tc
        row[nk - 1] = tl
        A.append(row)
        b.append(t - (tc if ki == 0 else 0.0))
    have = [any(ki == j for ki, *_ in pts) for j in range(nk)]
    if not pts or not have[0]:
        return [1.0] * nk, 0.0, len(pts), [0.0], None
    A, b = np.array(A), np.array(b)
    cols = [j - 1 for j in range(1, nk) if have[j]] + [nk - 1]
    sol, *_ = np.linalg.lstsq(A[:, cols], b, rcond=None)
    u = {j: 1.0 for j in range(nk)}
    for col, val in zip(cols[:-1], sol[:-1]):
        u[col + 1] = float(val)
    v = float(sol[-1])
    eff = [min(1.0, 1.0 / u[j]) if u[j] > 0 else 1.0 for j in range(nk)]
    alpha = float(min(0.999, max(0.0, 1.0 - v)))
    resid = [((tc / eff[ki]) + (1 - alpha) * tl - t) / t for ki, tc, tl, t in pts]
    return eff, alpha, len(pts), resid, 1.0 - v


def calibrate(workload: str, reps: int = 5, c_grid=None, log=print, rounds: int = 3) -> dict:
    shape = W.WORKLOADS[workload]
    N = torch.cuda.get_device_properties(0).multi_processor_count
    c_grid = c_grid or [c for c in range(8, 129, 8) if c < N]
    x = W.tokens(shape)
    wg = W.gate(shape, 0)
    bias = W.zipf_log_prior(shape, 0)
    w1, w3, w2 = W.experts(shape, 0)
    ws = W.shared_experts(shape, 0)
    layer = B.MoeLayer(shape, w1, w3, w2, *ws)
    try:
        xd = x.cuda()
        idx = torch.empty((shape.T, shape.top_k), dtype=torch.int32, device="cuda")
        w = torch.empty((shape.T, shape.top_k), dtype=torch.float32, device="cuda")
        y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        layer.route(xd, wg.cuda(), None if bias is None else bias.cuda(), idx, w)
        layer.forward(xd, idx, w, y, "serial")
        torch.cuda.synchronize()
        st = layer.ws_view("stats", torch.int32, 16).cpu().numpy()
        X, U = int(st[0]), int(st[3] + st[4])
        H, F = shape.hidden, shape.ffn
        w_comp = (X + shape.n_shared_experts * shape.tokens_per_rank) * 6.0 * H * F
        w_move = (U + X) * 2.0 * H
        run = lambda stages, n, K=1: B.moe_run_stages(layer.h, xd, idx, w, layer.packed, y, stages, n, K)

        tm = {c: [] for c in c_grid}
        tc = {c: [] for c in c_grid}
        rng = np.random.default_rng(0)
        for _ in range(rounds):
            for c in rng.permutation(c_grid):
                c = int(c)
                tm[c].append(_time(lambda: run(1 | 8, c), reps))
                tc[c].append(_time(lambda: run(2 | 4, N - c), reps))
        bw_raw = [w_move / float(np.median(tm[c])) for c in c_grid]
        fl_raw = [w_comp / float(np.median(tc[c])) for c in c_grid]
        bw = isotonic(bw_raw, increasing=True)
        fl = isotonic(fl_raw, increasing=False)
        for i, c in enumerate(c_grid):
            log(f"[calib] c={c:3d}: BW {bw_raw[i] / 1e9:8.1f} -> {bw[i] / 1e9:8.1f} GB/s  "
                f"TFLOPS(N-c) {fl_raw[i] / 1e12:7.1f} -> {fl[i] / 1e12:7.1f}")
        # the rate of all N workers moving together (the final combine)
        bw_all = w_move / _time(lambda: run(1 | 8, N), reps)
        log(f"[calib] all {N} workers: BW {bw_all / 1e9:8.1f} GB/s")
        Ks = [1, 2, 4, 8]
        t_k = [_time(lambda: run(2 | 4, N, K), reps) for K in Ks]
        eff_gemm = [min(1.0, t_k[0] / t) for t in t_k]
        log(f"[calib] GEMM-only chunk efficiency {dict(zip(Ks, [round(e, 3) for e in eff_gemm]))}")

        # the megakernel over a (c, K) grid of forced plans, movement workers
        # stealing GEMM tiles freely after dispatch
        steal_all = 1 << 20
        sweep = []
        for c in c_grid[:: max(1, len(c_grid) // 6)]:
            for K in Ks:
                p = B.moe_plan(c, K, steal_all, 1, 0.0)
                t = _time(lambda: layer.forward(xd, idx, w, y, "dynamic", forced=p), reps)
                sweep.append((c_grid.index(c), Ks.index(K), t))
        assert B.moe_sync_status(layer.h) == B.MOE_OK, B.moe_last_error()
        best_k = [min(t for _, ki, t in sweep if ki == j) for j in range(len(Ks))]
        eff_total = [min(1.0, best_k[0] / t) for t in best_k]
        log(f"[calib] whole-layer chunk ratio (free stealing) {dict(zip(Ks, [round(e, 3) for e in eff_total]))}")

        # the grid Eq 15 describes: no bubble stealing, the last combine on
        # every worker (section 4)
        sweep0 = []
        for c in c_grid[:: max(1, len(c_grid) // 6)]:
            for K in Ks:
                p = B.moe_plan(c, K, 0, 1, 0.0)
                t = _time(lambda: layer.forward(xd, idx, w, y, "dynamic", forced=p), reps)
                sweep0.append((c_grid.index(c), Ks.index(K), t))
        assert B.moe_sync_status(layer.h) == B.MOE_OK, B.moe_last_error()
        w_comb = X * 2.0 * H
        eff, alpha, n_fit, resid, alpha_raw = fit_eff_alpha(sweep0, Ks, w_comp, w_move, w_comb, fl, bw, bw_all)
        log(f"[calib] eff_chunk {dict(zip(Ks, [round(e, 3) for e in eff]))}, alpha {alpha:.3f} "
            f"(unclipped {alpha_raw if alpha_raw is None else round(alpha_raw, 3)}; fit over {n_fit} "
            f"compute-bound plans without stealing; residuals {min(resid) * 100:+.1f}% .. {max(resid) * 100:+.1f}%)")
        best = min(sweep, key=lambda s: s[2])
        log(f"[calib] measured best forced plan c={c_grid[best[0]]} K={Ks[best[1]]} {best[2] * 1e6:.1f} us")
        static_c = max(1, min(N - 1, int(round(N * 20 / 132 / 8)) * 8))
        return {
            "workload": workload, "N": N, "c": c_grid, "bw": bw, "flops": fl, "K": Ks, "eff": eff,
            "alpha": alpha, "static_c": static_c, "literal": 0, "bw_all": bw_all, "steal_window": 1, "steal_ceil": 1,
            "eff_gemm": eff_gemm, "eff_total": eff_total, "bw_raw": bw_raw, "flops_raw": fl_raw, "rounds": rounds,
            "w_comp": w_comp, "w_move": w_move, "w_combine": w_comb, "alpha_unclipped": alpha_raw,
            "fit_points": n_fit, "fit_residual_range": [min(resid), max(resid)],
            "sweep": [[c_grid[ci], Ks[ki], t] for ci, ki, t in sweep],
            "sweep_no_steal": [[c_grid[ci], Ks[ki], t] for ci, ki, t in sweep0],
            "device": torch.cuda.get_device_name(0), "date": time.strftime("%Y-%m-%d"),
        }
    finally:
        layer.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", nargs="+", default=["mixtral_ep4"])
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--rounds", type=int, default=3, help="interleaved rounds of the BW / TFLOPS curves")
    ap.add_argument("--out", default=CALIB_DIR, help="directory for the <workload>.json tables")
    args = ap.parse_args()
    os.makedirs(args.out, exist_ok=True)
    for wl in args.workload:
        print(f"[calib] {wl}", flush=True)
        d = calibrate(wl, args.reps, log=lambda s: print(s, flush=True), rounds=args.rounds)
        path = os.path.join(args.out, f"{wl}.json")
        with open(path, "w") as f:
            json.dump(d, f, indent=1)
        print(f"[calib] wrote {path}", flush=True)


if __name__ == "__main__":
    sys.exit(main())
