"""Measures the cost model's hardware input on this GPU (paper section 3:
calibrated communication bandwidth and GEMM throughput curves, Fig 4a/b; the
chunked-GEMM efficiency of Fig 7a; the overlap ratio alpha of Eq 6).

    python -m paper_2609_21483_amd.calibrate --workload mixtral_ep4

For a workload share (layer 0, its own routing):
  BW(c)         = (W_dispatch + W_combine) / time of dispatch + combine run as
                  separate kernels on c workgroups (the volumes the cost model
                  uses, Eq 2-3 as counted on one GPU);
  TFLOPS(N - c) = W_comp / time of GEMM0 + GEMM1 on N - c workgroups (Eq 1);
  BW(N)         = the same movement on all N workgroups (the final combine
                  runs on every worker, section 4);
  eff_chunk(K)  = the megakernel's best time over c at K = 1 / its best time
                  over c at K, on a (c, K) grid of forced plans whose movement
                  workers steal GEMM tiles freely: the throughput the chunk
                  pipeline keeps in the megakernel itself, where chunk
                  boundaries add dependency waits and ragged row tiles that
                  GEMM-only runs do not show (their ratio, GEMM time at K = 1 /
                  GEMM time with the tiling of K chunks, is kept as eff_gemm);
  alpha         = least-squares fit of Eq 15 to the same grid.
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


def calibrate(workload: str, reps: int = 5, c_grid=None, log=print) -> dict:
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

        bw, fl = [], []
        for c in c_grid:
            t_m = _time(lambda: run(1 | 8, c), reps)
            t_c = _time(lambda: run(2 | 4, N - c), reps)
            bw.append(w_move / t_m)
            fl.append(w_comp / t_c)
            log(f"[calib] c={c:3d}: BW {bw[-1] / 1e9:8.1f} GB/s  TFLOPS(N-c) {fl[-1] / 1e12:7.1f}")
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
        eff = [min(1.0, best_k[0] / t) for t in best_k]
        log(f"[calib] eff_chunk {dict(zip(Ks, [round(e, 3) for e in eff]))}")

        def predict(alpha, ci, ki):
            t_comp = w_comp / (fl[ci] * eff[ki])
            t_comm = w_move / bw[ci]
            t_tail = (1 - alpha) * (X * 2.0 * H) / (bw_all * Ks[ki])
            return max(t_comp + t_tail, t_comm)

        alphas = np.linspace(0.0, 1.0, 101)
        errs = [sum((predict(a, ci, ki) - t) ** 2 for ci, ki, t in sweep) for a in alphas]
        alpha = float(alphas[int(np.argmin(errs))])
        best = min(sweep, key=lambda s: s[2])
        log(f"[calib] alpha {alpha:.2f}; measured best forced plan c={c_grid[best[0]]} K={Ks[best[1]]} "
            f"{best[2] * 1e6:.1f} us")
        static_c = max(1, min(N - 1, int(round(N * 20 / 132 / 8)) * 8))
        return {
            "workload": workload, "N": N, "c": c_grid, "bw": bw, "flops": fl, "K": Ks, "eff": eff,
            "alpha": alpha, "static_c": static_c, "literal": 0, "bw_all": bw_all, "steal_window": 1, "steal_ceil": 1,
            "eff_gemm": eff_gemm,
            "sweep": [[c_grid[ci], Ks[ki], t] for ci, ki, t in sweep],
            "device": torch.cuda.get_device_name(0), "date": time.strftime("%Y-%m-%d"),
        }
    finally:
        layer.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", nargs="+", default=["mixtral_ep4"])
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--out", default=CALIB_DIR, help="directory for the <workload>.json tables")
    args = ap.parse_args()
    os.makedirs(args.out, exist_ok=True)
    for wl in args.workload:
        print(f"[calib] {wl}", flush=True)
        d = calibrate(wl, args.reps, log=lambda s: print(s, flush=True))
        path = os.path.join(args.out, f"{wl}.json")
        with open(path, "w") as f:
            json.dump(d, f, indent=1)
        print(f"[calib] wrote {path}", flush=True)


if __name__ == "__main__":
    sys.exit(main())
