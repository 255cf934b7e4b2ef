"""MoE-layer benchmark on one MI355X.

One step = one pass of the whole hot path over one batch: top-k routing
(moe_route: gate logits, softmax, top-k, routing tables) followed by the MoE
layer (moe_forward: dispatch, GEMM0 + SiLU*up, GEMM1, combine) in the
dynamic-split megakernel.  Inputs are resident in HBM before timing starts.

Prints one JSON line.  `value` is tokens/s of whole steps; `layer_us` is the
MoE-layer time alone (the megakernel, from HIP events on its launch stream,
the window the paper times: end of routing to end of combine).  `baselines`
holds the static-split and serial modes and the dynamic mode again, all timed
as back-to-back forward launches in interleaved rounds; `dynamic_speedup` is a
baseline's time over the dynamic time measured that way.  `roofline` rates the
megakernel (the dominant kernel) against the bf16 MFMA peak; `phases` comes
from one extra traced launch after the timed region and gives the movement
workers' HBM rate, the compute workers' MFMA utilisation, and SM Active and
movement/compute overlap (paper_2609_21483_amd.timeline).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "MoE-layer µs + tokens/s at 1 GPU; HBM GB/s & MFMA util vs peak"
# sources of the megakernel: a traffic figure measured on other sources is stale
KERNEL_SOURCES = ("paper_2609_21483_amd/csrc/forward.hip", "paper_2609_21483_amd/csrc/gemm.h",
                  "paper_2609_21483_amd/csrc/common.h", "paper_2609_21483_amd/csrc/kernels.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "megakernel_traffic.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixtral_ep4")
    ap.add_argument("--layer", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=128)
    ap.add_argument("--modes", default="static,serial", help="baselines timed next to the dynamic mode")
    ap.add_argument("--rounds", type=int, default=3, help="interleaved rounds of the baseline comparison")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run a plain torch copy of this many MiB (the scale for PMC byte counters)")
    return ap.parse_args()


def kernel_sources_hash() -> str:
    """Hash of the megakernel's sources with comments and whitespace removed,
    so that an edit of comments alone keeps a traffic measurement valid."""
    import re
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), encoding="utf-8") as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update("".join(src.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per megakernel launch from the committed PMC measurement, or
    None when there is none for this workload or the kernel changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    rec = d.get(workload)
    if not rec or rec.get("sources") != kernel_sources_hash():
        return None
    return float(rec["bytes_per_launch"])


def time_forward(B, layer, x, idx, w, y, mode, steps, warmup, stream):
    import torch
    for _ in range(warmup):
        layer.forward(x, idx, w, y, mode, stream=stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        layer.forward(x, idx, w, y, mode, stream=stream)
        b.record(stream)
    torch.cuda.synchronize()
    st = B.moe_sync_status(layer.h, stream)
    if st != B.MOE_OK:
        raise RuntimeError(f"{mode}: {B.moe_last_error()}")
    return [a.elapsed_time(b) * 1e3 for a, b in ev]  # us


def traced_phases(B, layer, x, idx, w, y, stream, shape, stats, flops):
    """One traced launch: movement bytes over the movers' dispatch window and
    the compute workers' MFMA utilisation over their busy time."""
    import numpy as np
    import torch
    buf = torch.zeros(64 + 32 * (1 << 17), dtype=torch.uint8, device="cuda")
    B.moe_set_trace(layer.h, buf)
    try:
        layer.forward(x, idx, w, y, "dynamic", stream=stream)
        torch.cuda.synchronize()
    finally:
        B.moe_set_trace(layer.h, None)
    tr = B.read_trace(buf)
    wgs, tiles, disp, comb = (tr[tr["kind"] == k] for k in (1, 2, 3, 4))
    if len(wgs) == 0:
        return None
    t0 = wgs["t0"].min()
    us = lambda t: (t - t0) / 100.0
    H = shape.hidden
    X, U = int(stats[0]), int(stats[3] + stats[4])
    disp_bytes = (U + X) * 2.0 * H
    comb_bytes = (X + shape.tokens_per_rank * shape.n_shared_experts) * 2.0 * H + shape.T * 2.0 * H
    disp_end = float(us(disp["t1"]).max()) if len(disp) else float("nan")
    busy = float(((tiles["t2"] - tiles["t1"]) / 100.0).sum())
    n_comp = int((wgs["id"] == 0).sum())
    span = float(us(wgs["t2"]).max())
    comb_span = float((us(comb["t2"]).max() - us(comb["t1"]).min())) if len(comb) else float("nan")
    per_cu_peak = PEAK_BF16_TFLOPS / 256.0
    from paper_2609_21483_amd import timeline as TL
    tl = TL.metrics(tr)
    return {
        "traced_layer_us": span,
        "dispatch_us": disp_end,
        "dispatch_hbm_gbs": disp_bytes / (disp_end * 1e-6) / 1e9,
        "dispatch_frac_of_peak": disp_bytes / (disp_end * 1e-6) / 1e9 / PEAK_HBM_GBS,
        "combine_us": comb_span,
        "combine_hbm_gbs": comb_bytes / (comb_span * 1e-6) / 1e9,
        "compute_workers": n_comp,
        "compute_busy_frac": busy / (n_comp * span) if n_comp else None,
        "mfma_util_while_busy": flops / (busy * 1e-6) / 1e12 / per_cu_peak,
        "sm_active": tl["sm_active"],
        "overlap": tl["overlap"],
        "overlap_of_movement": tl["overlap_of_mov"],
        "prologue_us": tl["prologue_us"],
        "note": "one traced launch (tracing adds overhead); dispatch includes rows moved by compute workers "
                "that steal movement while their tiles wait",
    }


def cpu_baseline(shape, c, rows_n):
    """The oracle as it stands, single-threaded, on a bounded sample: routing
    of every token (scaled to the sample's share) plus the layer for the first
    rows_n/R tokens of each rank."""
    import numpy as np
    from oracle import oracle as O
    from paper_2609_21483_amd import workloads as W

    xu = W.as_u16_numpy(c["x"])
    t0 = time.perf_counter()
    lg = O.gate_logits(xu, W.as_u16_numpy(c["wg"]), None if c["bias"] is None else c["bias"].numpy())
    idx, w = O.softmax_topk(lg, shape.top_k)
    tab = O.route_tables(idx, shape.n_src_ranks, shape.tokens_per_rank, 0, shape.n_local_experts)
    t_route = time.perf_counter() - t0
    per = max(1, rows_n // shape.n_src_ranks)
    rows = np.concatenate([r * shape.tokens_per_rank + np.arange(per) for r in range(shape.n_src_ranks)])
    t1 = time.perf_counter()
    O.layer_rows(xu, idx, w, *(W.as_u16_numpy(c[k]) for k in ("w1", "w3", "w2")),
                 *(W.as_u16_numpy(c[k]) for k in ("ws1", "ws3", "ws2")), Tr=shape.tokens_per_rank, rows=rows)
    t_rows = time.perf_counter() - t1
    n = rows.shape[0]
    t = t_route * n / shape.T + t_rows
    return {"value": n / t, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"routing+tables of all {shape.T} tokens ({t_route:.2f}s, scaled by {n}/{shape.T}) + "
                      f"layer rows of {n} tokens ({per} per rank, {t_rows:.2f}s), {tab.X} local pairs in total"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's share of the expert-parallel layer; --gpus {args.gpus} is not "
              "supported (this build runs on exactly one GPU)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2609_21483_amd import binding as B
    from paper_2609_21483_amd import workloads as W

    shape = W.WORKLOADS[args.workload]
    layer_id = args.layer
    torch.cuda.init()
    N = torch.cuda.get_device_properties(0).multi_processor_count
    print(f"[bench] workload {shape.name} layer {layer_id}: generating inputs", file=sys.stderr, flush=True)
    c = {"x": W.tokens(shape), "wg": W.gate(shape, layer_id), "bias": W.zipf_log_prior(shape, layer_id)}
    c["w1"], c["w3"], c["w2"] = W.experts(shape, layer_id)
    c["ws1"], c["ws3"], c["ws2"] = W.shared_experts(shape, layer_id)
    from paper_2609_21483_amd.calibrate import load_calib
    calib = load_calib(shape.name, N)
    layer = B.MoeLayer(shape, c["w1"], c["w3"], c["w2"], c["ws1"], c["ws3"], c["ws2"], calib=calib)
    stream = torch.cuda.current_stream()
    x = c["x"].cuda()
    wg = c["wg"].cuda()
    bias = None if c["bias"] is None else c["bias"].cuda()
    idx = torch.empty((shape.T, shape.top_k), dtype=torch.int32, device="cuda")
    w = torch.empty((shape.T, shape.top_k), dtype=torch.float32, device="cuda")
    y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    print("[bench] inputs resident; warmup", file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        layer.route(x, wg, bias, idx, w, stream=stream)
        layer.forward(x, idx, w, y, "dynamic", stream=stream)
    torch.cuda.synchronize()
    # timed region: whole steps, with events around each megakernel launch
    fwd_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in fwd_ev:
        layer.route(x, wg, bias, idx, w, stream=stream)
        a.record(stream)
        layer.forward(x, idx, w, y, "dynamic", stream=stream)
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = B.moe_sync_status(layer.h, stream)
    if st != B.MOE_OK:
        raise RuntimeError(B.moe_last_error())
    print("[bench] timed steps done", file=sys.stderr, flush=True)
    layer_us = [a.elapsed_time(b) * 1e3 for a, b in fwd_ev]
    ms_per_step = wall * 1e3 / args.steps
    plan = B.moe_get_plan(layer.h, stream)
    stats = layer.ws_view("stats", torch.int32, 16).cpu().numpy()
    X = int(stats[0])
    S, Tr, H, F = shape.n_shared_experts, shape.tokens_per_rank, shape.hidden, shape.ffn
    flops = (X + S * Tr) * 6.0 * H * F
    lat = float(np.median(layer_us))
    achieved = flops / (float(np.mean(layer_us)) * 1e-6) / 1e12

    # route alone (events), for the report
    r_ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    r_ev[0].record(stream)
    for _ in range(args.steps):
        layer.route(x, wg, bias, idx, w, stream=stream)
    r_ev[1].record(stream)
    torch.cuda.synchronize()
    route_us = r_ev[0].elapsed_time(r_ev[1]) * 1e3 / args.steps

    # the baselines next to the dynamic forward, timed the same way (forward
    # launches back to back on the same routing) in interleaved rounds, so
    # that clock drift spreads over all modes alike
    baselines = {}
    modes = [m for m in args.modes.split(",") if m]
    if modes:
        runs = {m: [] for m in ["dynamic"] + modes}
        for _ in range(args.rounds):
            for m in runs:
                runs[m] += time_forward(B, layer, x, idx, w, y, m, args.steps, 2, stream)
        dyn = float(np.median(runs["dynamic"]))
        baselines["dynamic_same_timing"] = {"layer_us_median": dyn}
        for m in modes:
            med = float(np.median(runs[m]))
            baselines[m] = {"layer_us_median": med, "tokens_per_s": shape.T / (med * 1e-6),
                            "dynamic_speedup": med / dyn}
        print(f"[bench] baselines done ({args.rounds} interleaved rounds)", file=sys.stderr, flush=True)
    phases = traced_phases(B, layer, x, idx, w, y, stream, shape, stats, flops)
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    out = {
        "metric": METRIC,
        "value": shape.T / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) tokens, N(0,0.02) weights, gate-logit routing)",
        "config": {"workload": f"{shape.name}: EP=4 rank share, E={shape.n_experts} k={shape.top_k} H={H} F={F}, "
                               f"{shape.n_local_experts} local experts, {shape.n_src_ranks} ranks x {Tr} tokens",
                   "tokens": shape.T, "local_pairs": X, "layer": layer_id},
        "layer_us": lat,
        "layer_us_p10_p90": [float(np.percentile(layer_us, 10)), float(np.percentile(layer_us, 90))],
        "layer_tokens_per_s": shape.T / (lat * 1e-6),
        "route_us": route_us,
        "plan": {"c": plan.c, "K": plan.K, "n_steal": plan.n_steal, "final_all": plan.final_all,
                 "t_pred_us": plan.t_pred_s * 1e6, "N": N, "calibrated": calib is not None},
        "baselines": baselines,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": measured_traffic(shape.name),
                     "kernel": "moe_megakernel", "flop_per_launch": flops,
                     "flop_per_unit": "6*H*F per routed (token, local expert) row and per shared-expert row"},
        "phases": phases,
        "context": "paper: 2.89x geomean MoE-layer speedup on 4xH100 SXM, EP=4, BF16 - different hardware and "
                   "baselines, not a target",
    }
    if not args.no_cpu_baseline:
        print("[bench] oracle CPU baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(shape, c, args.cpu_rows)
    layer.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
