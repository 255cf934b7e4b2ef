"""MoE-layer benchmark on one MI355X.

One step = one pass of the whole hot path over one batch of T tokens through
the workload's stack of layers: for each layer, top-k routing (moe_route: gate
logits, softmax, top-k, routing tables) and then the MoE layer (moe_forward:
dispatch, GEMM0 + SiLU*up, GEMM1, combine) in the dynamic-split megakernel.
The default workload is the 8-layer large fine-grained stack (E=128, k=8,
H=4096, F=1536, 32 local experts, 4 source ranks x 8192 tokens, a Zipf
routing skew drawn per layer), the largest configuration that fits one GPU;
its layers are independent draws sharing one x and run back to back on one
stream.  Inputs are resident in HBM before timing starts.

Prints one JSON line.  `value` is tokens/s of whole steps (T tokens through
every layer of the stack, routing included).  `layers` gives each layer's
plan (c*, K*, n_steal), MoE-layer time (the megakernel, from HIP events on its
launch stream: the window the paper times, end of routing to end of combine),
its time with L2 and MALL flushed before each launch, routing time and the
static-split and serial baselines, all timed as back-to-back stacks in
interleaved rounds.  `roofline` rates the megakernel (the dominant kernel)
against the bf16 MFMA peak over the stack's launches; `phases` comes from one
extra traced launch per layer after the timed region.  `per_config` holds the
other workloads (one layer each).  `cpu_baseline` times the oracle on a
bounded sample of rows, single-threaded and on the host cores; the oracle's
sampled rows are then compared with the GPU's routing and y (`y_check`).
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
TOL = 2e-2  # max|y - y_ref| <= TOL * max|y_ref| over the checked rows


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large_stack")
    ap.add_argument("--layers", default="", help="comma list of layers of the stack (default: all)")
    ap.add_argument("--extra", default="tiny,mixtral_ep4,fine_zipf,shared_routed",
                    help="other workloads measured one layer each (per_config)")
    ap.add_argument("--modes", default="static,serial", help="baselines timed next to the dynamic mode")
    ap.add_argument("--rounds", type=int, default=3, help="interleaved rounds of the baseline comparison")
    ap.add_argument("--reps", type=int, default=5, help="stack runs per mode and round")
    ap.add_argument("--flush-mib", type=int, default=512, help="scratch written before each flushed launch")
    ap.add_argument("--no-trace", action="store_true")
    ap.add_argument("--no-stack", action="store_true",
                    help="run the layers of a timed step as one launch per layer (default: one stacked launch)")
    ap.add_argument("--route-streams", type=int, default=3,
                    help="streams (default priority) the layers of a step are routed on; the layers are independent")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=8, help="oracle rows per rank and layer, single-thread leg")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="wall time the host-cores leg of the CPU baseline is sized for")
    ap.add_argument("--no-ceiling", action="store_true", help="skip the dense-GEMM ceiling measurement")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run a plain torch copy of this many MiB (the scale for PMC byte counters)")
    return ap.parse_args()


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


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


class Stack:
    """The layers of one workload on the GPU: per layer a handle with its own
    workspace and packed weights, its gate and bias, and its routing and output
    buffers; x is shared by every layer."""

    def __init__(self, B, W, shape, layers, N, keep_host: bool):
        import torch
        from paper_2609_21483_amd.calibrate import load_calib
        self.shape, self.ids = shape, list(layers)
        self.calib = load_calib(shape.name, N)
        self.x_host = W.tokens(shape)
        self.x = self.x_host.cuda()
        self.L, self.host = [], []
        for l in self.ids:
            log(f"{shape.name} layer {l}: drawing and packing weights")
            wg, bias = W.gate(shape, l), W.zipf_log_prior(shape, l)
            ex, sh = W.experts(shape, l), W.shared_experts(shape, l)
            layer = B.MoeLayer(shape, *ex, *sh, calib=self.calib)
            d = dict(layer=layer, wg=wg.cuda(), bias=None if bias is None else bias.cuda(),
                     idx=torch.empty((shape.T, shape.top_k), dtype=torch.int32, device="cuda"),
                     w=torch.empty((shape.T, shape.top_k), dtype=torch.float32, device="cuda"),
                     y=torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda"))
            self.L.append(d)
            self.host.append(dict(wg=wg, bias=bias, ex=ex, sh=sh) if keep_host else None)
        torch.cuda.synchronize()

    def route(self, i, stream):
        d = self.L[i]
        d["layer"].route(self.x, d["wg"], d["bias"], d["idx"], d["w"], stream=stream)

    def forward(self, i, mode, stream):
        d = self.L[i]
        d["layer"].forward(self.x, d["idx"], d["w"], d["y"], mode, stream=stream)

    def forward_stacked(self, B, mode, stream):
        """Every layer in one persistent launch (moe_forward_stack)."""
        B.moe_forward_stack([d["layer"].h for d in self.L], self.x, [d["idx"] for d in self.L],
                            [d["w"] for d in self.L], [d["layer"].packed for d in self.L],
                            [d["y"] for d in self.L], B.MODES[mode], stream=stream)

    def check(self, B, stream):
        for d in self.L:
            st = B.moe_sync_status(d["layer"].h, stream)
            if st != B.MOE_OK:
                raise RuntimeError(B.moe_last_error())

    def close(self):
        import torch
        torch.cuda.synchronize()
        for d in self.L:
            d["layer"].close()
        self.L = []
        self.x = None
        torch.cuda.synchronize()


def time_stack(stack, mode, reps, stream):
    """Back-to-back stacks of forward launches on the current routing: per
    layer, the launch durations (us) from HIP events on the launch stream."""
    import torch
    n = len(stack.L)
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
          for _ in range(reps)]
    for r in range(reps):
        for i in range(n):
            ev[r][i][0].record(stream)
            stack.forward(i, mode, stream)
            ev[r][i][1].record(stream)
    torch.cuda.synchronize()
    return [[ev[r][i][0].elapsed_time(ev[r][i][1]) * 1e3 for r in range(reps)] for i in range(n)]


def time_stacked(B, stack, reps, stream):
    """Back-to-back stacked launches: the duration (us) of each."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record(stream)
        stack.forward_stacked(B, "dynamic", stream)
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e3 for a, b in ev]


def time_flushed(stack, reps, stream, flush):
    """Per layer, dynamic launches with L2 and MALL flushed before each one (a
    scratch write outside the events)."""
    import torch
    out = []
    for i in range(len(stack.L)):
        ts = []
        for _ in range(reps):
            flush.zero_()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            stack.forward(i, "dynamic", stream)
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        out.append(ts)
    return out


def traced_phases(B, stack, i, stream, stats, flops):
    """One traced launch: movement bytes over the movers' dispatch window and
    the compute workers' MFMA utilisation over their busy time."""
    import torch
    from paper_2609_21483_amd import timeline as TL
    d = stack.L[i]
    shape = stack.shape
    buf = torch.zeros(64 + 32 * (1 << 18), dtype=torch.uint8, device="cuda")
    B.moe_set_trace(d["layer"].h, buf)
    try:
        stack.forward(i, "dynamic", stream)
        torch.cuda.synchronize()
    finally:
        B.moe_set_trace(d["layer"].h, None)
    tr = B.read_trace(buf)
    del buf
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
    tl = TL.metrics(tr)
    gemm_end = float(us(tiles["t2"]).max()) if len(tiles) else float("nan")
    return {
        "first_tile_start_us": float(us(tiles["t1"]).min()) if len(tiles) else None,
        "last_tile_end_us": gemm_end,
        "tail_after_gemm_us": span - gemm_end,
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
    }


def serial_stages(B, stack, i, stream, reps=3):
    """The serial mode's four kernels timed one at a time on every worker
    (moe_run_stages: a stage reads what the earlier ones wrote, so this is
    timing only; the forward before it leaves every stage's inputs in place)."""
    import numpy as np
    import torch
    d = stack.L[i]
    n = torch.cuda.get_device_properties(0).multi_processor_count
    out = {}
    for name, mask in (("dispatch", 1), ("gemm0", 2), ("gemm1", 4), ("combine", 8)):
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            B.moe_run_stages(d["layer"].h, stack.x, d["idx"], d["w"], d["layer"].packed, d["y"], mask, n, 1, stream)
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        out[name] = float(np.median(ts))
    stack.forward(i, "dynamic", stream)  # leaves y and the tables as the timed forwards did
    torch.cuda.synchronize()
    return out


def layer_stats(stack, i):
    return stack.L[i]["layer"].ws_view("stats", __import__("torch").int32, 16).cpu().numpy()


def layer_flops(shape, stats):
    return (int(stats[0]) + shape.n_shared_experts * shape.tokens_per_rank) * 6.0 * shape.hidden * shape.ffn


def dense_ceiling(shape, rows: int, reps: int = 5):
    """The library bf16 GEMM (hipBLASLt through torch.matmul) on dense GEMMs
    of the layer's two expert products with all `rows` routed rows stacked:
    [rows, H] x [H, 2F] (gate and up) and [rows, F] x [F, H] (down), operands
    drawn like the layer's (x ~ N(0,1), weights ~ N(0, 0.02^2)).  The part is
    power-limited, and MFMA power depends on the operand bits, so this rate,
    not the nominal peak, is what a bf16 GEMM of these shapes reaches on this
    GPU.  Returns TFLOP/s of each product and of the two together."""
    import numpy as np
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(1234)
    H, F = shape.hidden, shape.ffn
    m = max(256, rows // 256 * 256)

    def rate(M, K, N):
        a = torch.randn(M, K, device="cuda", dtype=torch.float32, generator=g).to(torch.bfloat16)
        b = (torch.randn(K, N, device="cuda", dtype=torch.float32, generator=g) * 0.02).to(torch.bfloat16)
        for _ in range(2):
            torch.matmul(a, b)
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            torch.matmul(a, b)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        del a, b
        return float(np.median(ts))

    t0 = rate(m, H, 2 * F)
    t1 = rate(m, F, H)
    torch.cuda.empty_cache()
    f0, f1 = 4.0 * m * H * F, 2.0 * m * F * H
    return {"what": "torch.matmul (hipBLASLt) bf16 on the dense GEMMs of one layer's routed rows stacked: "
                    "[rows,H]x[H,2F] and [rows,F]x[F,H], random operands of the layer's distributions",
            "rows": m, "gemm0_tflops": f0 / t0 / 1e12, "gemm1_tflops": f1 / t1 / 1e12,
            "tflops": (f0 + f1) / (t0 + t1) / 1e12}


def host_info():
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    aff = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return {"cpu_model": model, "nproc": os.cpu_count(), "affinity_cpus": aff}


def cpu_baseline(stack, W, per_rank, cores, seconds):
    """The oracle as it stands on a bounded sample, timed on the host: for
    `per_rank` seeded tokens of each source rank and every layer of the stack,
    routing (gate logits, softmax, top-k of those rows: rows are independent)
    and the layer's output rows.  First on one thread, then on `cores`
    threads, each taking its own rows (the C oracle releases the interpreter
    lock, so the threads run in parallel), with as many rows as the
    single-thread rate says fill about `seconds` of wall time.  tokens/s =
    sampled tokens through all layers / wall time.  Returns the baseline and
    the oracle's rows of the single-thread leg (for the check against the
    GPU)."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oracle as O

    shape = stack.shape
    xu = W.as_u16_numpy(stack.x_host)
    Tr = shape.tokens_per_rank
    u16 = W.as_u16_numpy

    def run_rows(li, rows):
        hst = stack.host[li]
        lg = O.gate_logits(xu[rows], u16(hst["wg"]), None if hst["bias"] is None else hst["bias"].numpy())
        idx, w = O.softmax_topk(lg, shape.top_k)
        ws = [u16(t) for t in hst["sh"]]
        y = np.empty((len(rows), shape.hidden), np.float64)
        r0 = rows < Tr  # shared experts apply to rank-0 tokens
        for sel, tr in ((r0, int(r0.sum())), (~r0, 0)):
            if sel.any():
                y[sel] = O.layer_rows(xu[rows[sel]], idx[sel], w[sel], *(u16(t) for t in hst["ex"]), *ws, Tr=tr)
        return idx, w, y

    samples = [W.sample_tokens(shape, per_rank, seed=900 + l) for l in stack.ids]
    t0 = time.perf_counter()
    ref = [run_rows(i, rows) for i, rows in enumerate(samples)]
    t1 = time.perf_counter() - t0
    n1 = len(samples[0])
    # host cores: each thread takes its own rows of every layer, sized from
    # the single-thread rate to about `seconds` of wall time
    rate1 = len(samples[0]) / t1
    mt_rank = int(rate1 * cores * seconds / shape.n_src_ranks)
    mt_rank = max(per_rank, min(Tr, (mt_rank // cores) * cores))
    big = [W.sample_tokens(shape, mt_rank, seed=1900 + l) for l in stack.ids]
    shards = [[(i, b[c::cores]) for i, b in enumerate(big)] for c in range(cores)]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(cores) as ex:
        list(ex.map(lambda sh: [run_rows(i, r) for i, r in sh if len(r)], shards))
    tc = time.perf_counter() - t0
    nc = len(big[0])
    info = host_info()
    base = {"value": nc / tc, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{nc} seeded tokens ({nc // shape.n_src_ranks} per rank) through all {len(stack.ids)} "
                      f"layers (routing of those rows + the layer's output rows), {cores} threads, {tc:.1f} s",
            "single_thread": {"value": n1 / t1, "unit": "tokens/s", "cores": 1,
                              "sample": f"{n1} tokens through all {len(stack.ids)} layers, {t1:.1f} s"},
            **info}
    return base, samples, ref


def y_check(stack, samples, ref):
    """The oracle's sampled rows (from the CPU-baseline leg) against the GPU's
    routing and output of the last step, layer by layer."""
    import numpy as np
    worst, exact, n = 0.0, True, 0
    for i, (rows, (idx, w, y)) in enumerate(zip(samples, ref)):
        d = stack.L[i]
        sel = __import__("torch").from_numpy(rows).cuda()
        idx_g = d["idx"][sel].cpu().numpy()
        exact &= bool(np.array_equal(idx_g, idx))
        yg = d["y"][sel].float().cpu().numpy().astype(np.float64)
        m = float(np.max(np.abs(y)))
        worst = max(worst, float(np.max(np.abs(yg - y))) / (m if m > 0 else 1.0))
        n += len(rows)
    return {"rows": n, "layers": len(samples), "routing_ids_exact": exact, "max_err_over_max_ref": worst,
            "tolerance": TOL, "ok": bool(exact and worst <= TOL)}


def measure_stack(B, stack, args, stream, flush, trace: bool):
    """Timed steps, then the baselines, flushed launches and traces.  A step
    routes every layer and runs the MoE layers in one stacked launch (or, with
    --no-stack, one launch per layer)."""
    import numpy as np
    import torch
    n = len(stack.L)
    stacked = n > 1 and not args.no_stack

    def layers_forward():
        if stacked:
            stack.forward_stacked(B, "dynamic", stream)
        else:
            for i in range(n):
                stack.forward(i, "dynamic", stream)

    # the layers' routings are independent (each layer routes the same tokens
    # with its own gate): with several streams, one layer's small table
    # kernels and the last round of its chain kernel run beside the next
    # layer's routing; the stream of the MoE launch waits for all of them
    n_rs = max(1, min(args.route_streams, n))
    side = [torch.cuda.Stream() for _ in range(n_rs)] if n_rs > 1 else []

    def route_step():
        if not side:
            for i in range(n):
                stack.route(i, stream)
            return
        fork = torch.cuda.Event()
        fork.record(stream)
        for sd in side:
            sd.wait_event(fork)
        for i in range(n):
            stack.route(i, side[i % n_rs])
        for sd in side:
            join = torch.cuda.Event()
            join.record(sd)
            stream.wait_event(join)

    for _ in range(args.warmup):
        route_step()
        layers_forward()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    ev_r = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        ev_r[s].record(stream)
        route_step()
        ev[s][0].record(stream)
        layers_forward()
        ev[s][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    stack.check(B, stream)
    moe_us = [a.elapsed_time(b) * 1e3 for a, b in ev]  # the MoE layers of a step (one launch or n)
    step_route_us = [r.elapsed_time(a) * 1e3 for r, (a, _) in zip(ev_r, ev)]  # the routing of a step
    log(f"{stack.shape.name}: timed steps done ({wall * 1e3 / args.steps:.2f} ms per step)")
    plans = [B.moe_get_plan(d["layer"].h, stream) for d in stack.L]
    stats = [layer_stats(stack, i) for i in range(n)]
    flops = [layer_flops(stack.shape, st) for st in stats]
    # routing alone, per layer
    route_us = []
    for i in range(n):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(args.steps):
            stack.route(i, stream)
        b.record(stream)
        torch.cuda.synchronize()
        route_us.append(a.elapsed_time(b) * 1e3 / args.steps)
    # one launch per layer in each mode, and the stacked launch, timed the
    # same way (back to back on the same routing) in interleaved rounds
    modes = ["dynamic"] + [m for m in args.modes.split(",") if m]
    runs = {m: [[] for _ in range(n)] for m in modes}
    stacked_runs = []
    for _ in range(args.rounds):
        for m in modes:
            t = time_stack(stack, m, args.reps, stream)
            for i in range(n):
                runs[m][i] += t[i]
        if n > 1:
            stacked_runs += time_stacked(B, stack, args.reps, stream)
    stack.check(B, stream)
    log(f"{stack.shape.name}: baselines done ({args.rounds} interleaved rounds)")
    fl = time_flushed(stack, args.reps, stream, flush) if flush is not None else None
    layers = []
    for i in range(n):
        p = plans[i]
        dyn = runs["dynamic"][i]
        rec = {"layer": stack.ids[i], "plan": {"c": p.c, "K": p.K, "n_steal": p.n_steal, "final_all": p.final_all,
                                                "t_pred_us": p.t_pred_s * 1e6},
               "local_pairs": int(stats[i][0]), "gflop": flops[i] / 1e9,
               "route_exact_chains": int(stats[i][8]),
               "layer_us": float(np.median(dyn)),
               "layer_us_p10_p90": [float(np.percentile(dyn, 10)), float(np.percentile(dyn, 90))],
               "layer_us_flushed": float(np.median(fl[i])) if fl else None,
               "route_us": route_us[i],
               "tflops": flops[i] / (float(np.median(dyn)) * 1e-6) / 1e12}
        rec["baselines"] = {}
        for m in modes[1:]:
            med = float(np.median(runs[m][i]))
            rec["baselines"][m] = {"layer_us": med, "dynamic_speedup": med / rec["layer_us"]}
        if trace:
            rec["phases"] = traced_phases(B, stack, i, stream, stats[i], flops[i])
            rec["serial_stages_us"] = serial_stages(B, stack, i, stream)
        layers.append(rec)
    tot = {m: float(sum(np.median(runs[m][i]) for i in range(n))) for m in modes}
    summary = {
        "steps": args.steps, "ms_per_step": wall * 1e3 / args.steps,
        "moe_us_per_step": float(np.median(moe_us)),
        "moe_launches_per_step": 1 if stacked else n,
        "stack_flops": float(sum(flops)),
        "stack_route_us_total": float(sum(route_us)),
        "route_streams": n_rs,
        "route_us_per_step": float(np.median(step_route_us)),
        "one_launch_per_layer_us_total": tot,
        "dynamic_speedup_vs": {m: tot[m] / tot["dynamic"] for m in modes[1:]},
    }
    if stacked_runs:
        st_med = float(np.median(stacked_runs))
        summary["stacked_launch_us"] = st_med
        summary["stacked_speedup_vs"] = {("one_launch_per_layer_" + m): tot[m] / st_med for m in modes}
    return summary, layers


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's share of the expert-parallel layer; --gpus {args.gpus} is not "
              "supported: this benchmark runs on exactly one GPU", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2609_21483_amd import binding as B
    from paper_2609_21483_amd import workloads as W

    shape = W.WORKLOADS[args.workload]
    ids = [int(v) for v in args.layers.split(",") if v] or list(range(shape.n_layers))
    torch.cuda.init()
    N = torch.cuda.get_device_properties(0).multi_processor_count
    stream = torch.cuda.current_stream()
    flush = torch.empty(args.flush_mib << 20, dtype=torch.uint8, device="cuda") if args.flush_mib else None
    want_cpu = not args.no_cpu_baseline
    stack = Stack(B, W, shape, ids, N, keep_host=want_cpu)
    log(f"{shape.name}: inputs resident ({len(ids)} layers); warmup")
    summary, layers = measure_stack(B, stack, args, stream, flush, trace=not args.no_trace)

    n = len(ids)
    # the dominant kernel: the stacked megakernel (one launch holds every
    # layer), else the megakernel of the one layer
    launches = summary["moe_launches_per_step"]
    rs_txt = f" (on {summary['route_streams']} streams)" if summary["route_streams"] > 1 else ""
    flops_per_launch = summary["stack_flops"] / launches
    achieved = flops_per_launch / (summary["moe_us_per_step"] / launches * 1e-6) / 1e12
    kernel = "moe_megakernel_stack" if launches == 1 and n > 1 else "moe_megakernel"
    out = {
        "metric": METRIC,
        "value": shape.T / (summary["ms_per_step"] * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": summary["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) tokens, N(0,0.02) weights, gate-logit routing with a seeded per-layer "
                "Zipf log-prior)",
        "config": {"workload": f"{shape.name}: {n}-layer stack of EP=4 rank shares, E={shape.n_experts} "
                               f"k={shape.top_k} H={shape.hidden} F={shape.ffn}, {shape.n_local_experts} local "
                               f"experts, {shape.n_src_ranks} ranks x {shape.tokens_per_rank} tokens; a step is "
                               f"the routing of every layer{rs_txt}, then the MoE layers "
                               f"({'in one stacked launch' if launches == 1 and n > 1 else 'one launch per layer'})",
                   "tokens": shape.T, "layers": ids},
        "stack": {**summary, "moe_tokens_per_s": shape.T / (summary["moe_us_per_step"] * 1e-6)},
        "layers": layers,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": measured_traffic(f"{shape.name}:{kernel}"),
                     "kernel": kernel, "flop_per_launch": flops_per_launch,
                     "flop_per_unit": "6*H*F per routed (token, local expert) row and per shared-expert row, "
                                      "summed over the layers one launch holds"},
        "context": "paper: 2.89x geomean MoE-layer speedup on 4xH100 SXM, EP=4, BF16 - different hardware and "
                   "baselines, not a target",
    }
    if not args.no_ceiling:
        rows = int(round(summary["stack_flops"] / n / (6.0 * shape.hidden * shape.ffn)))
        ceil = dense_ceiling(shape, rows)
        ceil["megakernel_frac_of_ceiling"] = achieved / ceil["tflops"]
        out["roofline"]["ceiling"] = ceil
        log(f"dense GEMM ceiling: {ceil['tflops']:.0f} TFLOP/s; megakernel at {achieved:.0f}")
    if want_cpu:
        log("oracle CPU baseline")
        cores = max(1, min(16, host_info()["affinity_cpus"]))
        base, samples, ref = cpu_baseline(stack, W, args.cpu_rows, cores, args.cpu_seconds)
        out["cpu_baseline"] = base
        out["y_check"] = y_check(stack, samples, ref)
        log(f"y check: {out['y_check']}")
    stack.close()
    del stack

    per = {}
    for name in [w for w in args.extra.split(",") if w and w != shape.name]:
        sh = W.WORKLOADS[name]
        st = Stack(B, W, sh, [0], N, keep_host=False)
        sargs = argparse.Namespace(**{**vars(args), "steps": max(5, args.steps)})
        s, l = measure_stack(B, st, sargs, stream, flush, trace=False)
        per[name] = {"tokens": sh.T, "step_tokens_per_s": sh.T / (s["ms_per_step"] * 1e-3), **l[0]}
        st.close()
        del st
    out["per_config"] = per
    if args.copy_probe_mib:
        nb = args.copy_probe_mib << 20
        src = torch.empty(nb, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    del flush
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
