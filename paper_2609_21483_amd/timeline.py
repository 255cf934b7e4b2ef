"""Timeline metrics of one traced megakernel launch (moe_set_trace records).

The paper places overlap systems along two utilisation dimensions (section 2,
Fig 2): how busy the SMs are ("SM Active") and how much communication runs
alongside computation ("comm-comp overlap").  It gives no formulas; the
readings used here, on one GPU where movement is dispatch and combine:

  sm_active      = sum over workgroups of the time the workgroup executes a
                   GEMM tile (inputs ready .. finished) or has a wavefront
                   copying a dispatch unit (start .. end) or a combine unit
                   (inputs ready .. end), over N x layer time;
  overlap        = time during which some movement unit and some GEMM tile
                   run at once, over layer time;
  overlap_of_mov = the same time over the time some movement unit runs (the
                   share of movement hidden under computation).

Layer time runs from the first workgroup's entry to the last one's exit, so
the prologue (plan + schedule) counts as idle.  Times are in microseconds.
"""
from __future__ import annotations

import numpy as np

TICKS_PER_US = 100.0  # the device clock of the trace runs at 100 MHz


def _union(iv: np.ndarray) -> np.ndarray:
    """Sorted, disjoint union of [start, end) intervals (n x 2)."""
    if len(iv) == 0:
        return np.zeros((0, 2))
    iv = iv[np.argsort(iv[:, 0], kind="stable")]
    out = [list(iv[0])]
    for s, e in iv[1:]:
        if s <= out[-1][1]:
            out[-1][1] = max(out[-1][1], e)
        else:
            out.append([s, e])
    return np.array(out, dtype=np.float64)


def _length(u: np.ndarray) -> float:
    return float((u[:, 1] - u[:, 0]).sum()) if len(u) else 0.0


def _intersection(a: np.ndarray, b: np.ndarray) -> float:
    """Length of the intersection of two disjoint sorted unions."""
    i = j = 0
    tot = 0.0
    while i < len(a) and j < len(b):
        lo, hi = max(a[i, 0], b[j, 0]), min(a[i, 1], b[j, 1])
        if hi > lo:
            tot += hi - lo
        if a[i, 1] < b[j, 1]:
            i += 1
        else:
            j += 1
    return tot


def metrics(tr: np.ndarray) -> dict | None:
    """SM Active and overlap of one traced launch (read_trace output)."""
    wgs = tr[tr["kind"] == 1]
    if len(wgs) == 0:
        return None
    t0 = int(wgs["t0"].min())
    us = lambda t: (np.asarray(t, dtype=np.float64) - t0) / TICKS_PER_US
    layer = float(us(wgs["t2"]).max())
    tiles = tr[tr["kind"] == 2]
    mov = tr[(tr["kind"] == 4) | (tr["kind"] == 5)]
    comp_iv = np.stack([us(tiles["t1"]), us(tiles["t2"])], axis=1) if len(tiles) else np.zeros((0, 2))
    # a dispatch unit copies from its start; a combine unit from the moment
    # its row tiles are done (before that it waits)
    mov_start = np.where(mov["kind"] == 4, mov["t1"], mov["t0"])
    mov_iv = np.stack([us(mov_start), us(mov["t2"])], axis=1) if len(mov) else np.zeros((0, 2))
    C, M = _union(comp_iv), _union(mov_iv)
    both = _intersection(C, M)
    busy = 0.0
    for t in np.unique(wgs["ticket"]):
        sel_c = tiles["ticket"] == t
        sel_m = mov["ticket"] == t
        iv = np.concatenate([comp_iv[sel_c], mov_iv[sel_m]])
        busy += _length(_union(iv))
    n = len(wgs)
    movers = wgs[wgs["id"] == 1]
    return {
        "layer_us": layer,
        "prologue_us": float((us(wgs["t1"]) - us(wgs["t0"])).mean()),
        "sm_active": busy / (n * layer),
        "overlap": both / layer,
        "overlap_of_mov": both / _length(M) if len(M) else None,
        "movement_active_us": _length(M),
        "compute_active_us": _length(C),
        "workers": n,
        "movement_workers": int(len(movers)),
    }
