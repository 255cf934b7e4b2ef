"""Python face of the CPU oracle (ctypes over ``libmoe_oracle.so``).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg import this module.  The HIP path never does.

The arithmetic lives in ``moe_oracle.c`` (plain single-threaded C); this file
only marshals numpy arrays.  See ``moe_oracle.h`` for what each stage computes
and which part of the paper it follows.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "moe_oracle.c")
LIB = os.path.join(HERE, "libmoe_oracle.so")

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (single thread, no fast-math, no contraction)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        srcs = [os.path.join(HERE, f) for f in ("moe_oracle.c", "moe_oracle.h")]
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < max(os.path.getmtime(f) for f in srcs):
            build()
        L = C.CDLL(LIB)
        P = C.c_void_p
        i = C.c_int
        L.orc_gate_logits.argtypes = [P, P, P, i, i, i, P]
        L.orc_softmax_topk.argtypes = [P, i, i, i, P, P]
        L.orc_route_tables.argtypes = [P, i, i, i, i, i, i, P, P, P, P, P, P]
        L.orc_route_tables.restype = i
        L.orc_chunk_offsets.argtypes = [P, P, i, i, i, i, P]
        L.orc_dispatch.argtypes = [P, P, i, i, i, P]
        L.orc_expert_ffn.argtypes = [P, P, P, P, i, i, P]
        L.orc_layer_rows.argtypes = [P, P, P, P, P, P, P, P, P, i, i, i, i, i, i, i, P, i, P]
        L.orc_tile_count.argtypes = [P, i, i, i, i, i]
        L.orc_tile_count.restype = C.c_int64
        L.orc_plan.argtypes = [C.POINTER(PlanIn), C.POINTER(PlanOut)]
        L.orc_t_total.argtypes = [C.POINTER(PlanIn), i, i]
        L.orc_t_total.restype = C.c_double
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


# ---- routing -------------------------------------------------------------

def gate_logits(x_u16: np.ndarray, wg_u16: np.ndarray, bias: Optional[np.ndarray] = None) -> np.ndarray:
    x = _c(x_u16, np.uint16)
    wg = _c(wg_u16, np.uint16)
    T, H = x.shape
    H2, E = wg.shape
    assert H == H2
    b = None if bias is None else _c(bias, np.float32)
    out = np.empty((T, E), np.float32)
    lib().orc_gate_logits(_p(x), _p(wg), _p(b), T, H, E, _p(out))
    return out


def softmax_topk(logits: np.ndarray, k: int):
    lg = _c(logits, np.float32)
    T, E = lg.shape
    idx = np.empty((T, k), np.int32)
    w = np.empty((T, k), np.float64)
    lib().orc_softmax_topk(_p(lg), T, E, k, _p(idx), _p(w))
    return idx, w


@dataclass
class Tables:
    X: int
    cnt_rank: np.ndarray   # [El, R]
    uniq: np.ndarray       # [R]
    off: np.ndarray        # [El+1]
    slot: np.ndarray       # [T, k]
    inv: np.ndarray        # [X]
    first_slot: np.ndarray  # [T]

    @property
    def counts(self) -> np.ndarray:
        return self.cnt_rank.sum(axis=1)


def route_tables(idx: np.ndarray, R: int, Tr: int, e0: int, El: int) -> Tables:
    idx = _c(idx, np.int32)
    T, k = idx.shape
    assert T == R * Tr
    cnt_rank = np.empty((El, R), np.int32)
    uniq = np.empty(R, np.int32)
    off = np.empty(El + 1, np.int32)
    slot = np.empty((T, k), np.int32)
    inv = np.empty(max(1, T * k), np.int32)
    first = np.empty(T, np.int32)
    X = lib().orc_route_tables(_p(idx), T, k, R, Tr, e0, El, _p(cnt_rank), _p(uniq), _p(off),
                               _p(slot), _p(inv), _p(first))
    return Tables(X, cnt_rank, uniq, off, slot, inv[:X].copy(), first)


def chunk_offsets(tab: Tables, T: int, k: int, K: int) -> np.ndarray:
    El = tab.off.shape[0] - 1
    out = np.empty((El, K + 1), np.int32)
    inv = tab.inv if tab.X else np.zeros(1, np.int32)
    lib().orc_chunk_offsets(_p(_c(inv, np.int32)), _p(tab.off), T, k, El, K, _p(out))
    return out


def dispatch(x_u16: np.ndarray, tab: Tables, k: int) -> np.ndarray:
    x = _c(x_u16, np.uint16)
    H = x.shape[1]
    A = np.empty((tab.X, H), np.uint16)
    if tab.X:
        lib().orc_dispatch(_p(x), _p(_c(tab.inv, np.int32)), tab.X, k, H, _p(A))
    return A


# ---- expert FFN and combine ---------------------------------------------

def expert_ffn(a_u16: np.ndarray, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray) -> np.ndarray:
    a = _c(a_u16, np.uint16)
    w1 = _c(w1, np.uint16)
    w3 = _c(w3, np.uint16)
    w2 = _c(w2, np.uint16)
    H, F = w1.shape
    out = np.empty(H, np.float64)
    lib().orc_expert_ffn(_p(a), _p(w1), _p(w3), _p(w2), H, F, _p(out))
    return out


def layer_rows(x_u16, idx, w, w1, w3, w2, ws1=None, ws3=None, ws2=None, *, Tr: int,
               e0: int = 0, rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Layer output y (fp64) for the given token rows (all rows when None)."""
    x = _c(x_u16, np.uint16)
    idx = _c(idx, np.int32)
    w = _c(w, np.float64)
    T, H = x.shape
    k = idx.shape[1]
    w1 = _c(w1, np.uint16)
    w3 = _c(w3, np.uint16)
    w2 = _c(w2, np.uint16)
    El, H2, F = w1.shape
    assert H2 == H and w2.shape == (El, F, H)
    S = 0 if ws1 is None else ws1.shape[0]
    ws1 = None if ws1 is None else _c(ws1, np.uint16)
    ws3 = None if ws3 is None else _c(ws3, np.uint16)
    ws2 = None if ws2 is None else _c(ws2, np.uint16)
    rows = np.arange(T, dtype=np.int64) if rows is None else _c(rows, np.int64)
    y = np.empty((rows.shape[0], H), np.float64)
    lib().orc_layer_rows(_p(x), _p(idx), _p(w), _p(w1), _p(w3), _p(w2), _p(ws1), _p(ws3), _p(ws2),
                         k, Tr, H, F, e0, El, S, _p(rows), int(rows.shape[0]), _p(y))
    return y


# ---- cost model ------------------------------------------------------------

class PlanIn(C.Structure):
    _fields_ = [
        ("n_c", C.c_int), ("c", C.c_void_p), ("bw", C.c_void_p), ("flops", C.c_void_p),
        ("n_k", C.c_int), ("K", C.c_void_p), ("eff", C.c_void_p), ("alpha", C.c_double),
        ("N", C.c_int),
        ("w_comp", C.c_double), ("w_dispatch", C.c_double), ("w_combine", C.c_double),
        ("n_tiles", C.c_void_p), ("bw_all", C.c_double), ("steal_window", C.c_int),
        ("steal_ceil", C.c_int),
    ]


class PlanOut(C.Structure):
    _fields_ = [("c", C.c_int), ("K", C.c_int), ("n_steal", C.c_int), ("ci", C.c_int),
                ("ki", C.c_int), ("t_total", C.c_double)]


@dataclass
class Plan:
    c: int
    K: int
    n_steal: int
    ci: int
    ki: int
    t_total: float


class _PlanArgs:
    def __init__(self, c, bw, flops, K, eff, alpha, N, w_comp, w_dispatch, w_combine, n_tiles, bw_all=0.0,
                 steal_window=0, steal_ceil=0):
        self.c = _c(c, np.int32)
        self.bw = _c(bw, np.float64)
        self.flops = _c(flops, np.float64)
        self.K = _c(K, np.int32)
        self.eff = _c(eff, np.float64)
        self.n_tiles = _c(n_tiles, np.int64)
        assert self.c.shape == self.bw.shape == self.flops.shape
        assert self.K.shape == self.eff.shape == self.n_tiles.shape
        self.s = PlanIn(len(self.c), _p(self.c), _p(self.bw), _p(self.flops), len(self.K), _p(self.K),
                        _p(self.eff), float(alpha), int(N), float(w_comp), float(w_dispatch),
                        float(w_combine), _p(self.n_tiles), float(bw_all), int(steal_window),
                        int(steal_ceil))


def plan(c, bw, flops, K, eff, alpha, N, w_comp, w_dispatch, w_combine, n_tiles, bw_all=0.0, steal_window=0,
         steal_ceil=0) -> Plan:
    """Eq 5, 9, 10, 15, 16 over the (c, K) grid, then Eq 11-14 at (c*, K*).

    The defaults are the plain reading of the printed equations: the exposed
    tail moves at BW(c) (bw_all = 0), Eq 11's window holds W_dispatch +
    W_combine (steal_window = 0) and Eq 14's share is taken as whole tiles
    (steal_ceil = 0).  The other values are the readings for one GPU (see
    moe_oracle.h)."""
    a = _PlanArgs(c, bw, flops, K, eff, alpha, N, w_comp, w_dispatch, w_combine, n_tiles, bw_all, steal_window,
                  steal_ceil)
    o = PlanOut()
    lib().orc_plan(C.byref(a.s), C.byref(o))
    return Plan(o.c, o.K, o.n_steal, o.ci, o.ki, o.t_total)


def t_total(ci, ki, c, bw, flops, K, eff, alpha, N, w_comp, w_dispatch, w_combine, n_tiles, bw_all=0.0) -> float:
    a = _PlanArgs(c, bw, flops, K, eff, alpha, N, w_comp, w_dispatch, w_combine, n_tiles, bw_all)
    return lib().orc_t_total(C.byref(a.s), int(ci), int(ki))


def tile_count(rows_seg: np.ndarray, BM: int, nt0: int, nt1: int) -> int:
    """rows_seg: [n_seg, K] rows of each (segment, chunk)."""
    r = _c(rows_seg, np.int32)
    n_seg, K = r.shape
    return int(lib().orc_tile_count(_p(r), n_seg, K, BM, nt0, nt1))


# ---- whole-share helpers built from the stages above ----------------------

def volumes(tab: Tables, H: int, F: int, shared_rows: int, literal: bool = False):
    """Workload volumes of section 3.1.

    W_comp = (pairs + shared rows) * 6HF flop (Eq 1).  With ``literal`` the
    movement volumes are Eq 2-3 as printed (remote tokens only: unique remote
    tokens * 2H and remote pairs * 2H).  Otherwise every source rank's rows
    are moved (on one GPU rank 0's rows also go through the movement workers):
    unique tokens * 2H and pairs * 2H.
    """
    B = 2.0 * H
    X = float(tab.cnt_rank.sum())
    X_in = float(tab.cnt_rank[:, 1:].sum())
    U_in = float(tab.uniq[1:].sum())
    U_all = float(tab.uniq.sum())
    w_comp = (X + shared_rows) * 6.0 * H * F
    if literal:
        return w_comp, U_in * B, X_in * B
    return w_comp, U_all * B, X * B
