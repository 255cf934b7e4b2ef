"""Thin Python binding of the C ABI in include/moe.h (ctypes; marshalling only).

Every function here has the name of the C entry point it calls and does no
arithmetic of the layer: tensors are passed as device pointers, streams as
``torch.cuda.Stream.cuda_stream``.  PyTorch only provides device memory and
streams.  If ``libmoe.so`` is missing the import of this module fails; there is
no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
import re
from typing import Optional

import torch  # imported before libmoe.so so both bind the same HIP runtime

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "moe.h")

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_UNSUPPORTED = -2
MOE_ERR_HIP = -3
MOE_ERR_TIMEOUT = -4
MOE_ERR_ROUTING = -5
MOE_ERR_STATE = -6

MOE_WINDOW_PLAIN = 0
MOE_WINDOW_MOVE_STEAL = 1
MOE_WINDOW_LAST_COMBINE = 2

MOE_MODE_DYNAMIC = 0
MOE_MODE_STATIC = 1
MOE_MODE_SERIAL = 2
MODES = {"dynamic": MOE_MODE_DYNAMIC, "static": MOE_MODE_STATIC, "serial": MOE_MODE_SERIAL}

CALIB_MAX_C = 32
CALIB_MAX_K = 4


class moe_config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_src_ranks", "tokens_per_rank", "hidden", "ffn", "n_experts", "top_k",
        "n_local_experts", "first_local_expert", "n_shared_experts", "n_workers",
                                    "gemm1_split")]


class moe_calib(C.Structure):
    _fields_ = [
        ("n_c", C.c_int32), ("c", C.c_int32 * CALIB_MAX_C),
        ("bw_bytes_per_s", C.c_double * CALIB_MAX_C), ("comp_flop_per_s", C.c_double * CALIB_MAX_C),
        ("n_k", C.c_int32), ("k_chunks", C.c_int32 * CALIB_MAX_K), ("eff_chunk", C.c_double * CALIB_MAX_K),
        ("alpha", C.c_double), ("literal_volumes", C.c_int32), ("static_c", C.c_int32),
        ("bw_all_bytes_per_s", C.c_double), ("steal_window", C.c_int32), ("steal_ceil", C.c_int32),
    ]


class moe_plan(C.Structure):
    _fields_ = [("c", C.c_int32), ("K", C.c_int32), ("n_steal", C.c_int32), ("final_all", C.c_int32),
                ("t_pred_s", C.c_double)]

    def as_tuple(self):
        return (self.c, self.K, self.n_steal, self.final_all)


class moe_ws_layout(C.Structure):
    _fields_ = [(n, C.c_size_t) for n in (
        "total", "slot", "inv", "first_slot", "off", "sub_off", "row_off", "cnt_rank", "uniq", "stats", "plan",
        "err", "A", "Hbuf", "O")]


class MoeError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed ({status}): {msg}")
        self.status = status


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                      "(python -c 'import __graft_entry__ as g; g.build()')")

_lib = C.CDLL(LIB_PATH)
_P = C.c_void_p
_H = C.c_void_p  # moe_handle*
_SIGS = {
    "moe_init": ([C.POINTER(moe_config), C.POINTER(moe_calib), C.POINTER(_H)], C.c_int),
    "moe_destroy": ([_H], C.c_int),
    "moe_last_error": ([], C.c_char_p),
    "moe_set_calib": ([_H, C.POINTER(moe_calib)], C.c_int),
    "moe_get_calib": ([_H, C.POINTER(moe_calib)], C.c_int),
    "moe_set_timeout_ms": ([_H, C.c_double, C.c_int32], C.c_int),
    "moe_set_jitter": ([_H, C.c_uint32, C.c_int32], C.c_int),
    "moe_set_trace": ([_H, C.c_void_p, C.c_int64], C.c_int),
    "moe_workspace_size": ([_H, C.POINTER(C.c_size_t)], C.c_int),
    "moe_workspace_layout": ([_H, C.POINTER(moe_ws_layout)], C.c_int),
    "moe_set_workspace": ([_H, _P, C.c_size_t, _P], C.c_int),
    "moe_packed_weights_size": ([_H, C.POINTER(C.c_size_t)], C.c_int),
    "moe_pack_weights": ([_H, _P, _P, _P, _P, _P, _P, _P, _P], C.c_int),
    "moe_route": ([_H, _P, _P, _P, C.c_int32, _P, _P, _P], C.c_int),
    "moe_build_tables": ([_H, _P, _P], C.c_int),
    "moe_route_topk_static": ([C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P, _P, _P, _P, _P, _P], C.c_int),
    "moe_forward": ([_H, _P, _P, _P, _P, _P, C.c_int32, C.POINTER(moe_plan), _P], C.c_int),
    "moe_run_stages": ([_H, _P, _P, _P, _P, _P, C.c_int32, C.c_int32, C.c_int32, _P], C.c_int),
    "moe_forward_stack": ([C.POINTER(_H), C.c_int32, _P, C.POINTER(_P), C.POINTER(_P), C.POINTER(_P), C.POINTER(_P),
                           C.c_int32, C.POINTER(moe_plan), _P], C.c_int),
    "moe_get_plan": ([_H, C.POINTER(moe_plan), _P], C.c_int),
    "moe_sync_status": ([_H, _P], C.c_int),
    "moe_plan_host": ([_H, C.c_double, C.c_double, C.c_double, C.POINTER(C.c_int64), C.POINTER(moe_plan)], C.c_int),
    "moe_tile_geometry": ([_H, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32)], C.c_int),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res


def header_functions() -> list:
    """Names of the functions include/moe.h declares."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:moe_status|const char\*|size_t)\s+(moe_\w+)\s*\(", txt, re.M)))


def library():
    return _lib


def _check(fn: str, st: int) -> None:
    if st != MOE_OK:
        raise MoeError(fn, st, _lib.moe_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the MoE library must be contiguous")
    return C.c_void_p(t.data_ptr())


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


# ---- one wrapper per C entry point -------------------------------------------

def moe_init(cfg: moe_config, calib: Optional[moe_calib] = None) -> int:
    h = _H()
    _check("moe_init", _lib.moe_init(C.byref(cfg), C.byref(calib) if calib is not None else None, C.byref(h)))
    return h.value


def moe_destroy(h: int) -> None:
    _check("moe_destroy", _lib.moe_destroy(h))


def moe_last_error() -> str:
    return _lib.moe_last_error().decode()


def moe_set_calib(h: int, calib: moe_calib) -> None:
    _check("moe_set_calib", _lib.moe_set_calib(h, C.byref(calib)))


def moe_get_calib(h: int) -> moe_calib:
    k = moe_calib()
    _check("moe_get_calib", _lib.moe_get_calib(h, C.byref(k)))
    return k


def moe_set_trace(h: int, buf, nbytes: int = 0) -> None:
    """Point the megakernel's timeline trace at a device buffer (None: off)."""
    ptr = None if buf is None else _ptr(buf)
    n = 0 if buf is None else int(nbytes or buf.numel() * buf.element_size())
    _check("moe_set_trace", _lib.moe_set_trace(h, ptr, n))


TRACE_KINDS = {1: "workgroup", 2: "tile", 3: "dispatch", 4: "combine", 5: "dispatch unit"}


TRACE_MAGIC = 0x31435254


def read_trace(buf) -> "np.ndarray":
    """Decode a trace buffer (see moe_set_trace) into one structured array
    (kind, ticket, xcd, id, t0, t1, t2) of every wavefront's records, times in
    device-clock ticks of 10 ns.  An empty array if no launch wrote it."""
    import numpy as np
    dt = [("kind", "i4"), ("ticket", "i4"), ("xcd", "i4"), ("id", "i8"), ("t0", "i8"), ("t1", "i8"), ("t2", "i8")]
    raw = buf.cpu().numpy().view(np.uint8)
    hdr = raw[:64].view(np.int32)
    if int(hdr[0]) != TRACE_MAGIC:
        return np.zeros(0, dtype=dt)
    nseg, cap, rec0 = int(hdr[1]), int(hdr[2]), int(hdr[3])
    counts = raw[64:64 + 4 * nseg].view(np.int32)
    recs = raw[rec0 * 8:rec0 * 8 + nseg * cap * 32].view(np.int64).reshape(nseg, cap, 4)
    rec = np.concatenate([recs[i, :min(int(counts[i]), cap)] for i in range(nseg)] + [np.zeros((0, 4), np.int64)])
    w0 = rec[:, 0]
    out = np.zeros(len(rec), dtype=dt)
    out["kind"] = w0 & 0xFF
    out["ticket"] = (w0 >> 8) & 0xFFF
    out["xcd"] = (w0 >> 20) & 0xFFF
    out["id"] = w0 >> 32
    out["t0"], out["t1"], out["t2"] = rec[:, 1], rec[:, 2], rec[:, 3]
    return out


def moe_set_jitter(h: int, seed: int, max_sleeps: int) -> None:
    _check("moe_set_jitter", _lib.moe_set_jitter(h, C.c_uint32(seed & 0xFFFFFFFF), int(max_sleeps)))


def moe_set_timeout_ms(h: int, ms: float, inject_stall: int = 0) -> None:
    _check("moe_set_timeout_ms", _lib.moe_set_timeout_ms(h, float(ms), int(inject_stall)))


def moe_workspace_size(h: int) -> int:
    n = C.c_size_t()
    _check("moe_workspace_size", _lib.moe_workspace_size(h, C.byref(n)))
    return n.value


def moe_workspace_layout(h: int) -> moe_ws_layout:
    L = moe_ws_layout()
    _check("moe_workspace_layout", _lib.moe_workspace_layout(h, C.byref(L)))
    return L


def moe_set_workspace(h: int, ws: torch.Tensor, stream=None) -> None:
    _check("moe_set_workspace", _lib.moe_set_workspace(h, _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def moe_packed_weights_size(h: int) -> int:
    n = C.c_size_t()
    _check("moe_packed_weights_size", _lib.moe_packed_weights_size(h, C.byref(n)))
    return n.value


def moe_pack_weights(h: int, w1, w3, w2, ws1, ws3, ws2, packed: torch.Tensor, stream=None) -> None:
    _check("moe_pack_weights", _lib.moe_pack_weights(h, _ptr(w1), _ptr(w3), _ptr(w2), _ptr(ws1), _ptr(ws3),
                                                     _ptr(ws2), _ptr(packed), _stream(stream)))


def moe_route(h: int, x, wg, logit_bias, top_k: int, topk_idx, topk_w, stream=None) -> None:
    _check("moe_route", _lib.moe_route(h, _ptr(x), _ptr(wg), _ptr(logit_bias), int(top_k), _ptr(topk_idx),
                                       _ptr(topk_w), _stream(stream)))


def moe_route_topk_static(T: int, H: int, E: int, top_k: int, x, wg, logit_bias, topk_idx, topk_w,
                          stream=None) -> None:
    _check("moe_route_topk_static", _lib.moe_route_topk_static(int(T), int(H), int(E), int(top_k), _ptr(x),
                                                               _ptr(wg), _ptr(logit_bias), _ptr(topk_idx),
                                                               _ptr(topk_w), _stream(stream)))


def moe_build_tables(h: int, topk_idx, stream=None) -> None:
    _check("moe_build_tables", _lib.moe_build_tables(h, _ptr(topk_idx), _stream(stream)))


def moe_forward(h: int, x, topk_idx, topk_w, packed, y, mode: int = MOE_MODE_DYNAMIC,
                forced: Optional[moe_plan] = None, stream=None) -> None:
    _check("moe_forward", _lib.moe_forward(h, _ptr(x), _ptr(topk_idx), _ptr(topk_w), _ptr(packed), _ptr(y),
                                           int(mode), C.byref(forced) if forced is not None else None,
                                           _stream(stream)))


def moe_forward_stack(handles, x, topk_idx, topk_w, packed, y, mode: int = MOE_MODE_DYNAMIC,
                      forced: Optional[moe_plan] = None, stream=None) -> None:
    """handles, topk_idx, topk_w, packed, y: one entry per layer."""
    n = len(handles)
    hs = (_H * n)(*handles)
    arr = lambda ts: (_P * n)(*[_ptr(t) for t in ts])
    _check("moe_forward_stack", _lib.moe_forward_stack(hs, n, _ptr(x), arr(topk_idx), arr(topk_w), arr(packed),
                                                       arr(y), int(mode),
                                                       C.byref(forced) if forced is not None else None,
                                                       _stream(stream)))


def moe_run_stages(h: int, x, topk_idx, topk_w, packed, y, stages: int, n_workers: int, K: int = 1,
                   stream=None) -> None:
    _check("moe_run_stages", _lib.moe_run_stages(h, _ptr(x), _ptr(topk_idx), _ptr(topk_w), _ptr(packed), _ptr(y),
                                                 int(stages), int(n_workers), int(K), _stream(stream)))


def moe_get_plan(h: int, stream=None) -> moe_plan:
    p = moe_plan()
    _check("moe_get_plan", _lib.moe_get_plan(h, C.byref(p), _stream(stream)))
    return p


def moe_sync_status(h: int, stream=None) -> int:
    """Returns the status code (does not raise) so callers can test error paths."""
    return int(_lib.moe_sync_status(h, _stream(stream)))


def moe_plan_host(h: int, w_comp: float, w_dispatch: float, w_combine: float, n_tiles) -> moe_plan:
    arr = (C.c_int64 * CALIB_MAX_K)(*[int(v) for v in n_tiles])
    p = moe_plan()
    _check("moe_plan_host", _lib.moe_plan_host(h, float(w_comp), float(w_dispatch), float(w_combine), arr,
                                               C.byref(p)))
    return p


def moe_tile_geometry(h: int):
    bm, n0, n1 = C.c_int32(), C.c_int32(), C.c_int32()
    _check("moe_tile_geometry", _lib.moe_tile_geometry(h, C.byref(bm), C.byref(n0), C.byref(n1)))
    return bm.value, n0.value, n1.value


# ---- convenience --------------------------------------------------------------

def make_config(shape, n_workers: int = 0, first_local_expert: int = 0, gemm1_split: int = 0) -> moe_config:
    return moe_config(shape.n_src_ranks, shape.tokens_per_rank, shape.hidden, shape.ffn, shape.n_experts,
                      shape.top_k, shape.n_local_experts, first_local_expert, shape.n_shared_experts, n_workers,
                      gemm1_split)


def make_calib(c, bw, flops, K, eff, alpha: float, static_c: int, literal: int = 0, bw_all: float = 0.0,
               steal_window: int = 1, steal_ceil: int = 1) -> moe_calib:
    k = moe_calib()
    k.n_c = len(c)
    for i, (cv, b, f) in enumerate(zip(c, bw, flops)):
        k.c[i], k.bw_bytes_per_s[i], k.comp_flop_per_s[i] = int(cv), float(b), float(f)
    k.n_k = len(K)
    for j, (kv, e) in enumerate(zip(K, eff)):
        k.k_chunks[j], k.eff_chunk[j] = int(kv), float(e)
    k.alpha = float(alpha)
    k.literal_volumes = int(literal)
    k.static_c = int(static_c)
    k.bw_all_bytes_per_s = float(bw_all)
    k.steal_window = int(steal_window)
    k.steal_ceil = int(steal_ceil)
    return k


class MoeLayer:
    """Owns a handle plus torch-allocated workspace and packed weights on one device."""

    def __init__(self, shape, w1, w3, w2, ws1=None, ws3=None, ws2=None, calib: Optional[moe_calib] = None,
                 device="cuda", n_workers: int = 0, stream=None, gemm1_split: int = 0):
        self.shape = shape
        self.device = torch.device(device)
        self.h = moe_init(make_config(shape, n_workers, gemm1_split=gemm1_split), calib)
        self.ws = torch.empty(moe_workspace_size(self.h), dtype=torch.uint8, device=self.device)
        moe_set_workspace(self.h, self.ws, stream)
        self.packed = torch.empty(moe_packed_weights_size(self.h), dtype=torch.uint8, device=self.device)
        dev = [None if t is None else t.to(self.device).contiguous() for t in (w1, w3, w2, ws1, ws3, ws2)]
        moe_pack_weights(self.h, *dev, self.packed, stream)
        torch.cuda.synchronize(self.device)
        self.layout = moe_workspace_layout(self.h)

    def route(self, x, wg, bias, topk_idx, topk_w, stream=None):
        moe_route(self.h, x, wg, bias, self.shape.top_k, topk_idx, topk_w, stream)

    def forward(self, x, topk_idx, topk_w, y, mode="dynamic", forced: Optional[moe_plan] = None, stream=None):
        moe_forward(self.h, x, topk_idx, topk_w, self.packed, y, MODES[mode] if isinstance(mode, str) else mode,
                    forced, stream)

    def ws_view(self, name: str, dtype: torch.dtype, count: int) -> torch.Tensor:
        off = getattr(self.layout, name)
        nbytes = count * torch.empty((), dtype=dtype).element_size()
        return self.ws[off:off + nbytes].view(dtype)

    def close(self):
        if self.h:
            moe_destroy(self.h)
            self.h = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
