"""Test-side helpers: seeded cases and oracle references.

The oracle is single-threaded C; for the large workloads the tests shard rows
over a thread pool (ctypes releases the GIL, rows are independent), so each
call is still the plain oracle on a slice of tokens.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from oracle import oracle as O
from paper_2609_21483_amd import workloads as W

THREADS = max(1, min(16, os.cpu_count() or 1))


def _shards(n: int, parts: int):
    step = max(1, (n + parts - 1) // parts)
    return [(s, min(n, s + step)) for s in range(0, n, step)]


def oracle_logits(xu: np.ndarray, wgu: np.ndarray, bias: Optional[np.ndarray]) -> np.ndarray:
    T = xu.shape[0]
    out = np.empty((T, wgu.shape[1]), np.float32)

    def run(se):
        s, e = se
        out[s:e] = O.gate_logits(xu[s:e], wgu, bias)

    with ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(run, _shards(T, THREADS * 4)))
    return out


def oracle_rows(c: "Case", idx: np.ndarray, w: np.ndarray, rows: np.ndarray) -> np.ndarray:
    rows = np.asarray(rows, np.int64)
    out = np.empty((rows.shape[0], c.shape.hidden), np.float64)

    def run(se):
        s, e = se
        out[s:e] = O.layer_rows(c.xu, idx, w, c.w1u, c.w3u, c.w2u, c.ws1u, c.ws3u, c.ws2u,
                                Tr=c.shape.tokens_per_rank, rows=rows[s:e])

    with ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(run, _shards(rows.shape[0], THREADS * 2)))
    return out


@dataclass
class Case:
    shape: W.MoeShape
    layer: int
    x: torch.Tensor
    wg: torch.Tensor
    bias: Optional[torch.Tensor]
    w1: Optional[torch.Tensor] = None
    w3: Optional[torch.Tensor] = None
    w2: Optional[torch.Tensor] = None
    ws1: Optional[torch.Tensor] = None
    ws3: Optional[torch.Tensor] = None
    ws2: Optional[torch.Tensor] = None

    @property
    def xu(self):
        return W.as_u16_numpy(self.x)

    @property
    def wgu(self):
        return W.as_u16_numpy(self.wg)

    @property
    def w1u(self):
        return W.as_u16_numpy(self.w1)

    @property
    def w3u(self):
        return W.as_u16_numpy(self.w3)

    @property
    def w2u(self):
        return W.as_u16_numpy(self.w2)

    @property
    def ws1u(self):
        return W.as_u16_numpy(self.ws1)

    @property
    def ws3u(self):
        return W.as_u16_numpy(self.ws3)

    @property
    def ws2u(self):
        return W.as_u16_numpy(self.ws2)

    @property
    def bias_np(self):
        return None if self.bias is None else self.bias.numpy()

    def with_tokens(self, other: "Case") -> "Case":
        """other's tokens, gate and bias with this case's expert weights."""
        return Case(self.shape, self.layer, other.x, other.wg, other.bias,
                    self.w1, self.w3, self.w2, self.ws1, self.ws3, self.ws2)

    def oracle_route(self):
        lg = oracle_logits(self.xu, self.wgu, self.bias_np)
        return O.softmax_topk(lg, self.shape.top_k)


def make_case(shape: W.MoeShape, layer: int = 0, weights: bool = True) -> Case:
    x = W.tokens(shape)
    wg = W.gate(shape, layer)
    bias = W.zipf_log_prior(shape, layer)
    c = Case(shape, layer, x, wg, bias)
    if weights:
        c.w1, c.w3, c.w2 = W.experts(shape, layer)
        c.ws1, c.ws3, c.ws2 = W.shared_experts(shape, layer)
    return c


def pick_rows(shape: W.MoeShape, idx: np.ndarray, per_rank: int, seed: int) -> np.ndarray:
    """Seeded sample of tokens per rank that always includes tokens with 0, 1
    and >= 2 local experts when such tokens exist."""
    rows = set(W.sample_tokens(shape, per_rank, seed).tolist())
    nloc = (idx < shape.n_local_experts).sum(axis=1)
    for want in (0, 1, 2):
        cand = np.nonzero(nloc == want if want < 2 else nloc >= 2)[0]
        if cand.size:
            rows.add(int(cand[0]))
            rows.add(int(cand[-1]))
    return np.array(sorted(rows), np.int64)


def rel_err(y_gpu: np.ndarray, y_ref: np.ndarray) -> float:
    m = float(np.max(np.abs(y_ref)))
    return float(np.max(np.abs(y_gpu - y_ref))) / (m if m > 0 else 1.0)


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


# ---- the cost model on the oracle's tables (plan parity) -------------------

def oracle_tiles(B, h, shape, tab, K):
    T, k = shape.T, shape.top_k
    El, S, Tr = shape.n_local_experts, shape.n_shared_experts, shape.tokens_per_rank
    bm, nt0, nt1 = B.moe_tile_geometry(h)
    sub = O.chunk_offsets(tab, T, k, K)
    rows = [list(np.diff(sub[le])) for le in range(El)]
    for _ in range(S):
        bnd = [(q * T + K - 1) // K for q in range(K + 1)]
        rows.append([max(0, min(bnd[q + 1], Tr) - bnd[q]) for q in range(K)])
    return O.tile_count(np.array(rows, np.int32).reshape(El + S, K), bm, nt0, nt1)


def oracle_plan(B, h, shape, idx):
    El, S, Tr = shape.n_local_experts, shape.n_shared_experts, shape.tokens_per_rank
    tab = O.route_tables(idx, shape.n_src_ranks, Tr, 0, El)
    cal = B.moe_get_calib(h)
    Ks = [cal.k_chunks[j] for j in range(cal.n_k)]
    n_tiles = [oracle_tiles(B, h, shape, tab, K) for K in Ks]
    wc, wd, wb = O.volumes(tab, shape.hidden, shape.ffn, S * Tr, literal=bool(cal.literal_volumes))
    n = cal.n_c
    return O.plan([cal.c[i] for i in range(n)], [cal.bw_bytes_per_s[i] for i in range(n)],
                  [cal.comp_flop_per_s[i] for i in range(n)], Ks, [cal.eff_chunk[j] for j in range(cal.n_k)],
                  cal.alpha, n_workers(), wc, wd, wb, n_tiles, bw_all=cal.bw_all_bytes_per_s,
                  steal_window=cal.steal_window, steal_ceil=cal.steal_ceil)


def n_workers():
    # the persistent workers: one per CU
    return torch.cuda.get_device_properties(0).multi_processor_count


def plain_reading(cal):
    """The printed cost model as it stands: remote-only volumes (Eq 2-3), the
    tail at BW(c) (Eq 10), Eq 11's window W_dispatch + W_combine, Eq 14's share
    as whole tiles."""
    cal.literal_volumes, cal.bw_all_bytes_per_s, cal.steal_window, cal.steal_ceil = 1, 0.0, 0, 0
    return cal


def check_plan(B, h, shape, idx):
    """The plan of the last megakernel launch against the oracle's cost model
    on the oracle's tables: identical integers, identical fp64 bits."""
    p = B.moe_get_plan(h)
    o = oracle_plan(B, h, shape, idx)
    assert (p.c, p.K, p.n_steal, p.final_all) == (o.c, o.K, o.n_steal, 1)
    assert p.t_pred_s == o.t_total
    return p
