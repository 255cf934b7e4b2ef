"""Seeded synthetic inputs for one GPU's share of an expert-parallel MoE layer.

This module only draws inputs: token rows, gate matrix, expert weights and the
Zipf log-prior that skews expert choice.  It holds none of the layer's
arithmetic (no logits, no routing, no FFN), so both the CPU oracle and the HIP
path can take their inputs from here without sharing any computation.

Every tensor is drawn in fixed pieces of ``PIECE`` elements.  Each piece has its
own seed derived from ``(workload id, layer, tensor id, piece index)`` with
``numpy.random.SeedSequence``, is filled by a CPU ``torch.Generator``
(``randn``), scaled, and rounded to bf16 (round-to-nearest-even, torch's CPU
conversion).  The result does not depend on how many threads draw the pieces.

bf16 tensors are returned as ``torch.uint16``-compatible ``int16`` bit
patterns inside ``torch.bfloat16`` tensors; ``as_u16_numpy`` gives the raw
bits for the oracle.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np
import torch

PIECE = 1 << 24

# tensor ids used in the seed scheme
T_X, T_WG, T_W1, T_W3, T_W2, T_WS1, T_WS3, T_WS2, T_ZIPF_PERM, T_ZIPF_S, T_ROUTE = range(11)


@dataclasses.dataclass(frozen=True)
class MoeShape:
    """One GPU's share of an expert-parallel MoE layer.

    ``n_src_ranks`` ranks each send ``tokens_per_rank`` token rows; this GPU
    is EP rank 0 and holds local experts ``[0, n_local_experts)``.  Rank 0's
    tokens are its own (no transfer on a real cluster), ranks 1.. stand in for
    peers.  ``n_shared_experts`` always-on experts apply to rank-0 tokens.
    """

    name: str
    wid: int                     # workload id used in the seed scheme
    n_src_ranks: int
    tokens_per_rank: int
    hidden: int
    ffn: int
    n_experts: int
    top_k: int
    n_local_experts: int
    n_shared_experts: int = 0
    zipf_s: Optional[float] = None       # fixed Zipf exponent of the log-prior
    zipf_s_max: Optional[float] = None   # per-layer exponent drawn in [0, max)
    n_layers: int = 1
    x_std: float = 1.0
    w_std: float = 0.02

    @property
    def T(self) -> int:
        return self.n_src_ranks * self.tokens_per_rank

    def with_(self, **kw) -> "MoeShape":
        return dataclasses.replace(self, **kw)


# The five workloads: shapes, sizes and routing structure of the layer shares
# the method is evaluated on (Table 1 gives the Qwen3-30B and DSv2-Lite shapes
# reused by the fine-grained and shared+routed cases).
TINY = MoeShape("tiny", 1, 4, 16, 128, 256, 8, 2, 8)
MIXTRAL_EP4 = MoeShape("mixtral_ep4", 2, 4, 1024, 4096, 14336, 8, 2, 2)
FINE_ZIPF = MoeShape("fine_zipf", 3, 4, 2048, 2048, 768, 128, 8, 32, zipf_s=1.2)
SHARED_ROUTED = MoeShape("shared_routed", 4, 4, 4096, 2048, 1408, 64, 6, 16, n_shared_experts=2)
LARGE_STACK = MoeShape("large_stack", 5, 4, 8192, 4096, 1536, 128, 8, 32, zipf_s_max=1.5, n_layers=8)

WORKLOADS = {w.name: w for w in (TINY, MIXTRAL_EP4, FINE_ZIPF, SHARED_ROUTED, LARGE_STACK)}


def _seed(*key: int) -> int:
    return int(np.random.SeedSequence([int(k) for k in key]).generate_state(1, dtype=np.uint64)[0])


def _threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal_bf16(shape, std: float, *key: int) -> torch.Tensor:
    """bf16 tensor of N(0, std^2) draws, seeded by ``key``; deterministic."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = torch.empty(n, dtype=torch.bfloat16)
    npieces = (n + PIECE - 1) // PIECE

    def piece(i: int) -> None:
        s = i * PIECE
        e = min(n, s + PIECE)
        g = torch.Generator().manual_seed(_seed(*key, i))
        v = torch.randn(e - s, generator=g, dtype=torch.float32)
        if std != 1.0:
            v.mul_(std)
        out[s:e] = v.to(torch.bfloat16)

    if npieces <= 1:
        if n:
            piece(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(piece, range(npieces)))
    return out.view(*shape)


def zipf_log_prior(shape: MoeShape, layer: int) -> Optional[torch.Tensor]:
    """fp32 [E] bias added to the gate logits, or None for plain routing.

    A seeded permutation pi ranks the experts; expert e gets -s*ln(pi[e]+1), a
    Zipf(s) log-prior (its normalising constant cancels in the softmax).
    """
    if shape.zipf_s is None and shape.zipf_s_max is None:
        return None
    E = shape.n_experts
    g = torch.Generator().manual_seed(_seed(shape.wid, layer, T_ZIPF_PERM))
    pi = torch.randperm(E, generator=g).to(torch.float64)
    if shape.zipf_s is not None:
        s = float(shape.zipf_s)
    else:
        gs = torch.Generator().manual_seed(_seed(shape.wid, layer, T_ZIPF_S))
        s = float(shape.zipf_s_max) * float(torch.rand((), generator=gs, dtype=torch.float64))
    return (-s * torch.log(pi + 1.0)).to(torch.float32)


def zipf_exponent(shape: MoeShape, layer: int) -> float:
    if shape.zipf_s is not None:
        return float(shape.zipf_s)
    if shape.zipf_s_max is None:
        return 0.0
    gs = torch.Generator().manual_seed(_seed(shape.wid, layer, T_ZIPF_S))
    return float(shape.zipf_s_max) * float(torch.rand((), generator=gs, dtype=torch.float64))


def tokens(shape: MoeShape) -> torch.Tensor:
    """x: bf16 [T, H]; rank r's rows are [r*T_r, (r+1)*T_r).  Shared by all layers."""
    return normal_bf16((shape.T, shape.hidden), shape.x_std, shape.wid, 0, T_X)


def gate(shape: MoeShape, layer: int = 0) -> torch.Tensor:
    """Wg: bf16 [H, E]."""
    return normal_bf16((shape.hidden, shape.n_experts), shape.w_std, shape.wid, layer, T_WG)


def experts(shape: MoeShape, layer: int = 0):
    """(W1, W3, W2) for the local experts: bf16 [E_l,H,F], [E_l,H,F], [E_l,F,H]."""
    El, H, F = shape.n_local_experts, shape.hidden, shape.ffn
    w1 = normal_bf16((El, H, F), shape.w_std, shape.wid, layer, T_W1)
    w3 = normal_bf16((El, H, F), shape.w_std, shape.wid, layer, T_W3)
    w2 = normal_bf16((El, F, H), shape.w_std, shape.wid, layer, T_W2)
    return w1, w3, w2


def shared_experts(shape: MoeShape, layer: int = 0):
    """(Ws1, Ws3, Ws2) bf16 [S,H,F], [S,H,F], [S,F,H], or (None,)*3."""
    S, H, F = shape.n_shared_experts, shape.hidden, shape.ffn
    if S == 0:
        return None, None, None
    ws1 = normal_bf16((S, H, F), shape.w_std, shape.wid, layer, T_WS1)
    ws3 = normal_bf16((S, H, F), shape.w_std, shape.wid, layer, T_WS3)
    ws2 = normal_bf16((S, F, H), shape.w_std, shape.wid, layer, T_WS2)
    return ws1, ws3, ws2


def random_routing(T: int, E: int, k: int, seed: int, skew: float = 0.0):
    """A synthetic routing result (distinct expert ids per token, weights summing
    to one) for tests that feed routing directly instead of computing it."""
    g = np.random.default_rng(seed)
    pri = -skew * np.log(np.arange(1, E + 1, dtype=np.float64))
    score = pri[None, :] + g.gumbel(size=(T, E))
    idx = np.argsort(-score, axis=1, kind="stable")[:, :k].astype(np.int32)
    w = g.random((T, k)) + 0.05
    w = (w / w.sum(axis=1, keepdims=True)).astype(np.float32)
    return idx, w


def as_u16_numpy(t: Optional[torch.Tensor]) -> Optional[np.ndarray]:
    """Raw bf16 bit patterns of a CPU bf16 tensor as a contiguous uint16 array."""
    if t is None:
        return None
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def bf16_from_u16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)


def sample_tokens(shape: MoeShape, n_per_rank: int, seed: int) -> np.ndarray:
    """Seeded sorted sample of token indices, ``n_per_rank`` from each rank."""
    g = np.random.default_rng(seed)
    out = []
    for r in range(shape.n_src_ranks):
        m = min(n_per_rank, shape.tokens_per_rank)
        out.append(r * shape.tokens_per_rank + np.sort(g.choice(shape.tokens_per_rank, m, replace=False)))
    return np.concatenate(out).astype(np.int64)
