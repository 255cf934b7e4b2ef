"""The megakernel prologue's plan (c*, K*, n_steal, T_total) against the
oracle's cost model evaluated on the oracle's own routing tables and tile
counts: identical integers and identical fp64 bits."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_21483_amd import workloads as W
from tests.cases import make_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21483_amd import binding
    return binding


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
                  head_on_all=cal.head_on_all)


def n_workers():
    # the persistent workers: one per CU
    return torch.cuda.get_device_properties(0).multi_processor_count


@pytest.mark.parametrize("name,literal,head", [("tiny", 0, 1), ("fine_zipf", 0, 1), ("fine_zipf", 1, 1),
                                               ("fine_zipf", 0, 0), ("shared_routed", 0, 1)])
def test_prologue_plan_matches_oracle(B, name, literal, head):
    shape = W.WORKLOADS[name]
    c = make_case(shape)
    idx, w = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
    try:
        cal = B.moe_get_calib(layer.h)
        cal.literal_volumes = literal
        cal.head_on_all = head
        B.moe_set_calib(layer.h, cal)
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(layer.h, idx_d)
        y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        layer.forward(x, idx_d, w_d, y, "dynamic")
        assert B.moe_sync_status(layer.h) == B.MOE_OK
        p = B.moe_get_plan(layer.h)
        o = oracle_plan(B, layer.h, shape, idx)
        assert (p.c, p.K, p.n_steal, p.final_all) == (o.c, o.K, o.n_steal, 1)
        assert p.t_pred_s == o.t_total
        # static mode reports its fixed plan
        layer.forward(x, idx_d, w_d, y, "static")
        ps = B.moe_get_plan(layer.h)
        assert (ps.c, ps.K, ps.n_steal, ps.final_all) == (B.moe_get_calib(layer.h).static_c, 1, 0, 0)
    finally:
        layer.close()


@pytest.mark.parametrize("name", ["tiny", "fine_zipf", "shared_routed"])
def test_table_builder_tile_counts(B, name):
    """The GEMM tiles at each chunk option (the cost model's W_tile input,
    Eq 14), counted once by the table builder, against the oracle's count."""
    shape = W.WORKLOADS[name]
    c = make_case(shape)
    idx, w = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
    try:
        B.moe_build_tables(layer.h, torch.from_numpy(idx).cuda())
        torch.cuda.synchronize()
        st = layer.ws_view("stats", torch.int32, 16).cpu().numpy()
        tab = O.route_tables(idx, shape.n_src_ranks, shape.tokens_per_rank, 0, shape.n_local_experts)
        assert [int(v) for v in st[10:14]] == [oracle_tiles(B, layer.h, shape, tab, K) for K in (1, 2, 4, 8)]
    finally:
        layer.close()
