"""The megakernel prologue's plan (c*, K*, n_steal, T_total) against the
oracle's cost model evaluated on the oracle's own routing tables and tile
counts: identical integers and identical fp64 bits."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_21483_amd import workloads as W
from tests.cases import check_plan, make_case, oracle_tiles, plain_reading

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21483_amd import binding
    return binding


def check_plan_after_forward(B, layer, shape, idx, x, idx_d, w_d, y):
    layer.forward(x, idx_d, w_d, y, "dynamic")
    assert B.moe_sync_status(layer.h) == B.MOE_OK
    return check_plan(B, layer.h, shape, idx)


READINGS = [dict(), dict(literal_volumes=1), dict(steal_window=0), dict(steal_window=2), dict(steal_ceil=0),
            dict(bw_all_bytes_per_s=0.0), "plain"]


@pytest.mark.parametrize("name", ["tiny", "fine_zipf", "shared_routed"])
def test_prologue_plan_matches_oracle(B, name):
    """Every reading of the cost model (moe.h, moe_calib), on the built-in
    table and on the committed measured table of the workload."""
    from paper_2609_21483_amd.calibrate import load_calib
    shape = W.WORKLOADS[name]
    c = make_case(shape)
    idx, w = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
    try:
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(layer.h, idx_d)
        y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        tables = [B.moe_get_calib(layer.h)]
        measured = load_calib(name, torch.cuda.get_device_properties(0).multi_processor_count)
        if measured is not None:
            tables.append(measured)
        for base in tables:
            for r in READINGS:
                cal = B.moe_calib.from_buffer_copy(base)
                if r == "plain":
                    plain_reading(cal)
                else:
                    for k, v in r.items():
                        setattr(cal, k, v)
                B.moe_set_calib(layer.h, cal)
                check_plan_after_forward(B, layer, shape, idx, x, idx_d, w_d, y)
        # static mode reports its fixed plan
        layer.forward(x, idx_d, w_d, y, "static")
        ps = B.moe_get_plan(layer.h)
        assert (ps.c, ps.K, ps.n_steal, ps.final_all) == (B.moe_get_calib(layer.h).static_c, 1, 0, 0)
    finally:
        layer.close()


@pytest.mark.parametrize("name", ["tiny", "fine_zipf", "shared_routed", "mixtral_ep4"])
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


@pytest.mark.parametrize("name", ["tiny", "shared_routed"])
def test_stored_plan_matches_prologue(B, name):
    """The plan the routing's last kernel stores with the tables and the plan
    the prologue evaluates itself (after moe_set_calib, which makes the
    stored one stale) are identical, and both match the oracle's."""
    shape = W.WORKLOADS[name]
    c = make_case(shape)
    idx, w = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
    try:
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        plans = []
        for step in ("stored", "recomputed", "stored again"):
            if step == "recomputed":
                B.moe_set_calib(layer.h, B.moe_get_calib(layer.h))
            else:
                B.moe_build_tables(layer.h, idx_d)
            layer.forward(x, idx_d, w_d, y, "dynamic")
            assert B.moe_sync_status(layer.h) == B.MOE_OK
            p = B.moe_get_plan(layer.h)
            plans.append((p.as_tuple(), p.t_pred_s))
            check_plan(B, layer.h, shape, idx)
        assert plans[0] == plans[1] == plans[2]
    finally:
        layer.close()
