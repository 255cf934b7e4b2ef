"""The megakernel's timeline trace (moe_set_trace) on the device: one record
per workgroup, per compute tile, per movement worker's dispatch, per combine
unit and per dispatch unit, each time-ordered; every tile, dispatch unit and
combine unit appears exactly once; tracing leaves y unchanged bit for bit."""
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


def n_tiles(B, h, shape, idx, K):
    T, k = shape.T, shape.top_k
    El, S, Tr = shape.n_local_experts, shape.n_shared_experts, shape.tokens_per_rank
    tab = O.route_tables(idx, shape.n_src_ranks, Tr, 0, El)
    bm, nt0, nt1 = B.moe_tile_geometry(h)
    sub = O.chunk_offsets(tab, T, k, K)
    rows = [list(np.diff(sub[le])) for le in range(El)]
    for _ in range(S):
        bnd = [(q * T + K - 1) // K for q in range(K + 1)]
        rows.append([max(0, min(bnd[q + 1], Tr) - bnd[q]) for q in range(K)])
    return O.tile_count(np.array(rows, np.int32).reshape(El + S, K), bm, nt0, nt1)


@pytest.mark.parametrize("name,plan", [("fine_zipf", (16, 1, 100, 1)), ("shared_routed", (24, 2, 3, 1))])
def test_trace_records(B, name, plan):
    shape = W.WORKLOADS[name]
    c = make_case(shape)
    idx, w = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
    try:
        N = torch.cuda.get_device_properties(0).multi_processor_count
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(layer.h, idx_d)
        forced = B.moe_plan(*plan, 0.0)
        y0 = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        layer.forward(x, idx_d, w_d, y0, "dynamic", forced=forced)
        buf = torch.zeros(64 + 32 * 65536, dtype=torch.uint8, device="cuda")
        B.moe_set_trace(layer.h, buf)
        y1 = torch.empty_like(y0)
        layer.forward(x, idx_d, w_d, y1, "dynamic", forced=forced)
        B.moe_set_trace(layer.h, None)
        assert B.moe_sync_status(layer.h) == B.MOE_OK, B.moe_last_error()
        assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
        tr = B.read_trace(buf)
        nt = n_tiles(B, layer.h, shape, idx, plan[1])
    finally:
        layer.close()

    units = N * 8                      # wavefronts on the workers
    per = max(1, shape.T // units)
    dt, ct = min(per, 8), min(per, 4)  # movement unit sizes chosen by the host
    kinds = {k: tr[tr["kind"] == k] for k in (1, 2, 3, 4, 5)}
    assert set(np.unique(tr["kind"])) <= {1, 2, 3, 4, 5}
    # one record per workgroup, tickets 0..N-1
    assert sorted(kinds[1]["ticket"]) == list(range(N))
    # every compute tile once (tile codes are unique)
    assert len(kinds[2]) == nt and len(np.unique(kinds[2]["id"])) == nt
    # one dispatch record per movement worker, movement workers first
    assert sorted(kinds[3]["ticket"]) == list(range(plan[0]))
    # every combine unit and every dispatch unit once
    cu = kinds[4]["id"] & 0xFFFFFF
    du = kinds[5]["id"] & 0xFFFFFF
    assert sorted(cu) == list(range(-(-shape.T // ct)))
    assert sorted(du) == list(range(-(-shape.T // dt)))
    # time order inside every record
    for k in (1, 2, 4, 5):
        r = kinds[k]
        assert np.all(r["t0"] <= r["t1"]) and np.all(r["t1"] <= r["t2"]), k
    # a workgroup's records lie inside its own entry .. exit window
    wg = {int(t): (a, b) for t, a, b in zip(kinds[1]["ticket"], kinds[1]["t0"], kinds[1]["t2"])}
    for k in (2, 4, 5):
        for rec in kinds[k]:
            a, b = wg[int(rec["ticket"])]
            assert a <= rec["t0"] and rec["t2"] <= b
