"""moe_route_topk_static (routing with its scratch in a static device array,
for callers that cannot allocate) against moe_route (the same routing with
the scratch in the handle's workspace), called through the C ABI on two
inputs in a row, the second smaller: routing ids bit for bit, weights within
1e-6; and the ids of the second call against the oracle."""
import numpy as np
import pytest
import torch

from paper_2609_21483_amd import workloads as W
from tests.cases import make_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21483_amd import binding
    return binding


def route_with_handle(B, shape, x, wg, bias):
    h = B.moe_init(B.make_config(shape))
    try:
        ws = torch.empty(B.moe_workspace_size(h), dtype=torch.uint8, device="cuda")
        B.moe_set_workspace(h, ws)
        idx = torch.empty((shape.T, shape.top_k), dtype=torch.int32, device="cuda")
        w = torch.empty((shape.T, shape.top_k), dtype=torch.float32, device="cuda")
        B.moe_route(h, x, wg, bias, shape.top_k, idx, w)
        assert B.moe_sync_status(h) == B.MOE_OK
        return idx.cpu().numpy(), w.cpu().numpy()
    finally:
        B.moe_destroy(h)


def test_static_routing_matches_moe_route(B):
    shapes = [W.FINE_ZIPF.with_(tokens_per_rank=1024),
              W.MoeShape("static_small", 89, 3, 333, 1024, 256, 64, 6, 16, zipf_s=0.7)]
    for i, shape in enumerate(shapes):
        c = make_case(shape, weights=False)
        x, wg = c.x.cuda(), c.wg.cuda()
        bias = None if c.bias is None else c.bias.cuda()
        idx_ref, w_ref = route_with_handle(B, shape, x, wg, bias)
        idx = torch.full((shape.T, shape.top_k), -7, dtype=torch.int32, device="cuda")
        w = torch.full((shape.T, shape.top_k), float("nan"), dtype=torch.float32, device="cuda")
        B.moe_route_topk_static(shape.T, shape.hidden, shape.n_experts, shape.top_k, x, wg, bias, idx, w)
        torch.cuda.synchronize()
        assert np.array_equal(idx.cpu().numpy(), idx_ref), shape.name
        assert np.max(np.abs(w.cpu().numpy() - w_ref)) <= 1e-6, shape.name
        if i == 1:
            idx_o, _ = c.oracle_route()
            assert np.array_equal(idx_ref, idx_o)
