"""GPU regression test of the row map of A, Hbuf and O (moe.h, row_off).

Each (segment, chunk) of the dispatched rows, h and the expert outputs starts
on a 32-row group, so that no 128-byte line holds rows of two segments or
chunks.  Workers on different XCDs (each with its own L2) wait on different
readiness counters; a line shared by two segments could be cached by one XCD
while the other segment's rows are still being written.  The routing here is
supplied so that every local expert has an odd number of rows, so in slot
space every expert after the first starts on an odd slot, and the movement
workers are few (c = 8) and, in the forced plans without stealing, keep their
roles, so later segments become ready while earlier ones are still being
dispatched.  Every launch is relaunched with
fresh tokens on the same workspace.  y must equal the oracle within the bar
and be bit-identical across modes and plans."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_21483_amd import workloads as W
from tests.cases import bf16_to_f64, make_case, oracle_rows, rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21483_amd import binding
    return binding


def odd_boundary_routing(T, E, k, El, seed):
    """Distinct ids per token; the local experts' row counts are all odd and
    every chunk boundary of K = 2, 4, 8 falls on an odd slot of each expert."""
    rng = np.random.default_rng(seed)
    idx = np.zeros((T, k), np.int32)
    for g in range(T):
        idx[g] = rng.choice(E, k, replace=False)
    tab = O.route_tables(idx, 4, T // 4, 0, El)
    # make every local expert's count odd by moving one pair of the first
    # token without that expert onto it, where needed
    counts = tab.cnt_rank.sum(axis=1)
    for le in range(El):
        if counts[le] % 2 == 0:
            for g in range(T):
                if le not in idx[g] and idx[g, 0] >= El:
                    idx[g, 0] = le
                    break
    w = rng.random((T, k)) + 0.1
    return idx, (w / w.sum(axis=1, keepdims=True)).astype(np.float64)


@pytest.mark.parametrize("S", [0, 1])
def test_odd_segment_boundaries_relaunched(B, S):
    shape = W.MoeShape("rowmap", 91, 4, 500, 256, 320, 8, 2, 4, n_shared_experts=S)
    c1 = make_case(shape.with_(w_std=0.05))
    c2 = make_case(shape.with_(wid=shape.wid + 40, w_std=0.05))
    idx, w = odd_boundary_routing(shape.T, 8, 2, 4, seed=11)
    tab = O.route_tables(idx, 4, shape.tokens_per_rank, 0, 4)
    assert all(n % 2 == 1 for n in tab.cnt_rank.sum(axis=1))
    plans = [B.moe_plan(8, K, 0, 0, 0.0) for K in (1, 2, 4, 8)] + [B.moe_plan(8, 2, 4, 1, 0.0)]
    layer = B.MoeLayer(shape, c1.w1, c1.w3, c1.w2, c1.ws1, c1.ws3, c1.ws2)
    try:
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(layer.h, idx_d)
        rows = np.arange(shape.T)
        for c in (c1, c2, c1):
            x = c.x.cuda()
            y_ref = oracle_rows(c1.with_tokens(c), idx, w, rows)
            first = None
            runs = [("static", None)] + [("dynamic", p) for p in plans] + [("serial", None)]
            for mode, p in runs:
                y = torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
                layer.forward(x, idx_d, w_d, y, mode, forced=p)
                assert B.moe_sync_status(layer.h) == B.MOE_OK, (mode, p and p.as_tuple(), B.moe_last_error())
                assert rel_err(bf16_to_f64(y), y_ref) <= TOL, (mode, p and p.as_tuple())
                if first is None:
                    first = y
                else:
                    assert torch.equal(y.view(torch.int16), first.view(torch.int16)), (mode, p and p.as_tuple())
        # every segment and chunk starts on a 32-row group
        rof = layer.ws_view("row_off", torch.int32, 4 * (4 + S) * 9).cpu().numpy()
        assert np.all(rof % 32 == 0)
    finally:
        layer.close()
