"""GPU tests of the stacked launch (moe_forward_stack: several independent
layers in one persistent megakernel launch): every layer's y equals its own
moe_forward bit for bit, and the oracle within the bar on sampled rows."""
import numpy as np
import pytest
import torch

from paper_2609_21483_amd import workloads as W
from tests.cases import bf16_to_f64, make_case, oracle_rows, pick_rows, rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21483_amd import binding
    return binding


def build_stack(B, shape, n_layers):
    cases, layers, idx, w = [], [], [], []
    for l in range(n_layers):
        c = make_case(shape, l)
        i, ww = c.oracle_route()
        ml = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
        idx_d = torch.from_numpy(np.ascontiguousarray(i, np.int32)).cuda()
        w_d = torch.from_numpy(np.ascontiguousarray(ww, np.float32)).cuda()
        B.moe_build_tables(ml.h, idx_d)
        cases.append((c, i, ww))
        layers.append(ml)
        idx.append(idx_d)
        w.append(w_d)
    return cases, layers, idx, w


@pytest.mark.parametrize("shape,n_layers,mode", [
    (W.FINE_ZIPF.with_(tokens_per_rank=512), 3, "dynamic"),
    (W.FINE_ZIPF.with_(tokens_per_rank=512), 3, "static"),
    (W.MoeShape("stack_shared", 88, 3, 300, 256, 384, 16, 4, 6, n_shared_experts=1, w_std=0.05), 4, "dynamic"),
], ids=["fine-dynamic", "fine-static", "shared-dynamic"])
def test_stack_matches_single_launches_and_oracle(B, shape, n_layers, mode):
    cases, layers, idx, w = build_stack(B, shape, n_layers)
    try:
        x = cases[0][0].x.cuda()
        singles = []
        for l, ml in enumerate(layers):
            y = torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
            ml.forward(x, idx[l], w[l], y, mode)
            assert B.moe_sync_status(ml.h) == B.MOE_OK
            singles.append(y)
        for rep in range(2):  # twice: both control sets of every layer
            ys = [torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
                  for _ in layers]
            B.moe_forward_stack([ml.h for ml in layers], x, idx, w, [ml.packed for ml in layers], ys,
                                B.MODES[mode])
            for l, ml in enumerate(layers):
                assert B.moe_sync_status(ml.h) == B.MOE_OK, (rep, l, B.moe_last_error())
                assert torch.equal(ys[l].view(torch.int16), singles[l].view(torch.int16)), (rep, l)
        for l, (c, i, ww) in enumerate(cases):
            rows = pick_rows(shape, i, per_rank=20, seed=40 + l)
            y_ref = oracle_rows(c, i, ww, rows)
            assert rel_err(bf16_to_f64(ys[l][torch.from_numpy(rows).cuda()]), y_ref) <= TOL, l
    finally:
        for ml in layers:
            ml.close()


@pytest.mark.parametrize("plan", [(8, 2, 3, 1), (4, 4, 0, 0), "stale"], ids=["K2", "K4", "stale-calibration"])
def test_stack_dispatch_ahead_plans(B, plan):
    """A layer's movement workers dispatch the next layer ahead under that
    layer's chunk count: forced plans with K = 2 and 4 (chunked readiness
    counts), and a layer whose calibration changed after its tables were built
    (its prologue evaluates the model again, so nothing is dispatched ahead for
    it).  Each layer's y equals its own launch's, bit for bit."""
    shape = W.FINE_ZIPF.with_(tokens_per_rank=512)
    cases, layers, idx, w = build_stack(B, shape, 3)
    try:
        forced = None if plan == "stale" else B.moe_plan(*plan, 0.0)
        if plan == "stale":
            B.moe_set_calib(layers[1].h, B.moe_get_calib(layers[1].h))
        x = cases[0][0].x.cuda()
        singles = []
        for l, ml in enumerate(layers):
            y = torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
            ml.forward(x, idx[l], w[l], y, "dynamic", forced=forced)
            assert B.moe_sync_status(ml.h) == B.MOE_OK
            singles.append(y)
        if plan == "stale":  # the single launch stored nothing: the stack's layer 1 is still stale
            B.moe_set_calib(layers[1].h, B.moe_get_calib(layers[1].h))
        for rep in range(2):
            ys = [torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
                  for _ in layers]
            B.moe_forward_stack([ml.h for ml in layers], x, idx, w, [ml.packed for ml in layers], ys,
                                B.MOE_MODE_DYNAMIC, forced=forced)
            for l, ml in enumerate(layers):
                assert B.moe_sync_status(ml.h) == B.MOE_OK, (rep, l, B.moe_last_error())
                assert torch.equal(ys[l].view(torch.int16), singles[l].view(torch.int16)), (rep, l)
    finally:
        for ml in layers:
            ml.close()


def test_large_stack_all_layers_in_one_launch(B):
    """The 8 layers of the large fine-grained stack in one launch: each layer's
    y equals its own launch's, bit for bit (each launch is checked against the
    oracle in test_gpu_forward)."""
    shape = W.LARGE_STACK
    x = W.tokens(shape).cuda()
    layers, idx, w, singles = [], [], [], []
    try:
        for l in range(shape.n_layers):
            ml = B.MoeLayer(shape, *W.experts(shape, l))
            i = torch.empty((shape.T, shape.top_k), dtype=torch.int32, device="cuda")
            ww = torch.empty((shape.T, shape.top_k), dtype=torch.float32, device="cuda")
            ml.route(x, W.gate(shape, l).cuda(), W.zipf_log_prior(shape, l).cuda(), i, ww)
            y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
            ml.forward(x, i, ww, y, "dynamic")
            assert B.moe_sync_status(ml.h) == B.MOE_OK
            layers.append(ml), idx.append(i), w.append(ww), singles.append(y)
        ys = [torch.empty_like(singles[0]) for _ in layers]
        B.moe_forward_stack([ml.h for ml in layers], x, idx, w, [ml.packed for ml in layers], ys)
        for l, ml in enumerate(layers):
            assert B.moe_sync_status(ml.h) == B.MOE_OK
            assert torch.equal(ys[l].view(torch.int16), singles[l].view(torch.int16)), l
    finally:
        for ml in layers:
            ml.close()


def test_stack_refuses_bad_arguments(B):
    shape = W.TINY
    cases, layers, idx, w = build_stack(B, shape, 2)
    try:
        x = cases[0][0].x.cuda()
        ys = [torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda") for _ in layers]
        hs, packed = [ml.h for ml in layers], [ml.packed for ml in layers]
        with pytest.raises(B.MoeError) as ei:  # the same handle twice
            B.moe_forward_stack([hs[0], hs[0]], x, idx, w, packed, ys)
        assert ei.value.status == B.MOE_ERR_INVALID_ARG
        with pytest.raises(B.MoeError) as ei:  # tables built from another routing array
            B.moe_forward_stack(hs, x, [idx[1], idx[0]], w, packed, ys)
        assert ei.value.status == B.MOE_ERR_STATE
        with pytest.raises(B.MoeError) as ei:  # the serial mode is not a megakernel
            B.moe_forward_stack(hs, x, idx, w, packed, ys, B.MOE_MODE_SERIAL)
        assert ei.value.status == B.MOE_ERR_INVALID_ARG
    finally:
        for ml in layers:
            ml.close()
