"""Scheduler stress (section 4: dynamic claiming tolerates CUs that run at
different speeds).  The megakernel runs with seeded random delays before
every arrival ticket, GEMM tile, dispatch unit and combine unit
(moe_set_jitter), under the cost model's plan and forced plans that cover
few and many movement workers, every chunk count, bubble stealing from none
to all, and the final combine on or off.  Every output must be bit-identical
to the serial kernels' (each output element is computed by the same
operations in the same order whatever the claim order), and the serial
output must match the oracle.  A second test draws many random layer shapes
and routings and does the same."""
import numpy as np
import pytest
import torch

from paper_2609_21483_amd import workloads as W
from tests.cases import bf16_to_f64, make_case, oracle_rows, rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-2
PLANS = [None, (1, 1, 0, 1), (8, 2, 3, 1), (64, 4, 0, 0), (255, 8, 1000, 1), (40, 1, 0, 0), (128, 8, 2, 0),
         (16, 2, 1000, 0), (200, 1, 5, 1)]


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21483_amd import binding
    return binding


def _setup(B, shape, gemm1_split=0):
    c = make_case(shape.with_(w_std=0.05))
    idx, w = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2, gemm1_split=gemm1_split)
    x = c.x.cuda()
    idx_d = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).cuda()
    w_d = torch.from_numpy(np.ascontiguousarray(w, np.float32)).cuda()
    B.moe_build_tables(layer.h, idx_d)
    return c, idx, w, layer, x, idx_d, w_d


def _run(B, layer, shape, x, idx_d, w_d, mode, plan=None):
    y = torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
    layer.forward(x, idx_d, w_d, y, mode, forced=None if plan is None else B.moe_plan(*plan, 0.0))
    st = B.moe_sync_status(layer.h)
    assert st == B.MOE_OK, (mode, plan, B.moe_last_error())
    return y


@pytest.mark.parametrize("shape,split", [
    (W.WORKLOADS["tiny"], 0),
    (W.MoeShape("wide_tail", 94, 2, 200, 320, 576, 12, 2, 3, n_shared_experts=2), 0),
    (W.MoeShape("split_k", 93, 4, 96, 256, 1024, 16, 4, 8, n_shared_experts=1), 4),
], ids=lambda v: v.name if hasattr(v, "name") else str(v))
def test_jittered_plans_bit_identical(B, shape, split):
    c, idx, w, layer, x, idx_d, w_d = _setup(B, shape, split)
    try:
        ref = _run(B, layer, shape, x, idx_d, w_d, "serial")
        y_ref = oracle_rows(c, idx, w, np.arange(shape.T))
        assert rel_err(bf16_to_f64(ref), y_ref) <= TOL
        for seed in range(1, 19):
            B.moe_set_jitter(layer.h, seed * 7919, 64 + 37 * (seed % 8))
            plan = PLANS[seed % len(PLANS)]
            for mode in (("dynamic", "static") if seed % 3 == 0 else ("dynamic",)):
                y = _run(B, layer, shape, x, idx_d, w_d, mode, plan if mode == "dynamic" else None)
                assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), (seed, mode, plan)
        B.moe_set_jitter(layer.h, 0, 0)
    finally:
        layer.close()


def _random_shape(rng, i):
    E = int(rng.integers(2, 33))
    k = int(rng.integers(1, min(8, E) + 1))
    El = int(rng.integers(1, E + 1))
    return W.MoeShape(f"rand{i}", 300 + i, int(rng.integers(1, 5)), int(rng.integers(1, 260)),
                      int(rng.choice([128, 192, 256, 320])), int(rng.choice([128, 192, 320, 576])), E, k, El,
                      n_shared_experts=int(rng.integers(0, 3)),
                      zipf_s=float(rng.choice([0.0, 1.2, 3.0])) or None)


def test_random_shapes_and_routings_jittered(B):
    rng = np.random.default_rng(2024)
    for i in range(16):
        shape = _random_shape(rng, i)
        c, idx, w, layer, x, idx_d, w_d = _setup(B, shape)
        try:
            ref = _run(B, layer, shape, x, idx_d, w_d, "serial")
            y_ref = oracle_rows(c, idx, w, np.arange(shape.T))
            assert rel_err(bf16_to_f64(ref), y_ref) <= TOL, shape
            for j, plan in enumerate((None, PLANS[1 + i % (len(PLANS) - 1)])):
                B.moe_set_jitter(layer.h, 1000 * i + j + 1, 128)
                y = _run(B, layer, shape, x, idx_d, w_d, "dynamic", plan)
                assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), (shape, plan)
        finally:
            layer.close()


def test_jitter_hook_is_active(B):
    """The delays really happen: at up to 4096 sleeps of 64 cycles per event
    (about 55 us on average before each workgroup's ticket alone) a launch
    takes measurably longer than without them, and y is unchanged."""
    shape = W.WORKLOADS["tiny"]
    c, idx, w, layer, x, idx_d, w_d = _setup(B, shape)
    try:
        ref = _run(B, layer, shape, x, idx_d, w_d, "dynamic")

        def timed(max_sleeps):
            B.moe_set_jitter(layer.h, 12345, max_sleeps)
            ts = []
            for _ in range(5):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                y = torch.empty_like(ref)
                a.record()
                layer.forward(x, idx_d, w_d, y, "dynamic")
                b.record()
                torch.cuda.synchronize()
                assert B.moe_sync_status(layer.h) == B.MOE_OK
                assert torch.equal(y.view(torch.int16), ref.view(torch.int16))
                ts.append(a.elapsed_time(b) * 1e3)
            return float(np.median(ts))

        t0, t1 = timed(0), timed(4096)
        B.moe_set_jitter(layer.h, 0, 0)
        assert t1 > t0 + 25.0, (t0, t1)
        with pytest.raises(B.MoeError):
            B.moe_set_jitter(layer.h, 1, 4097)
    finally:
        layer.close()
