"""GPU parity of the MoE layer (dispatch, GEMM0 + SiLU*up, GEMM1, combine)
against the CPU oracle, in the three execution modes and under forced plans.

Bar: max|y_gpu - y_ref| <= 2e-2 * max|y_ref| over the checked rows (bf16
inputs, fp32 accumulation, bf16 intermediates).  The dispatched rows are
checked bit for bit.  Every plan computes each output element with the same
operations in the same order, so y must also be bit-identical across modes
and plans."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2609_21483_amd import workloads as W
from tests.cases import bf16_to_f64, check_plan, make_case, oracle_rows, pick_rows, plain_reading, rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21483_amd import binding
    return binding


def run_modes(B, layer, c, idx, w, modes=("dynamic", "static", "serial"), forced=()):
    shape = c.shape
    x = c.x.cuda()
    idx_d = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).cuda()
    w_d = torch.from_numpy(np.ascontiguousarray(w, np.float32)).cuda()
    B.moe_build_tables(layer.h, idx_d)
    outs = {}
    for m in modes:
        y = torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
        layer.forward(x, idx_d, w_d, y, m)
        st = B.moe_sync_status(layer.h)
        assert st == B.MOE_OK, (m, B.moe_last_error())
        outs[m] = y
    for p in forced:
        y = torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
        layer.forward(x, idx_d, w_d, y, "dynamic", forced=B.moe_plan(*p, 0.0))
        st = B.moe_sync_status(layer.h)
        assert st == B.MOE_OK, (p, B.moe_last_error())
        outs[p] = y
    return outs


def check_case(B, c, rows=None, forced=(), check_A=False, gemm1_split=0):
    shape = c.shape
    idx, w = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2, gemm1_split=gemm1_split)
    try:
        outs = run_modes(B, layer, c, idx, w, forced=forced)
        rows = np.arange(shape.T) if rows is None else rows
        y_ref = oracle_rows(c, idx, w, rows)
        first = None
        for key, y in outs.items():
            yg = bf16_to_f64(y[torch.from_numpy(rows).cuda()])
            assert np.all(np.isfinite(yg)), key
            err = rel_err(yg, y_ref)
            assert err <= TOL, (key, err)
            if first is None:
                first = y
            else:
                assert torch.equal(y.view(torch.int16), first.view(torch.int16)), f"{key} differs from dynamic"
        if check_A:
            check_dispatched_rows(B, layer, c, idx, w)
        return err
    finally:
        layer.close()


def check_dispatched_rows(B, layer, c, idx, w):
    """After a forward at each chunk count K, A holds the oracle's dispatched
    rows (slot order) at the rows of the row map of moe.h, and the row map is
    the segment-major prefix of the (segment, chunk) row counts, each rounded
    up to 32 rows."""
    shape = c.shape
    El, S, Tr, T, H = shape.n_local_experts, shape.n_shared_experts, shape.tokens_per_rank, shape.T, shape.hidden
    tab = O.route_tables(idx, shape.n_src_ranks, Tr, 0, El)
    ref = O.dispatch(c.xu, tab, shape.top_k)
    x = c.x.cuda()
    idx_d = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).cuda()
    w_d = torch.from_numpy(np.ascontiguousarray(w, np.float32)).cuda()
    B.moe_build_tables(layer.h, idx_d)
    y = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
    nseg = El + S
    rof = layer.ws_view("row_off", torch.int32, 4 * nseg * 9).cpu().numpy().reshape(4, nseg, 9)
    for ki, K in enumerate((1, 2, 4, 8)):
        sub = O.chunk_offsets(tab, T, shape.top_k, K)
        bnd = [(q * T + K - 1) // K for q in range(K + 1)]
        rows = [[int(sub[le][q + 1] - sub[le][q]) for q in range(K)] for le in range(El)]
        rows += [[max(0, min(bnd[q + 1], Tr) - bnd[q]) for q in range(K)] for _ in range(S)]
        start, at = np.zeros((nseg, K), np.int64), 0
        for seg in range(nseg):
            for q in range(K):
                start[seg, q] = at
                at += -(-rows[seg][q] // 32) * 32
        assert np.array_equal(rof[ki, :, :K], start), K
        assert not rof[ki, :, K:].any()
        layer.forward(x, idx_d, w_d, y, "dynamic", forced=B.moe_plan(8, K, 3, 1, 0.0))
        assert B.moe_sync_status(layer.h) == B.MOE_OK
        # 32-row groups, each group's 32-column k-steps one 32 x 32 block after the other
        G = -(-int(at) // 32)
        A = layer.ws_view("A", torch.int16, G * 32 * H).cpu().numpy().view(np.uint16)
        A = A.reshape(G, H // 32, 32, 32).transpose(0, 2, 1, 3).reshape(G * 32, H)
        for le in range(El):
            for q in range(K):
                n, s0, r0 = rows[le][q], int(sub[le][q]), int(start[le, q])
                assert np.array_equal(A[r0:r0 + n], ref[s0:s0 + n]), (K, le, q)


FORCED_SMALL = [(1, 1, 0, 1), (8, 2, 3, 1), (64, 4, 0, 0), (255, 8, 1000, 1), (40, 1, 0, 0), (128, 8, 2, 0)]


def test_tiny_all_rows_all_plans(B):
    c = make_case(W.TINY)
    check_case(B, c, forced=FORCED_SMALL, check_A=True)


@pytest.mark.parametrize("shape", [
    W.MoeShape("ragged", 98, 3, 45, 192, 320, 10, 3, 4, n_shared_experts=1),
    W.MoeShape("one_token", 97, 1, 1, 128, 128, 8, 2, 8),
    W.MoeShape("all_local", 96, 2, 150, 256, 192, 4, 4, 4),
    W.MoeShape("skew_empty", 95, 4, 77, 128, 256, 32, 8, 5, zipf_s=3.0),
    W.MoeShape("wide_tail", 94, 2, 200, 320, 576, 12, 2, 3, n_shared_experts=2),
], ids=lambda s: s.name)
def test_edge_shapes(B, shape):
    c = make_case(shape.with_(w_std=0.05))
    check_case(B, c, forced=FORCED_SMALL, check_A=True)


@pytest.mark.parametrize("split", [1, 2, 4, 8])
def test_gemm1_split_factors(B, split):
    """GEMM1 split 1, 2, 4 or 8 ways over F (the last split of a tile adds
    the fp32 partials in split order); shared experts and a ragged row tail
    included."""
    shape = W.MoeShape("split", 92, 3, 70, 128, 512, 8, 2, 4, n_shared_experts=1)
    c = make_case(shape.with_(w_std=0.05))
    check_case(B, c, forced=[(8, 2, 3, 1), (100, 4, 0, 0)], gemm1_split=split)


def test_no_local_pairs(B):
    """Every token routed off this GPU: y must be all zeros (no shared experts),
    or only the shared output on rank 0."""
    for S in (0, 1):
        shape = W.MoeShape("nolocal", 93, 2, 64, 128, 128, 16, 2, 4, n_shared_experts=S)
        c = make_case(shape.with_(w_std=0.05))
        idx, w = W.random_routing(shape.T, 12, 2, seed=5)
        idx = (idx + 4).astype(np.int32)  # experts 4..15, all remote
        layer = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
        try:
            outs = run_modes(B, layer, c, idx, w.astype(np.float64))
            y_ref = oracle_rows(c, idx, w.astype(np.float64), np.arange(shape.T))
            for y in outs.values():
                yg = bf16_to_f64(y)
                if S == 0:
                    assert np.all(yg == 0.0)
                else:
                    assert np.all(yg[shape.tokens_per_rank:] == 0.0)
                    assert rel_err(yg, y_ref) <= TOL
        finally:
            layer.close()


FULL = [("mixtral_ep4", 0), ("fine_zipf", 0), ("shared_routed", 0)] + [("large_stack", l) for l in range(8)]


@pytest.mark.parametrize("name,layer", FULL, ids=[f"{n}-L{l}" for n, l in FULL])
def test_full_size_sampled_rows(B, name, layer):
    """A whole layer share at full size, y checked on sampled rows (rows are
    independent, so a sample is exact) in every mode, under forced chunked
    plans, and under the cost model's plans on the built-in table, the
    committed measured table and the plain reading of the printed equations;
    each plan against the oracle's cost model on the oracle's tables."""
    from paper_2609_21483_amd.calibrate import load_calib
    shape = W.WORKLOADS[name]
    c = make_case(shape, layer)
    idx, w = c.oracle_route()
    rows = pick_rows(shape, idx, per_rank=16, seed=100 + layer)
    forced = [(8, 8, 4, 1), (120, 2, 0, 1)] if name == "fine_zipf" else [(40, 2, 4, 1), (64, 4, 2, 1)]
    ml = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
    try:
        x = c.x.cuda()
        idx_d = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).cuda()
        w_d = torch.from_numpy(np.ascontiguousarray(w, np.float32)).cuda()
        B.moe_build_tables(ml.h, idx_d)

        def fwd(mode, plan=None):
            y = torch.full((shape.T, shape.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
            ml.forward(x, idx_d, w_d, y, mode, forced=None if plan is None else B.moe_plan(*plan, 0.0))
            assert B.moe_sync_status(ml.h) == B.MOE_OK, (mode, plan, B.moe_last_error())
            return y

        outs = {"dynamic": fwd("dynamic")}
        check_plan(B, ml.h, shape, idx)
        outs["static"] = fwd("static")
        outs["serial"] = fwd("serial")
        for p in forced:
            outs[p] = fwd("dynamic", p)
        measured = load_calib(name, torch.cuda.get_device_properties(0).multi_processor_count)
        if measured is not None:
            B.moe_set_calib(ml.h, measured)
            outs["measured"] = fwd("dynamic")
            check_plan(B, ml.h, shape, idx)
            B.moe_set_calib(ml.h, plain_reading(B.moe_calib.from_buffer_copy(measured)))
            outs["plain"] = fwd("dynamic")
            check_plan(B, ml.h, shape, idx)
        y_ref = oracle_rows(c, idx, w, rows)
        first = outs["dynamic"]
        sel = torch.from_numpy(rows).cuda()
        for key, y in outs.items():
            yg = bf16_to_f64(y[sel])
            assert np.all(np.isfinite(yg)), key
            assert rel_err(yg, y_ref) <= TOL, key
            assert torch.equal(y.view(torch.int16), first.view(torch.int16)), f"{key} differs from dynamic"
    finally:
        ml.close()


@pytest.mark.parametrize("K", [1, 2, 4])
def test_run_stages_reproduces_forward(B, K):
    """moe_run_stages (the stages as separate kernels on n workers, used by
    the calibration) with every stage gives the forward's y bit for bit."""
    shape = W.SHARED_ROUTED.with_(tokens_per_rank=512)
    c = make_case(shape)
    idx, w = c.oracle_route()
    ml = B.MoeLayer(shape, c.w1, c.w3, c.w2, c.ws1, c.ws3, c.ws2)
    try:
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(ml.h, idx_d)
        y0 = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        ml.forward(x, idx_d, w_d, y0, "dynamic")
        assert B.moe_sync_status(ml.h) == B.MOE_OK
        rows = pick_rows(shape, idx, per_rank=24, seed=3)
        assert rel_err(bf16_to_f64(y0[torch.from_numpy(rows).cuda()]), oracle_rows(c, idx, w, rows)) <= TOL
        for n in (torch.cuda.get_device_properties(0).multi_processor_count, 37):
            y = torch.full_like(y0, float("nan"))
            B.moe_run_stages(ml.h, x, idx_d, w_d, ml.packed, y, 15, n, K)
            assert B.moe_sync_status(ml.h) == B.MOE_OK
            assert torch.equal(y.view(torch.int16), y0.view(torch.int16)), (K, n)
    finally:
        ml.close()


def test_route_then_forward_end_to_end(B):
    """moe_route output fed straight into moe_forward."""
    shape = W.FINE_ZIPF.with_(tokens_per_rank=256)
    c = make_case(shape)
    idx_ref, w_ref = c.oracle_route()
    layer = B.MoeLayer(shape, c.w1, c.w3, c.w2)
    try:
        x = c.x.cuda()
        idx = torch.empty((shape.T, shape.top_k), dtype=torch.int32, device="cuda")
        w = torch.empty((shape.T, shape.top_k), dtype=torch.float32, device="cuda")
        layer.route(x, c.wg.cuda(), c.bias.cuda(), idx, w)
        y = torch.empty((shape.T, shape.hidden), dtype=torch.bfloat16, device="cuda")
        layer.forward(x, idx, w, y, "dynamic")
        assert B.moe_sync_status(layer.h) == B.MOE_OK
        assert np.array_equal(idx.cpu().numpy(), idx_ref)
        y_ref = oracle_rows(c, idx_ref, w_ref, np.arange(shape.T))
        assert rel_err(bf16_to_f64(y), y_ref) <= TOL
        # forward refuses routing the tables were not built from
        other = idx.clone()
        with pytest.raises(B.MoeError) as ei:
            layer.forward(x, other, w, y, "dynamic")
        assert ei.value.status == B.MOE_ERR_STATE
    finally:
        layer.close()


def test_repeat_launches_deterministic(B):
    c = make_case(W.FINE_ZIPF.with_(tokens_per_rank=512))
    idx, w = c.oracle_route()
    layer = B.MoeLayer(c.shape, c.w1, c.w3, c.w2)
    try:
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(layer.h, idx_d)
        ys = []
        for i in range(6):
            y = torch.empty((c.shape.T, c.shape.hidden), dtype=torch.bfloat16, device="cuda")
            layer.forward(x, idx_d, w_d, y, ("dynamic", "static", "serial")[i % 3])
            ys.append(y)
        assert B.moe_sync_status(layer.h) == B.MOE_OK
        for y in ys[1:]:
            assert torch.equal(y.view(torch.int16), ys[0].view(torch.int16))
    finally:
        layer.close()


def test_relaunch_with_new_inputs(B):
    """The same workspace and control sets serve launches whose tokens and
    routing change: each result matches the oracle for its own inputs (no
    stale rows from the previous launch)."""
    shape = W.FINE_ZIPF.with_(tokens_per_rank=384)
    c1 = make_case(shape)
    c2 = make_case(shape.with_(wid=shape.wid + 50))
    layer = B.MoeLayer(shape, c1.w1, c1.w3, c1.w2)
    try:
        for c in (c1, c2, c1):
            idx, w = c.oracle_route()
            outs = run_modes(B, layer, c, idx, w, modes=("dynamic", "serial"))
            rows = pick_rows(shape, idx, per_rank=24, seed=7)
            # c2 shares c1's expert weights (the layer packs them once)
            y_ref = oracle_rows(c1.with_tokens(c), idx, w, rows)
            for y in outs.values():
                assert rel_err(bf16_to_f64(y[torch.from_numpy(rows).cuda()]), y_ref) <= TOL
    finally:
        layer.close()


def test_more_workers_than_the_gpu_holds_is_refused(B):
    """The megakernel's workgroups wait on each other, so all of them must be
    resident at once: a worker count beyond what the GPU holds is refused
    before any launch (one workgroup fits a CU)."""
    c = make_case(W.TINY)
    idx, w = c.oracle_route()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    layer = B.MoeLayer(c.shape, c.w1, c.w3, c.w2, n_workers=2 * cus)
    try:
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(layer.h, idx_d)
        y = torch.zeros((c.shape.T, c.shape.hidden), dtype=torch.bfloat16, device="cuda")
        with pytest.raises(B.MoeError) as ei:
            layer.forward(x, idx_d, w_d, y, "dynamic")
        assert ei.value.status == B.MOE_ERR_UNSUPPORTED
        assert "holds at once" in B.moe_last_error()
        # the serial kernels have no such constraint
        layer.forward(x, idx_d, w_d, y, "serial")
        assert B.moe_sync_status(layer.h) == B.MOE_OK
        assert rel_err(bf16_to_f64(y), oracle_rows(c, idx, w, np.arange(c.shape.T))) <= TOL
    finally:
        layer.close()


def test_timeout_path_recovers(B):
    """Host-forced stall: every wait targets an unreachable value, so the
    launch times out on its own bounded waits, reports MOE_ERR_TIMEOUT, and the
    next launch (other control set) is correct again."""
    c = make_case(W.TINY)
    idx, w = c.oracle_route()
    layer = B.MoeLayer(c.shape, c.w1, c.w3, c.w2)
    try:
        x = c.x.cuda()
        idx_d = torch.from_numpy(idx).cuda()
        w_d = torch.from_numpy(w.astype(np.float32)).cuda()
        B.moe_build_tables(layer.h, idx_d)
        y = torch.empty((c.shape.T, c.shape.hidden), dtype=torch.bfloat16, device="cuda")
        B.moe_set_timeout_ms(layer.h, 20.0, 1)
        layer.forward(x, idx_d, w_d, y, "dynamic")
        assert B.moe_sync_status(layer.h) == B.MOE_ERR_TIMEOUT
        B.moe_set_timeout_ms(layer.h, 2000.0, 0)
        for _ in range(2):
            layer.forward(x, idx_d, w_d, y, "dynamic")
            assert B.moe_sync_status(layer.h) == B.MOE_OK
            y_ref = oracle_rows(c, idx, w, np.arange(c.shape.T))
            assert rel_err(bf16_to_f64(y), y_ref) <= TOL
    finally:
        layer.close()
