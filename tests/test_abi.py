"""CPU tests of the C ABI: the library loads, exports every function that
include/moe.h declares, validates arguments on the host before touching the
GPU, and its host cost model agrees bit for bit with the oracle's.  No kernel
is launched here."""
import ctypes as C
import math

import numpy as np
import pytest

from paper_2609_21483_amd import workloads as W

B = pytest.importorskip("paper_2609_21483_amd.binding", reason="libmoe.so not built")


def test_exports_every_declared_function():
    names = B.header_functions()
    assert len(names) >= 18
    lib = B.library()
    for n in names:
        assert hasattr(lib, n), n
    assert set(B._SIGS) == set(names)


def cfg_for(shape, **kw):
    c = B.make_config(shape, n_workers=256)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("field,value", [
    ("hidden", 100), ("hidden", 0), ("ffn", 96), ("top_k", 0), ("top_k", 9), ("n_experts", 0),
    ("n_local_experts", 0), ("first_local_expert", 7), ("n_src_ranks", 0), ("tokens_per_rank", 0),
    ("n_shared_experts", 9), ("n_workers", -1), ("gemm1_split", 3), ("gemm1_split", 16),
])
def test_init_rejects_bad_config(field, value):
    c = cfg_for(W.TINY, **{field: value})
    with pytest.raises(B.MoeError) as ei:
        B.moe_init(c)
    assert ei.value.status in (B.MOE_ERR_INVALID_ARG, B.MOE_ERR_UNSUPPORTED)
    assert B.moe_last_error()


def test_init_rejects_row_buffer_over_4gib():
    # T * min(k, E_l) rows of H bf16 must stay under 4 GiB (32-bit offsets)
    c = cfg_for(W.TINY, n_src_ranks=16, tokens_per_rank=65536, hidden=4096, n_experts=8, top_k=1,
                n_local_experts=1)
    with pytest.raises(B.MoeError) as ei:
        B.moe_init(c)
    assert ei.value.status == B.MOE_ERR_UNSUPPORTED


def test_init_rejects_bad_calib():
    c = cfg_for(W.TINY)
    good = dict(c=[8, 16], bw=[1e11, 2e11], flops=[1e14, 1e14], K=[1, 2], eff=[1.0, 0.9], alpha=0.5, static_c=40)
    h = B.moe_init(c, B.make_calib(**good))
    B.moe_destroy(h)
    for bad in [dict(c=[16, 8]), dict(c=[8, 256]), dict(bw=[0.0, 1.0]), dict(K=[1, 3]), dict(eff=[1.0, 1.5]),
                dict(alpha=2.0), dict(static_c=0), dict(bw_all=-1.0), dict(bw_all=float("inf")),
                dict(steal_window=3), dict(steal_window=-1), dict(steal_ceil=2)]:
        kw = {**good, **bad}
        with pytest.raises(B.MoeError):
            B.moe_init(c, B.make_calib(**kw))


@pytest.mark.parametrize("shape", list(W.WORKLOADS.values()) + [
    W.MoeShape("padded_slabs", 98, 3, 45, 192, 320, 10, 3, 4, n_shared_experts=1)], ids=lambda s: s.name)
def test_workspace_layout_covers_buffers(shape):
    h = B.moe_init(cfg_for(shape))
    try:
        L = B.moe_workspace_layout(h)
        size = B.moe_workspace_size(h)
        assert size == L.total
        T, k, El, S = shape.T, shape.top_k, shape.n_local_experts, shape.n_shared_experts
        xmax = T * min(k, El)
        # the row map rounds each of at most 8 chunks of every segment up to 32 rows
        arows = xmax + El * 8 * 31
        rows = arows + S * (shape.tokens_per_rank + 8 * 31)
        offs = sorted((getattr(L, n), n) for n in ("slot", "inv", "first_slot", "off", "sub_off", "row_off",
                                                    "cnt_rank", "uniq", "stats", "plan", "err", "A", "Hbuf", "O"))
        assert all(o % 256 == 0 for o, _ in offs)
        assert L.slot + 4 * T * k <= L.inv
        assert L.sub_off + 4 * 4 * El * 9 <= L.row_off
        assert L.row_off + 4 * 4 * (El + S) * 9 <= L.cnt_rank
        assert L.A + 2 * arows * shape.hidden <= L.Hbuf
        assert L.Hbuf + 2 * rows * shape.ffn <= L.O
        assert L.O + 2 * rows * shape.hidden <= size
        # weight slabs of the GEMM tiles are padded to 256 rows
        slab = lambda n: math.ceil(n / 256) * 256
        assert B.moe_packed_weights_size(h) == (shape.n_local_experts + shape.n_shared_experts) * 2 * \
            (slab(2 * shape.ffn) * shape.hidden + slab(shape.hidden) * shape.ffn)
        bm, nt0, nt1 = B.moe_tile_geometry(h)
        assert nt0 == math.ceil(2 * shape.ffn / 256) and bm > 0
        # GEMM1 tiles per row tile: column tiles over H times a split-K factor of 1, 2, 4 or 8
        assert nt1 // math.ceil(shape.hidden / 256) in (1, 2, 4) and nt1 % math.ceil(shape.hidden / 256) == 0
    finally:
        B.moe_destroy(h)


def test_calls_without_workspace_fail_cleanly():
    h = B.moe_init(cfg_for(W.TINY))
    try:
        with pytest.raises(B.MoeError) as ei:
            B._check("moe_build_tables", B.library().moe_build_tables(h, C.c_void_p(16), None))
        assert ei.value.status == B.MOE_ERR_STATE
        with pytest.raises(B.MoeError):
            B._check("moe_set_timeout_ms", B.library().moe_set_timeout_ms(h, -1.0, 0))
    finally:
        B.moe_destroy(h)


def test_trace_buffer_must_hold_a_record_per_wavefront():
    h = B.moe_init(cfg_for(W.TINY))  # 256 workers x 8 wavefronts
    try:
        lib = B.library()
        need = 64 + 4 * 2048 + 32 * 2048
        with pytest.raises(B.MoeError) as ei:
            B._check("moe_set_trace", lib.moe_set_trace(h, C.c_void_p(1 << 20), need - 1))
        assert ei.value.status == B.MOE_ERR_INVALID_ARG
        B._check("moe_set_trace", lib.moe_set_trace(h, C.c_void_p(1 << 20), need))
        B._check("moe_set_trace", lib.moe_set_trace(h, None, 0))
    finally:
        B.moe_destroy(h)


def test_default_calibration_is_valid_and_static_split_is_deepep_fraction():
    h = B.moe_init(cfg_for(W.MIXTRAL_EP4))
    try:
        k = B.moe_get_calib(h)
        assert k.n_c >= 1 and all(1 <= k.c[i] < 256 for i in range(k.n_c))
        assert k.static_c == 40  # 20 of 132 SMs scaled to 256 CUs, multiple of 8
    finally:
        B.moe_destroy(h)


def test_host_cost_model_matches_oracle(orc):
    """The library's host mirror of the prologue cost model against the oracle
    on random volumes and calibration tables: identical plan, identical bits."""
    rng = np.random.default_rng(0)
    h = B.moe_init(cfg_for(W.FINE_ZIPF))
    try:
        for trial in range(200):
            n_c = int(rng.integers(1, 17))
            cs = np.sort(rng.choice(np.arange(1, 256), n_c, replace=False)).astype(np.int32)
            bw = rng.uniform(1e10, 6e12, n_c)
            fl = rng.uniform(1e13, 2.5e15, n_c)
            Ks = [1, 2, 4, 8][: int(rng.integers(1, 5))]
            eff = np.sort(rng.uniform(0.5, 1.0, len(Ks)))[::-1]
            alpha = float(rng.uniform(0, 1))
            wc, wd, wb = float(rng.uniform(0, 1e13)), float(rng.uniform(0, 2e9)), float(rng.uniform(0, 2e9))
            nt = rng.integers(0, 5000, len(Ks))
            bw_all = 0.0 if trial % 3 == 0 else float(rng.uniform(1e11, 8e12))
            window, ceil_ = trial % 3, (trial // 3) % 2
            B.moe_set_calib(h, B.make_calib(cs, bw, fl, Ks, eff, alpha, static_c=int(cs[0]), bw_all=bw_all,
                                            steal_window=window, steal_ceil=ceil_))
            p = B.moe_plan_host(h, wc, wd, wb, list(nt) + [0] * (4 - len(Ks)))
            o = orc.plan(cs, bw, fl, Ks, eff, alpha, 256, wc, wd, wb, nt, bw_all=bw_all, steal_window=window,
                         steal_ceil=ceil_)
            assert (p.c, p.K, p.n_steal) == (o.c, o.K, o.n_steal), trial
            assert p.t_pred_s == o.t_total, trial
    finally:
        B.moe_destroy(h)


def test_static_routing_refuses_what_its_scratch_cannot_hold():
    """moe_route_topk_static checks its arguments and the size of its static
    scratch on the host and launches nothing when they do not fit."""
    import types
    import torch
    x = torch.zeros(8, dtype=torch.int16)
    null_stream = types.SimpleNamespace(cuda_stream=0)  # the null stream, without initialising a GPU
    dummy = [x, x, None, x, x, null_stream]
    with pytest.raises(B.MoeError) as ei:
        B.moe_route_topk_static(1 << 21, 4096, 512, 8, *dummy)
    assert ei.value.status == B.MOE_ERR_UNSUPPORTED and "static scratch" in B.moe_last_error()
    for T, H, E, k in [(0, 64, 8, 2), (16, 96, 8, 2), (16, 64, 0, 1), (16, 64, 8, 9), (16, 64, 4, 5)]:
        with pytest.raises(B.MoeError) as ei:
            B.moe_route_topk_static(T, H, E, k, *dummy)
        assert ei.value.status == B.MOE_ERR_INVALID_ARG, (T, H, E, k)
