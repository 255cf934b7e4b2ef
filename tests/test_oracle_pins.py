"""Pins of the CPU oracle against things other than itself.

Each test checks one oracle stage against an exact result (integer-valued
sums, IEEE-exact orderings), an independent brute force (Python sorts, numpy
/ torch fp64 dense evaluation), a closed form of the cost model, a hand-derived
worked example (tests/golden/), or an invariant the paper states (e.g. the
deduplicated remote count never exceeds the remote count, section 3.1).
All CPU-only.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from paper_2609_21483_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16_bits(a) -> np.ndarray:
    """Round fp64/fp32 values to bf16 (RNE) bit patterns via torch (test-side helper)."""
    t = torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- gate logits

def test_logits_exact_integer_sums(orc):
    """Small-integer bf16 inputs make every sum exact; the oracle must equal the
    exact integer dot product x[g,:] . Wg[:,e] (pins operand roles and indexing)."""
    rng = np.random.default_rng(0)
    T, H, E = 7, 96, 11
    xi = rng.integers(-8, 9, size=(T, H))
    wi = rng.integers(-8, 9, size=(H, E))
    bias = rng.integers(-4, 5, size=E).astype(np.float32)
    got = orc.gate_logits(bf16_bits(xi), bf16_bits(wi), bias)
    want = (xi.astype(np.int64) @ wi.astype(np.int64)) + bias.astype(np.int64)
    assert np.array_equal(got.astype(np.int64), want)
    assert np.array_equal(got, want.astype(np.float32))


def test_logits_ascending_order_pin(orc):
    """In fp32, (0 + 2^24) + 1 - 2^24 = 0 while summing in the opposite order
    gives 1: the oracle's pinned order is ascending hidden index."""
    x = bf16_bits([[1.0, 1.0, 1.0]])
    wg = bf16_bits([[2.0 ** 24], [1.0], [-(2.0 ** 24)]])
    assert orc.gate_logits(x, wg)[0, 0] == 0.0
    wg_rev = bf16_bits([[-(2.0 ** 24)], [1.0], [2.0 ** 24]])
    assert orc.gate_logits(x, wg_rev)[0, 0] == 1.0


def test_logits_within_fp32_error_bound(orc):
    """Random case: |l32 - l_exact| <= gamma_H * sum|x w| (standard recursive
    summation bound, u = 2^-24), with l_exact from an fp64 matmul of the same
    bf16 values (fp64 is exact here up to 2^-53 relative per term)."""
    rng = np.random.default_rng(1)
    T, H, E = 64, 512, 16
    x = bf16_bits(rng.standard_normal((T, H)))
    wg = bf16_bits(0.02 * rng.standard_normal((H, E)))
    got = orc.gate_logits(x, wg).astype(np.float64)
    xf, wf = bits_to_f64(x), bits_to_f64(wg)
    exact = xf @ wf
    u = 2.0 ** -24
    gamma = H * u / (1 - H * u)
    bound = gamma * (np.abs(xf) @ np.abs(wf)) + 1e-30
    assert np.all(np.abs(got - exact) <= bound)


# ------------------------------------------------------ softmax / top-k / w

def _brute_topk(l: np.ndarray, k: int):
    order = sorted(range(l.shape[0]), key=lambda e: (-float(l[e]), e))
    return order[:k]


def test_topk_bruteforce_sort(orc):
    rng = np.random.default_rng(2)
    T, E, k = 200, 24, 5
    lg = rng.standard_normal((T, E)).astype(np.float32)
    lg[::7, 3] = lg[::7, 9]  # exact ties
    idx, w = orc.softmax_topk(lg, k)
    for g in range(T):
        assert list(idx[g]) == _brute_topk(lg[g], k)
        p = np.exp(lg[g].astype(np.float64) - lg[g].max())
        p /= p.sum()
        sel = p[idx[g]]
        assert np.allclose(w[g], sel / sel.sum(), rtol=1e-13, atol=0)


def test_topk_ties_prefer_lower_id(orc):
    lg = np.array([[1.0, 3.0, 3.0, 0.5, 3.0]], np.float32)
    idx, w = orc.softmax_topk(lg, 3)
    assert list(idx[0]) == [1, 2, 4]
    assert np.allclose(w[0], [1 / 3] * 3, rtol=1e-15)


def test_topk_k_equals_E_is_full_softmax(orc):
    rng = np.random.default_rng(3)
    lg = rng.standard_normal((10, 8)).astype(np.float32)
    idx, w = orc.softmax_topk(lg, 8)
    ref = torch.softmax(torch.from_numpy(lg.astype(np.float64)), dim=1).numpy()
    for g in range(10):
        assert sorted(idx[g]) == list(range(8))
        assert np.allclose(w[g], ref[g, idx[g]], rtol=1e-13)


def test_topk_invariants(orc):
    rng = np.random.default_rng(4)
    lg = (0.9 * rng.standard_normal((500, 64))).astype(np.float32)
    idx, w = orc.softmax_topk(lg, 6)
    assert np.all((idx >= 0) & (idx < 64))
    assert all(len(set(r)) == 6 for r in idx)
    assert np.allclose(w.sum(axis=1), 1.0, atol=1e-12)
    assert np.all(np.diff(w, axis=1) <= 0)


# ------------------------------------------------------------ route tables

def _brute_tables(idx, R, Tr, e0, El):
    T, k = idx.shape
    pairs = sorted((int(idx[g, j]) - e0, g, j) for g in range(T) for j in range(k)
                   if 0 <= int(idx[g, j]) - e0 < El)
    slot = -np.ones((T, k), np.int64)
    inv = []
    for s, (le, g, j) in enumerate(pairs):
        slot[g, j] = s
        inv.append(g * k + j)
    off = [0]
    for le in range(El):
        off.append(off[-1] + sum(1 for p in pairs if p[0] == le))
    cnt = np.zeros((El, R), np.int64)
    for le, g, j in pairs:
        cnt[le, g // Tr] += 1
    first = -np.ones(T, np.int64)
    for g in range(T):
        loc = [(int(idx[g, j]) - e0, j) for j in range(k) if 0 <= int(idx[g, j]) - e0 < El]
        if loc:
            le, j = min(loc)
            first[g] = slot[g, j]
    uniq = np.array([sum(1 for g in range(r * Tr, (r + 1) * Tr) if first[g] >= 0) for r in range(R)])
    return slot, np.array(inv, np.int64), np.array(off), cnt, first, uniq


@pytest.mark.parametrize("R,Tr,E,k,e0,El,skew", [
    (4, 16, 8, 2, 0, 8, 0.0),     # tiny workload shape: every pair is local
    (4, 37, 16, 3, 4, 5, 0.0),    # ragged token counts, offset local range
    (3, 50, 32, 8, 0, 8, 1.5),    # skewed routing, empty experts likely
    (2, 9, 6, 6, 0, 3, 0.0),      # k = E
])
def test_route_tables_bruteforce(orc, R, Tr, E, k, e0, El, skew):
    idx, _ = W.random_routing(R * Tr, E, k, seed=R * 100 + Tr, skew=skew)
    tab = orc.route_tables(idx, R, Tr, e0, El)
    slot, inv, off, cnt, first, uniq = _brute_tables(idx, R, Tr, e0, El)
    assert tab.X == len(inv)
    assert np.array_equal(tab.slot, slot)
    assert np.array_equal(tab.inv, inv)
    assert np.array_equal(tab.off, off)
    assert np.array_equal(tab.cnt_rank, cnt)
    assert np.array_equal(tab.first_slot, first)
    assert np.array_equal(tab.uniq, uniq)


def test_route_tables_invariants(orc):
    R, Tr, E, k, El = 4, 64, 16, 4, 6
    idx, _ = W.random_routing(R * Tr, E, k, seed=7, skew=0.7)
    tab = orc.route_tables(idx, R, Tr, 0, El)
    T = R * Tr
    local = (idx >= 0) & (idx < El)
    assert tab.X == int(local.sum()) == int(tab.cnt_rank.sum())
    # global histogram over all experts is T*k
    assert np.bincount(idx.ravel(), minlength=E).sum() == T * k
    # the slot map is a bijection between local pairs and [0, X)
    s = tab.slot[local]
    assert np.array_equal(np.sort(s), np.arange(tab.X))
    assert np.all(tab.slot[~local] == -1)
    assert np.array_equal(tab.slot.ravel()[tab.inv], np.arange(tab.X))
    assert np.all(np.diff(tab.off) >= 0) and tab.off[0] == 0 and tab.off[-1] == tab.X
    # deduplicated remote tokens never exceed remote pairs (section 3.1)
    assert tab.uniq[1:].sum() <= tab.cnt_rank[:, 1:].sum()


def test_route_tables_all_local(orc):
    idx, _ = W.random_routing(64, 8, 2, seed=11)
    tab = orc.route_tables(idx, 4, 16, 0, 8)
    assert tab.X == 128 and tab.uniq.sum() == 64


@pytest.mark.parametrize("K", [1, 2, 3, 4, 8])
def test_chunk_offsets_bruteforce(orc, K):
    R, Tr, E, k, El = 3, 41, 12, 3, 5
    T = R * Tr
    idx, _ = W.random_routing(T, E, k, seed=K, skew=0.5)
    tab = orc.route_tables(idx, R, Tr, 0, El)
    sub = orc.chunk_offsets(tab, T, k, K)
    for le in range(El):
        toks = [g for g in range(T) for j in range(k) if idx[g, j] == le]
        for q in range(K + 1):
            n_before = sum(1 for g in toks if (g * K) // T < q)
            assert sub[le, q] == tab.off[le] + n_before
        assert sub[le, 0] == tab.off[le] and sub[le, K] == tab.off[le + 1]


def test_dispatch_is_row_gather(orc):
    rng = np.random.default_rng(5)
    T, H, E, k = 30, 64, 8, 3
    x = bf16_bits(rng.standard_normal((T, H)))
    idx, _ = W.random_routing(T, E, k, seed=5)
    tab = orc.route_tables(idx, 3, 10, 0, 4)
    A = orc.dispatch(x, tab, k)
    for s in range(tab.X):
        g, j = divmod(int(tab.inv[s]), k)
        assert tab.slot[g, j] == s
        assert np.array_equal(A[s], x[g])


# -------------------------------------------------------- expert FFN, combine

def _torch_swiglu(x_bits, w1_bits, w3_bits, w2_bits):
    """Textbook SwiGLU FFN in fp64 with torch.nn.functional.silu."""
    X = torch.from_numpy(bits_to_f64(x_bits))
    W1 = torch.from_numpy(bits_to_f64(w1_bits))
    W3 = torch.from_numpy(bits_to_f64(w3_bits))
    W2 = torch.from_numpy(bits_to_f64(w2_bits))
    return ((torch.nn.functional.silu(X @ W1) * (X @ W3)) @ W2).numpy()


def test_expert_ffn_matches_textbook_swiglu(orc):
    rng = np.random.default_rng(6)
    H, F = 64, 96
    a = bf16_bits(rng.standard_normal(H))
    w1 = bf16_bits(0.1 * rng.standard_normal((H, F)))
    w3 = bf16_bits(0.1 * rng.standard_normal((H, F)))
    w2 = bf16_bits(0.1 * rng.standard_normal((F, H)))
    got = orc.expert_ffn(a, w1, w3, w2)
    want = _torch_swiglu(a[None, :], w1, w3, w2)[0]
    assert np.allclose(got, want, rtol=1e-12, atol=1e-14)


def _dense_masked(x, idx, w, w1, w3, w2, ws, Tr, e0):
    """Every local expert on every token (dense), masked by top-k."""
    T, k = idx.shape
    El = w1.shape[0]
    y = np.zeros((T, x.shape[1]))
    for le in range(El):
        Y = _torch_swiglu(x, w1[le], w3[le], w2[le])
        m = np.zeros(T)
        for j in range(k):
            m += np.where(idx[:, j] == le + e0, w[:, j], 0.0)
        y += m[:, None] * Y
    if ws is not None:
        for s in range(ws[0].shape[0]):
            Ys = _torch_swiglu(x[:Tr], ws[0][s], ws[1][s], ws[2][s])
            y[:Tr] += Ys
    return y


@pytest.mark.parametrize("shared", [False, True])
def test_layer_sparse_equals_dense_masked(orc, shared):
    """Brute force: dense evaluation of every local expert, masked by
    top-k, equals the oracle's sparse path."""
    sh = W.TINY.with_(hidden=64, ffn=64, n_local_experts=5, n_shared_experts=2 if shared else 0)
    rng = np.random.default_rng(8)
    x = bf16_bits(rng.standard_normal((sh.T, sh.hidden)))
    idx, w32 = W.random_routing(sh.T, sh.n_experts, sh.top_k, seed=9)
    w = w32.astype(np.float64)
    E_l, H, F = sh.n_local_experts, sh.hidden, sh.ffn
    w1 = bf16_bits(0.1 * rng.standard_normal((E_l, H, F)))
    w3 = bf16_bits(0.1 * rng.standard_normal((E_l, H, F)))
    w2 = bf16_bits(0.1 * rng.standard_normal((E_l, F, H)))
    ws = None
    if shared:
        ws = tuple(bf16_bits(0.1 * rng.standard_normal(s)) for s in [(2, H, F), (2, H, F), (2, F, H)])
    y = orc.layer_rows(x, idx, w, w1, w3, w2, *(ws or (None, None, None)), Tr=sh.tokens_per_rank)
    yd = _dense_masked(x, idx, w, w1, w3, w2, ws, sh.tokens_per_rank, 0)
    assert np.max(np.abs(y - yd)) <= 1e-12 * np.max(np.abs(yd))
    # tokens with no local expert (and not rank 0 with shared experts) are zero
    for g in range(sh.T):
        if not np.any(idx[g] < E_l) and not (shared and g < sh.tokens_per_rank):
            assert np.all(y[g] == 0.0)


def test_layer_special_cases(orc):
    rng = np.random.default_rng(10)
    T, H, F = 12, 32, 48
    x = bf16_bits(rng.standard_normal((T, H)))
    w1 = bf16_bits(0.2 * rng.standard_normal((1, H, F)))
    w3 = bf16_bits(0.2 * rng.standard_normal((1, H, F)))
    w2 = bf16_bits(0.2 * rng.standard_normal((1, F, H)))
    # E = E_l = 1, k = 1: a dense SwiGLU FFN
    idx = np.zeros((T, 1), np.int32)
    w = np.ones((T, 1))
    y = orc.layer_rows(x, idx, w, w1, w3, w2, Tr=T)
    assert np.allclose(y, _torch_swiglu(x, w1[0], w3[0], w2[0]), rtol=1e-12, atol=1e-14)
    # x = 0 gives y = 0
    z = np.zeros_like(x)
    assert np.all(orc.layer_rows(z, idx, w, w1, w3, w2, Tr=T) == 0.0)
    # doubling W2 (a power of two) doubles y exactly
    w2x2 = bf16_bits(2.0 * bits_to_f64(w2))
    y2 = orc.layer_rows(x, idx, w, w1, w3, w2x2, Tr=T)
    assert np.array_equal(y2, 2.0 * y)


def test_layer_identical_experts(orc):
    """With identical experts and all k choices local, y = FFN(x) since the
    renormalised weights sum to one."""
    rng = np.random.default_rng(12)
    T, H, F, E, k = 16, 32, 32, 4, 3
    x = bf16_bits(rng.standard_normal((T, H)))
    one = [bf16_bits(0.2 * rng.standard_normal(s)) for s in [(H, F), (H, F), (F, H)]]
    w1, w3, w2 = (np.stack([m] * E) for m in one)
    idx, w32 = W.random_routing(T, E, k, seed=13)
    y = orc.layer_rows(x, idx, w32.astype(np.float64), w1, w3, w2, Tr=T)
    ref = _torch_swiglu(x, *one)
    assert np.allclose(y, ref, rtol=1e-6, atol=1e-9)


# ------------------------------------------------------------------ cost model

def _linear_grid(N, beta, phi, cs):
    cs = np.asarray(cs, np.int32)
    return cs, beta * cs.astype(np.float64), phi * (N - cs).astype(np.float64)


WINDOWS = {"plain": 0, "move_steal": 1, "last_combine": 2}


def test_cost_model_hand_example(orc):
    d = json.load(open(os.path.join(GOLDEN, "cost_model_hand_example.json")))
    args = dict(c=d["c"], bw=d["bw"], flops=d["flops"], K=d["K"], eff=d["eff"], alpha=d["alpha"],
                N=d["N"], w_comp=d["w_comp"], w_dispatch=d["w_dispatch"], w_combine=d["w_combine"])
    for ki in range(3):
        t16 = orc.t_total(1, ki, n_tiles=[1, 1, 1], **args)
        t32 = orc.t_total(2, ki, n_tiles=[1, 1, 1], **args)
        assert math.isclose(t16, d["expected_t_total_c16"][ki], rel_tol=4e-16)
        assert math.isclose(t32, d["expected_t_total_c32"][ki], rel_tol=4e-16)
    assert orc.t_total(1, 0, n_tiles=[1, 1, 1], **args) == 4.5
    assert orc.t_total(2, 2, n_tiles=[1, 1, 1], **args) == 12.0625
    for case in d["cases_n_tiles"]:
        for reading, n_steal in case["n_steal"].items():
            window, rounding = reading.rsplit("_", 1)
            p = orc.plan(n_tiles=case["n_tiles"], steal_window=WINDOWS[window], steal_ceil=int(rounding == "ceil"),
                         **args)
            num, den = d["expected_t_total_min_num_den"]
            assert (p.c, p.K) == (d["expected_c"], d["expected_K"])
            assert math.isclose(p.t_total, num / den, rel_tol=5e-16)
            assert p.n_steal == n_steal, reading


def test_cost_model_hand_example_all_worker_tail(orc):
    """The same hand example with the last chunk's combine moving at the rate
    of all N = 64 workers, bw_all = 2^30 * 64 = 2^36 (section 4 runs the final
    combine on every worker): Eq 10 becomes 0.5 * 2^34 / (2^36 K) = 1/(8K) s.
    c=16: K=1 max(4 + 1/8, 1.5) = 4.125; K=2 4/0.75 + 1/16 = 259/48; K=4 8 + 1/32.
    c=32: 6.125; 8.0625; 12.03125.  c=8, K=1: 192/56 + 1/8 = 199/56 (minimum).
    n_steal (Eq 11-14) does not use the tail: the same counts as without it."""
    d = json.load(open(os.path.join(GOLDEN, "cost_model_hand_example.json")))
    args = dict(c=d["c"], bw=d["bw"], flops=d["flops"], K=d["K"], eff=d["eff"], alpha=d["alpha"],
                N=d["N"], w_comp=d["w_comp"], w_dispatch=d["w_dispatch"], w_combine=d["w_combine"],
                bw_all=float(2 ** 36))
    assert orc.t_total(1, 0, n_tiles=[1, 1, 1], **args) == 4.125
    assert math.isclose(orc.t_total(1, 1, n_tiles=[1, 1, 1], **args), 259 / 48, rel_tol=4e-16)
    assert orc.t_total(1, 2, n_tiles=[1, 1, 1], **args) == 8.03125
    assert orc.t_total(2, 0, n_tiles=[1, 1, 1], **args) == 6.125
    assert orc.t_total(2, 1, n_tiles=[1, 1, 1], **args) == 8.0625
    assert orc.t_total(2, 2, n_tiles=[1, 1, 1], **args) == 12.03125
    for case in d["cases_n_tiles"]:
        p = orc.plan(n_tiles=case["n_tiles"], **args)
        assert (p.c, p.K) == (8, 1)
        assert math.isclose(p.t_total, 199 / 56, rel_tol=5e-16)
        assert p.n_steal == case["n_steal"]["plain_floor"]


def test_cost_model_balance_point(orc):
    """BW(c) = beta*c, TFLOPS(N-c) = phi*(N-c), eff = 1, alpha = 1: T_total is
    max(Wc/(phi(N-c)), Wm/(beta c)); the continuous optimum is the balance
    c0 = N*(Wm/beta)/((Wm/beta)+(Wc/phi)), so c* is one of the two grid points
    around c0."""
    N, beta, phi = 256, 30e9, 9e12
    grid = list(range(8, 129, 8))
    rng = np.random.default_rng(14)
    for _ in range(50):
        wc = float(rng.uniform(1e10, 3e12))
        wm = float(rng.uniform(1e7, 2e9))
        cs, bw, fl = _linear_grid(N, beta, phi, grid)
        p = orc.plan(cs, bw, fl, [1], [1.0], 1.0, N, wc, wm / 2, wm / 2, [100])
        c0 = N * (wm / beta) / ((wm / beta) + (wc / phi))
        lo = max([c for c in grid if c <= c0], default=grid[0])
        hi = min([c for c in grid if c >= c0], default=grid[-1])
        assert p.c in (lo, hi)
        f = lambda c: max(wc / (phi * (N - c)), wm / (beta * c))
        assert p.t_total == pytest.approx(min(f(lo), f(hi)), rel=1e-12)


def test_cost_model_special_cases(orc):
    N = 256
    cs, bw, fl = _linear_grid(N, 30e9, 9e12, [8, 16, 32, 64, 128])
    Ks, eff_dec, eff_one = [1, 2, 4, 8], [1.0, 0.95, 0.85, 0.73], [1.0] * 4
    nt = [1000] * 4
    # no movement work: fewest movement workers, K = 1 by the tie-break
    p = orc.plan(cs, bw, fl, Ks, eff_dec, 0.5, N, 1e12, 0.0, 0.0, nt)
    assert (p.c, p.K) == (8, 1)
    # no compute work, BW strictly increasing: most movement workers
    p = orc.plan(cs, bw, fl, Ks, eff_dec, 0.5, N, 0.0, 1e9, 1e9, nt)
    assert p.c == 128 and p.n_steal == 0
    # alpha = 1 hides the whole tail: chunking only costs, K* = 1
    p = orc.plan(cs, bw, fl, Ks, eff_dec, 1.0, N, 1e12, 1e8, 1e8, nt)
    assert p.K == 1
    # alpha = 0 and no chunking penalty, compute-dominated: the tail shrinks as 1/K
    p = orc.plan(cs, bw, fl, Ks, eff_one, 0.0, N, 1e12, 1e8, 1e8, nt)
    assert p.K == 8
    # movement-dominated: nothing to steal
    p = orc.plan(cs, bw, fl, Ks, eff_dec, 0.5, N, 1e9, 5e10, 5e10, nt)
    assert p.t_total == pytest.approx(1e11 / bw[-1]) and p.n_steal == 0
    # a tail moved by all workers at a high rate is worth less than any
    # chunking loss: K* = 1 where the printed BW(c) tail would chunk
    p_lit = orc.plan(cs, bw, fl, Ks, [1.0, 0.9, 0.8, 0.7], 0.0, N, 1e12, 2e8, 2e8, nt)
    p_all = orc.plan(cs, bw, fl, Ks, [1.0, 0.9, 0.8, 0.7], 0.0, N, 1e12, 2e8, 2e8, nt, bw_all=5e12)
    assert p_lit.K > 1 and p_all.K == 1


def test_cost_model_tie_break_first_minimum(orc):
    """Equal T_total everywhere: c ascending then K ascending, first wins."""
    p = orc.plan([8, 16], [1e9, 1e9], [1e12, 1e12], [1, 2], [1.0, 1.0], 1.0, 64, 0.0, 0.0, 0.0, [1, 1])
    assert (p.c, p.K, p.ci, p.ki) == (8, 1, 0, 0)


def test_n_steal_formula_by_hand(orc):
    # The plain reading of Eq 11: W_comm = W_dispatch + W_combine, the volume
    # of Eq 5, whatever K; Eq 14's share taken as whole tiles.
    # t_comm = 2e9/1e12 = 2 ms; W_partial = 2e-3 * 5e14 = 1e12; W_steal = 4e12 - 1e12 = 3e12;
    # W_tile = 4e12/4000 = 1e9; share = 3e12 / (100 * 1e9) = 30
    for K in (1, 2, 4):
        p = orc.plan([20], [1e12], [5e14], [K], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000])
        assert p.n_steal == 30
    # a share that is not whole: W_comp = 4.05e12 -> W_steal = 3.05e12, W_tile = 1.0125e9,
    # share = 3.05e12 / 1.0125e11 = 30.12..: 30 whole tiles, 31 rounded up
    p = orc.plan([20], [1e12], [5e14], [1], [1.0], 1.0, 100, 4.05e12, 1e9, 1e9, [4000])
    assert p.n_steal == 30
    p = orc.plan([20], [1e12], [5e14], [1], [1.0], 1.0, 100, 4.05e12, 1e9, 1e9, [4000], steal_ceil=1)
    assert p.n_steal == 31
    # communication longer than the GEMMs: W_partial > W_comp, nothing to steal (Eq 13's max)
    p = orc.plan([20], [1e10], [5e14], [1], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_ceil=1)
    assert p.n_steal == 0


def test_n_steal_formula_by_hand_last_combine_window(orc):
    # Eq 11 window without the last chunk's combine (it runs on every worker
    # after the GEMMs, section 4): W_dispatch + W_combine (K-1)/K.
    # K = 1: t_comm = 1e9/1e12 = 1 ms; W_partial = 5e11; W_steal = 3.5e12;
    # W_tile = 1e9; n_steal = 3.5e12 / (100 * 1e9) = 35
    p = orc.plan([20], [1e12], [5e14], [1], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_window=2)
    assert p.n_steal == 35
    # K = 2: t_comm = (1e9 + 1e9/2)/1e12 = 1.5 ms; W_partial = 7.5e11; W_steal = 3.25e12;
    # share 32.5: 32 whole tiles, 33 rounded up
    p = orc.plan([20], [1e12], [5e14], [2], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_window=2)
    assert p.n_steal == 32
    p = orc.plan([20], [1e12], [5e14], [2], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_window=2, steal_ceil=1)
    assert p.n_steal == 33


def test_n_steal_formula_by_hand_move_steal_window(orc):
    # With every worker dispatching the first chunk before any GEMM tile can
    # start, Eq 11's window is (W_dispatch + W_combine)(K-1)/K.
    # K = 1: empty window; W_steal = W_comp = 4e12; n_steal = 4e12 / (100 * 1e9) = 40
    p = orc.plan([20], [1e12], [5e14], [1], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_window=1)
    assert p.n_steal == 40
    # K = 2: window 2e9 / 2 = 1e9 bytes -> 1 ms; W_partial = 5e11; W_steal = 3.5e12; n_steal = 35
    p = orc.plan([20], [1e12], [5e14], [2], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_window=1)
    assert p.n_steal == 35
    # K = 4: window 2e9 * 3/4 = 1.5e9 bytes -> 1.5 ms; W_partial = 7.5e11; W_steal = 3.25e12;
    # share 32.5: 32 whole tiles, 33 rounded up
    p = orc.plan([20], [1e12], [5e14], [4], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_window=1)
    assert p.n_steal == 32
    p = orc.plan([20], [1e12], [5e14], [4], [1.0], 1.0, 100, 4e12, 1e9, 1e9, [4000], steal_window=1, steal_ceil=1)
    assert p.n_steal == 33
    # the window does not enter T_total (Eq 15): same plan and prediction under every reading
    plans = [orc.plan([8, 16], [1e11, 2e11], [1e15, 9e14], [1, 2], [1.0, 0.9], 0.5, 64, 1e12, 2e8, 2e8,
                      [1000, 1100], steal_window=w) for w in (0, 1, 2)]
    assert len({(p.c, p.K, p.t_total) for p in plans}) == 1


def test_tile_count_bruteforce(orc):
    rng = np.random.default_rng(15)
    rows = rng.integers(0, 700, size=(9, 4)).astype(np.int32)
    rows[2, :] = 0
    BM, nt0, nt1 = 128, 7, 3
    n = 0
    for seg in range(9):
        for q in range(4):
            m = int(rows[seg, q])
            while m > 0:
                n += nt0 + nt1
                m -= BM
    assert orc.tile_count(rows, BM, nt0, nt1) == n


def test_volumes_invariants(orc):
    R, Tr, E, k, El = 4, 128, 32, 8, 8
    idx, _ = W.random_routing(R * Tr, E, k, seed=16)
    tab = orc.route_tables(idx, R, Tr, 0, El)
    H, F = 256, 512
    wc, wd, wcb = orc.volumes(tab, H, F, 0, literal=True)
    X_in = tab.cnt_rank[:, 1:].sum()
    assert wc == tab.X * 6 * H * F
    assert wcb == X_in * 2 * H
    assert wd <= wcb   # X_in^uniq <= X_in (section 3.1)
    wc2, wd2, wcb2 = orc.volumes(tab, H, F, 0, literal=False)
    assert wc2 == wc and wd2 >= wd and wcb2 >= wcb
    # every row moved: one row per unique token of any rank (brute force over
    # the routing) and one per local pair
    U_all = sum(1 for g in range(R * Tr) if np.any(idx[g] < El))
    assert wd2 == U_all * 2 * H and wcb2 == tab.X * 2 * H


def test_volumes_hand_example(orc):
    """Eq 1-3 on the hand-made routing of tests/golden/volumes_hand_example.json,
    exact, under both readings of the movement volumes."""
    d = json.load(open(os.path.join(GOLDEN, "volumes_hand_example.json")))
    idx = np.array(d["topk_idx"], np.int32)
    tab = orc.route_tables(idx, d["R"], d["Tr"], d["e0"], d["El"])
    for shared_rows, w_comp in d["shared_rows_cases"]:
        for literal, key in ((True, "literal"), (False, "all_rows")):
            wc, wd, wb = orc.volumes(tab, d["H"], d["F"], shared_rows, literal=literal)
            assert wc == w_comp
            assert (wd, wb) == (d[key]["w_dispatch"], d[key]["w_combine"]), key
