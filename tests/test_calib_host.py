"""Host logic of the calibration: the monotone fit of the measured BW(c) and
TFLOPS(N - c) curves (no GPU)."""
import itertools

import numpy as np

from paper_2609_21483_amd.calibrate import isotonic


def _brute(y, increasing):
    # least-squares monotone fit by brute force over step functions whose
    # levels are block means (the optimum is one of them)
    n = len(y)
    best, arg = None, None
    for cuts in itertools.product([0, 1], repeat=n - 1):
        blocks, cur = [], [y[0]]
        for i, c in enumerate(cuts):
            if c:
                blocks.append(cur)
                cur = [y[i + 1]]
            else:
                cur.append(y[i + 1])
        blocks.append(cur)
        fit = sum(([float(np.mean(b))] * len(b) for b in blocks), [])
        d = np.diff(fit)
        if (increasing and np.any(d < -1e-12)) or (not increasing and np.any(d > 1e-12)):
            continue
        err = float(np.sum((np.array(fit) - np.array(y)) ** 2))
        if best is None or err < best - 1e-12:
            best, arg = err, fit
    return arg


def test_isotonic_matches_brute_force():
    rng = np.random.default_rng(3)
    for _ in range(40):
        n = int(rng.integers(1, 8))
        y = list(rng.normal(size=n) + np.linspace(0, 1, n) * rng.choice([-1, 1]))
        for inc in (True, False):
            np.testing.assert_allclose(isotonic(y, inc), _brute(y, inc), rtol=0, atol=1e-9)


def test_isotonic_keeps_monotone_input_and_mean():
    y = [1.0, 2.0, 2.0, 5.0]
    assert isotonic(y, True) == y
    z = [3.0, 1.0, 2.0, 0.5]
    f = isotonic(z, False)
    assert all(a >= b for a, b in zip(f, f[1:]))
    assert abs(sum(f) - sum(z)) < 1e-12


def test_eff_alpha_fit_recovers_a_planted_model():
    """Eq 15 on a synthetic no-stealing grid built from known eff_chunk and
    alpha (compute-bound points, plus communication-bound ones the fit must
    leave out) is identified back."""
    from paper_2609_21483_amd.calibrate import fit_eff_alpha
    Ks = [1, 2, 4, 8]
    eff_true, alpha_true = [1.0, 0.95, 0.85, 0.7], 0.35
    cs = [8, 24, 40, 56, 72, 88, 104, 120]
    fl = [1.0e15 * (1 - c / 400) for c in cs]
    bw = [2.0e10 * c for c in cs]
    w_comp, w_move, w_comb, bw_all = 2.0e12, 2.4e9, 1.2e9, 3.0e12
    sweep = []
    for ci, c in enumerate(cs):
        for ki, K in enumerate(Ks):
            tc = w_comp / fl[ci]
            t = max(tc / eff_true[ki] + (1 - alpha_true) * w_comb / (bw_all * K), w_move / bw[ci])
            if w_move / bw[ci] > tc:
                t *= 0.3  # what the model cannot describe: must not enter the fit
            sweep.append((ci, ki, t))
    eff, alpha, n, resid, raw = fit_eff_alpha(sweep, Ks, w_comp, w_move, w_comb, fl, bw, bw_all)
    assert n == sum(1 for ci in range(len(cs)) if w_move / bw[ci] <= w_comp / fl[ci]) * len(Ks)
    np.testing.assert_allclose(eff, eff_true, rtol=1e-9)
    assert abs(alpha - alpha_true) < 1e-9 and abs(raw - alpha_true) < 1e-9
    assert max(abs(r) for r in resid) < 1e-9
